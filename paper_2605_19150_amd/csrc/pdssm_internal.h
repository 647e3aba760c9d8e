// pdssm_internal.h -- host-side launch interface shared by the C ABI layer and
// the kernel translation units.  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pdssm {

// Everything a scan launch needs.  Pointers are device pointers; complex
// tensors are float2 (re, im).  seq = b*H + h indexes a sequence; per-chunk
// buffers are [seq][chunk][N].
struct ScanArgs {
    int B, L, H, N, K;
    int tau;  // chunk length
    int C;    // ceil(L / tau)
    const int* idx;
    const int* pi;
    const float2* D;
    const float2* b;
    const float2* c;
    const float2* h0;
    const float* dy;
    const float2* dhf;
    float* y;
    float2* hfinal;
    float2* dD;
    float2* db;
    float2* dc;
    float2* dh0;
    float2* carry;   // [seq][C][N] state entering each chunk (saved or workspace)
    // per-chunk operator (pi_c, d_c) and local term (bias B_c in fwd, local
    // adjoint gamma_c in bwd)
    int* agg_p;
    float2* agg_d;
    float2* agg_v;
    float2* U;       // bwd: gradient reaching the last state of each chunk from later chunks
    int* status;
};

struct ComposeArgs {
    int B, L, H, N, K;
    int tau, C;
    const int* idx;
    const int* pi;
    const float2* D;
    int* pi_out;
    float2* d_out;
    int* status;
};

// Each returns hipSuccess or the launch error.
hipError_t launch_fwd_chunked(const ScanArgs& a, hipStream_t s);
hipError_t launch_bwd_chunked(const ScanArgs& a, hipStream_t s);
hipError_t launch_compose(const ComposeArgs& a, hipStream_t s);

// LDS bytes the chunked backward's emit kernel needs per workgroup.
inline size_t bwd_emit_lds_bytes(int N, int tau) { return (size_t)(tau + 2) * N * 8; }
constexpr size_t kMaxLdsPerGroup = 65536;

}  // namespace pdssm
