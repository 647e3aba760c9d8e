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
    int io;   // row format of D, b, c, dD, db, dc, z (kIoC64, kIoBf16, kIoReal: pdssm_io.h; z stays
              // complex64 with kIoBf16); the float2 pointers below are reinterpreted for the 4-byte formats
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
    // adjoint gamma_c in bwd); the forward keeps pi_c in sorted form (srt_word)
    int* agg_p;
    float2* agg_d;
    float2* agg_v;
    float2* U;       // bwd: gradient reaching the last state of each chunk from later chunks
    // per-entry dictionary tables of the prep kernel (PrepArgs), [H][K][N]
    // words and [H][K] classes: the scatter-adds of the dictionary steps
    const uint64_t* rec;
    const uint8_t* mtab;
    int* status;
    // bwd, optional: the scaled states z = D_t .* h_{t-1} [B,L,H,N] that
    // the straight-through gradients need (Sec. 3.1 Prop. 2)
    float2* z;
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

// Straight-through surrogate inputs (Sec. 3.1 Prop. 2): the dictionary
// gradient G[h,k] = sum over the steps (b,t) with idx[b,t,h] == k of
// Re(g_t z_t^H), and the scores q[b,t,h,k] = sum_j Re(g_t[pi_k(j)] conj(z_t[j])).
// The steps of every head are first grouped by map (a stable counting sort),
// then each group is cut into items of at most P steps; an item sums its
// steps' outer products on the matrix cores and writes G[h,k] itself when it
// is the group's only item, else a partial that a last pass adds up in item
// order.  All sums run in a fixed order (deterministic results).
struct DictPlan {
    int seg, S;      // steps per counting segment (a multiple of 256), segments per head (<= 64)
    int P;           // steps per item
    int max_items;   // bound on the number of items (grid size)
    int max_slots;   // bound on the partials of groups with several items
    size_t off_order, off_hist, off_n, off_pos, off_item, off_slot, off_partial, bytes;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// segment counts the dictionary planning kernel holds in LDS (64 KiB)
constexpr int kDictPlanLds = 16384;

inline DictPlan dict_plan(int B, int L, int H, int N, int K) {
    DictPlan p;
    const size_t BL = (size_t)B * L, total = BL * H;
    // segments of about 512 steps (two tiles of the scatter), at most 64 per
    // head and at most kDictPlanLds counts in all: enough workgroups for the
    // grouping kernels to fill the chip, each with a short serial walk, and
    // the counts fit the planning kernel's LDS
    size_t s_want = BL >= 64 * 512 ? 64 : (BL + 511) / 512;
    const size_t s_lds = (size_t)kDictPlanLds / ((size_t)H * K);
    if (s_want > s_lds) s_want = s_lds > 0 ? s_lds : 1;
    p.seg = (int)(((BL + s_want - 1) / s_want + 255) & ~(size_t)255);
    p.S = (int)((BL + p.seg - 1) / p.seg);
    const size_t cell = (size_t)N * N * 4;
    // About 2048 items (fewer idle CUs at the grid's end than with 1024:
    // measured 6% faster at fsa-perm, 12% at timeseries), with the average
    // group cut into m equal pieces plus 20% slack, so that groups leave no
    // short remainder items (their partials and their reduction cost more
    // than their steps: hybrid-lm's groups of ~512 steps stay whole).
    const size_t groups = (size_t)H * K;
    const size_t gs = (total + groups - 1) / groups;            // average group size
    const size_t P0 = (total + 2047) / 2048;
    size_t m = (gs + P0 / 2) / P0;
    if (m < 1) m = 1;
    size_t P = (gs * 6 / 5 + m - 1) / m;
    const size_t Pmem = (2 * total * cell + (1u << 28) - 1) >> 28;  // partials <= 256 MiB
    if (P < Pmem) P = Pmem;
    if (P < 64) P = 64;
    P = (P + 63) & ~(size_t)63;
    p.P = (int)P;
    // a group of n > P steps has ceil(n/P) <= 2n/P items; others have at most one
    p.max_slots = (int)(2 * total / P);
    p.max_items = (int)((total + P - 1) / P + (size_t)H * K);
    size_t o = 0;
    p.off_order = o; o = align256(o + total * 4);
    p.off_hist = o; o = align256(o + (size_t)H * p.S * K * 4);
    p.off_n = o; o = align256(o + (size_t)H * K * 4);
    p.off_pos = o; o = align256(o + (size_t)H * K * 4);
    p.off_item = o; o = align256(o + ((size_t)H * K + 1) * 4);
    p.off_slot = o; o = align256(o + (size_t)H * K * 4);
    p.off_partial = o; o = align256(o + (size_t)p.max_slots * cell);
    p.bytes = o;
    return p;
}

struct SteGradArgs {
    int B, L, H, N, K;
    const int* idx;    // [B,L,H]
    const int* pi;     // [H,K,N] (scores only)
    int io;            // row format of g: kIoC64, kIoReal (real fp32; z too) or kIoBf16 (bf16
                       // pairs; z complex64), pdssm_io.h
    const float2* g;   // [B,L,H,N] gradient reaching h_t (db of the backward)
    const float2* z;   // [B,L,H,N] D_t .* h_{t-1}
    float* q;          // [B,L,H,K] scores of every map, or null
    float* G;          // [H,K,N,N] or null
    DictPlan plan;
    unsigned char* ws;
    int* status;
};

// Each returns hipSuccess or the launch error.
hipError_t launch_fwd_chunked(const ScanArgs& a, hipStream_t s);
hipError_t launch_bwd_chunked(const ScanArgs& a, hipStream_t s);
hipError_t launch_compose(const ComposeArgs& a, hipStream_t s);
hipError_t launch_ste_grads(const SteGradArgs& a, hipStream_t s);
// gx = s .* (gy - <s, gy>) * inv_temp along the middle axis of [outer, len, inner],
// s = softmax(x * inv_temp).
hipError_t launch_softmax_vjp(const float* x, const float* gy, float* gx, int64_t outer, int len,
                              int64_t inner, float inv_temp, hipStream_t s);

// LDS bytes the chunked backward's emit kernel needs per workgroup: tau + 1
// states and an exchange row of N + 1 entries.
inline size_t bwd_emit_lds_bytes(int N, int tau) { return ((size_t)(tau + 1) * N + N + 1) * 8; }
constexpr size_t kMaxLdsPerGroup = 65536;

}  // namespace pdssm
