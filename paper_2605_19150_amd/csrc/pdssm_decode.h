// pdssm_decode.h -- host-side launch interface of the single-step decode
// kernel (pdssm_decode.hip).  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>

namespace pdssm {

// One recurrence step per (batch, head) sequence (token-by-token decode).
struct DecodeArgs {
    int B, H, N, K;
    const int* idx;      // [B,H]
    const int* pi;       // [H,K,N]
    const float2* D;     // [B,H,N]
    const float2* b;
    const float2* c;
    const float2* h_in;  // [B,H,N] or null (zero state)
    float2* h_out;       // [B,H,N], may equal h_in
    float* y;            // [B,H]
    int* status;
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t s);

}  // namespace pdssm
