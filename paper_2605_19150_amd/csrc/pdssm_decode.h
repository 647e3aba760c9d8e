// pdssm_decode.h -- host-side launch interface of the single-step decode
// kernel (pdssm_decode.hip).  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>

namespace pdssm {

// One recurrence step per (batch, head) sequence (token-by-token decode).
struct DecodeArgs {
    int B, H, N, K;
    int io;              // row format of D, b, c (kIoC64, kIoBf16, kIoReal: pdssm_io.h)
    const int* idx;      // [B,H]
    const int* pi;       // [H,K,N]
    const void* D;       // [B,H,N] in the row format
    const void* b;
    const void* c;
    const float2* h_in;  // [B,H,N] or null (zero state)
    float2* h_out;       // [B,H,N], may equal h_in
    float* y;            // [B,H]
    int* status;
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t s);

}  // namespace pdssm
