// pdssm_select.h -- host-side launch interface of the selection front end
// (pdssm_select.hip).  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pdssm {

// Routing: logits[t, h*K + k] = sum_d u[t,d] S[h*K + k, d] (bf16 operands,
// fp32 result), idx[t, h] = first argmax over k.
struct RouteArgs {
    int T, Dm, H, K;       // tokens (B*L), contraction length, heads, maps per head
    const uint16_t* u;     // [T, Dm] bf16
    const uint16_t* S;     // [H*K, Dm] bf16
    float* logits;         // [T, H*K] or null
    int* idx;              // [T, H]
};

hipError_t launch_route(const RouteArgs& a, hipStream_t s);
// pi[g, j] = first argmax_i M[g, i, j] for g < HK (M: [HK, N, N]).
hipError_t launch_dict_argmax(const float* M, int* pi, int HK, int N, hipStream_t s);

}  // namespace pdssm
