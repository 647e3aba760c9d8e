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

// The token projections of a layer in one product on the matrix cores:
// routing logits and choices as launch_route (S non-null), and up to three
// per-head complex projections P = u W^T of weights W [H*2N, Dm] bf16 (rows
// 2n, 2n+1 = real and imaginary part of entry n), written as [T, H*2N]
// floats = [T, H, N] complex: b and c as they are, the diagonal generator as
// sigmoid(P[2n]) exp(i P[2n+1]).  Dm a multiple of 32.
enum ProjKind { kProjPlain = 0, kProjGen = 1 };
struct ProjectArgs {
    int T, Dm, H, K, N;
    const uint16_t* u;      // [T, Dm] bf16
    const uint16_t* S;      // [H*K, Dm] bf16, or null (no routing tiles)
    float* logits;          // [T, H*K] or null
    int* idx;               // [T, H] (when S)
    int nproj;              // projections present (0..3), in order
    const uint16_t* W[3];   // their weights [H*2N, Dm]
    float* out[3];          // their outputs [T, H*2N]
    int kind[3];            // kProjPlain (b, c) or kProjGen (the diagonal generator)
};

hipError_t launch_project(const ProjectArgs& a, hipStream_t s);
// pi[g, j] = first argmax_i M[g, i, j] for g < HK (M: [HK, N, N]).
hipError_t launch_dict_argmax(const float* M, int* pi, int HK, int N, hipStream_t s);

}  // namespace pdssm
