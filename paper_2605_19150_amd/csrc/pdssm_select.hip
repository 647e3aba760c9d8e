// pdssm_select.hip -- the selection front end of the scan (Sec. 3.1 eqs. (5)-(8),
// App. E.2.1):
//
//   maps      pi[h,k,j] = argmax_i M[h,k,i,j]   (column argmax of the dense
//                                                dictionary, once per step of
//                                                the optimizer)
//   routing   logits[t,h,k] = sum_d u[t,d] S[h,k,d],   idx[t,h] = argmax_k logits[t,h,k]
//
// Ties go to the first maximal index (numpy's and torch's rule).
//
// k_route: the routing product on the matrix cores (v_mfma_f32_32x32x16_bf16:
// bf16 operands, fp32 accumulation) with the argmax fused into the epilogue.
// A workgroup computes a 128-token x (whole heads, at most 256 columns)
// tile: four waves own 64 x 128 blocks (2 x 4 tiles of 32 x 32).  The
// contraction goes in slices of 64, copied by the workgroup into LDS (two
// stages: the next slice's global loads run while the current one is
// multiplied).  The fp32 tile then goes to LDS in two halves, from where it is
// written out coalesced and each (token, head) takes its argmax, so the
// logits are read back from nowhere.
#include "pdssm_device.h"
#include "pdssm_select.h"

namespace pdssm {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kRouteTM = 128;  // tokens per workgroup
constexpr int kRouteTN = 256;  // column capacity per workgroup (whole heads)
constexpr int kRouteKS = 64;   // contraction slice staged in LDS (one 128-byte line per row)
constexpr int kRoutePitch = kRouteKS + 8;  // padded LDS row (bf16): 16-byte reads without bank conflicts
constexpr int kRouteStageElems = (kRouteTM + kRouteTN) * kRoutePitch;
// two stages of bf16; the epilogue tile (half the tokens, fp32) aliases them
constexpr size_t kRouteStages = 2 * kRouteStageElems * 2, kRouteTile = (size_t)kRouteTM / 2 * kRouteTN * 4;
constexpr size_t kRouteLds = kRouteStages > kRouteTile ? kRouteStages : kRouteTile;

// Lane layout of v_mfma_f32_32x32x16_bf16: lane l supplies A[l%32][8(l/32) .. 8(l/32)+7]
// and B[8(l/32) .. +7][l%32]; accumulator element r of lane l is
// C[8(r/4) + 4(l/32) + r%4][l%32].
// Waves form a 2 x 2 grid of 64-token x 128-column blocks.  Each slice of 64
// of the contraction is copied by the whole workgroup from global memory
// (coalesced 16-byte chunks, rows past the tensor clamped, chunks past the
// contraction zero) into one of two LDS stages while the other stage is
// multiplied; one barrier per slice.
__global__ __launch_bounds__(256) void k_route(RouteArgs a) {
    extern __shared__ __align__(16) unsigned char lds[];
    uint16_t* stage_base = reinterpret_cast<uint16_t*>(lds);
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wv >> 1, wn = wv & 1;
    const int hpb = kRouteTN / a.K;              // heads per workgroup
    const int h0 = blockIdx.y * hpb;
    const int nh = min(hpb, a.H - h0);
    const int ncol = nh * a.K;                   // valid columns of this tile
    const int m0 = blockIdx.x * kRouteTM;
    const int HK = a.H * a.K;

    f32x16 acc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // copy plan: the stage holds kRouteTM rows of u then kRouteTN rows of S,
    // kRouteKS/8 chunks of 16 bytes per row; thread t takes chunks t, t + 256, ...
    constexpr int kCpr = kRouteKS / 8;
    constexpr int kChunks = (kRouteTM + kRouteTN) * kCpr;
    constexpr int kPer = kChunks / 256;
    static_assert(kChunks % 256 == 0, "whole chunks per thread");
    const uint16_t* src[kPer];
    int dst[kPer], col[kPer];
#pragma unroll
    for (int c = 0; c < kPer; ++c) {
        const int e = threadIdx.x + 256 * c;
        const int row = e / kCpr, ch = e % kCpr;
        col[c] = 8 * ch;
        dst[c] = row * kRoutePitch + 8 * ch;
        if (row < kRouteTM) {
            src[c] = a.u + (size_t)min(m0 + row, a.T - 1) * a.Dm;
        } else {
            const int n = min(row - kRouteTM, ncol - 1);
            src[c] = a.S + ((size_t)h0 * a.K + n) * a.Dm;
        }
    }
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    u32x4 reg[kPer];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int c = 0; c < kPer; ++c) {
            const int k = k0 + col[c];
            reg[c] = k < a.Dm ? *reinterpret_cast<const u32x4*>(src[c] + k) : u32x4{0, 0, 0, 0};
        }
    };
    auto store = [&](int st) {
        uint16_t* base = stage_base + st * kRouteStageElems;
#pragma unroll
        for (int c = 0; c < kPer; ++c) *reinterpret_cast<u32x4*>(base + dst[c]) = reg[c];
    };

    const int nslice = (a.Dm + kRouteKS - 1) / kRouteKS;
    const int c0 = wn * 128;  // this wave's first column of the tile
    const bool work = c0 < ncol;
    fetch(0);
    store(0);
    __syncthreads();
    const int kl = 8 * (lane >> 5);
    for (int sl = 0; sl < nslice; ++sl) {
        if (sl + 1 < nslice) fetch((sl + 1) * kRouteKS);
        if (work) {
            const uint16_t* As = stage_base + (sl & 1) * kRouteStageElems;
            const uint16_t* Bs = As + kRouteTM * kRoutePitch;
#pragma unroll
            for (int ks = 0; ks < kRouteKS; ks += 16) {
                bf16x8 A[2], B[4];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    A[i] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + 32 * i + (lane & 31)) * kRoutePitch + ks + kl);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    B[j] = *reinterpret_cast<const bf16x8*>(Bs + (c0 + 32 * j + (lane & 31)) * kRoutePitch + ks + kl);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[i], B[j], acc[i][j], 0, 0, 0);
            }
        }
        if (sl + 1 < nslice) store((sl + 1) & 1);
        __syncthreads();
    }

    float(*tile)[kRouteTN] = reinterpret_cast<float(*)[kRouteTN]>(lds);  // aliases the stages
    for (int half = 0; half < 2; ++half) {
        if (half) __syncthreads();  // the first half's readers are done
        if (wm == half && work) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        tile[32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)][c0 + 32 * j + (lane & 31)] =
                            acc[i][j][r];
        }
        __syncthreads();
        const int mb = m0 + half * (kRouteTM / 2);
        const int nm = max(0, min(kRouteTM / 2, a.T - mb));
        // logits: row m of the tile is ncol contiguous floats of the output
        if (a.logits)
            for (int e = threadIdx.x; e < nm * ncol; e += 256) {
                const int m = e / ncol, c = e - m * ncol;
                a.logits[(size_t)(mb + m) * HK + (size_t)h0 * a.K + c] = tile[m][c];
            }
        // argmax per (token, head): first maximal index
        for (int e = threadIdx.x; e < nm * nh; e += 256) {
            const int m = e / nh, hh = e - m * nh;
            const float* v = &tile[m][hh * a.K];
            int best = 0;
            float bv = v[0];
            for (int k = 1; k < a.K; ++k)
                if (v[k] > bv) bv = v[k], best = k;
            a.idx[(size_t)(mb + m) * a.H + h0 + hh] = best;
        }
    }
}

// pi[h,k,j] = argmax_i M[h,k,i,j]: a thread per (h,k,j), loads coalesced over j.
__global__ __launch_bounds__(256) void k_dict_argmax(const float* __restrict__ M, int* __restrict__ pi, int HK,
                                                     int N) {
    const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (id >= (int64_t)HK * N) return;
    const int64_t g = id / N;
    const int j = (int)(id - g * N);
    const float* col = M + (size_t)g * N * N + j;
    int best = 0;
    float bv = col[0];
    for (int i = 1; i < N; ++i) {
        const float v = col[(size_t)i * N];
        if (v > bv) bv = v, best = i;
    }
    pi[id] = best;
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t st) {
    const int hpb = kRouteTN / a.K;
    dim3 grid((a.T + kRouteTM - 1) / kRouteTM, (a.H + hpb - 1) / hpb);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_route),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kRouteLds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_route, grid, dim3(256), kRouteLds, st, a);
    return hipGetLastError();
}

hipError_t launch_dict_argmax(const float* M, int* pi, int HK, int N, hipStream_t st) {
    const int64_t n = (int64_t)HK * N;
    hipLaunchKernelGGL(k_dict_argmax, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, M, pi, HK, N);
    return hipGetLastError();
}

}  // namespace pdssm
