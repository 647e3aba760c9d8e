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

// ------------------------------------------------------------------ k_project_dma
// The routing product -- and the token projections b, c and the diagonal
// generator, as further column tiles of the same product -- for contraction
// sizes that are a multiple of 32, with
// direct buffer-to-LDS loads (buffer_load_dwordx4 ... lds: every lane of a
// wave moves 16 bytes to LDS at a wave-uniform base + 16 * lane), so that
// several slices are in flight without holding them in registers.  Rows past
// the end of u or S lie past their buffer descriptors and read as 0.
//
// A workgroup computes BM tokens x 256 columns (whole heads) with eight
// waves in a WGM x WGN grid.  The contraction goes in slices of 32 through
// NS = 4 LDS stages: while slice s is multiplied, slices s+1 .. s+3 are
// loading.  A stage holds BM rows of u, then 256 rows of S, 64 bytes of each;
// every 16 consecutive rows form a 1 KB block laid out chunk-major (byte
// (r/16)*1024 + c*256 + (r%16)*16 for row r, 16-byte chunk c), which is
// exactly what one wave-wide load instruction writes (lane l: row l%16, chunk
// l/16) and makes the operand reads (32 rows at one chunk) conflict-free.
// (Measured: loads of half cache lines, as here, reach about half the L2 rate
// of full ones, and the slices' loads set the pace of the kernel.)
//
// Tiles are numbered so that each XCD (workgroups are dealt round-robin over
// the 8 XCDs) takes a contiguous range, all column tiles of a few token tiles
// at a time: u streams from HBM once and the rows of S are shared in L2.
typedef __attribute__((address_space(3))) void* lds_void_t;

// One wave-wide 16-byte-per-lane load from a buffer into LDS at dst + 16*lane.
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, unsigned char* dst, uint32_t voff,
                                           uint32_t soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t)dst, 16, voff, soff, 0, 0);
}

template <int BM>
struct RouteDma {
    static constexpr int BN = 256, BK = 32, NS = 4, NW = 8;
    static constexpr int WGM = BM / 64, WGN = NW / WGM;  // wave grid: 64-row blocks of the tile
    static constexpr int TM = BM / WGM, TN = BN / WGN;   // a wave's block
    static constexpr int WM = TM / 32, WN = TN / 32;     // its 32 x 32 products
    static constexpr int ROWS = BM + BN;                 // rows of a stage
    static constexpr int STAGE = ROWS * BK * 2;          // bytes of a stage
    static constexpr int PER_WAVE = ROWS / 16 / NW;      // load instructions per wave per stage
    // epilogue tile pitch (floats): 16-byte aligned rows; 16 consecutive rows
    // start in distinct 16-byte bank groups
    static constexpr int PITCH = BN + 4;
    static constexpr size_t kStages = (size_t)NS * STAGE, kTile = (size_t)BM / 2 * PITCH * 4;
    static constexpr size_t LDS = kStages > kTile ? kStages : kTile;
    static_assert(ROWS % (16 * NW) == 0, "whole blocks per wave");
    static_assert(WGM * WGN == NW && TM == 64, "wave grid");
    static_assert(LDS <= 160 * 1024, "fits the LDS of a CU");
};

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier without the memory fence of __syncthreads, whose release
// half would wait for every outstanding load, the later slices' included.
// The loads a slice needs are waited for explicitly before it; the compiler
// fences keep LDS accesses on their side of the barrier.
__device__ __forceinline__ void barrier_no_fence() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Column tiles of the product: first the routing tiles (whole heads of K
// columns, 256 / K heads each), then for each projection its rows of
// H*2N in tiles of 256.  All scalar.
struct ColTile {
    int kind;   // -1: routing; else the projection's index
    int r0;     // first weight row of the tile
    int ncol;   // valid columns
    int h0, nh; // routing: first head, heads
};

__device__ __forceinline__ ColTile col_tile(const ProjectArgs& a, int nt, int BN) {
    ColTile c;
    const int hpb = a.S ? BN / a.K : 1;
    const int NTr = a.S ? (a.H + hpb - 1) / hpb : 0;
    if (nt < NTr) {
        c.kind = -1;
        c.h0 = nt * hpb;
        c.nh = min(hpb, a.H - c.h0);
        c.r0 = c.h0 * a.K;
        c.ncol = c.nh * a.K;
    } else {
        const int R = 2 * a.H * a.N, NTp = (R + BN - 1) / BN;
        const int j = nt - NTr;
        c.kind = j / NTp;
        c.r0 = (j - c.kind * NTp) * BN;
        c.ncol = min(BN, R - c.r0);
        c.h0 = c.nh = 0;
    }
    return c;
}

__device__ __forceinline__ int col_tiles(const ProjectArgs& a, int BN) {
    const int hpb = a.S ? BN / a.K : 1;
    const int NTr = a.S ? (a.H + hpb - 1) / hpb : 0;
    const int R = 2 * a.H * a.N;
    return NTr + a.nproj * ((R + BN - 1) / BN);
}

// D = sigmoid(m) exp(i p): the diagonal generator of one entry from its two
// projected values (magnitude logit m, phase p).
__device__ __forceinline__ float2 diag_gen(float m, float p) {
    const float r = 1.f / (1.f + expf(-m));
    float s, c;
    sincosf(p, &s, &c);
    return make_float2(r * c, r * s);
}

template <int BM>
__global__ __launch_bounds__(512) void k_project_dma(ProjectArgs a) {
    using C = RouteDma<BM>;
    constexpr int NT_ = C::NW * 64;
    extern __shared__ __align__(16) unsigned char lds[];
    // wave-uniform in a scalar register: the load instructions' LDS base and
    // descriptor depend on it
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int wm = wv / C::WGN, wn = wv % C::WGN;
    const int NT = col_tiles(a, C::BN), MT = (a.T + BM - 1) / BM;
    const int total = NT * MT;
    int t = blockIdx.x;
    if (total % 8 == 0) t = (t % 8) * (total / 8) + t / 8;
    const int nt = t % NT, mt = t / NT;
    const ColTile ct = col_tile(a, nt, C::BN);
    const int ncol = ct.ncol;
    const int m0 = mt * BM;
    const int HK = a.H * a.K;
    const int R = 2 * a.H * a.N;

    // this lane's byte offset of each of its load instructions: row
    // (wv * PER_WAVE + i) * 16 + lane % 16 of the stage, chunk lane / 16
    const uint32_t row_bytes = (uint32_t)a.Dm * 2;
    const __amdgpu_buffer_rsrc_t ru = row_block(a.u, (uint32_t)a.T * row_bytes);
    const __amdgpu_buffer_rsrc_t rs =
        ct.kind < 0 ? row_block(a.S, (uint32_t)HK * row_bytes) : row_block(a.W[ct.kind], (uint32_t)R * row_bytes);
    uint32_t voff[C::PER_WAVE];
#pragma unroll
    for (int i = 0; i < C::PER_WAVE; ++i) {
        const int row = (wv * C::PER_WAVE + i) * 16 + (lane & 15);
        const uint32_t r = row < BM ? (uint32_t)(m0 + row) : (uint32_t)(ct.r0 + row - BM);
        voff[i] = r * row_bytes + 16u * (uint32_t)(lane >> 4);
    }
    auto issue = [&](int s) {
        unsigned char* st = lds + (s % C::NS) * C::STAGE;
        const uint32_t so = (uint32_t)s * C::BK * 2;
#pragma unroll
        for (int i = 0; i < C::PER_WAVE; ++i)
            load_lds16((wv * C::PER_WAVE + i) * 16 >= BM ? rs : ru, st + (wv * C::PER_WAVE + i) * 1024, voff[i], so);
    };

    f32x16 acc[C::WM][C::WN];
#pragma unroll
    for (int i = 0; i < C::WM; ++i)
#pragma unroll
        for (int j = 0; j < C::WN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int c0 = wn * C::TN;     // this wave's first column of the tile
    const bool work = c0 < ncol;  // a wave past the tile's columns multiplies zeros and stores nothing
    const int ra = wm * C::TM + (lane & 31);  // operand rows: A tile i at ra + 32 i
    const int rb = BM + c0 + (lane & 31);     // B tile j at rb + 32 j
    auto off = [](int r, int c) { return (r >> 4) * 1024 + c * 256 + (r & 15) * 16; };
    // every operand read of a slice is issued before its first product, so
    // the reads of the second half of the slice overlap the products of the first
    auto compute = [&](int s) {
        const unsigned char* st = lds + (s % C::NS) * C::STAGE;
        bf16x8 A[2][C::WM], B[2][C::WN];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int c = 2 * kk + (lane >> 5);
#pragma unroll
            for (int i = 0; i < C::WM; ++i) A[kk][i] = *reinterpret_cast<const bf16x8*>(st + off(ra + 32 * i, c));
#pragma unroll
            for (int j = 0; j < C::WN; ++j) B[kk][j] = *reinterpret_cast<const bf16x8*>(st + off(rb + 32 * j, c));
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int i = 0; i < C::WM; ++i)
#pragma unroll
                for (int j = 0; j < C::WN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[kk][i], B[kk][j], acc[i][j], 0, 0, 0);
    };

    const int nsl = a.Dm / C::BK;
#pragma unroll
    for (int s = 0; s < C::NS - 1; ++s)
        if (s < nsl) issue(s);
    for (int s = 0; s < nsl; ++s) {
        // this wave's loads of slice s are done once at most the later issued slices are outstanding
        const int ahead = min(C::NS - 2, nsl - 1 - s);
        if (ahead >= 2) wait_vmcnt<2 * C::PER_WAVE>();
        else if (ahead == 1) wait_vmcnt<C::PER_WAVE>();
        else wait_vmcnt<0>();
        barrier_no_fence();  // every wave's slice s is in LDS; every wave is done with slice s-1
        if (s + C::NS - 1 < nsl) issue(s + C::NS - 1);  // into slice s-1's stage
        compute(s);
    }
    __syncthreads();  // the stages are free for the epilogue tile

    float* tile = reinterpret_cast<float*>(lds);
    constexpr int HALF = BM / 2;
    // 16-byte logits stores and argmax reads when K % 4 == 0 (then every head,
    // every tile and every output row starts on a 16-byte boundary)
    const bool vec = a.K % 4 == 0;
    for (int half = 0; half < 2; ++half) {
        if (half) __syncthreads();  // the first half's readers are done
        const int rlo = wm * C::TM - half * HALF;  // this wave's first row within the half
        if (rlo >= 0 && rlo < HALF && work) {
#pragma unroll
            for (int i = 0; i < C::WM; ++i)
#pragma unroll
                for (int j = 0; j < C::WN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        tile[(rlo + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * C::PITCH + c0 + 32 * j +
                             (lane & 31)] = acc[i][j][r];
        }
        __syncthreads();
        const int mb = m0 + half * HALF;
        const int nm = max(0, min(HALF, a.T - mb));
        if (ct.kind >= 0) {
            // a projection: rows of [T, H*2N] floats; R, r0 and ncol are
            // multiples of 4 (2N >= 16), so every row piece is 16-byte aligned
            float* orow = a.out[ct.kind] + (size_t)mb * R + ct.r0;
            const int nq = ncol / 4;
            const bool gen = a.kind[ct.kind] == kProjGen;
            for (int e = threadIdx.x; e < nm * nq; e += NT_) {
                const int m = e / nq, q = e - m * nq;
                float4 v = *reinterpret_cast<const float4*>(tile + m * C::PITCH + 4 * q);
                if (gen) {
                    const float2 d0 = diag_gen(v.x, v.y), d1 = diag_gen(v.z, v.w);
                    v = make_float4(d0.x, d0.y, d1.x, d1.y);
                }
                *reinterpret_cast<float4*>(orow + (size_t)m * R + 4 * q) = v;
            }
            continue;
        }
        float* lrow = a.logits ? a.logits + (size_t)mb * HK + (size_t)ct.h0 * a.K : nullptr;  // row mb, first column
        if (vec) {
            const int nq = ncol / 4;
            if (lrow)
                for (int e = threadIdx.x; e < nm * nq; e += NT_) {
                    const int m = e / nq, q = e - m * nq;
                    *reinterpret_cast<float4*>(lrow + (size_t)m * HK + 4 * q) =
                        *reinterpret_cast<const float4*>(tile + m * C::PITCH + 4 * q);
                }
        } else if (lrow) {
            for (int e = threadIdx.x; e < nm * ncol; e += NT_) {
                const int m = e / ncol, c = e - m * ncol;
                lrow[(size_t)m * HK + c] = tile[m * C::PITCH + c];
            }
        }
        // first maximal index per (token, head); neighbouring lanes take
        // neighbouring tokens
        for (int e = threadIdx.x; e < HALF * ct.nh; e += NT_) {
            const int m = e % HALF, hh = e / HALF;
            if (m >= nm) continue;
            const float* v = tile + m * C::PITCH + hh * a.K;
            int best = 0;
            float bv = v[0];
            if (vec) {
                for (int q = 0; q < a.K / 4; ++q) {
                    const float4 x = reinterpret_cast<const float4*>(v)[q];
                    if (x.x > bv) bv = x.x, best = 4 * q;
                    if (x.y > bv) bv = x.y, best = 4 * q + 1;
                    if (x.z > bv) bv = x.z, best = 4 * q + 2;
                    if (x.w > bv) bv = x.w, best = 4 * q + 3;
                }
            } else {
                for (int k = 1; k < a.K; ++k)
                    if (v[k] > bv) bv = v[k], best = k;
            }
            a.idx[(size_t)(mb + m) * a.H + ct.h0 + hh] = best;
        }
    }
}

template <int BM>
hipError_t project_dma_launch(const ProjectArgs& a, hipStream_t st) {
    using C = RouteDma<BM>;
    const int hpb = a.S ? C::BN / a.K : 1;
    const int NT = (a.S ? (a.H + hpb - 1) / hpb : 0) + a.nproj * ((2 * a.H * a.N + C::BN - 1) / C::BN);
    const int MT = (a.T + BM - 1) / BM;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_project_dma<BM>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::LDS);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_project_dma<BM>, dim3((unsigned)(NT * MT)), dim3(C::NW * 64), C::LDS, st, a);
    return hipGetLastError();
}

// 256-token tiles when they still give every CU two of them
hipError_t project_dma(const ProjectArgs& a, hipStream_t st) {
    const int hpb = a.S ? 256 / a.K : 1;
    const long long NT = (a.S ? (a.H + hpb - 1) / hpb : 0) + (long long)a.nproj * ((2LL * a.H * a.N + 255) / 256);
    const long long tiles256 = (long long)((a.T + 255) / 256) * NT;
    return tiles256 >= 512 ? project_dma_launch<256>(a, st) : project_dma_launch<128>(a, st);
}

// pi[h,k,j] = argmax_i M[h,k,i,j].  A workgroup takes 64 columns of one
// matrix (h,k) (loads coalesced over j); its four waves each scan a quarter
// of the rows with eight loads in flight, and wave 0 combines the quarters in
// row order, so the first maximal row wins as in a single pass.
constexpr int kArgCols = 64;
__global__ __launch_bounds__(256) void k_dict_argmax(const float* __restrict__ M, int* __restrict__ pi, int HK,
                                                     int N) {
    __shared__ float sv[4][kArgCols];
    __shared__ int si[4][kArgCols];
    const int lane = threadIdx.x & 63, part = threadIdx.x >> 6;
    const int per = (N + kArgCols - 1) / kArgCols;  // column blocks per matrix
    const int g = blockIdx.x / per;
    const int j = (blockIdx.x - g * per) * kArgCols + lane;
    const bool on = g < HK && j < N;
    const int rows = N / 4;  // N is a power of two >= 8
    const int i0 = part * rows;
    const float* col = M + ((size_t)(on ? g : 0) * N + i0) * N + (on ? j : 0);
    int best = i0;
    float bv = col[0];
#pragma unroll 8
    for (int i = 1; i < rows; ++i) {
        const float v = col[(size_t)i * N];
        if (v > bv) bv = v, best = i0 + i;
    }
    sv[part][lane] = bv;
    si[part][lane] = best;
    __syncthreads();
    if (part == 0 && on) {
#pragma unroll
        for (int q = 1; q < 4; ++q)
            if (sv[q][lane] > bv) bv = sv[q][lane], best = si[q][lane];
        pi[(size_t)g * N + j] = best;
    }
}

}  // namespace

// byte offsets of the direct-load kernel are 32-bit, rows past the end included
bool project_fits(long long T, long long rows, long long Dm) {
    return (T + 256) * Dm * 2 < (1LL << 32) && (rows + 256) * Dm * 2 < (1LL << 32);
}

hipError_t launch_route(const RouteArgs& a, hipStream_t st) {
    if (a.Dm % RouteDma<128>::BK == 0 && project_fits(a.T, (long long)a.H * a.K, a.Dm)) {
        ProjectArgs p = {};
        p.T = a.T;
        p.Dm = a.Dm;
        p.H = a.H;
        p.K = a.K;
        p.N = 8;
        p.u = a.u;
        p.S = a.S;
        p.logits = a.logits;
        p.idx = a.idx;
        p.nproj = 0;
        return project_dma(p, st);
    }
    const int hpb = kRouteTN / a.K;
    dim3 grid((a.T + kRouteTM - 1) / kRouteTM, (a.H + hpb - 1) / hpb);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_route),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kRouteLds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_route, grid, dim3(256), kRouteLds, st, a);
    return hipGetLastError();
}

hipError_t launch_project(const ProjectArgs& a, hipStream_t st) {
    const long long rows = a.S ? (long long)a.H * a.K : 0;
    if (a.Dm % RouteDma<128>::BK != 0 || !project_fits(a.T, rows > 2LL * a.H * a.N ? rows : 2LL * a.H * a.N, a.Dm))
        return hipErrorInvalidValue;
    return project_dma(a, st);
}

hipError_t launch_dict_argmax(const float* M, int* pi, int HK, int N, hipStream_t st) {
    const int64_t blocks = (int64_t)HK * ((N + kArgCols - 1) / kArgCols);
    hipLaunchKernelGGL(k_dict_argmax, dim3((unsigned)blocks), dim3(256), 0, st, M, pi, HK, N);
    return hipGetLastError();
}

}  // namespace pdssm
