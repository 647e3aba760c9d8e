// pdssm_ste.hip -- straight-through surrogate gradients for gfx950 (Sec. 3.1
// Prop. 2 and its derivation in the appendix).
//
// The backward scan emits, per step, the gradient g_t reaching h_t (db) and,
// when asked, the scaled state z_t = D_t .* h_{t-1}.  This file holds what
// follows from them:
//
//   dictionary gradient  G[h,k] = sum over the steps (b,t) with
//                        idx[b,t,h] == k of Re(g_t z_t^H)   (an N x N matrix)
//     k_dict_hist     per (head, segment of steps): how many steps chose each map
//     k_dict_plan     one workgroup: per group (h,k) its step count, its first
//                     position in the grouped order, its first item and, for
//                     groups of several items, its first partial slot; per
//                     (head, segment, map) the segment's first position
//     k_dict_scatter  per (head, segment): step ids into the grouped order,
//                     stable (ranks from ballots over the key bits)
//     k_ste_gemm      per item (at most P steps of one group): the sum of the
//                     steps' outer products on the matrix cores,
//                     v_mfma_f32_32x32x2f32 with the contraction pair
//                     (re, im): Re(g_i conj(z_j)) = g_i.re z_j.re + g_i.im z_j.im;
//                     and, from the same g and z rows staged transposed in
//                     LDS (lane = step), the scores
//                     q_t[k] = sum_j Re(g_t[pi_k(j)] conj(z_t[j])) of every
//                     map at each of its steps
//     k_dict_reduce   groups of several items: their partials added in item
//                     order; groups no step chose: zeros
//   tempered softmax    gx = s .* (gy - <s, gy>) / temp along one axis,
//                     s = softmax(x / temp) -- the backward stand-in for a hard
//                     argmax -- in two passes with an online (max, sums)
//                     state: k_softmax_rows for a contiguous axis (routing
//                     logits over k), k_softmax_cols / k_softmax_cols4 for a
//                     strided one (down each column of the dense dictionary
//                     M[h,k]).
//
// Every sum runs in a fixed order, so the results do not change from run to run.
#include "pdssm_device.h"
#include "pdssm_internal.h"

namespace pdssm {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x32 __attribute__((ext_vector_type(32)));

struct SteWs {
    int* order;      // [B*L*H] step ids u = b*L + t, grouped by (head, map)
    int* hist;       // [H][S][K] step counts; k_dict_plan turns them into each
                     // segment's first position in the grouped order
    int* n;          // [H*K] steps per group
    int* pos;        // [H*K] first position of the group in order
    int* item;       // [H*K + 1] first item of the group; item[H*K] = number of items
    int* slot;       // [H*K] first partial slot (groups of several items), else -1
    float* partial;  // [max_slots][N*N]
};

__device__ __forceinline__ SteWs ste_ws(const SteGradArgs& a) {
    SteWs w;
    w.order = reinterpret_cast<int*>(a.ws + a.plan.off_order);
    w.hist = reinterpret_cast<int*>(a.ws + a.plan.off_hist);
    w.n = reinterpret_cast<int*>(a.ws + a.plan.off_n);
    w.pos = reinterpret_cast<int*>(a.ws + a.plan.off_pos);
    w.item = reinterpret_cast<int*>(a.ws + a.plan.off_item);
    w.slot = reinterpret_cast<int*>(a.ws + a.plan.off_slot);
    w.partial = reinterpret_cast<float*>(a.ws + a.plan.off_partial);
    return w;
}

// An idx entry outside [0,K) counts as map 0 (and is reported) so that every
// access stays in bounds; the histogram and the scatter treat it alike.
__device__ __forceinline__ int map_key(int k, int K, bool& bad) {
    const bool b = (unsigned)k >= (unsigned)K;
    bad |= b;
    return b ? 0 : k;
}

// ------------------------------------------------------------------ grouping
// Block x = h * S + segment: steps u in [segment*seg, min(+seg, B*L)).  Each
// thread reads its steps' indices in batches of 8 independent loads.
__global__ __launch_bounds__(256) void k_dict_hist(SteGradArgs a) {
    constexpr int UB = 8;
    __shared__ int cnt[256];
    const int h = blockIdx.x / a.plan.S, sg = blockIdx.x - h * a.plan.S;
    for (int k = threadIdx.x; k < a.K; k += 256) cnt[k] = 0;
    __syncthreads();
    const long BL = (long)a.B * a.L;
    const long u0 = (long)sg * a.plan.seg, u1 = min(u0 + (long)a.plan.seg, BL);
    bool bad = false;
    for (long ub = u0 + threadIdx.x; ub < u1; ub += 256 * UB) {
        int v[UB];
#pragma unroll
        for (int e = 0; e < UB; ++e) {
            const long u = ub + (long)e * 256;
            v[e] = u < u1 ? a.idx[u * a.H + h] : 0;
        }
#pragma unroll
        for (int e = 0; e < UB; ++e)
            if (ub + (long)e * 256 < u1) atomicAdd(&cnt[map_key(v[e], a.K, bad)], 1);
    }
    __syncthreads();
    const SteWs w = ste_ws(a);
    for (int k = threadIdx.x; k < a.K; k += 256) w.hist[((size_t)h * a.plan.S + sg) * a.K + k] = cnt[k];
    if (bad) report_index_error(a.status);
}

// One workgroup: exclusive prefix sums over the groups gi = h*K + k of their
// step counts (positions; head h starts at h*B*L), item counts and partial
// slots.  Thread t owns a contiguous range of groups.  Last, each segment
// count in hist is replaced by the segment's first position in the grouped
// order (the group's position plus the counts of its earlier segments).  The
// counts are first copied into LDS when they fit (the plan keeps H*S*K at
// most kDictPlanLds), so that the walks down the segments read LDS.
__global__ __launch_bounds__(1024) void k_dict_plan(SteGradArgs a) {
    constexpr int T = 1024, SB = 16;
    __shared__ int sh[3][T / 64];
    __shared__ int hs[kDictPlanLds];
    const SteWs w = ste_ws(a);
    const int HK = a.H * a.K, t = threadIdx.x, P = a.plan.P, S = a.plan.S;
    const int nh = HK * S;
    const bool in_lds = nh <= kDictPlanLds;
    if (in_lds) {
#pragma unroll 4
        for (int e = t; e < nh; e += T) hs[e] = w.hist[e];
        __syncthreads();
    }
    auto count = [&](size_t e) { return in_lds ? hs[e] : w.hist[e]; };
    const int per = (HK + T - 1) / T;
    const int g0 = min(t * per, HK), g1 = min(g0 + per, HK);
    // entry of segment sg of group gi in hist
    auto at = [&](int gi, int sg) {
        const int h = gi / a.K, k = gi - h * a.K;
        return ((size_t)h * S + sg) * a.K + k;
    };
    int sn = 0, si = 0, ss = 0;
    for (int gi = g0; gi < g1; ++gi) {
        int n = 0;
        for (int s0 = 0; s0 < S; s0 += SB) {
            int c[SB];
#pragma unroll
            for (int e = 0; e < SB; ++e) c[e] = s0 + e < S ? count(at(gi, s0 + e)) : 0;
#pragma unroll
            for (int e = 0; e < SB; ++e) n += c[e];
        }
        w.n[gi] = n;
        const int pieces = (n + P - 1) / P;
        sn += n;
        si += pieces;
        ss += pieces >= 2 ? pieces : 0;
    }
    // prefix sums over the threads: within each wave by shuffles, then over
    // the waves' totals
    const int lane = t & 63, wv = t >> 6;
    int x0 = sn, x1 = si, x2 = ss;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int y0 = __shfl_up(x0, d), y1 = __shfl_up(x1, d), y2 = __shfl_up(x2, d);
        if (lane >= d) {
            x0 += y0;
            x1 += y1;
            x2 += y2;
        }
    }
    if (lane == 63) {
        sh[0][wv] = x0;
        sh[1][wv] = x1;
        sh[2][wv] = x2;
    }
    __syncthreads();
    for (int v = 0; v < wv; ++v) {
        x0 += sh[0][v];
        x1 += sh[1][v];
        x2 += sh[2][v];
    }
    int pn = x0 - sn, pi = x1 - si, ps = x2 - ss;
    for (int gi = g0; gi < g1; ++gi) {
        const int n = w.n[gi];
        const int pieces = (n + P - 1) / P;
        w.pos[gi] = pn;
        w.item[gi] = pi;
        w.slot[gi] = pieces >= 2 ? ps : -1;
        int run = pn;
        for (int s0 = 0; s0 < S; s0 += SB) {
            int c[SB];
#pragma unroll
            for (int e = 0; e < SB; ++e) c[e] = s0 + e < S ? count(at(gi, s0 + e)) : 0;
#pragma unroll
            for (int e = 0; e < SB; ++e) {
                if (s0 + e < S) w.hist[at(gi, s0 + e)] = run;
                run += c[e];
            }
        }
        pn += n;
        pi += pieces;
        if (pieces >= 2) ps += pieces;
    }
    if (t == T - 1) w.item[HK] = x1;  // the inclusive total
}

// Block x = h * S + segment.  Tiles of 256 steps in order; within a tile a
// step's rank among the earlier steps with the same map comes from ballots
// over the key bits (wave) and per-wave counts in LDS (tile), so the grouped
// order keeps the steps of each group in increasing u.  The next tile's
// indices are loaded while a tile is ranked.
__global__ __launch_bounds__(256) void k_dict_scatter(SteGradArgs a) {
    __shared__ int base[256];
    __shared__ int wc[4][256];
    const int h = blockIdx.x / a.plan.S, sg = blockIdx.x - h * a.plan.S;
    const int t = threadIdx.x, wv = t >> 6, lane = t & 63;
    const SteWs w = ste_ws(a);
    for (int k = t; k < a.K; k += 256) {
        base[k] = w.hist[((size_t)h * a.plan.S + sg) * a.K + k];  // the segment's first position
        wc[0][k] = wc[1][k] = wc[2][k] = wc[3][k] = 0;
    }
    __syncthreads();
    const long BL = (long)a.B * a.L;
    const long u0 = (long)sg * a.plan.seg, u1 = min(u0 + (long)a.plan.seg, BL);
    int nbits = 0;
    while ((1 << nbits) < a.K) ++nbits;
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    bool bad = false;
    int raw_next = u0 + t < u1 ? a.idx[(u0 + t) * a.H + h] : 0;
    for (long tb = u0; tb < u1; tb += 256) {
        const long u = tb + t;
        const bool valid = u < u1;
        const int raw = raw_next;
        if (u + 256 < u1) raw_next = a.idx[(u + 256) * a.H + h];
        const int key = valid ? map_key(raw, a.K, bad) : 0;
        uint64_t peers = __ballot(valid);
        for (int bit = 0; bit < nbits; ++bit) {
            const bool on = (key >> bit) & 1;
            const uint64_t m = __ballot(on);
            peers &= on ? m : ~m;
        }
        const int rank = __popcll(peers & below);
        if (valid && rank == 0) wc[wv][key] = __popcll(peers);
        __syncthreads();
        if (valid) {
            int p = base[key] + rank;
            for (int w2 = 0; w2 < wv; ++w2) p += wc[w2][key];
            w.order[p] = (int)u;
        }
        __syncthreads();
        for (int k = t; k < a.K; k += 256) {
            base[k] += wc[0][k] + wc[1][k] + wc[2][k] + wc[3][k];
            wc[0][k] = wc[1][k] = wc[2][k] = wc[3][k] = 0;
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ outer products and scores
// An item's steps go in runs of RS steps that every wave of the workgroup
// works on together.
//   Outer products: a wave owns an NB x NB block of G[h,k] (NB = 64: 2 x 2
//   tiles of 32 x 32; NB = 32 for N <= 32, rows and columns past N zero).
//   N <= 64: one block, the four waves take a quarter of each run and add up
//   in LDS at the end; N = 128 / 256: 4 / 16 waves, one block each, every step.
//   Scores: the run's g and z rows are staged in LDS transposed, Gt[i][t] and
//   Zt[j][t] (t = step of the run); lane t then reads Gt[pi_k(j)][t] for every
//   (j, k): all lanes read one row, so the reads are contiguous and free of
//   bank conflicts, and each lane sums its own step (no cross-lane
//   reduction).  The waves split the maps in blocks of 16.
template <int N>
struct DictCfg {
    static constexpr int NB = N >= 64 ? 64 : 32;
    static constexpr int GRID = N >= 64 ? N / 64 : 1;  // blocks per edge
    static constexpr int BLOCKS = GRID * GRID;
    static constexpr int SPLIT = BLOCKS >= 4 ? 1 : 4;
    static constexpr int WAVES = BLOCKS * SPLIT;
    static constexpr int TILES = NB / 32;
    static constexpr int RS = N <= 64 ? 64 : (N == 128 ? 32 : 16);  // steps per run (staged tiles <= ~70 KB)
    static constexpr int SLOTS = 64 / RS;                            // score tasks a wave runs side by side
    static constexpr int MY = RS / SPLIT;                            // steps of a run one wave multiplies
    static constexpr int U = (N >= 256 || N == 64) ? 4 : 8;          // steps per load batch (N = 64: 4 measured 3% faster)
    static constexpr int NBAT = MY / U;                              // load batches per run (even)
    static constexpr int GP = RS + 1;                                // padded tile row (complex entries)
    static constexpr int TILE_BYTES = 2 * N * GP * 8;
    // the cross-wave sum after the loop aliases the tiles
    static constexpr int RED_BYTES = SPLIT > 1 ? (SPLIT - 1) * NB * NB * 4 : 0;
    static_assert(NBAT % 2 == 0 && NBAT >= 2, "runs are processed in pairs of batches");
};

__host__ __device__ inline int score_kp(int K) { return (K + 15) & ~15; }

template <int N>
size_t ste_gemm_lds(int K, bool q) {
    using Cfg = DictCfg<N>;
    const size_t stage = q ? (size_t)Cfg::TILE_BYTES + (size_t)N * score_kp(K) : 0;
    return stage > (size_t)Cfg::RED_BYTES ? stage : (size_t)Cfg::RED_BYTES;
}

// One step's operands: lane l holds g[i0 + l] and z[j0 + l] (NB = 64) or
// g[i0 + l%32], z[j0 + l%32] (NB = 32; lanes past N repeat entry N-1, which
// only reaches rows and columns of the tile past N, never stored).  The loads
// are unconditional (u is always a valid step) so that the compiler's wait
// counts stay exact and the loads of later batches stay in flight.
// Real rows (the real-valued model) widen to (x, 0).
template <int N, int IO>
__device__ __forceinline__ void load_step(const SteGradArgs& a, int u, int h, int i0, int j0, int lane,
                                          float2& gv, float2& zv) {
    constexpr int NB = DictCfg<N>::NB;
    const int r = NB == 64 ? lane : min(lane & 31, N - 1);
    const size_t row = ((size_t)u * a.H + h) * N;
    if constexpr (IO == kIoReal) {
        const float gq = __builtin_nontemporal_load(reinterpret_cast<const float*>(a.g) + row + i0 + r);
        const float zq = __builtin_nontemporal_load(reinterpret_cast<const float*>(a.z) + row + j0 + r);
        gv = make_float2(gq, 0.f);
        zv = make_float2(zq, 0.f);
    } else if constexpr (IO == kIoBf16) {
        // g = db in bf16 (re, im) pairs, widened exactly; z complex64
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const uint32_t gw = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(a.g) + row + i0 + r);
        const f32x2 zq = __builtin_nontemporal_load(reinterpret_cast<const f32x2*>(a.z + row + j0 + r));
        gv = bf2_to_f2(gw);
        zv = make_float2(zq.x, zq.y);
    } else {
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const f32x2 gq = __builtin_nontemporal_load(reinterpret_cast<const f32x2*>(a.g + row + i0 + r));
        const f32x2 zq = __builtin_nontemporal_load(reinterpret_cast<const f32x2*>(a.z + row + j0 + r));
        gv = make_float2(gq.x, gq.y);
        zv = make_float2(zq.x, zq.y);
    }
}

// acc[ti][tj] += A_ti B_tj with A[m][0..1] = (g[m].re, g[m].im) and
// B[0..1][n] = (z[n].re, z[n].im): lane l supplies A[l%32][l/32] and
// B[l/32][l%32].  NB = 64: a permlane32 swap of (re, im) gives both tiles'
// operands: lanes 0-31 keep re of rows 0-31 and get im of rows 0-31 (tile 0),
// and the other half the same for rows 32-63 (tile 1).
template <int N>
__device__ __forceinline__ void mfma_step(f32x16 (&acc)[DictCfg<N>::TILES][DictCfg<N>::TILES], float2 gv, float2 zv,
                                          int lane) {
    if constexpr (DictCfg<N>::NB == 64) {
        const auto ga = __builtin_amdgcn_permlane32_swap(__float_as_uint(gv.x), __float_as_uint(gv.y), false, false);
        const auto zb = __builtin_amdgcn_permlane32_swap(__float_as_uint(zv.x), __float_as_uint(zv.y), false, false);
        const float A[2] = {__uint_as_float(ga[0]), __uint_as_float(ga[1])};
        const float Bv[2] = {__uint_as_float(zb[0]), __uint_as_float(zb[1])};
#pragma unroll
        for (int ti = 0; ti < 2; ++ti)
#pragma unroll
            for (int tj = 0; tj < 2; ++tj)
                acc[ti][tj] = __builtin_amdgcn_mfma_f32_32x32x2f32(A[ti], Bv[tj], acc[ti][tj], 0, 0, 0);
    } else {
        const float A = lane < 32 ? gv.x : gv.y;
        const float Bv = lane < 32 ? zv.x : zv.y;
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(A, Bv, acc[0][0], 0, 0, 0);
    }
}

// Staged score tiles hold complex64 entries, or fp32 for real rows (the
// real model), whose scores then take one multiply-add per gathered entry:
// the complex form's second one, 0 * 0 + v, returns v unchanged (v is never
// -0), so both give the same bits.
template <int IO>
struct TileOf {
    using T = float2;
};
template <>
struct TileOf<kIoReal> {
    using T = float;
};
__device__ __forceinline__ float tile_elem(float2 x, float) { return x.x; }
__device__ __forceinline__ float2 tile_elem(float2 x, float2) { return x; }
__device__ __forceinline__ float score_fma(float g, float z, float v) { return fmaf(g, z, v); }
__device__ __forceinline__ float score_fma(float2 g, float2 z, float v) { return fmaf(g.x, z.x, fmaf(g.y, z.y, v)); }

// Real rows (NB = 64): G += g z^T needs no second contraction term, so one
// v_mfma_f32_32x32x1f32 (two 32 x 32 blocks, K = 1) does the work of two
// tiles.  accR[tj] holds tiles (0, tj) and (1, tj) as its blocks: lane l
// supplies A = g[l] (block l/32, row l%32) and B = z of column 32 tj + l%32
// for both blocks, i.e. the low (tj = 0) or high (tj = 1) half of z in both
// halves of the wave, which one permlane32 swap of z with itself gives.
// Block b's registers 16 b .. 16 b + 15 follow the 32x32 single-block
// layout below, so accR[tj][16 ti + r] is element r of tile (ti, tj).
__device__ __forceinline__ void mfma_step_real(f32x32 (&accR)[2], float g, float z) {
    const auto zs = __builtin_amdgcn_permlane32_swap(__float_as_uint(z), __float_as_uint(z), false, false);
    accR[0] = __builtin_amdgcn_mfma_f32_32x32x1f32(g, __uint_as_float(zs[0]), accR[0], 0, 0, 0);
    accR[1] = __builtin_amdgcn_mfma_f32_32x32x1f32(g, __uint_as_float(zs[1]), accR[1], 0, 0, 0);
}

// Element r of tile (ti, tj) in lane l sits at row 32 ti + 8 (r/4) + 4 (l/32) + r%4,
// column 32 tj + l%32 of the wave's block.
__device__ __forceinline__ int acc_row(int ti, int r, int lane) { return 32 * ti + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }
__device__ __forceinline__ int acc_col(int tj, int lane) { return 32 * tj + (lane & 31); }

// Per item: the outer products of its steps into G[h,k] (DO_G) and the
// scores q[b,t,h,k] = sum_j Re(g_t[pi_k(j)] conj(z_t[j])) of every map at
// each of its steps (KW > 0: tasks of KW maps, spread over the waves; every
// step of the call belongs to one item).
template <int N, int KW, bool DO_G, int IO>
__global__ __launch_bounds__(DictCfg<N>::WAVES * 64) void k_ste_gemm(SteGradArgs a) {
    using Cfg = DictCfg<N>;
    constexpr bool DO_Q = KW > 0;
    constexpr int NB = Cfg::NB, T = Cfg::TILES, U = Cfg::U, RS = Cfg::RS, GP = Cfg::GP;
    extern __shared__ __align__(16) unsigned char lds[];
    float* red = reinterpret_cast<float*>(lds);
    using TE = typename TileOf<IO>::T;
    TE* Gt = reinterpret_cast<TE*>(lds);
    TE* Zt = Gt + N * GP;
    uint8_t* dT = lds + Cfg::TILE_BYTES;
    const SteWs w = ste_ws(a);
    const int HK = a.H * a.K, KP = score_kp(a.K);
    const int item = blockIdx.x;
    if (item >= w.item[HK]) return;
    // the group holding this item: the last gi with item[gi] <= item
    int lo = 0, hi = HK;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (w.item[mid] <= item) lo = mid;
        else hi = mid;
    }
    const int gi = lo, h = gi / a.K;
    const int pieces = w.item[gi + 1] - w.item[gi], piece = item - w.item[gi];
    const int first = piece * a.plan.P;
    const int cnt = min(a.plan.P, w.n[gi] - first);
    const int* ord = w.order + w.pos[gi] + first;

    const int wv = wave_id(), lane = lane_id();
    const int blk = wv / Cfg::SPLIT, part = wv - blk * Cfg::SPLIT;
    const int bi = blk / Cfg::GRID, bj = blk % Cfg::GRID;
    const int i0 = bi * NB, j0 = bj * NB;
    const int my0 = part * Cfg::MY;  // this wave's first step within a run

    if constexpr (DO_Q) {
        // the head's maps, transposed: dT[j*KP + k] = pi[h,k,j] (0 for k >= K)
        const int* pih = a.pi + (size_t)h * a.K * N;
        for (int e = threadIdx.x; e < N * KP; e += Cfg::WAVES * 64) {
            const int k = e / N, j = e - k * N;
            const int p = k < a.K ? pih[(size_t)k * N + j] : 0;
            dT[j * KP + k] = (uint8_t)((unsigned)p < (unsigned)N ? p : 0);
        }
    }

    f32x16 acc[T][T];
#pragma unroll
    for (int ti = 0; ti < T; ++ti)
#pragma unroll
        for (int tj = 0; tj < T; ++tj)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[ti][tj][r] = 0.f;
    constexpr bool kRealG = IO == kIoReal && NB == 64;
    f32x32 accR[2];
    if constexpr (kRealG) {
#pragma unroll
        for (int tj = 0; tj < 2; ++tj)
#pragma unroll
            for (int r = 0; r < 32; ++r) accR[tj][r] = 0.f;
    }

    // step ids of run r (lane t: step t; past the item: the item's last step,
    // so every load below stays valid and unconditional)
    auto run_ids = [&](int r) { return ord[min(r * RS + lane, cnt - 1)]; };
    // batch b of run r (sidv = run_ids(r))
    auto issue = [&](float2 (&gq)[U], float2 (&zq)[U], int sidv, int b) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            load_step<N, IO>(a, readlane_i(sidv, my0 + b * U + u), h, i0, j0, lane, gq[u], zq[u]);
    };
    // rows of batch b into the tiles: column t = the step's place in the run
    auto stage = [&](const float2 (&gq)[U], const float2 (&zq)[U], int b) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int t = my0 + b * U + u;
            if constexpr (Cfg::SPLIT > 1) {
                if (lane < N) {
                    Gt[lane * GP + t] = tile_elem(gq[u], TE());
                    Zt[lane * GP + t] = tile_elem(zq[u], TE());
                }
            } else {
                if (bj == 0) Gt[(i0 + lane) * GP + t] = tile_elem(gq[u], TE());
                if (bi == 0) Zt[(j0 + lane) * GP + t] = tile_elem(zq[u], TE());
            }
        }
    };
    auto multiply = [&](const float2 (&gq)[U], const float2 (&zq)[U], int r, int b) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (r * RS + my0 + b * U + u < cnt) {
                if constexpr (kRealG) mfma_step_real(accR, gq[u].x, zq[u].x);
                else mfma_step<N>(acc, gq[u], zq[u], lane);
            }
    };
    // scores of the run's steps, KW maps per task: lane l takes step l % RS
    // of the run, and the 64 / RS lane groups of a wave take different tasks
    // (every lane reads: a run shorter than the wave leaves none idle)
    auto scores = [&](int sidv, int r) {
        const int slot = lane / RS, tt = lane % RS;
        const int sidt = __shfl(sidv, tt);  // step id of this lane's step
        const bool step_on = r * RS + tt < cnt;
        constexpr int KWD = KW > 0 ? KW : 1;
        const int ntask = (a.K + KWD - 1) / KWD;
        for (int tg = wv; tg * Cfg::SLOTS < ntask; tg += Cfg::WAVES) {
            const int task = tg * Cfg::SLOTS + slot;
            const bool on = step_on && task < ntask;
            const int kb = min(task, ntask - 1) * KW;  // a lane past the tasks reads the last one and stores nothing
            float v[KW > 0 ? KW : 1];
#pragma unroll
            for (int u = 0; u < KW; ++u) v[u] = 0.f;
            // column j: z_t[j], the KW maps' rows at j (packed bytes), then
            // the KW gathered g_t[pi(j)]; the next column's z and map bytes
            // are read with this column's gathers, so each column waits for
            // one LDS round trip
            constexpr int NW4 = KW / 4 > 0 ? KW / 4 : 1;
            auto ld_col = [&](int j, uint32_t (&wds)[NW4], TE& zt) {
                zt = Zt[j * GP + tt];
                if constexpr (KW == 16) {
                    const uint4 pk = *reinterpret_cast<const uint4*>(dT + j * KP + kb);
                    wds[0] = pk.x, wds[1] = pk.y, wds[2] = pk.z, wds[3] = pk.w;
                } else if constexpr (KW == 8) {
                    const uint2 pk = *reinterpret_cast<const uint2*>(dT + j * KP + kb);
                    wds[0] = pk.x, wds[1] = pk.y;
                } else {
                    wds[0] = *reinterpret_cast<const uint32_t*>(dT + j * KP + kb);
                }
            };
            auto column = [&](const uint32_t (&wc)[NW4], TE zc) {
                TE g[KW > 0 ? KW : 1];
#pragma unroll
                for (int u = 0; u < KW; ++u) g[u] = Gt[((wc[u >> 2] >> (8 * (u & 3))) & 0xff) * GP + tt];
#pragma unroll
                for (int u = 0; u < KW; ++u) v[u] = score_fma(g[u], zc, v[u]);
            };
            if constexpr (N == 128 && KW == 4) {
                // blocks of 8 columns: their z and map bytes first, then
                // their gathers (timeseries-like shapes: measured 9% faster
                // for the whole call than one column ahead; slower at N = 64
                // and with 8 maps per task)
                constexpr int JB = 8;
#pragma unroll 1
                for (int jb = 0; jb < N; jb += JB) {
                    uint32_t wc[JB][NW4];
                    TE zc[JB];
#pragma unroll
                    for (int jj = 0; jj < JB; ++jj) ld_col(jb + jj, wc[jj], zc[jj]);
#pragma unroll
                    for (int jj = 0; jj < JB; ++jj) column(wc[jj], zc[jj]);
                }
            } else if constexpr (N < 256 && (KW >= 8 || N == 128)) {
                uint32_t wc[NW4];
                TE zc;
                ld_col(0, wc, zc);
#pragma unroll 2
                for (int j = 0; j < N; ++j) {
                    uint32_t wn[NW4];
                    TE zn;
                    ld_col(min(j + 1, N - 1), wn, zn);
                    column(wc, zc);
#pragma unroll
                    for (int q = 0; q < NW4; ++q) wc[q] = wn[q];
                    zc = zn;
                }
            } else {
                // few maps per task (or 16 waves, 128 registers): each gather
                // added as it arrives, two columns unrolled (measured faster
                // here than batching the gathers)
#pragma unroll 2
                for (int j = 0; j < N; ++j) {
                    uint32_t wc[NW4];
                    TE zc;
                    ld_col(j, wc, zc);
#pragma unroll
                    for (int u = 0; u < KW; ++u) {
                        const TE g = Gt[((wc[u >> 2] >> (8 * (u & 3))) & 0xff) * GP + tt];
                        v[u] = score_fma(g, zc, v[u]);
                    }
                }
            }
            if (on) {
                float* qrow = a.q + ((size_t)sidt * a.H + h) * a.K + kb;
                if (kb + KW <= a.K && (a.K & 3) == 0) {
#pragma unroll
                    for (int u = 0; u < KW; u += 4)
                        *reinterpret_cast<float4*>(qrow + u) = make_float4(v[u], v[u + 1], v[u + 2], v[u + 3]);
                } else {
#pragma unroll
                    for (int u = 0; u < KW; ++u)
                        if (kb + u < a.K) qrow[u] = v[u];
                }
            }
        }
    };

    // Two load batches are always in flight or ready: batch b is multiplied,
    // then its registers take batch b + 2 (of the next run for the last two,
    // so those loads run during the scores).  Step ids come two runs ahead.
    const int nrun = (cnt + RS - 1) / RS;
    int sid = run_ids(0), sidn = run_ids(1);
    float2 ga[U], za[U], gb[U], zb[U];
    issue(ga, za, sid, 0);
    issue(gb, zb, sid, 1);
    for (int r = 0; r < nrun; ++r) {
        const int sidnn = run_ids(r + 2);
        for (int b = 0; b < Cfg::NBAT; b += 2) {
            if constexpr (DO_G) multiply(ga, za, r, b);
            if constexpr (DO_Q) stage(ga, za, b);
            if (b + 2 < Cfg::NBAT) issue(ga, za, sid, b + 2);
            else issue(ga, za, sidn, 0);
            issue_fence();
            if constexpr (DO_G) multiply(gb, zb, r, b + 1);
            if constexpr (DO_Q) stage(gb, zb, b + 1);
            if (b + 3 < Cfg::NBAT) issue(gb, zb, sid, b + 3);
            else issue(gb, zb, sidn, 1);
            issue_fence();
        }
        if constexpr (DO_Q) {
            __syncthreads();  // tiles (and, in the first run, the maps) complete
            scores(sid, r);
            __syncthreads();  // tiles free for the next run
        }
        sid = sidn;
        sidn = sidnn;
    }
    if constexpr (!DO_G) return;
    if constexpr (kRealG) {
#pragma unroll
        for (int ti = 0; ti < 2; ++ti)
#pragma unroll
            for (int tj = 0; tj < 2; ++tj)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[ti][tj][r] = accR[tj][16 * ti + r];
    }

    if constexpr (Cfg::SPLIT > 1) {
        __syncthreads();  // red aliases the tiles
        if (part > 0) {
#pragma unroll
            for (int ti = 0; ti < T; ++ti)
#pragma unroll
                for (int tj = 0; tj < T; ++tj)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        red[(part - 1) * NB * NB + acc_row(ti, r, lane) * NB + acc_col(tj, lane)] = acc[ti][tj][r];
        }
        __syncthreads();
        if (part > 0) return;
#pragma unroll 1
        for (int p = 0; p < Cfg::SPLIT - 1; ++p)
#pragma unroll
            for (int ti = 0; ti < T; ++ti)
#pragma unroll
                for (int tj = 0; tj < T; ++tj)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        acc[ti][tj][r] += red[p * NB * NB + acc_row(ti, r, lane) * NB + acc_col(tj, lane)];
    }
    float* dst = pieces == 1 ? a.G + (size_t)gi * N * N : w.partial + (size_t)(w.slot[gi] + piece) * N * N;
#pragma unroll
    for (int ti = 0; ti < T; ++ti)
#pragma unroll
        for (int tj = 0; tj < T; ++tj)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = i0 + acc_row(ti, r, lane), col = j0 + acc_col(tj, lane);
                if (NB == 64 || (row < N && col < N)) dst[(size_t)row * N + col] = acc[ti][tj][r];
            }
}

// Block (gi, y): groups of several items add their partials in item order;
// groups no step chose get zeros; single-item groups were written directly.
// A thread takes 4 consecutive entries (one 16-byte load per partial when G
// is 16-byte aligned) and issues the loads of 4 partials before it adds them,
// in item order.
template <int N>
__global__ __launch_bounds__(256) void k_dict_reduce(SteGradArgs a) {
    constexpr int PB = 4;
    const SteWs w = ste_ws(a);
    const int gi = blockIdx.x;
    const int pieces = w.item[gi + 1] - w.item[gi];
    if (pieces == 1) return;
    constexpr int NN = N * N;
    float* dst = a.G + (size_t)gi * NN;
    const float* src = w.partial + (size_t)(pieces ? w.slot[gi] : 0) * NN;
    const bool vec = (reinterpret_cast<uintptr_t>(a.G) & 15) == 0;
    for (int e = 4 * (blockIdx.y * 256 + threadIdx.x); e < NN; e += 4 * 256 * gridDim.y) {
        float sum[4] = {0.f, 0.f, 0.f, 0.f};
        for (int p0 = 0; p0 < pieces; p0 += PB) {
            float4 v[PB];
#pragma unroll
            for (int i = 0; i < PB; ++i)
                v[i] = p0 + i < pieces ? *reinterpret_cast<const float4*>(src + (size_t)(p0 + i) * NN + e)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int i = 0; i < PB; ++i) {
                if (p0 + i < pieces) {
                    sum[0] += v[i].x;
                    sum[1] += v[i].y;
                    sum[2] += v[i].z;
                    sum[3] += v[i].w;
                }
            }
        }
        if (vec) {
            *reinterpret_cast<float4*>(dst + e) = make_float4(sum[0], sum[1], sum[2], sum[3]);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) dst[e + i] = sum[i];
        }
    }
}

template <int N, int KW, bool DO_G>
hipError_t gemm_launch(const SteGradArgs& a, hipStream_t st) {
    auto kern = a.io == kIoReal   ? k_ste_gemm<N, KW, DO_G, kIoReal>
                : a.io == kIoBf16 ? k_ste_gemm<N, KW, DO_G, kIoBf16>
                                  : k_ste_gemm<N, KW, DO_G, kIoC64>;
    const size_t lds = ste_gemm_lds<N>(a.K, KW > 0);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.plan.max_items), dim3(DictCfg<N>::WAVES * 64), lds, st, a);
    return hipGetLastError();
}

template <int N>
hipError_t dict_launch(const SteGradArgs& a, hipStream_t st) {
    // score tasks of 16, 8 or 4 maps: wide enough to amortise each z read,
    // many enough to keep every lane group of every wave busy
    const int waves = DictCfg<N>::WAVES * DictCfg<N>::SLOTS;
    hipError_t e;
    constexpr int KW16 = N < 256 ? 16 : 4, KW8 = N < 256 ? 8 : 4;  // N = 256 (16 waves): 4 maps per task
    if (!a.q) e = gemm_launch<N, 0, true>(a, st);
    else if (a.K >= 16 * waves) e = a.G ? gemm_launch<N, KW16, true>(a, st) : gemm_launch<N, KW16, false>(a, st);
    else if (a.K >= 8 * waves) e = a.G ? gemm_launch<N, KW8, true>(a, st) : gemm_launch<N, KW8, false>(a, st);
    else e = a.G ? gemm_launch<N, 4, true>(a, st) : gemm_launch<N, 4, false>(a, st);
    if (e != hipSuccess || !a.G) return e;
    const int ys = (N * N + 1023) / 1024 < 64 ? (N * N + 1023) / 1024 : 64;  // one 4-entry piece per thread
    hipLaunchKernelGGL(k_dict_reduce<N>, dim3(a.H * a.K, ys), dim3(256), 0, st, a);
    return hipGetLastError();
}

// ------------------------------------------------------------------ tempered softmax
// Online softmax state of one fibre: m = max(x * it), s = sum exp(x*it - m),
// d = sum exp(x*it - m) * gy.
struct SoftState {
    float m, s, d;
};

__device__ __forceinline__ void soft_add(SoftState& a, float xi, float gi) {
    const float mn = fmaxf(a.m, xi);
    const float r = __expf(a.m - mn), e = __expf(xi - mn);
    a.s = a.s * r + e;
    a.d = a.d * r + e * gi;
    a.m = mn;
}

__device__ __forceinline__ void soft_merge(SoftState& a, const SoftState& b) {
    const float mn = fmaxf(a.m, b.m);
    if (mn == -INFINITY) return;  // both empty
    const float ra = __expf(a.m - mn), rb = __expf(b.m - mn);
    a.s = a.s * ra + b.s * rb;
    a.d = a.d * ra + b.d * rb;
    a.m = mn;
}

// inner == 1 (the axis is contiguous, e.g. routing logits over k): a team of
// T lanes (T = min(64, len rounded up to a power of two)) per row, lane t
// taking entries t, t + T, ...; the team merges its states with butterfly
// shuffles.  Loads of a wave cover 64 consecutive floats.
template <int T>
__global__ __launch_bounds__(256) void k_softmax_rows(const float* __restrict__ x, const float* __restrict__ gy,
                                                      float* __restrict__ gx, int64_t rows, int len, float it) {
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t row = gid / T;
    const int t = (int)(gid % T);
    const bool on = row < rows;
    const int64_t base = (on ? row : 0) * len;
    SoftState st = {-INFINITY, 0.f, 0.f};
    if (on)
        for (int i = t; i < len; i += T) soft_add(st, x[base + i] * it, gy[base + i]);
#pragma unroll
    for (int off = T / 2; off > 0; off >>= 1) {
        SoftState o;
        o.m = __shfl_xor(st.m, off, T);
        o.s = __shfl_xor(st.s, off, T);
        o.d = __shfl_xor(st.d, off, T);
        soft_merge(st, o);
    }
    if (!on) return;
    const float rs = 1.f / st.s, dot = st.d * rs;
    for (int i = t; i < len; i += T) gx[base + i] = __expf(x[base + i] * it - st.m) * rs * (gy[base + i] - dot) * it;
}

// inner == 1, len % 4 == 0, len <= 4 T, 16-byte aligned rows (the routing
// logits over k): a team of T lanes per row, lane t holding entries
// 4t .. 4t+3 (one 16-byte load of x and one of gy); the row's max, then its
// two sums, each reduced across the team with butterfly shuffles -- one
// exponential per entry.
template <int T>
__global__ __launch_bounds__(256) void k_softmax_rows4(const float* __restrict__ x, const float* __restrict__ gy,
                                                       float* __restrict__ gx, int64_t rows, int len, float it) {
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t row = gid / T;
    const int t = (int)(gid % T);
    const bool on = row < rows && 4 * t < len;
    const int64_t off = on ? row * len + 4 * t : 0;
    float4 xv = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY), gv = make_float4(0.f, 0.f, 0.f, 0.f);
    if (on) {
        xv = *reinterpret_cast<const float4*>(x + off);
        gv = *reinterpret_cast<const float4*>(gy + off);
        xv = make_float4(xv.x * it, xv.y * it, xv.z * it, xv.w * it);
    }
    float m = fmaxf(fmaxf(xv.x, xv.y), fmaxf(xv.z, xv.w));
#pragma unroll
    for (int o = T / 2; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, T));
    float4 e = make_float4(0.f, 0.f, 0.f, 0.f);
    if (on) e = make_float4(__expf(xv.x - m), __expf(xv.y - m), __expf(xv.z - m), __expf(xv.w - m));
    float sum = (e.x + e.y) + (e.z + e.w);
    float dt = fmaf(e.x, gv.x, fmaf(e.y, gv.y, fmaf(e.z, gv.z, e.w * gv.w)));
#pragma unroll
    for (int o = T / 2; o > 0; o >>= 1) {
        sum += __shfl_xor(sum, o, T);
        dt += __shfl_xor(dt, o, T);
    }
    if (!on) return;
    const float rs = 1.f / sum, dot = dt * rs, c = rs * it;
    *reinterpret_cast<float4*>(gx + off) = make_float4(e.x * c * (gv.x - dot), e.y * c * (gv.y - dot),
                                                       e.z * c * (gv.z - dot), e.w * c * (gv.w - dot));
}

// inner > 1 (e.g. down the columns of M[h,k]): a thread per fibre (o, j);
// neighbouring threads take neighbouring j, so every load is coalesced.
__global__ __launch_bounds__(256) void k_softmax_cols(const float* __restrict__ x, const float* __restrict__ gy,
                                                      float* __restrict__ gx, int64_t outer, int len, int64_t inner,
                                                      float it) {
    const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (id >= outer * inner) return;
    const int64_t o = id / inner, j = id - o * inner;
    const int64_t base = o * len * inner + j;
    SoftState st = {-INFINITY, 0.f, 0.f};
#pragma unroll 4
    for (int i = 0; i < len; ++i) soft_add(st, x[base + i * inner] * it, gy[base + i * inner]);
    const float rs = 1.f / st.s, dot = st.d * rs;
#pragma unroll 4
    for (int i = 0; i < len; ++i)
        gx[base + i * inner] = __expf(x[base + i * inner] * it - st.m) * rs * (gy[base + i * inner] - dot) * it;
}

// inner > 1 with a long axis (the columns of M[h,k] at N >= 32): four
// threads per fibre, each folding a quarter of the axis; the quarters'
// states merge in LDS in quarter order and each thread writes its quarter.
// Neighbouring threads of a wave take neighbouring fibres (coalesced), and
// the chip gets four times the waves of one thread per fibre.
__global__ __launch_bounds__(256) void k_softmax_cols4(const float* __restrict__ x, const float* __restrict__ gy,
                                                       float* __restrict__ gx, int64_t outer, int len, int64_t inner,
                                                       float it) {
    __shared__ SoftState part_st[4][64];
    const int f = threadIdx.x & 63, part = threadIdx.x >> 6;
    const int64_t id = (int64_t)blockIdx.x * 64 + f;
    const bool on = id < outer * inner;
    const int64_t o = on ? id / inner : 0, j = on ? id - o * inner : 0;
    const int64_t base = o * len * inner + j;
    const int qn = (len + 3) / 4, i0 = min(len, part * qn), i1 = min(len, i0 + qn);
    SoftState st = {-INFINITY, 0.f, 0.f};
    if (on) {
#pragma unroll 4
        for (int i = i0; i < i1; ++i) soft_add(st, x[base + i * inner] * it, gy[base + i * inner]);
    }
    part_st[part][f] = st;
    __syncthreads();
    SoftState m = part_st[0][f];
#pragma unroll
    for (int p = 1; p < 4; ++p) soft_merge(m, part_st[p][f]);
    if (!on) return;
    const float rs = 1.f / m.s, dot = m.d * rs;
#pragma unroll 4
    for (int i = i0; i < i1; ++i)
        gx[base + i * inner] = __expf(x[base + i * inner] * it - m.m) * rs * (gy[base + i * inner] - dot) * it;
}

template <int T>
void softmax_rows4_launch(const float* x, const float* gy, float* gx, int64_t rows, int len, float it,
                          hipStream_t st) {
    const int64_t lanes = rows * T;
    hipLaunchKernelGGL(k_softmax_rows4<T>, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, st, x, gy, gx, rows,
                       len, it);
}

template <int T>
void softmax_rows_launch(const float* x, const float* gy, float* gx, int64_t rows, int len, float it,
                         hipStream_t st) {
    const int64_t lanes = rows * T;
    hipLaunchKernelGGL(k_softmax_rows<T>, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, st, x, gy, gx, rows,
                       len, it);
}

}  // namespace

hipError_t launch_ste_grads(const SteGradArgs& a, hipStream_t st) {
    const int nb = a.H * a.plan.S;
    hipLaunchKernelGGL(k_dict_hist, dim3(nb), dim3(256), 0, st, a);
    hipLaunchKernelGGL(k_dict_plan, dim3(1), dim3(1024), 0, st, a);
    hipLaunchKernelGGL(k_dict_scatter, dim3(nb), dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    switch (a.N) {
        case 8: return dict_launch<8>(a, st);
        case 16: return dict_launch<16>(a, st);
        case 32: return dict_launch<32>(a, st);
        case 64: return dict_launch<64>(a, st);
        case 128: return dict_launch<128>(a, st);
        case 256: return dict_launch<256>(a, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_softmax_vjp(const float* x, const float* gy, float* gx, int64_t outer, int len, int64_t inner,
                              float inv_temp, hipStream_t st) {
    const int64_t n = outer * inner;
    if (n == 0) return hipSuccess;
    const bool al16 = ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(gy) |
                        reinterpret_cast<uintptr_t>(gx)) & 15) == 0;
    if (inner == 1 && len % 4 == 0 && len <= 256 && al16) {
        if (len <= 4) softmax_rows4_launch<1>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 8) softmax_rows4_launch<2>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 16) softmax_rows4_launch<4>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 32) softmax_rows4_launch<8>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 64) softmax_rows4_launch<16>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 128) softmax_rows4_launch<32>(x, gy, gx, outer, len, inv_temp, st);
        else softmax_rows4_launch<64>(x, gy, gx, outer, len, inv_temp, st);
    } else if (inner == 1) {
        if (len <= 2) softmax_rows_launch<2>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 4) softmax_rows_launch<4>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 8) softmax_rows_launch<8>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 16) softmax_rows_launch<16>(x, gy, gx, outer, len, inv_temp, st);
        else if (len <= 32) softmax_rows_launch<32>(x, gy, gx, outer, len, inv_temp, st);
        else softmax_rows_launch<64>(x, gy, gx, outer, len, inv_temp, st);
    } else if (len >= 32) {
        hipLaunchKernelGGL(k_softmax_cols4, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, st, x, gy, gx, outer, len,
                           inner, inv_temp);
    } else {
        hipLaunchKernelGGL(k_softmax_cols, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, x, gy, gx, outer, len,
                           inner, inv_temp);
    }
    return hipGetLastError();
}

}  // namespace pdssm
