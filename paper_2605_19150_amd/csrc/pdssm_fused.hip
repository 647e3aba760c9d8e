// pdssm_fused.hip -- single-read fused PD scan for gfx950.
//
// Layout of the work.  One workgroup owns one (batch, head) sequence, or one
// segment of it when there are too few sequences to fill the chip (see the
// work units below).  The sequence is cut into chunks of TAU steps (App. E.1
// Algorithm 1).
//
// Forward: W chunk waves plus one frontier wave.  Chunk wave w takes chunks
// w, w+W, w+2W, ...; for each chunk it
//   1. loads the chunk's D, b, c rows (and idx) into registers -- the only
//      time they are read from HBM -- while it still computes the previous
//      chunk (two register buffers);
//   2. runs the chunk once from a zero state (Algorithm 1 Phase A): the local
//      state B_c, the chunk's PD operator (Pi, Delta) built by the App. E.3.1
//      accumulator update, and per step the local readout Re<c_t, x_t^loc>
//      and the weights w_t[j] = Delta_t[j] c_t[Pi_t(j)] that carry the
//      entering state to y_t (Phase C in Algorithm 1's form);
//   3. publishes (B_c, Pi_c, Delta_c) in an LDS slot; the frontier wave, which
//      keeps the running state in registers, applies
//      carry_{c+1} = B_c + (Pi_c, Delta_c) carry_c (Phase B) and hands carry_c
//      back through an LDS ring;
//   4. finishes y_t = Re<c_t, x_t^loc> + Re sum_j w_t[j] carry_c[j]; h_t
//      never reaches memory.  The frontier keeps the chunk-entering states
//      (the saved states) in LDS and the workgroup writes them out once all
//      its rows are read.
// Backward: W waves, chunks in reverse order, the adjoint recurrence (a
// gather: g_{t-1}[j] = conj(D_t[j]) g_t[pi_t[j]] + readout term) folded the
// same way, the chunk-to-chunk hand-off passed wave to wave, and the chunk's
// states recomputed from its saved entering state.
//
// Scatter as gathers.  The forward step h'[r] = b[r] + sum_{j: pi(j)=r}
// D[j] h[j] adds up every source that lands on row r.  For each dictionary
// entry a prep kernel lists, per destination row, its sources in ascending
// order (up to 7, plus the in-degree) once per call; the step then writes
// D .* h to LDS once and every lane gathers its row's sources.  The number of
// gathers per step is fixed per head (1, 3 or 7, the head's largest in-degree
// rounded up), so the step has no branches: unused record slots point at a
// row that stays zero.  An entry with a row of in-degree above 7 (rare for
// random maps, e.g. an all-to-one map) is stored in sorted form instead and
// its steps sum each row's run with a segmented scan across lanes; a head
// with such entries runs the step-by-step chunk pass, whose steps test their
// map's class (heads without them never test for it).  No sum uses float
// atomics, so results are deterministic.
//
// The last chunk of a sequence may be short; its missing steps run as exact
// no-ops (D = 1, b = 0, an identity dictionary entry at index K), so no step
// tests its own index either.
//
// Row formats.  D, b, c and the gradients come as complex64, bf16 (re, im)
// pairs or real fp32 (the real-valued model of App. B).  The first two run
// complex (float2) arithmetic; the real model runs with float elements
// throughout (state, LDS staging, published operators), rounding every
// operation as the complex arithmetic does on zero imaginary parts.
#include "pdssm_device.h"
#include "pdssm_fused.h"

namespace pdssm {

namespace {

// ------------------------------------------------------------------ prep
// One wave per dictionary entry (h, k): byte dictionary, per-row source
// records, per-entry max in-degree; an entry with a row of more than kMaxSrc
// sources gets its sorted form instead of records.  Every source finds its
// rank among the sources of its row (ascending source order) from lane-mask
// tables (map_ranks), so no lane walks the whole map.
template <int N>
__global__ __launch_bounds__(256) void k_prep(PrepArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ uint64_t smt[4][SL][N];  // per wave: lane-mask tables
    __shared__ uint64_t srec[4][N];     // per wave: the records being filled
    __shared__ int soff[4][N];          // per wave: sorted form, first position of each row's run
    __shared__ uint8_t sst[4][N];       // per wave: sorted form, run-start flags by position
    const int wv = wave_id(), lane = lane_id();
    const int e = blockIdx.x * 4 + wv;
    if (e >= a.H * a.K) return;
    const bool act = lane < LANES;
    bool bad = false;
    IV<SL> p;
#pragma unroll
    for (int s = 0; s < SL; ++s) p.v[s] = 0;
    if (act) {
        p = ld_iv<SL>(a.pi + (size_t)e * N, lane);
        bad = sanitize_map<N, SL>(p);
#pragma unroll
        for (int s = 0; s < SL; ++s) a.dict[(size_t)e * N + lane * SL + s] = (uint8_t)p.v[s];
    }
    uint64_t* MT[SL];
#pragma unroll
    for (int q = 0; q < SL; ++q) MT[q] = smt[wv][q];
    int rank[SL], cnt[SL];
    map_ranks<N>(p, lane, act, MT, rank, cnt);
    int maxdeg = 0;
    if (act) {
#pragma unroll
        for (int s = 0; s < SL; ++s) maxdeg = max(maxdeg, cnt[s]);
    }
    for (int off = 32; off >= 1; off >>= 1) maxdeg = max(maxdeg, __shfl_xor(maxdeg, off));
    uint64_t* out = a.rec + (size_t)e * N;
    if (maxdeg <= kMaxSrc) {
        // record of row r: its sources in ascending order in bytes 0..6
        // (unused ones name the sentinel), its in-degree in byte 7; each
        // source writes its own byte at its rank
        uint64_t* R = srec[wv];
        uint64_t empty = 0;
#pragma unroll
        for (int m = 0; m < kMaxSrc; ++m) empty |= (uint64_t)Sentinel<N>::kByte << (8 * m);
        wave_sync();
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) R[lane * SL + s] = empty | (uint64_t)cnt[s] << 56;
        }
        wave_sync();
        if (act) {
            uint8_t* RB = reinterpret_cast<uint8_t*>(R);
#pragma unroll
            for (int s = 0; s < SL; ++s) RB[p.v[s] * 8 + rank[s]] = (uint8_t)(lane * SL + s);
        }
        wave_sync();
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) out[lane * SL + s] = R[lane * SL + s];
        }
    } else {
        uint64_t w[SL];
        map_sorted_words<N>(p, lane, act, MT, soff[wv], sst[wv], w);
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) out[lane * SL + s] = w[s];
        }
    }
    if (lane == 0) a.mtab[e] = (uint8_t)(maxdeg <= kMaxSrc ? maxdeg : kFallback);
    if (bad) report_index_error(a.status);
}

// ------------------------------------------------------------------ shared pieces
// Element of the state and of the rows as the kernels compute them: complex
// (float2) for complex64 and bf16 pairs, float for the real-valued model,
// whose states stay real (half the arithmetic and LDS bytes).  Every
// buffer keeps its place in the layout; the real model uses its first half.
template <int IO>
struct ElemOf {
    using T = float2;
};
template <>
struct ElemOf<kIoReal> {
    using T = float;
};

struct Smem {
    uint64_t* rec;  // [K+1][N]
    uint8_t* dict;  // [K+1][N]
    uint8_t* mtab;  // [K+1]
    float2* ring;   // [W+1][N] carry slots
    int* ready;     // carry counter, followed by the operator-slot flags
    float4* agg;    // [2W][N] published chunk operator: local state (xy), diagonal (zw)
    uint8_t* agp;   // [2W][N] published chunk map, or the sorted position of each source
    uint16_t* age;  // [2W][N] last sorted position of each destination's run (kNoRun: none)
    uint8_t* agh;   // [2W][N] 1 where a sorted position starts a destination's run
    uint8_t* agm;   // [2W][N] the chunk map itself (aggregate pass)
    int* aflag;     // [2W] chunk id held by each operator slot
    int* prog;      // chunks finished by the workgroup's waves (bounded waits)
    float4* vd;     // [W][N+1] per wave: staged values V[N+1], then Z[N+1] (see Stage)
    float2* x;      // [W][N]
    float2* cs;     // [W][2][N] (forward: staged c_t, two steps)
    uint8_t* pa;    // [W][N] (backward)
    float2* sb;     // [sbM][N] forward: staged saved states (complex64 rows; the real model's
                    // are narrowed to their real parts when written out)
};

__device__ __forceinline__ Smem carve_smem(unsigned char* base, const LdsLayout& l) {
    Smem s;
    s.rec = reinterpret_cast<uint64_t*>(base + l.rec);
    s.dict = base + l.dict;
    s.mtab = base + l.mtab;
    s.ring = reinterpret_cast<float2*>(base + l.ring);
    s.ready = reinterpret_cast<int*>(base + l.ready);
    s.agg = reinterpret_cast<float4*>(base + l.agg);
    s.agp = base + l.agp;
    s.age = reinterpret_cast<uint16_t*>(base + l.age);
    s.agh = base + l.agh;
    s.agm = base + l.agm;
    s.aflag = reinterpret_cast<int*>(base + l.aflag);
    s.prog = reinterpret_cast<int*>(base + l.prog);
    s.vd = reinterpret_cast<float4*>(base + l.vd);
    s.x = reinterpret_cast<float2*>(base + l.x);
    s.cs = reinterpret_cast<float2*>(base + l.cs);
    s.pa = base + l.pa;
    s.sb = reinterpret_cast<float2*>(base + l.sb);
    return s;
}

// A wave's staging rows: values V[0..N] (V[N] stays zero, the target of
// unused gather slots) and a second operand Z[0..N] (D_t, or the backward's
// diagonal), as two arrays of 8-byte words so that a 64-lane gather from V
// spreads over all 32 bank pairs.
template <class E>
struct Stage {
    E* V;
    E* Z;
};

template <int N, class E = float2>
__device__ __forceinline__ Stage<E> stage_of(const Smem& s, int wv) {
    float2* base = reinterpret_cast<float2*>(s.vd + wv * (N + 1));
    return Stage<E>{reinterpret_cast<E*>(base), reinterpret_cast<E*>(base + N + 1)};
}

// Copy head hh's dictionary tables into LDS and append the identity entry
// (all threads; a barrier follows).  The tables sit at the start of every
// layout of one (N, K), whatever its wave count.
template <int N>
__device__ __forceinline__ void stage_tables(const FusedArgs& a, const Smem& s, int hh) {
    const int nthr = blockDim.x, tid = threadIdx.x;
    const int K = a.K;
    const size_t e0 = (size_t)hh * K;
    const uint64_t* rsrc = a.rec + e0 * N;
    for (int i = tid; i < K * N; i += nthr) s.rec[i] = rsrc[i];
    const uint32_t* dsrc = reinterpret_cast<const uint32_t*>(a.dict + e0 * N);
    uint32_t* ddst = reinterpret_cast<uint32_t*>(s.dict);
    for (int i = tid; i < K * N / 4; i += nthr) ddst[i] = dsrc[i];
    for (int i = tid; i < K; i += nthr) s.mtab[i] = a.mtab[e0 + i];
    for (int j = tid; j < N; j += nthr) {
        uint64_t rec = (uint64_t)1 << 56 | (uint64_t)j;
#pragma unroll
        for (int m = 1; m < kMaxSrc; ++m) rec |= (uint64_t)Sentinel<N>::kByte << (8 * m);
        s.rec[(size_t)K * N + j] = rec;
        s.dict[K * N + j] = (uint8_t)j;
    }
    if (tid == 0) s.mtab[K] = 1;
}

// Clear the zero row V[N] of the first nw waves' staging rows.
template <int N, class E>
__device__ __forceinline__ void clear_zero_rows(const Smem& s, int nw) {
    for (int w = threadIdx.x; w < nw; w += blockDim.x) stage_of<N, E>(s, w).V[N] = ezero<E>();
}

// Gather variant of a head: the smallest of 1, 3, 7 sources covering every
// entry's in-degree, and whether some entry needs the atomic scatter.
__device__ __forceinline__ int head_variant(const Smem& s, int K, bool& fallback) {
    const int lane = lane_id();
    int m = 0, fb = 0;
    for (int i = lane; i < K; i += kWave) {
        const int v = s.mtab[i];
        if (v == (int)kFallback) fb = 1;
        else m = max(m, v);
    }
    for (int off = 32; off >= 1; off >>= 1) {
        m = max(m, __shfl_xor(m, off));
        fb |= __shfl_xor(fb, off);
    }
    // the same in every lane: scalar values, so that everything derived
    // from them (branches, layout offsets) stays scalar
    fallback = __builtin_amdgcn_readfirstlane(fb) != 0;
    return __builtin_amdgcn_readfirstlane(m <= 1 ? 1 : (m <= 3 ? 3 : 7));
}

// Sequence handled by this workgroup.  Workgroups are dispatched round-robin
// over the 8 XCDs; consecutive sequences (neighbouring heads of one batch
// row, whose rows of D/b/c/y sit next to each other in memory) are kept on
// one XCD so they share its L2.
__device__ __forceinline__ int xcd_seq(int nseq) {
    const int i = blockIdx.x;
    if (nseq % 8 != 0) return i;
    return (i % 8) * (nseq / 8) + i / 8;
}

// Spin on a workgroup hand-off flag until it reaches `want`.  Every flag only
// grows (atomic max), so a late or early publish can never hide a value
// another wave waits for.  Bounded: a wave gives up only after two windows
// of kSpinLimit polls without the flag, the second one also without progress
// of the workgroup (*prog did not move: a long but live wait, e.g. for a run
// of thousands of chunks, keeps going).  It then reports PDSSM_ERR_HIP and raises every flag of the
// workgroup (the nflags ints at `all`) to INT_MAX, so that all other waiting
// waves are released at once and the grid drains.
constexpr int kSpinLimit = 1 << 22;
constexpr int kErrHang = -4;  // PDSSM_ERR_HIP

__device__ __forceinline__ void wait_ready(int* ready, int want, int* status, int* all, int nflags, const int* prog) {
    int spins = 0;
    int seen = -1;  // progress count at the end of the last window (none yet)
    while (__hip_atomic_load(ready, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < want) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinLimit) {
            // a window without the flag: keep waiting while the workgroup
            // finishes chunks, give up after a window in which none finished
            const int now = __hip_atomic_load(prog, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            if (seen < 0 || now != seen) {
                seen = now;
                spins = 0;
                continue;
            }
            if (status && lane_id() == 0) *status = kErrHang;
            for (int i = lane_id(); i < nflags; i += kWave)
                __hip_atomic_fetch_max(all + i, 0x7fffffff, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            return;
        }
    }
}

// One more chunk folded by this wave.  Only the aggregate pass's run folds
// count: they are the one place where a wave waits for another's many chunks
// (every other hand-off waits for a single chunk, far below one window).
__device__ __forceinline__ void note_progress(const Smem& s) {
    if (lane_id() == 0) __hip_atomic_fetch_add(s.prog, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void publish_ready(int* ready, int v) {
    __hip_atomic_fetch_max(ready, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// acc[j] += sum of V[src] over the G listed sources of destination row j;
// V = the wave's staged values.  Straight-line: G reads, no tests.
template <int N, int G, class E>
__device__ __forceinline__ void gather_rows(const E* V, const uint64_t* recrow, int lane, CV<Lay<N>::SL, E>& acc) {
    constexpr int SL = Lay<N>::SL;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const uint64_t r = recrow[lane * SL + s];
        const unsigned lo = (unsigned)r, hi = (unsigned)(r >> 32);
#pragma unroll
        for (int m = 0; m < G; ++m) {
            const unsigned src = m < 4 ? (lo >> (8 * m)) & 255u : (hi >> (8 * (m - 4))) & 255u;
            E v = V[src];
            if constexpr (!Sentinel<N>::kZeroRow) {
                const bool use = m < (int)(hi >> 24);
                v = use ? v : ezero<E>();
            }
            acc.v[s] = cadd(acc.v[s], v);
        }
    }
}

// Per-chunk registers of one wave.
template <int N, int TAU, class E = float2>
struct Chunk {
    static constexpr int SL = Lay<N>::SL;
    CV<SL, E> D[TAU], b[TAU], c[TAU];
    int kv, mv, len;
};

// The same sums reading only as many sources as the step's map needs: gk is
// that map's max in-degree (wave-uniform), and every record byte past a
// row's own sources names the zero row or an unused slot, so stopping after
// gk of them changes nothing.  Heads of the 7-source class pick 3, 4, 5 or 7
// reads with a scalar branch per step (uniform maps at N = 64..128 mostly
// need 4 or 5).  The forward's pipelined chunk pass keeps its fixed count:
// there the branch splits the step's one batch of LDS reads and measured
// slower.
template <int N, int G, class E>
__device__ __forceinline__ void gather_rows_k(const E* V, const uint64_t* recrow, int lane, CV<Lay<N>::SL, E>& acc,
                                              int gk) {
    if constexpr (G <= 3) {
        gather_rows<N, G>(V, recrow, lane, acc);
    } else {
        if (gk <= 3) gather_rows<N, 3>(V, recrow, lane, acc);
        else if (gk <= 4) gather_rows<N, 4>(V, recrow, lane, acc);
        else if (gk <= 5) gather_rows<N, 5>(V, recrow, lane, acc);
        else gather_rows<N, G>(V, recrow, lane, acc);
    }
}

// One step h <- bt + P(k) (Dt .* h).  With STAGE_D the step also leaves D_t
// in Z for a map composition.  FB: the head has entries in sorted form
// (a row of more than kMaxSrc sources), tested per step.  M: the step's
// in-degree class (its map's max in-degree, or kFallback).
template <int N, int G, bool FB, bool STAGE_D, class E>
__device__ __forceinline__ void pd_step(const Smem& s, const Stage<E>& st, int lane, bool act, int k, int M,
                                        CV<Lay<N>::SL, E>& h, const CV<Lay<N>::SL, E>& Dt,
                                        const CV<Lay<N>::SL, E>& bt) {
    constexpr int SL = Lay<N>::SL;
    if constexpr (FB) {
        if (M == (int)kFallback) {
            uint64_t w[SL];
#pragma unroll
            for (int q = 0; q < SL; ++q) w[q] = act ? s.rec[(size_t)k * N + lane * SL + q] : 0;
            if constexpr (STAGE_D) {
                wave_sync();
                if (act) {
#pragma unroll
                    for (int q = 0; q < SL; ++q) st.Z[lane * SL + q] = Dt.v[q];
                }
            }
            sorted_step<N, E>(st.V, w, h, Dt, bt, lane, act);
            return;
        }
    }
    wave_sync();
    if (act) {
#pragma unroll
        for (int q = 0; q < SL; ++q) {
            st.V[lane * SL + q] = cmul(Dt.v[q], h.v[q]);
            if constexpr (STAGE_D) st.Z[lane * SL + q] = Dt.v[q];
        }
    }
    wave_sync();
    if (act) {
        CV<SL, E> acc = bt;
        gather_rows_k<N, G>(st.V, s.rec + (size_t)k * N, lane, acc, M);
        h = acc;
    }
}

// Issues the loads of chunk ch of sequence (bb, hh) into registers and
// consumes none of them, so a wave can prefetch one chunk while it computes
// another.  Steps past the end of a short last chunk read through a null
// buffer descriptor (zero records): out-of-range buffer reads return 0, so
// their b and c rows are 0; their D row is taken as 1 at use (Dt()).
//
// The issue itself never branches (a chunk number >= C issues a chunk with no
// steps, all through the null descriptor): the compiler can then count the
// outstanding loads exactly and a wave waits only for the chunk it computes.
// AUX: cache policy of the row loads (the forward streams them, kLoadStream).
template <int N, int TAU, bool LOAD_B, bool LOAD_C, int AUX = 0, int IO = kIoC64>
__device__ __forceinline__ void issue_chunk(const FusedArgs& a, int bb, int hh, int ch, int lane, bool act,
                                            Chunk<N, TAU, typename ElemOf<IO>::T>& q) {
    using E = typename ElemOf<IO>::T;
    constexpr int SL = Lay<N>::SL;
    const int chc = min(ch, a.C - 1);  // addresses stay inside the tensors
    const int s0 = chc * TAU;
    const int lenc = min(TAU, a.L - s0);
    q.len = ch < a.C ? lenc : 0;
    const size_t base = (((size_t)bb * a.L + s0) * a.H + hh) * N;
    q.kv = a.idx[((size_t)bb * a.L + s0 + min(lane, lenc - 1)) * a.H + hh];
    constexpr uint32_t ESZ = IO == kIoC64 ? 8 : 4;    // bytes per entry
    const uint32_t rstride = (uint32_t)a.H * N * ESZ;  // bytes between consecutive steps
    const uint32_t extent = (uint32_t)(lenc - 1) * rstride + N * ESZ;
    const __amdgpu_buffer_rsrc_t rD = row_block(reinterpret_cast<const char*>(a.D) + base * ESZ, extent);
    const __amdgpu_buffer_rsrc_t rb = row_block(reinterpret_cast<const char*>(a.b) + base * ESZ, extent);
    const __amdgpu_buffer_rsrc_t rc = row_block(reinterpret_cast<const char*>(a.c) + base * ESZ, extent);
    const __amdgpu_buffer_rsrc_t rnull = row_block(a.D, 0);
    const uint32_t voff = (uint32_t)lane * SL * ESZ;
    auto ld = [&](__amdgpu_buffer_rsrc_t r, uint32_t so) {
        if constexpr (IO == kIoReal) return ld_row_r<SL, AUX>(r, voff, so);
        else if constexpr (IO == kIoBf16) return ld_row_w<SL, AUX, IO>(r, voff, so);
        else return ld_row<SL, AUX>(r, voff, so);
    };
#pragma unroll
    for (int t = 0; t < TAU; ++t) {
        const bool in = t < q.len;
        const uint32_t soff = (uint32_t)t * rstride;
        if (act) {
            q.D[t] = ld(in ? rD : rnull, soff);
            if constexpr (LOAD_B) q.b[t] = ld(in ? rb : rnull, soff);
            if constexpr (LOAD_C) q.c[t] = ld(in ? rc : rnull, soff);
        } else {
            q.D[t] = cv_zero<SL, E>();
            if constexpr (LOAD_B) q.b[t] = cv_zero<SL, E>();
            if constexpr (LOAD_C) q.c[t] = cv_zero<SL, E>();
        }
    }
}

// D row of step t as used by the step: 1 for the padded steps of a short chunk.
template <int N, int TAU, class E>
__device__ __forceinline__ CV<Lay<N>::SL, E> Dt(const Chunk<N, TAU, E>& q, int t) {
    CV<Lay<N>::SL, E> d = q.D[t];
    const bool in = t < q.len;
#pragma unroll
    for (int r = 0; r < Lay<N>::SL; ++r) d.v[r] = in ? d.v[r] : eone<E>();
    return d;
}

// Completes an issued chunk: checks the dictionary indices (an index outside
// [0,K) becomes 0 and is reported) and looks up the steps' in-degree class;
// padded steps use the identity dictionary entry K.
template <int N, int TAU, class E>
__device__ __forceinline__ void finish_chunk(const FusedArgs& a, const Smem& s, int lane, Chunk<N, TAU, E>& q,
                                             bool& bad) {
    if (lane < q.len) {
        const bool bk = (unsigned)q.kv >= (unsigned)a.K;
        bad |= bk;
        q.kv = bk ? 0 : q.kv;
    } else {
        q.kv = a.K;
    }
    q.mv = s.mtab[q.kv];
}


// ================================================================== forward
// ------------------------------------------------------------------ sorted chunk maps
// For a many-to-one chunk map the frontier applies carry -> Pi (Delta .* carry)
// without float atomics: the chunk wave orders the map's sources by
// (destination, source); the frontier stores Delta_j carry_j at source j's
// sorted position (a permutation, no collisions), adds up each
// destination's run with a segmented scan across lanes, and every
// destination reads the total at the end of its run.  Runs add their sources
// in ascending source order, so the result is deterministic.
constexpr uint16_t kNoRun = 0xffff;

// Sorted form of the map pm (source j = lane*SL + r goes to row pm[r]),
// written into operator slot `slot`: agp = sorted position of every source,
// age = last position of every destination's run (kNoRun if it has no
// source), agh = run-start flags of the positions.  Runs list their sources
// in ascending order; the ranks come from lane-mask tables (map_ranks).
// OFF: N ints of this wave's scratch; MT: SL tables of N words in this
// wave's staging buffers, free outside the pass.
template <int N>
__device__ __forceinline__ void publish_sorted_map(const Smem& s, int slot, const IV<Lay<N>::SL>& pm, int lane,
                                                   bool act, int* OFF, uint64_t* const (&MT)[Lay<N>::SL]) {
    constexpr int SL = Lay<N>::SL;
    int rank[SL], cnt[SL];
    map_ranks<N>(pm, lane, act, MT, rank, cnt);
    int tot = 0;
#pragma unroll
    for (int r = 0; r < SL; ++r) tot += cnt[r];
    int off = wave_incl_scan_i(tot) - tot;  // first position of this lane's first row
    uint16_t* AE = s.age + slot * N;
    uint8_t* AH = s.agh + slot * N;
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            OFF[lane * SL + r] = off;
            AE[lane * SL + r] = cnt[r] ? (uint16_t)(off + cnt[r] - 1) : kNoRun;
            AH[lane * SL + r] = 0;
            off += cnt[r];
        }
    }
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            const int p = OFF[pm.v[r]] + rank[r];
            s.agp[slot * N + lane * SL + r] = (uint8_t)p;
            if (rank[r] == 0) AH[p] = 1;
        }
    }
}

// ------------------------------------------------------------------ work units
// The chunk range of one workgroup: chunks [c0, c0 + nc) of sequence seq,
// segment sg of S (S = 1: the whole sequence).  A grid of B*H*nseg
// workgroups covers segments first_sg .. first_sg + nseg - 1 of every
// sequence; the segments of one sequence sit on one XCD.
struct Work {
    int seq, bb, hh, sg, c0, nc;
    int wa;   // chunk waves the forward uses (<= W; the rest stay idle); its LDS layout is built for wa
    int sbm;  // saved-state rows the forward stages in LDS (0: stored as computed)
};

// The chunk waves a forward workgroup uses: w.wa in a wide kernel (a head of
// permutations may run fewer), else W itself as a compile-time constant (so
// that slot numbers and buffer offsets fold into the instructions).
template <int W>
__device__ __forceinline__ int active_waves(const Work& w) {
    if constexpr (W > kPermWaves) return w.wa;
    else return W;
}

__device__ __forceinline__ Work work_of(const FusedArgs& a, int nseg, int first_sg) {
    Work w;
    const int u = xcd_seq(a.B * a.H * nseg);
    w.seq = u / nseg;
    w.sg = u - w.seq * nseg + first_sg;
    w.bb = w.seq / a.H;
    w.hh = w.seq - w.bb * a.H;
    w.c0 = w.sg * a.Cs;
    w.nc = min(a.C - w.c0, a.Cs);
    w.wa = 0;
    w.sbm = 0;
    return w;
}

// The state entering segment w.sg: h0 (or 0) pushed through the aggregates
// of segments 0 .. w.sg-1, carry <- B_s + Phi_s carry, each row adding its
// sources in ascending order (cross-lane values by readlane).
template <int N, class E>
__device__ __forceinline__ CV<Lay<N>::SL, E> seg_enter_fwd(const FusedArgs& a, const Work& w, int lane, bool act) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    CV<SL, E> carry = cv_zero<SL, E>();
    if (a.h0 && act) carry = ld_state<E, SL>(a.h0 + (size_t)w.seq * N, lane);
    for (int sp = 0; sp < w.sg; ++sp) {
        const size_t base = ((size_t)w.seq * a.S + sp) * N;
        CV<SL, E> acc = cv_zero<SL, E>(), v = cv_zero<SL, E>();
        IV<SL> P;
#pragma unroll
        for (int r = 0; r < SL; ++r) P.v[r] = 0;
        if (act) {
            acc = ld_state<E, SL>(a.segA + base, lane);
            const CV<SL, E> d = ld_state<E, SL>(a.segD + base, lane);
            P = ld_iv<SL>(a.segP + base, lane);
#pragma unroll
            for (int r = 0; r < SL; ++r) v.v[r] = cmul(d.v[r], carry.v[r]);
        }
        for (int jl = 0; jl < LANES; ++jl) {
#pragma unroll
            for (int q = 0; q < SL; ++q) {
                const int pj = readlane_i(P.v[q], jl);
                const E vj = readlane_e(v.v[q], jl);
#pragma unroll
                for (int r = 0; r < SL; ++r) {
                    const bool hit = pj == lane * SL + r;
                    acc.v[r] = cadd(acc.v[r], hit ? vj : ezero<E>());
                }
            }
        }
        carry = acc;
    }
    return carry;
}

// A wave's running fold in the aggregate pass: map, diagonal and local state
// of the chunks it has folded so far (identity and zero at its first one).
template <int SL, class E>
struct RunState {
    IV<SL> pm;
    CV<SL, E> dm, Bm;
};

// A published operator entry: local state and diagonal side by side (one
// 16-byte word for complex values, 8 bytes for real ones).
__device__ __forceinline__ void put_op(float4* agg, int i, float2 B, float2 d) {
    agg[i] = make_float4(B.x, B.y, d.x, d.y);
}
__device__ __forceinline__ void put_op(float4* agg, int i, float B, float d) {
    reinterpret_cast<float2*>(agg)[i] = make_float2(B, d);
}
__device__ __forceinline__ void get_op(const float4* agg, int i, float2& B, float2& d) {
    const float4 e = agg[i];
    B = make_float2(e.x, e.y);
    d = make_float2(e.z, e.w);
}
__device__ __forceinline__ void get_op(const float4* agg, int i, float& B, float& d) {
    const float2 e = reinterpret_cast<const float2*>(agg)[i];
    B = e.x;
    d = e.y;
}

// Writes an operator (local state Bm, diagonal dm, map pm) into operator slot
// `slot` (and its sorted map, many-to-one heads), then raises the slot's flag
// to `flag`.  AGG also keeps the plain map for the frontier's composition.
template <int N, int G, bool FB, bool AGG, class E>
__device__ __forceinline__ void publish_op(const Smem& s, int wa, int wv, int slot, int flag, const IV<Lay<N>::SL>& pm,
                                           const CV<Lay<N>::SL, E>& dm, const CV<Lay<N>::SL, E>& Bm, int lane,
                                           bool act) {
    constexpr int SL = Lay<N>::SL;
    // scratch for the sorted map: the wave's buffers in their complex
    // layout, whatever the element type (no other wave's buffers overlap)
    const Stage<float2> st = stage_of<N>(s, wv);
    float2* X = s.x + wv * N;
    float2* CS = s.cs + wv * N;
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            put_op(s.agg, slot * N + lane * SL + r, Bm.v[r], dm.v[r]);
            if constexpr (G == 1 && !FB) s.agp[slot * N + lane * SL + r] = (uint8_t)pm.v[r];
            if constexpr (AGG) s.agm[slot * N + lane * SL + r] = (uint8_t)pm.v[r];
        }
    }
    if constexpr (!(G == 1 && !FB)) {
        uint64_t* mt[SL];
        mt[0] = reinterpret_cast<uint64_t*>(CS);
        if constexpr (SL > 1) mt[1] = reinterpret_cast<uint64_t*>(CS + wa * N);
        if constexpr (SL > 2) {
            mt[2] = reinterpret_cast<uint64_t*>(st.Z);
            mt[3] = reinterpret_cast<uint64_t*>(st.V);  // rows 0..N-1: the zero row V[N] stays
        }
        publish_sorted_map<N>(s, slot, pm, lane, act, reinterpret_cast<int*>(X), mt);
    }
    wave_sync();
    if (lane == 0) publish_ready(s.aflag + slot, flag);
}

// One chunk is run once, from a zero state (Algorithm 1 Phase A), while the
// readout is split as in Phase C: with M_t = A_t ... A_s in PD form
// (Pi_t, Delta_t) and x_t = x_t^loc + M_t carry,
//   y_t = Re<c_t, x_t^loc> + Re sum_j w_t[j] carry[j],  w_t[j] = Delta_t[j] c_t[Pi_t[j]].
// The wave keeps w_t and the local readout partials, hands the carry on as
// soon as the chunk is folded, and finishes y once its own carry arrives.
// AGG: the aggregate pass of a segment -- the wave only builds and publishes
// the chunk operator (c is not loaded, no readout).  RUN (with AGG): the pass
// starts from and returns to *run instead, and publishes nothing.
template <int N, int TAU, int W, int G, bool FB, bool AGG, bool RUN = false, class E>
__device__ __forceinline__ void fwd_chunk(const FusedArgs& a, const Smem& s, const Work& w, int lc,
                                          Chunk<N, TAU, E>& q, bool& bad, RunState<Lay<N>::SL, E>* run = nullptr) {
    static_assert(!RUN || AGG, "a run fold is an aggregate pass");
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    const int wv = wave_id(), lane = lane_id();
    const bool act = lane < LANES;
    const int ch = w.c0 + lc;
    const Stage<E> st = stage_of<N, E>(s, wv);
    const int WA = active_waves<W>(w);
    // c staging buffer 0, and buffer 1 Wa*N complex slots further (the
    // layout's wave count), in elements
    E* CS = reinterpret_cast<E*>(s.cs + wv * N);
    const int csb = WA * N * (int)(sizeof(float2) / sizeof(E));
    finish_chunk<N, TAU>(a, s, lane, q, bad);

    // ---- 2. one pass: local state B, chunk operator (Pi, Delta), w_t, local readout
    IV<SL> pm;
    CV<SL, E> dm, Bm = cv_zero<SL, E>();
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        pm.v[r] = lane * SL + r;
        dm.v[r] = eone<E>();
    }
    if constexpr (RUN) {
        pm = run->pm;
        dm = run->dm;
        Bm = run->Bm;
    }
    CV<SL, E> wt[TAU];
    float yl[TAU];
    // Pipelined form (no step of the chunk may use a sorted-form entry):
    // every step's gather records are read at chunk start; step t then issues
    // one batch of LDS reads -- its gathers, D_t and pi_t at Pi_{t-1}, and
    // c_{t-1} at Pi_{t-1} for w_{t-1} (c staged in two alternating buffers)
    // -- so each step waits for one round trip.  Otherwise the step-by-step
    // form, where each step waits for its own writes and reads.
    //
    // With real elements a head with sorted-form entries runs the pipelined
    // pass on every chunk none of whose steps uses one (one ballot over the
    // steps' classes per chunk; measured hybrid-lm 413.7 -> 385.7 us, within
    // 1% of the same maps without the entry).  With complex elements the two
    // passes in one kernel cost registers (measured: hybrid-lm in bf16 pairs
    // 580 -> 1209 us), so those heads keep the step-by-step form; a per-step
    // test inside the pipelined pass measured 13% slower at N = 128.
    constexpr bool kPipe = Sentinel<N>::kZeroRow && (!FB || sizeof(E) == sizeof(float));
    constexpr bool kStep = FB || !Sentinel<N>::kZeroRow;
    bool pipe = kPipe && !FB;
    if constexpr (kPipe && FB) pipe = __builtin_amdgcn_ballot_w64(q.mv == (int)kFallback) == 0;
    if constexpr (kPipe) {
        if (pipe) {
            uint64_t rec[TAU][SL];
#pragma unroll
            for (int t = 0; t < TAU; ++t) {
                const int k = readlane_i(q.kv, t);
#pragma unroll
                for (int r = 0; r < SL; ++r) rec[t][r] = act ? s.rec[(size_t)k * N + lane * SL + r] : 0;
            }
#pragma unroll
            for (int t = 0; t < TAU; ++t) {
                const int k = readlane_i(q.kv, t), gk = readlane_i(q.mv, t);
                E* CSt = CS + (t & 1) * csb;
                const E* CSp = CS + ((t + 1) & 1) * csb;
                const CV<SL, E> Dv = Dt(q, t);
                wave_sync();
                if (act) {
#pragma unroll
                    for (int r = 0; r < SL; ++r) {
                        if constexpr (!AGG) CSt[lane * SL + r] = q.c[t].v[r];
                        st.V[lane * SL + r] = cmul(Dv.v[r], Bm.v[r]);
                        st.Z[lane * SL + r] = Dv.v[r];
                    }
                }
                wave_sync();
                float part = 0.f;
                if (act) {
                    // the first GM sources of every row with the step's other
                    // reads in one batch; the 7-source class reads the rest only
                    // at steps whose map has a row with more than GM sources
                    constexpr int GM = G > 4 ? 4 : G;
                    E acc[SL], Dp[SL], Cp[SL];
                    int np[SL];
#pragma unroll
                    for (int r = 0; r < SL; ++r) {
                        acc[r] = q.b[t].v[r];
                        gather_rec_range<0, GM>(st.V, rec[t][r], acc[r]);
                        const int p = pm.v[r];
                        Dp[r] = st.Z[p];
                        np[r] = s.dict[k * N + p];
                        if constexpr (!AGG) Cp[r] = CSp[p];
                    }
                    if constexpr (G > GM) {
                        if (gk > GM) {
#pragma unroll
                            for (int r = 0; r < SL; ++r) gather_rec_range<GM, G>(st.V, rec[t][r], acc[r]);
                        }
                    }
#pragma unroll
                    for (int r = 0; r < SL; ++r) {
                        if constexpr (!AGG) {
                            if (t > 0) wt[t - 1].v[r] = cmul(dm.v[r], Cp[r]);
                        }
                        Bm.v[r] = acc[r];
                        dm.v[r] = cmul(Dp[r], dm.v[r]);
                        pm.v[r] = np[r];
                        if constexpr (!AGG) part = re_fma(part, q.c[t].v[r], Bm.v[r]);
                    }
                } else if constexpr (!AGG) {
                    if (t > 0) wt[t - 1] = cv_zero<SL, E>();
                }
                yl[t] = part;
            }
            if constexpr (!AGG) {
                const E* CSl = CS + ((TAU - 1) & 1) * csb;
                wave_sync();
                if (act) {
#pragma unroll
                    for (int r = 0; r < SL; ++r) wt[TAU - 1].v[r] = cmul(dm.v[r], CSl[pm.v[r]]);
                } else {
                    wt[TAU - 1] = cv_zero<SL, E>();
                }
            }
        }
    }
    if constexpr (kStep) {
        if (!pipe) {
#pragma unroll
            for (int t = 0; t < TAU; ++t) {
                const int k = readlane_i(q.kv, t);
                const int M = readlane_i(q.mv, t);
                if (!AGG && act) {
                    wave_sync();
#pragma unroll
                    for (int r = 0; r < SL; ++r) CS[lane * SL + r] = q.c[t].v[r];
                }
                pd_step<N, G, FB, true>(s, st, lane, act, k, M, Bm, Dt(q, t), q.b[t]);
                float part = 0.f;
                if (act) {
#pragma unroll
                    for (int r = 0; r < SL; ++r) {
                        // (Pi, Delta) <- (pi_t[Pi], D_t[Pi] * Delta), D_t staged in Z
                        const int p = pm.v[r];
                        dm.v[r] = cmul(st.Z[p], dm.v[r]);
                        pm.v[r] = s.dict[k * N + p];
                        if constexpr (!AGG) {
                            wt[t].v[r] = cmul(dm.v[r], CS[pm.v[r]]);
                            part = re_fma(part, q.c[t].v[r], Bm.v[r]);
                        }
                    }
                } else if constexpr (!AGG) {
                    wt[t] = cv_zero<SL, E>();
                }
                yl[t] = part;
            }
        }
    }

    // ---- 3. publish the chunk operator for the frontier wave, take carry_c.
    // Slot reuse (Wa = w.wa chunk waves, the stride of the chunks): the
    // operator of local chunk lc + 2Wa goes where that of lc went.  This wave
    // writes it only after carry_{lc+Wa} arrived, which the frontier
    // publishes after it read operator lc (the aggregate pass waits for that
    // hand-off count explicitly).  Carry slot lc % (Wa + 1) is rewritten with
    // carry_{lc+Wa+1} only after the frontier took operator lc + Wa from this
    // same wave, which this wave publishes after its read of carry_lc below
    // (one wave's LDS accesses complete in order).
    if constexpr (RUN) {
        run->pm = pm;
        run->dm = dm;
        run->Bm = Bm;
        note_progress(s);
        return;
    }
    {
        const int slot = lc % (2 * WA);
        if constexpr (AGG) wait_ready(s.ready, lc - 2 * WA + 1, a.status, s.ready, 1 + 2 * WA, s.prog);
        publish_op<N, G, FB, AGG>(s, WA, wv, slot, lc, pm, dm, Bm, lane, act);
    }
    if constexpr (AGG) return;
    wait_ready(s.ready, lc + 1, a.status, s.ready, 1 + 2 * WA, s.prog);
    CV<SL, E> carry = cv_zero<SL, E>();
    if (act) carry = ld_cv<SL>(reinterpret_cast<const E*>(s.ring) + (lc % (WA + 1)) * N, lane);
    if (act && a.saved && w.sbm == 0) {
        if constexpr (sizeof(E) == sizeof(float)) st_srow<SL>(a.saved, ((size_t)w.seq * a.C + ch) * N, lane, carry);
        else st_state<SL>(a.saved + ((size_t)w.seq * a.C + ch) * N, lane, carry);
    }

    // ---- 4. readout correction with the true carry, then one store per chunk
#pragma unroll
    for (int t = 0; t < TAU; ++t) {
#pragma unroll
        for (int r = 0; r < SL; ++r) yl[t] = re_fma(yl[t], wt[t].v[r], carry.v[r]);
    }
    const float yv = transpose_sum<TAU>(yl, lane);
    const int t = lane / (kWave / TAU);
    if (lane % (kWave / TAU) == 0 && t < q.len)
        a.y[((size_t)w.bb * a.L + ch * TAU + t) * a.H + w.hh] = yv;
}

// A published chunk operator as the frontier wave holds it: local state B
// and diagonal d; p = the map (permutation heads) or the sorted position of
// each source; e, h = run ends per destination and run-start flags per
// position (many-to-one heads).
template <int SL, class E>
struct ChunkOp {
    CV<SL, E> B, d;
    IV<SL> p, e, h;
};

template <int N, bool SORTED, class E>
__device__ __forceinline__ ChunkOp<Lay<N>::SL, E> read_op(const Smem& s, int slot, int lane, bool act) {
    constexpr int SL = Lay<N>::SL;
    ChunkOp<SL, E> o;
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        o.B.v[r] = o.d.v[r] = ezero<E>();
        o.p.v[r] = o.e.v[r] = o.h.v[r] = 0;
    }
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            const int i = slot * N + lane * SL + r;
            get_op(s.agg, i, o.B.v[r], o.d.v[r]);
            o.p.v[r] = s.agp[i];
            if constexpr (SORTED) {
                o.e.v[r] = s.age[i];
                o.h.v[r] = s.agh[i];
            }
        }
    }
    return o;
}

// nxt = B + Pi (Delta .* carry) for a sorted many-to-one operator; X: N
// complex values of LDS scratch.
template <int N, class E>
__device__ __forceinline__ CV<Lay<N>::SL, E> apply_sorted(const ChunkOp<Lay<N>::SL, E>& op,
                                                          const CV<Lay<N>::SL, E>& carry, E* X, int lane, bool act) {
    constexpr int SL = Lay<N>::SL;
    CV<SL, E> u = cv_zero<SL, E>();
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) X[op.p.v[r]] = cmul(op.d.v[r], carry.v[r]);
    }
    wave_sync();
    if (act) u = ld_cv<SL>(X, lane);
    bool st[SL];
    int e[SL];
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        st[r] = op.h.v[r] != 0;
        e[r] = op.e.v[r] == kNoRun ? -1 : op.e.v[r];
    }
    const CV<SL, E> tot = run_totals<N, E>(X, u, st, e, lane, act);
    CV<SL, E> nxt = cv_zero<SL, E>();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) nxt.v[r] = cadd(op.B.v[r], tot.v[r]);
    }
    return nxt;
}

// The frontier wave: keeps the running state in registers and, chunk by
// chunk, hands carry_c to the chunk's wave and applies the chunk's published
// operator: carry_{c+1} = B_c + (Pi_c, Delta_c) carry_c.  Per chunk its
// critical path is one pipelined batch of LDS accesses: the carry store, the
// scatter and the read-back, with the next chunk's operator read
// speculatively in the same batch (LDS accesses of one wave complete in issue
// order, so operator data read after a flag that shows it published is that
// operator's; a flag still behind sends the wave to a bounded wait and a
// re-read).  The wave runs at raised issue priority: it shares its SIMD with
// chunk waves whose long arithmetic runs would otherwise delay it.
template <int N, int W, int G, bool FB, bool AGG, class E>
__device__ __forceinline__ void fwd_frontier(const FusedArgs& a, const Smem& s, const Work& w) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    constexpr bool kPerm = G == 1 && !FB;
    const int lane = lane_id();
    const bool act = lane < LANES;
    const int WA = active_waves<W>(w);
    E* X = reinterpret_cast<E*>(s.x + WA * N);
    E* ring = reinterpret_cast<E*>(s.ring);
    int* flags = s.ready;
    const int nflags = 1 + 2 * WA;
    // The aggregate pass folds the segment from zero and composes its map;
    // the scan starts from the state entering its segment.
    CV<SL, E> carry = AGG ? cv_zero<SL, E>() : seg_enter_fwd<N, E>(a, w, lane, act);
    IV<SL> accP;
    CV<SL, E> accD;
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        accP.v[r] = lane * SL + r;
        accD.v[r] = eone<E>();
    }
    __builtin_amdgcn_s_setprio(3);
    wait_ready(s.aflag, 0, a.status, flags, nflags, s.prog);
    ChunkOp<SL, E> op = read_op<N, !kPerm, E>(s, 0, lane, act);
    const int M = AGG || !a.saved ? 0 : w.sbm;
    // slot indices c % (Wa + 1) (carry ring) and c % (2 Wa) (operators),
    // advanced by one per chunk
    const int nring = WA + 1, nops = 2 * WA;
    int rslot = 0, oslot = 0;
    for (int c = 0; c < w.nc; ++c) {
        wave_sync();
        if (!AGG && act) st_cv<SL>(ring + rslot * N, lane, carry);
        rslot = rslot + 1 == nring ? 0 : rslot + 1;
        if (M > 0 && act) {
            // the first M chunk states wait in LDS until the whole workgroup
            // has read its rows; later ones (near the end anyway) go out now.
            // (Staging the real model's states as floats measured 2% slower
            // at markov-manyone: the compiler spills more scalar registers.)
            if (c < M) st_state<SL>(s.sb + c * N, lane, carry);
            else if constexpr (sizeof(E) == sizeof(float))
                st_srow<SL>(a.saved, ((size_t)w.seq * a.C + w.c0 + c) * N, lane, carry);
            else st_state<SL>(a.saved + ((size_t)w.seq * a.C + w.c0 + c) * N, lane, carry);
        }
        CV<SL, E> nxt;
        if constexpr (kPerm) {
            // every entry is a permutation, so is Pi_c: scatter by plain stores
            if (act) {
#pragma unroll
                for (int r = 0; r < SL; ++r) X[op.p.v[r]] = cmul(op.d.v[r], carry.v[r]);
            }
        }
        const bool more = c + 1 < w.nc;
        [[maybe_unused]] const int slot = oslot;
        const int nslot = oslot + 1 == nops ? 0 : oslot + 1;
        oslot = nslot;
        int seen = 0x7fffffff;
        ChunkOp<SL, E> nx;
        if (more) {
            seen = __hip_atomic_load(s.aflag + nslot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            issue_fence();
            nx = read_op<N, !kPerm, E>(s, nslot, lane, act);
        }
        if constexpr (kPerm) {
            wave_sync();
            nxt = cv_zero<SL, E>();
            if (act) nxt = ld_cv<SL>(X, lane);
#pragma unroll
            for (int r = 0; r < SL; ++r) nxt.v[r] = cadd(nxt.v[r], op.B.v[r]);
        } else {
            nxt = apply_sorted<N, E>(op, carry, X, lane, act);
        }
        if constexpr (AGG) {
            // Phi_acc <- Phi_c Phi_acc: (Pi_c[Pi_acc], Delta_c[Pi_acc] * Delta_acc)
            if (act) {
#pragma unroll
                for (int r = 0; r < SL; ++r) {
                    const int p = accP.v[r];
                    E Bc, dc;
                    get_op(s.agg, slot * N + p, Bc, dc);
                    accD.v[r] = cmul(dc, accD.v[r]);
                    accP.v[r] = s.agm[slot * N + p];
                }
            }
        }
        wave_sync();
        if (lane == 0) publish_ready(s.ready, c + 1);
        carry = nxt;
        if (more) {
            if (__builtin_amdgcn_readfirstlane(seen) < c + 1) {
                wait_ready(s.aflag + nslot, c + 1, a.status, flags, nflags, s.prog);
                nx = read_op<N, !kPerm, E>(s, nslot, lane, act);
            }
            op = nx;
        }
    }
    __builtin_amdgcn_s_setprio(0);
    if constexpr (AGG) {
        const size_t base = ((size_t)w.seq * a.S + w.sg) * N;
        if (act) {
            st_state<SL>(a.segA + base, lane, carry);
            st_state<SL>(a.segD + base, lane, accD);
            st_iv<SL>(a.segP + base, lane, accP);
        }
    } else if (act && a.hfinal && w.sg == a.S - 1) {
        st_state<SL>(a.hfinal + (size_t)w.seq * N, lane, carry);
    }
}

// Wave wv owns local chunks wv, wv+W, ...; with PREFETCH the loads of its next
// chunk are in flight while it computes the current one (two register
// buffers).  A local chunk past the range issues an empty chunk.
template <int N, int TAU, int W, int G, bool FB, bool PREFETCH, bool AGG, int IO>
__device__ __forceinline__ void fwd_body(const FusedArgs& a, const Smem& s, const Work& w) {
    using E = typename ElemOf<IO>::T;
    constexpr int LANES = Lay<N>::LANES;
    const int wv = wave_id(), lane = lane_id();
    const bool act = lane < LANES;
    auto issue = [&](int lc, Chunk<N, TAU, E>& q) {
        issue_chunk<N, TAU, true, !AGG, kLoadStream, IO>(a, w.bb, w.hh, lc < w.nc ? w.c0 + lc : a.C, lane, act, q);
    };
    bool bad = false;
    if constexpr (AGG) {
        // The aggregate needs no chunk-by-chunk hand-off: wave wv folds a
        // contiguous run of chunks, carrying map, diagonal and local state
        // from chunk to chunk, and publishes the run's operator in slot wv
        // (flag wv); the frontier composes the runs in order, as it would
        // chunks.  Runs <= W < 2W slots, so no slot is reused.  The cut into
        // at most kFusedWaves runs does not depend on W, so the wide kernels
        // of the 4-byte formats add in the same order as complex64's (same
        // bits on the same values).
        constexpr int SL = Lay<N>::SL, RUNS = W < kFusedWaves ? W : kFusedWaves;
        const int per = max(1, (w.nc + RUNS - 1) / RUNS);
        const int runs = (w.nc + per - 1) / per;
        if (wv == W) {
            Work wr = w;
            wr.nc = runs;
            fwd_frontier<N, W, G, FB, true, E>(a, s, wr);
            return;
        }
        if (wv >= runs) return;
        const int r0 = wv * per, r1 = min(w.nc, r0 + per);
        RunState<SL, E> rs;
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            rs.pm.v[r] = lane * SL + r;
            rs.dm.v[r] = eone<E>();
            rs.Bm.v[r] = ezero<E>();
        }
        if constexpr (PREFETCH) {
            Chunk<N, TAU, E> qa, qb;
            issue(r0, qa);
            for (int lc = r0; lc < r1; lc += 2) {
                issue(lc + 1 < r1 ? lc + 1 : w.nc, qb);
                issue_fence();
                fwd_chunk<N, TAU, W, G, FB, true, true>(a, s, w, lc, qa, bad, &rs);
                if (lc + 1 >= r1) break;
                issue(lc + 2 < r1 ? lc + 2 : w.nc, qa);
                issue_fence();
                fwd_chunk<N, TAU, W, G, FB, true, true>(a, s, w, lc + 1, qb, bad, &rs);
            }
        } else {
            for (int lc = r0; lc < r1; ++lc) {
                Chunk<N, TAU, E> q;
                issue(lc, q);
                fwd_chunk<N, TAU, W, G, FB, true, true>(a, s, w, lc, q, bad, &rs);
            }
        }
        publish_op<N, G, FB, true>(s, active_waves<W>(w), wv, wv, wv, rs.pm, rs.dm, rs.Bm, lane, act);
        if (bad) report_index_error(a.status);
        return;
    }
    if (wv == W) {
        fwd_frontier<N, W, G, FB, AGG, E>(a, s, w);
        return;
    }
    const int WA = active_waves<W>(w);
    if (wv >= WA) return;
    if constexpr (PREFETCH) {
        Chunk<N, TAU, E> qa, qb;
        issue(wv, qa);
        for (int lc = wv; lc < w.nc; lc += 2 * WA) {
            issue(lc + WA, qb);
            issue_fence();
            fwd_chunk<N, TAU, W, G, FB, AGG>(a, s, w, lc, qa, bad);
            if (lc + WA >= w.nc) break;
            issue(lc + 2 * WA, qa);
            issue_fence();
            fwd_chunk<N, TAU, W, G, FB, AGG>(a, s, w, lc + WA, qb, bad);
        }
    } else {
        for (int lc = wv; lc < w.nc; lc += WA) {
            Chunk<N, TAU, E> q;
            issue(lc, q);
            fwd_chunk<N, TAU, W, G, FB, AGG>(a, s, w, lc, q, bad);
        }
    }
    if (bad) report_index_error(a.status);
}

template <int N, int TAU, int W, bool AGG, int IO>
__global__ __launch_bounds__((W + 1) * 64) void k_fwd_fused(FusedArgs a) {
    extern __shared__ __align__(16) unsigned char lds[];
    Smem s = carve_smem(lds, a.lds);
    Work w = AGG ? work_of(a, a.S - 1, 0) : work_of(a, a.S, 0);

    stage_tables<N>(a, s, w.hh);
    __syncthreads();
    bool fb;
    const int G = head_variant(s, a.K, fb);
    // Heads of permutations stream complex64 rows at the pace of HBM with
    // kPermWaves chunk waves: more waves only add loads in flight, and the
    // layout of fewer waves leaves LDS for more staged chunk states.  Other
    // heads are bound by their chunk passes and use all W.  The tables sit
    // at the same offsets in both layouts.
    const bool narrow = __builtin_amdgcn_readfirstlane(!AGG && IO == kIoC64 && G == 1 && !fb && W > kPermWaves) != 0;
    w.wa = narrow ? kPermWaves : W;
    w.sbm = narrow ? a.sbM_perm : a.sbM;
    if (narrow) s = carve_smem(lds, a.lds_perm);
    clear_zero_rows<N, typename ElemOf<IO>::T>(s, w.wa);
    if (threadIdx.x == 0) {
        *s.ready = 0;
        *s.prog = 0;
    }
    for (int i = threadIdx.x; i < 2 * w.wa; i += blockDim.x) s.aflag[i] = -1;
    __syncthreads();
    // The aggregate pass loads D and b only and keeps no readout state: its
    // runs prefetch the next chunk at every N (measured registers fit).
    constexpr bool PF = fused_prefetch(N, TAU) || AGG;
    if (fb) fwd_body<N, TAU, W, 7, true, PF, AGG, IO>(a, s, w);
    else if (G == 1) fwd_body<N, TAU, W, 1, false, PF, AGG, IO>(a, s, w);
    else if (G == 3) fwd_body<N, TAU, W, 3, false, PF, AGG, IO>(a, s, w);
    else fwd_body<N, TAU, W, 7, false, PF, AGG, IO>(a, s, w);
    if constexpr (!AGG) {
        // write out the staged chunk states, every wave a share of the rows
        if (w.sbm > 0 && a.saved) {
            constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
            const int lane = lane_id();
            __syncthreads();
            const int rows = min(w.sbm, w.nc);
            if constexpr (IO == kIoReal) {
                // the real model's states leave as their real parts
                const size_t dst = ((size_t)w.seq * a.C + w.c0) * N;
                if (lane < LANES)
                    for (int i = wave_id(); i < rows; i += W + 1)
                        st_srow<SL>(a.saved, dst + (size_t)i * N, lane, ld_state<float, SL>(s.sb + (size_t)i * N, lane));
            } else {
                float2* dst = a.saved + ((size_t)w.seq * a.C + w.c0) * N;
                if (lane < LANES)
                    for (int i = wave_id(); i < rows; i += W + 1)
                        st_cv<SL>(dst + (size_t)i * N, lane, ld_cv<SL>(s.sb + i * N, lane));
            }
        }
    }
}

// ================================================================== backward
// The backward streams its inputs and its gradient rows (each byte is read
// or written once): nontemporal loads and stores.
template <int IO, int SL, class E>
__device__ __forceinline__ void st_out(void* rows, size_t off, int lane, const CV<SL, E>& x) {
    if constexpr (IO == kIoReal) st_row_r_stream<SL>(reinterpret_cast<float*>(rows) + off, lane, x);
    else if constexpr (IO == kIoBf16) st_row_w_stream<SL, IO>(reinterpret_cast<uint32_t*>(rows) + off, lane, x);
    else st_cv_stream<SL>(reinterpret_cast<float2*>(rows) + off, lane, x);
}
// Per-chunk registers of the backward: the chunk's rows, the saved state
// entering it and its dy values (lane t holds dy of step t).
template <int N, int TAU, class E>
struct BwdChunk {
    Chunk<N, TAU, E> q;
    CV<Lay<N>::SL, E> hs;
    float dyv;
};

// Issues every load of reverse-order local chunk r (chunk c0 + nc - 1 - r);
// r >= nc issues an empty chunk through the null descriptor, as issue_chunk
// does.  The aggregate pass needs neither b nor the saved states.
template <int N, int TAU, bool AGG, int IO>
__device__ __forceinline__ void issue_bwd(const FusedArgs& a, const Work& w, int r, int lane, bool act,
                                          BwdChunk<N, TAU, typename ElemOf<IO>::T>& u) {
    using E = typename ElemOf<IO>::T;
    constexpr int SL = Lay<N>::SL;
    const int ch = r < w.nc ? w.c0 + w.nc - 1 - r : a.C;
    issue_chunk<N, TAU, !AGG, true, kLoadStream, IO>(a, w.bb, w.hh, ch, lane, act, u.q);
    const int chc = min(ch, a.C - 1);
    const int s0 = chc * TAU;
    const int lenc = min(TAU, a.L - s0);
    u.dyv = a.dy[((size_t)w.bb * a.L + s0 + min(lane, lenc - 1)) * a.H + w.hh];
    if constexpr (!AGG)
        u.hs = act ? ld_srow<SL, E>(a.saved, ((size_t)w.seq * a.C + chc) * N, lane) : cv_zero<SL, E>();  // real: fp32 rows
}

// AGG: the aggregate pass of a segment -- each chunk's adjoint operator is
// composed into the running aggregate passed from wave to wave.
template <int N, int TAU, int W, int G, bool FB, bool AGG, bool STE, int IO>
__device__ __forceinline__ void bwd_chunk(const FusedArgs& a, const Smem& s, const Work& w, int r,
                                          BwdChunk<N, TAU, typename ElemOf<IO>::T>& u, bool& bad) {
    using E = typename ElemOf<IO>::T;
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    const int wv = wave_id(), lane = lane_id();
    const bool act = lane < LANES;
    const Stage<E> st = stage_of<N, E>(s, wv);
    E* ringe = reinterpret_cast<E*>(s.ring);
    uint8_t* PA = s.pa + wv * N;
    const size_t stride = (size_t)a.H * N;
    const int ch = w.c0 + w.nc - 1 - r;
    const int s0 = ch * TAU;
    const size_t base = (((size_t)w.bb * a.L + s0) * a.H + w.hh) * N;
    const int seq = w.seq;
    Chunk<N, TAU, E>& q = u.q;
    finish_chunk<N, TAU>(a, s, lane, q, bad);
    const float dyv = lane < q.len ? u.dyv : 0.f;

    // ---- local adjoint from zero and the chunk operator, reverse time:
    // Phi <- Phi A_t: pa(j) <- pa[pi_t(j)], da(j) <- da[pi_t(j)] D_t(j)
    CV<SL, E> g = cv_zero<SL, E>(), da;
    IV<SL> pa;
#pragma unroll
    for (int i = 0; i < SL; ++i) {
        pa.v[i] = lane * SL + i;
        da.v[i] = eone<E>();
    }
#pragma unroll
    for (int t = TAU - 1; t >= 0; --t) {
        const int k = readlane_i(q.kv, t);
        const float dyt = readlane_f(dyv, t);
        IV<SL> pt;
        wave_sync();
        if (act) {
#pragma unroll
            for (int i = 0; i < SL; ++i) {
                pt.v[i] = s.dict[k * N + lane * SL + i];
                g.v[i] = add_sconj(g.v[i], dyt, q.c[t].v[i]);
                st.V[lane * SL + i] = g.v[i];
                st.Z[lane * SL + i] = da.v[i];
                PA[lane * SL + i] = (uint8_t)pa.v[i];
            }
        }
        wave_sync();
        if (act) {
#pragma unroll
            for (int i = 0; i < SL; ++i) {
                const E gv = st.V[pt.v[i]], dz = st.Z[pt.v[i]];
                pa.v[i] = PA[pt.v[i]];
                da.v[i] = cmul(dz, Dt(q, t).v[i]);
                g.v[i] = cmulc(Dt(q, t).v[i], gv);
            }
        }
    }

    // ---- hand-off: U_{c-1} = gamma_c + Phi_c^H U_c (a gather from the ring)
#pragma unroll
    for (int i = 0; i < SL; ++i) {
        materialize(pa.v[i]);
        materialize(da.v[i]);
        materialize(g.v[i]);
    }
    wait_ready(s.ready, r, a.status, s.ready, 1, s.prog);
    if constexpr (AGG) {
        // (Gamma, Pi, Delta)_acc <- (gamma_c + Phi_c^H Gamma_acc, Pi_acc[Pi_c], Delta_acc[Pi_c] Delta_c):
        // the aggregate of chunks c .. c1-1, mapping the gradient entering
        // the segment's last chunk to the one leaving chunk c.
        const E* GA = ringe + (r & 1) * N;
        const E* DA = ringe + (2 + (r & 1)) * N;
        const uint8_t* PAc = s.agp + (r & 1) * N;
        CV<SL, E> Gn, Dn;
        IV<SL> Pn;
        if (act) {
#pragma unroll
            for (int i = 0; i < SL; ++i) {
                const int p = pa.v[i];
                Gn.v[i] = cfmac(g.v[i], da.v[i], GA[p]);
                Dn.v[i] = cmul(DA[p], da.v[i]);
                Pn.v[i] = PAc[p];
            }
            st_cv<SL>(ringe + ((r + 1) & 1) * N, lane, Gn);
            st_cv<SL>(ringe + (2 + ((r + 1) & 1)) * N, lane, Dn);
#pragma unroll
            for (int i = 0; i < SL; ++i) s.agp[((r + 1) & 1) * N + lane * SL + i] = (uint8_t)Pn.v[i];
        }
        wave_sync();
        if (lane == 0) publish_ready(s.ready, r + 1);
        if (r == w.nc - 1 && act) {
            const size_t sb = ((size_t)seq * a.S + w.sg) * N;
            st_state<SL>(a.segA + sb, lane, Gn);
            st_state<SL>(a.segD + sb, lane, Dn);
            st_iv<SL>(a.segP + sb, lane, Pn);
        }
        return;
    }
    CV<SL, E> U = cv_zero<SL, E>(), Up;
    if (act) {
        const E* ring = ringe + (r & 1) * N;
        U = ld_cv<SL>(ring, lane);
#pragma unroll
        for (int i = 0; i < SL; ++i) Up.v[i] = cfmac(g.v[i], da.v[i], ring[pa.v[i]]);
        st_cv<SL>(ringe + ((r + 1) & 1) * N, lane, Up);
    }
    wave_sync();
    if (lane == 0) publish_ready(s.ready, r + 1);
    if (ch == 0 && a.dh0 && act) st_state<SL>(a.dh0 + (size_t)seq * N, lane, Up);

    // ---- recompute the chunk's states from the saved entering state
    CV<SL, E> Hs[TAU + 1];
    CV<SL, E> hs = u.hs;
    Hs[0] = hs;
#pragma unroll
    for (int t = 0; t < TAU; ++t) {
        const int k = readlane_i(q.kv, t);
        const int M = readlane_i(q.mv, t);
        pd_step<N, G, FB, false>(s, st, lane, act, k, M, hs, Dt(q, t), q.b[t]);
        Hs[t + 1] = hs;
    }

    // ---- final reverse walk with the true incoming gradient
    g = U;
#pragma unroll
    for (int t = TAU - 1; t >= 0; --t) {
        const int k = readlane_i(q.kv, t);
        const float dyt = readlane_f(dyv, t);
        IV<SL> pt;
        CV<SL, E> dct;
        wave_sync();
        if (act) {
#pragma unroll
            for (int i = 0; i < SL; ++i) {
                pt.v[i] = s.dict[k * N + lane * SL + i];
                g.v[i] = add_sconj(g.v[i], dyt, q.c[t].v[i]);
                dct.v[i] = sconj(dyt, Hs[t + 1].v[i]);
                st.V[lane * SL + i] = g.v[i];
            }
        }
        const bool in = t < q.len;
        const size_t off = base + (size_t)t * stride;
        if (act && in) {
            st_out<IO, SL>(a.db, off, lane, g);
            st_out<IO, SL>(a.dc, off, lane, dct);
        }
        wave_sync();
        if (act) {
            CV<SL, E> dDt;
#pragma unroll
            for (int i = 0; i < SL; ++i) {
                const E gp = st.V[pt.v[i]];
                dDt.v[i] = cmulc(Hs[t].v[i], gp);
                g.v[i] = cmulc(Dt(q, t).v[i], gp);
            }
            if (in) st_out<IO, SL>(a.dD, off, lane, dDt);
        }
        if constexpr (STE) {
            // the scaled state z_t = D_t .* h_{t-1} for the straight-through gradients
            if (act && in) {
                CV<SL, E> zt;
#pragma unroll
                for (int i = 0; i < SL; ++i) zt.v[i] = cmul(Dt(q, t).v[i], Hs[t].v[i]);
                // with bf16 pairs z stays complex64 (rounding it would round
                // the straight-through inputs)
                st_out<(IO == kIoBf16 ? kIoC64 : IO), SL>(a.z, off, lane, zt);
            }
        }
    }
}

// Wave wv owns reverse-order local chunks wv, wv+W, ...; with PREFETCH every
// load of its next chunk is in flight while it computes the current one.
template <int N, int TAU, int W, int G, bool FB, bool PREFETCH, bool AGG, bool STE, int IO>
__device__ __forceinline__ void bwd_body(const FusedArgs& a, const Smem& s, const Work& w) {
    using E = typename ElemOf<IO>::T;
    constexpr int LANES = Lay<N>::LANES;
    const int wv = wave_id(), lane = lane_id();
    const bool act = lane < LANES;
    bool bad = false;
    if constexpr (PREFETCH) {
        BwdChunk<N, TAU, E> ua, ub;
        issue_bwd<N, TAU, AGG, IO>(a, w, wv, lane, act, ua);
        for (int r = wv; r < w.nc; r += 2 * W) {
            issue_bwd<N, TAU, AGG, IO>(a, w, r + W, lane, act, ub);
            issue_fence();
            bwd_chunk<N, TAU, W, G, FB, AGG, STE, IO>(a, s, w, r, ua, bad);
            if (r + W >= w.nc) break;
            issue_bwd<N, TAU, AGG, IO>(a, w, r + 2 * W, lane, act, ua);
            issue_fence();
            bwd_chunk<N, TAU, W, G, FB, AGG, STE, IO>(a, s, w, r + W, ub, bad);
        }
    } else {
        for (int r = wv; r < w.nc; r += W) {
            BwdChunk<N, TAU, E> u;
            issue_bwd<N, TAU, AGG, IO>(a, w, r, lane, act, u);
            bwd_chunk<N, TAU, W, G, FB, AGG, STE, IO>(a, s, w, r, u, bad);
        }
    }
    if (bad) report_index_error(a.status);
}

// The gradient entering segment w.sg from the right: dh_final (or 0) pulled
// back through the aggregates of segments S-1 .. w.sg+1,
// U <- Gamma_s + Phi_s^H U (a gather through the wave's LDS buffer X).
template <int N, class E>
__device__ __forceinline__ CV<Lay<N>::SL, E> seg_enter_bwd(const FusedArgs& a, const Work& w, E* X, int lane,
                                                           bool act) {
    constexpr int SL = Lay<N>::SL;
    CV<SL, E> U = cv_zero<SL, E>();
    if (a.dhf && act) U = ld_state<E, SL>(a.dhf + (size_t)w.seq * N, lane);
    for (int sp = a.S - 1; sp > w.sg; --sp) {
        const size_t base = ((size_t)w.seq * a.S + sp) * N;
        CV<SL, E> Un = cv_zero<SL, E>();
        wave_sync();
        if (act) st_cv<SL>(X, lane, U);
        wave_sync();
        if (act) {
            const CV<SL, E> G = ld_state<E, SL>(a.segA + base, lane);
            const CV<SL, E> d = ld_state<E, SL>(a.segD + base, lane);
            const IV<SL> P = ld_iv<SL>(a.segP + base, lane);
#pragma unroll
            for (int i = 0; i < SL; ++i) Un.v[i] = cfmac(G.v[i], d.v[i], X[P.v[i]]);
        }
        U = Un;
    }
    return U;
}

template <int N, int TAU, int W, bool AGG, bool STE, int IO>
__global__ __launch_bounds__(W * 64) void k_bwd_fused(FusedArgs a) {
    using E = typename ElemOf<IO>::T;
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    extern __shared__ __align__(16) unsigned char lds[];
    const Smem s = carve_smem(lds, a.lds);
    const int wv = wave_id(), lane = lane_id();
    const bool act = lane < LANES;
    const Work w = AGG ? work_of(a, a.S - 1, 1) : work_of(a, a.S, 0);

    stage_tables<N>(a, s, w.hh);
    clear_zero_rows<N, E>(s, W);
    E* ring = reinterpret_cast<E*>(s.ring);
    if (wv == 0) {
        if constexpr (AGG) {
            // identity aggregate: Gamma = 0, Pi = id, Delta = 1
            if (act) {
                st_cv<SL>(ring, lane, cv_zero<SL, E>());
                CV<SL, E> one;
#pragma unroll
                for (int i = 0; i < SL; ++i) {
                    one.v[i] = eone<E>();
                    s.agp[lane * SL + i] = (uint8_t)(lane * SL + i);
                }
                st_cv<SL>(ring + 2 * N, lane, one);
            }
        } else {
            const CV<SL, E> u = seg_enter_bwd<N, E>(a, w, reinterpret_cast<E*>(s.x), lane, act);
            if (act) st_cv<SL>(ring, lane, u);
        }
        if (lane == 0) {
            *s.ready = 0;
            *s.prog = 0;
        }
    }
    __syncthreads();
    bool fb;
    const int G = head_variant(s, a.K, fb);
    constexpr bool PF = fused_prefetch(N, TAU);
    if (fb) bwd_body<N, TAU, W, 7, true, PF, AGG, STE, IO>(a, s, w);
    else if (G == 1) bwd_body<N, TAU, W, 1, false, PF, AGG, STE, IO>(a, s, w);
    else if (G == 3) bwd_body<N, TAU, W, 3, false, PF, AGG, STE, IO>(a, s, w);
    else bwd_body<N, TAU, W, 7, false, PF, AGG, STE, IO>(a, s, w);
}

// Segmented scans (S > 1) first run the aggregate pass over segments that
// have a neighbour to hand to, then the scan over every segment.
template <int N, int TAU, int W, int IO>
hipError_t fwd_launch_io(const FusedArgs& a, hipStream_t st) {
    if (a.S > 1) {
        auto agg = k_fwd_fused<N, TAU, W, true, IO>;
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(agg),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)a.lds.total);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(agg, dim3(a.B * a.H * (a.S - 1)), dim3((W + 1) * 64), a.lds.total, st, a);
    }
    // every workgroup gets the larger of the two layouts' bytes
    const uint32_t bytes = a.lds.total > a.lds_perm.total ? a.lds.total : a.lds_perm.total;
    auto kern = k_fwd_fused<N, TAU, W, false, IO>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.B * a.H * a.S), dim3((W + 1) * 64), bytes, st, a);
    return hipGetLastError();
}

template <int N, int TAU, int W, int IO>
hipError_t bwd_launch_io(const FusedArgs& a, hipStream_t st) {
    if (a.S > 1) {
        auto agg = k_bwd_fused<N, TAU, W, true, false, IO>;
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(agg),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)a.lds.total);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(agg, dim3(a.B * a.H * (a.S - 1)), dim3(W * 64), a.lds.total, st, a);
    }
    // the scaled states for the straight-through gradients come from the scan pass only
    auto kern = a.z ? k_bwd_fused<N, TAU, W, false, true, IO> : k_bwd_fused<N, TAU, W, false, false, IO>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)a.lds.total);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(a.B * a.H * a.S), dim3(W * 64), a.lds.total, st, a);
    return hipGetLastError();
}

// The chunk-wave count of a call: fused_waves(N, TAU), or kFusedWavesWide
// for the prefetching kernels when the caller's layout was built for it, or
// at N = 256 kFusedWavesNarrow / kFusedWavesNarrowest.
template <int N, int TAU, int IO>
hipError_t fwd_dispatch_io(const FusedArgs& a, hipStream_t st) {
    if constexpr (fused_prefetch(N, TAU)) {
        if (a.W == kFusedWavesWide) return fwd_launch_io<N, TAU, kFusedWavesWide, IO>(a, st);
    }
    if constexpr (N == 256) {
        if (a.W == kFusedWavesNarrow) return fwd_launch_io<N, TAU, kFusedWavesNarrow, IO>(a, st);
        if (a.W == kFusedWavesNarrowest) return fwd_launch_io<N, TAU, kFusedWavesNarrowest, IO>(a, st);
    }
    if (a.W != fused_waves(N, TAU)) return hipErrorInvalidValue;
    return fwd_launch_io<N, TAU, fused_waves(N, TAU), IO>(a, st);
}

// The backward's: fused_waves_bwd(N, TAU), or at N = 256 kFusedWavesNarrow
// or kFusedWavesNarrowest.
template <int N, int TAU, int IO>
hipError_t bwd_dispatch_io(const FusedArgs& a, hipStream_t st) {
    if constexpr (N == 256) {
        if (a.W == kFusedWavesNarrow) return bwd_launch_io<N, TAU, kFusedWavesNarrow, IO>(a, st);
        if (a.W == kFusedWavesNarrowest) return bwd_launch_io<N, TAU, kFusedWavesNarrowest, IO>(a, st);
    }
    if (a.W != fused_waves_bwd(N, TAU)) return hipErrorInvalidValue;
    return bwd_launch_io<N, TAU, fused_waves_bwd(N, TAU), IO>(a, st);
}

template <int N>
hipError_t prep_launch(const PrepArgs& p, hipStream_t st) {
    hipLaunchKernelGGL(k_prep<N>, dim3((p.H * p.K + 3) / 4), dim3(256), 0, st, p);
    return hipGetLastError();
}

// The row format (complex64, bf16 pairs, real fp32) picks the instantiation.
// Chunk lengths compiled per N: TAU * max(1, N/64) <= 16 keeps a chunk's
// D, b, c rows (and the backward's recomputed states) in registers.
template <int N, int TAU>
hipError_t fwd_dispatch_waves(const FusedArgs& a, hipStream_t st) {
    switch (a.io) {
        case kIoC64: return fwd_dispatch_io<N, TAU, kIoC64>(a, st);
        case kIoBf16: return fwd_dispatch_io<N, TAU, kIoBf16>(a, st);
        case kIoReal: return fwd_dispatch_io<N, TAU, kIoReal>(a, st);
        default: return hipErrorInvalidValue;
    }
}
template <int N, int TAU>
hipError_t bwd_dispatch_waves(const FusedArgs& a, hipStream_t st) {
    switch (a.io) {
        case kIoC64: return bwd_dispatch_io<N, TAU, kIoC64>(a, st);
        case kIoBf16: return bwd_dispatch_io<N, TAU, kIoBf16>(a, st);
        case kIoReal: return bwd_dispatch_io<N, TAU, kIoReal>(a, st);
        default: return hipErrorInvalidValue;
    }
}

template <int N, bool FWD>
hipError_t dispatch_tau(const FusedArgs& a, hipStream_t st) {
    constexpr int SL = Lay<N>::SL;
    switch (a.tau) {
        case 4:
            return FWD ? fwd_dispatch_waves<N, 4>(a, st) : bwd_dispatch_waves<N, 4>(a, st);
        case 8:
            if constexpr (8 * SL <= 16)
                return FWD ? fwd_dispatch_waves<N, 8>(a, st) : bwd_dispatch_waves<N, 8>(a, st);
            break;
        case 16:
            if constexpr (16 * SL <= 16)
                return FWD ? fwd_dispatch_waves<N, 16>(a, st) : bwd_dispatch_waves<N, 16>(a, st);
            break;
        default: break;
    }
    return hipErrorInvalidValue;
}

}  // namespace

// This file is compiled once per state size N (-DPDSSM_N=...), so the six
// sizes build in parallel; pdssm_api.cpp dispatches on N.
#ifndef PDSSM_N
#error "compile pdssm_fused.hip with -DPDSSM_N=<state size>"
#endif
template <>
hipError_t launch_prep_n<PDSSM_N>(const PrepArgs& p, hipStream_t st) {
    return prep_launch<PDSSM_N>(p, st);
}
template <>
hipError_t launch_fwd_fused_n<PDSSM_N>(const FusedArgs& a, hipStream_t st) {
    return dispatch_tau<PDSSM_N, true>(a, st);
}
template <>
hipError_t launch_bwd_fused_n<PDSSM_N>(const FusedArgs& a, hipStream_t st) {
    return dispatch_tau<PDSSM_N, false>(a, st);
}

}  // namespace pdssm
