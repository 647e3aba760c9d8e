// pdssm_chunked.hip -- chunk-parallel PD scan for gfx950 (three phases).
//
// Forward (App. E.1 Algorithm 1, App. E.3 kernels A/B/C, re-designed for
// 64-lane wavefronts):
//   k_fwd_agg    one wave per (sequence, chunk): folds the chunk's steps into
//                its PD operator (pi_c, d_c) and local term B_c (state reached
//                from zero), App. E.3.1 accumulator update.
//   k_fwd_carry  one wave per sequence: carry_{c+1} = B_c + (pi_c, d_c) carry_c,
//                storing the state entering every chunk (the saved states).
//   k_fwd_replay one wave per (sequence, chunk): replays the chunk from its
//                entering state and reduces the readout y_t on the fly; the
//                per-step state never leaves the wave.
// Backward (adjoint of the above; the paper gives no backward scan):
//   k_bwd_agg    per chunk, in reverse time: the local adjoint gamma_c
//                (gradient reaching the chunk's entering state from the chunk's
//                own readouts) and the chunk operator (pi_c, d_c).
//   k_bwd_carry  per sequence, reverse over chunks:
//                U_{c-1} = gamma_c + (pi_c, d_c)^H U_c; U_{-1} = dh0.
//   k_bwd_emit   per chunk: recomputes the chunk's states from the saved
//                entering state into LDS, then walks backwards emitting dD, db,
//                dc.
//
// Every scatter-add runs in a fixed order (no float atomics): dictionary steps
// use the per-entry tables of the prep kernel (source records, or the sorted
// form for maps with a row of more than kMaxSrc sources), read from the
// workspace; the carry pass uses the sorted form of every chunk's composed
// map, built once per chunk by k_fwd_agg.
#include "pdssm_device.h"
#include "pdssm_internal.h"

namespace pdssm {

namespace {

constexpr int kWavesPerGroup = 4;

// Rows of D, b, c (in) and dD, db, dc, z (out) in row format IO: off counts
// entries; the 4-byte formats widen to (and narrow from) complex in registers
// exactly as the single-read kernels do.
template <int SL, int IO>
__device__ __forceinline__ CV<SL> ld_io(const float2* base, size_t off, int lane) {
    if constexpr (IO == kIoC64) {
        return ld_cv<SL>(base + off, lane);
    } else {
        const uint32_t* p = reinterpret_cast<const uint32_t*>(base) + off + (size_t)lane * SL;
        CV<SL> out;
#pragma unroll
        for (int s = 0; s < SL; ++s) out.v[s] = word_to_f2<IO>(p[s]);
        return out;
    }
}
template <int SL, int IO>
__device__ __forceinline__ void st_io(float2* base, size_t off, int lane, const CV<SL>& v) {
    if constexpr (IO == kIoC64) {
        st_cv<SL>(base + off, lane, v);
    } else {
        uint32_t* p = reinterpret_cast<uint32_t*>(base) + off + (size_t)lane * SL;
#pragma unroll
        for (int s = 0; s < SL; ++s) p[s] = f2_to_word<IO>(v.v[s]);
    }
}

// This lane's prep words of dictionary entry k of head hh, and the entry's
// class (max in-degree, or kFallback for the sorted form).
template <int N>
__device__ __forceinline__ int load_entry(const ScanArgs& a, int hh, int k, int lane, bool act,
                                          uint64_t (&w)[Lay<N>::SL]) {
    constexpr int SL = Lay<N>::SL;
    const size_t e = (size_t)hh * a.K + k;
#pragma unroll
    for (int r = 0; r < SL; ++r) w[r] = act ? a.rec[e * N + lane * SL + r] : 0;
    return __builtin_amdgcn_readfirstlane((int)a.mtab[e]);
}

// ================================================================== forward
template <int N, int IO>
__global__ __launch_bounds__(256) void k_fwd_agg(ScanArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 xs[kWavesPerGroup][N + 1];
    __shared__ float2 dsh[kWavesPerGroup][N];
    __shared__ int psh[kWavesPerGroup][N];
    __shared__ uint64_t mts[kWavesPerGroup][SL][N];
    __shared__ uint8_t sts[kWavesPerGroup][N];
    const int wv = wave_id(), lane = lane_id();
    const int nseq = a.B * a.H;
    const int task = blockIdx.x * kWavesPerGroup + wv;
    if (task >= nseq * a.C) return;
    const int seq = task / a.C, ch = task - seq * a.C;
    const int bb = seq / a.H, hh = seq - bb * a.H;
    const int s0 = ch * a.tau, len = min(a.tau, a.L - s0);
    const bool act = lane < LANES;
    float2* X = xs[wv];
    float2* Ds = dsh[wv];
    int* Ps = psh[wv];
    if (lane == 0) X[N] = make_float2(0.f, 0.f);  // zero row of the source records

    bool bad = false;
    int kv = 0;
    if (lane < len) {
        kv = a.idx[((size_t)bb * a.L + s0 + lane) * a.H + hh];
        bool bk = (unsigned)kv >= (unsigned)a.K;
        bad |= bk;
        kv = bk ? 0 : kv;
    }

    IV<SL> pm;
    CV<SL> dm, bm;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        pm.v[s] = lane * SL + s;
        dm.v[s] = make_float2(1.f, 0.f);
        bm.v[s] = make_float2(0.f, 0.f);
    }
    const size_t stride = (size_t)a.H * N;
    const size_t base = (((size_t)bb * a.L + s0) * a.H + hh) * N;
    const int* pih = a.pi + (size_t)hh * a.K * N;

    CV<SL> Dn = cv_zero<SL>(), bn = cv_zero<SL>();
    IV<SL> pn = {};
    uint64_t wn[SL];
    int cn = load_entry<N>(a, hh, readlane_i(kv, 0), lane, act, wn);
    if (act) {
        int k = readlane_i(kv, 0);
        Dn = ld_io<SL, IO>(a.D, base, lane);
        bn = ld_io<SL, IO>(a.b, base, lane);
        pn = ld_iv<SL>(pih + (size_t)k * N, lane);
    }
    for (int t = 0; t < len; ++t) {
        CV<SL> Dt = Dn, bt = bn;
        IV<SL> pt = pn;
        uint64_t wt[SL];
#pragma unroll
        for (int r = 0; r < SL; ++r) wt[r] = wn[r];
        const int ct = cn;
        if (t + 1 < len) {
            int k = readlane_i(kv, t + 1);
            cn = load_entry<N>(a, hh, k, lane, act, wn);
            if (act) {
                Dn = ld_io<SL, IO>(a.D, base + (t + 1) * stride, lane);
                bn = ld_io<SL, IO>(a.b, base + (t + 1) * stride, lane);
                pn = ld_iv<SL>(pih + (size_t)k * N, lane);
            }
        }
        bad |= sanitize_map<N, SL>(pt);
        // B <- b_t + P_t (D_t .* B)
        table_step<N>(X, ct, wt, bm, Dt, bt, lane, act);
        // (pi, d) <- (pi_t[pi], D_t[pi] * d): stage D_t and pi_t for random access
        wave_sync();
        if (act) {
            st_cv<SL>(Ds, lane, Dt);
            st_iv<SL>(Ps, lane, pt);
        }
        wave_sync();
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                int q = pm.v[s];
                dm.v[s] = cmul(Ds[q], dm.v[s]);
                pm.v[s] = Ps[q];
            }
        }
    }
    // the composed map in sorted form, for the carry pass's scatter
    uint64_t* mt[SL];
#pragma unroll
    for (int q = 0; q < SL; ++q) mt[q] = mts[wv][q];
    uint64_t sw[SL];
    map_sorted_words<N>(pm, lane, act, mt, Ps, sts[wv], sw);
    if (act) {
        const size_t o = ((size_t)seq * a.C + ch) * N;
        IV<SL> packed;
#pragma unroll
        for (int s = 0; s < SL; ++s) packed.v[s] = (int)sw[s];
        st_iv<SL>(a.agg_p + o, lane, packed);
        st_cv<SL>(a.agg_d + o, lane, dm);
        st_cv<SL>(a.agg_v + o, lane, bm);
    }
    if (bad) report_index_error(a.status);
}

// The carries (chunk-entering states, the saved states when the caller
// keeps them): complex64, or their real parts as fp32 for the real model
// (whose states have imaginary parts 0 here too).
template <int SL>
__device__ __forceinline__ void st_carry(const ScanArgs& a, size_t off, int lane, const CV<SL>& h) {
    if (a.io == kIoReal) st_srow<SL>(a.carry, off, lane, to_elem<float>(h));
    else st_srow<SL>(a.carry, off, lane, h);
}
template <int SL>
__device__ __forceinline__ CV<SL> ld_carry(const ScanArgs& a, size_t off, int lane) {
    if (a.io == kIoReal) return to_c64<SL>(ld_srow<SL, float>(a.carry, off, lane));
    return ld_srow<SL, float2>(a.carry, off, lane);
}

template <int N>
__global__ __launch_bounds__(256) void k_fwd_carry(ScanArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 xs[kWavesPerGroup][N];
    const int wv = wave_id(), lane = lane_id();
    const int seq = blockIdx.x * kWavesPerGroup + wv;
    if (seq >= a.B * a.H) return;
    const bool act = lane < LANES;
    float2* X = xs[wv];

    CV<SL> h = cv_zero<SL>();
    if (a.h0 && act) h = ld_cv<SL>(a.h0 + (size_t)seq * N, lane);
    const size_t o0 = (size_t)seq * a.C * N;
    IV<SL> pn = {};
    CV<SL> dn = cv_zero<SL>(), vn = cv_zero<SL>();
    if (act) {
        pn = ld_iv<SL>(a.agg_p + o0, lane);
        dn = ld_cv<SL>(a.agg_d + o0, lane);
        vn = ld_cv<SL>(a.agg_v + o0, lane);
    }
    for (int ch = 0; ch < a.C; ++ch) {
        const size_t o = o0 + (size_t)ch * N;
        if (act) st_carry<SL>(a, o, lane, h);
        uint64_t wc[SL];
#pragma unroll
        for (int s = 0; s < SL; ++s) wc[s] = (uint32_t)pn.v[s];  // sorted form of the chunk map
        CV<SL> dc = dn, vc = vn;
        if (ch + 1 < a.C && act) {
            pn = ld_iv<SL>(a.agg_p + o + N, lane);
            dn = ld_cv<SL>(a.agg_d + o + N, lane);
            vn = ld_cv<SL>(a.agg_v + o + N, lane);
        }
        sorted_step<N>(X, wc, h, dc, vc, lane, act);
    }
    if (a.hfinal && act) st_cv<SL>(a.hfinal + (size_t)seq * N, lane, h);
}

template <int N, int IO>
__global__ __launch_bounds__(256) void k_fwd_replay(ScanArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 xs[kWavesPerGroup][N + 1];
    const int wv = wave_id(), lane = lane_id();
    const int nseq = a.B * a.H;
    const int task = blockIdx.x * kWavesPerGroup + wv;
    if (task >= nseq * a.C) return;
    const int seq = task / a.C, ch = task - seq * a.C;
    const int bb = seq / a.H, hh = seq - bb * a.H;
    const int s0 = ch * a.tau, len = min(a.tau, a.L - s0);
    const bool act = lane < LANES;
    float2* X = xs[wv];
    if (lane == 0) X[N] = make_float2(0.f, 0.f);  // zero row of the source records

    int kv = 0;
    if (lane < len) {
        kv = a.idx[((size_t)bb * a.L + s0 + lane) * a.H + hh];
        kv = (unsigned)kv >= (unsigned)a.K ? 0 : kv;  // reported by k_fwd_agg
    }
    CV<SL> h = cv_zero<SL>();
    if (act) h = ld_carry<SL>(a, ((size_t)seq * a.C + ch) * N, lane);

    const size_t stride = (size_t)a.H * N;
    const size_t base = (((size_t)bb * a.L + s0) * a.H + hh) * N;
    float* yrow = a.y + ((size_t)bb * a.L + s0) * a.H + hh;

    CV<SL> Dn = cv_zero<SL>(), bn = cv_zero<SL>(), cn = cv_zero<SL>();
    uint64_t wn[SL];
    int kn = load_entry<N>(a, hh, readlane_i(kv, 0), lane, act, wn);
    if (act) {
        Dn = ld_io<SL, IO>(a.D, base, lane);
        bn = ld_io<SL, IO>(a.b, base, lane);
        cn = ld_io<SL, IO>(a.c, base, lane);
    }
    for (int t = 0; t < len; ++t) {
        CV<SL> Dt = Dn, bt = bn, ct = cn;
        uint64_t wt[SL];
#pragma unroll
        for (int r = 0; r < SL; ++r) wt[r] = wn[r];
        const int kc = kn;
        if (t + 1 < len) {
            kn = load_entry<N>(a, hh, readlane_i(kv, t + 1), lane, act, wn);
            if (act) {
                const size_t off = base + (t + 1) * stride;
                Dn = ld_io<SL, IO>(a.D, off, lane);
                bn = ld_io<SL, IO>(a.b, off, lane);
                cn = ld_io<SL, IO>(a.c, off, lane);
            }
        }
        table_step<N>(X, kc, wt, h, Dt, bt, lane, act);
        float part = 0.f;
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) part += ct.v[s].x * h.v[s].x - ct.v[s].y * h.v[s].y;
        }
        float tot = wave_sum_last(part);
        if (lane == kWave - 1) yrow[(size_t)t * a.H] = tot;
    }
}

// ================================================================== backward
template <int N, int IO>
__global__ __launch_bounds__(256) void k_bwd_agg(ScanArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 gsh[kWavesPerGroup][N];
    __shared__ float2 dsh[kWavesPerGroup][N];
    __shared__ int psh[kWavesPerGroup][N];
    const int wv = wave_id(), lane = lane_id();
    const int nseq = a.B * a.H;
    const int task = blockIdx.x * kWavesPerGroup + wv;
    if (task >= nseq * a.C) return;
    const int seq = task / a.C, ch = task - seq * a.C;
    const int bb = seq / a.H, hh = seq - bb * a.H;
    const int s0 = ch * a.tau, len = min(a.tau, a.L - s0);
    const bool act = lane < LANES;
    float2* G = gsh[wv];
    float2* Dm = dsh[wv];
    int* Pm = psh[wv];

    bool bad = false;
    int kv = 0;
    float dyv = 0.f;
    if (lane < len) {
        const size_t o = ((size_t)bb * a.L + s0 + lane) * a.H + hh;
        kv = a.idx[o];
        bool bk = (unsigned)kv >= (unsigned)a.K;
        bad |= bk;
        kv = bk ? 0 : kv;
        dyv = a.dy[o];
    }
    const size_t stride = (size_t)a.H * N;
    const size_t base = (((size_t)bb * a.L + s0) * a.H + hh) * N;
    const int* pih = a.pi + (size_t)hh * a.K * N;

    // Phi_{[t..e)} = Phi_{[t+1..e)} A_t: pi(j) <- pi'[pi_t(j)], d(j) <- d'[pi_t(j)] D_t(j)
    IV<SL> pm;
    CV<SL> dm, g = cv_zero<SL>();
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        pm.v[s] = lane * SL + s;
        dm.v[s] = make_float2(1.f, 0.f);
    }
    CV<SL> Dn = cv_zero<SL>(), cn = cv_zero<SL>();
    IV<SL> pn = {};
    if (act) {
        int k = readlane_i(kv, len - 1);
        const size_t off = base + (len - 1) * stride;
        Dn = ld_io<SL, IO>(a.D, off, lane);
        cn = ld_io<SL, IO>(a.c, off, lane);
        pn = ld_iv<SL>(pih + (size_t)k * N, lane);
    }
    for (int t = len - 1; t >= 0; --t) {
        CV<SL> Dt = Dn, ct = cn;
        IV<SL> pt = pn;
        if (t > 0 && act) {
            int k = readlane_i(kv, t - 1);
            const size_t off = base + (t - 1) * stride;
            Dn = ld_io<SL, IO>(a.D, off, lane);
            cn = ld_io<SL, IO>(a.c, off, lane);
            pn = ld_iv<SL>(pih + (size_t)k * N, lane);
        }
        bad |= sanitize_map<N, SL>(pt);
        const float dyt = readlane_f(dyv, t);
        wave_sync();
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                g.v[s].x += dyt * ct.v[s].x;
                g.v[s].y -= dyt * ct.v[s].y;
            }
            st_cv<SL>(G, lane, g);
            st_cv<SL>(Dm, lane, dm);
            st_iv<SL>(Pm, lane, pm);
        }
        wave_sync();
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                int q = pt.v[s];
                float2 gp = G[q];
                dm.v[s] = cmul(Dm[q], Dt.v[s]);
                pm.v[s] = Pm[q];
                g.v[s] = cmulc(Dt.v[s], gp);
            }
        }
    }
    if (act) {
        const size_t o = ((size_t)seq * a.C + ch) * N;
        st_iv<SL>(a.agg_p + o, lane, pm);
        st_cv<SL>(a.agg_d + o, lane, dm);
        st_cv<SL>(a.agg_v + o, lane, g);
    }
    if (bad) report_index_error(a.status);
}

template <int N>
__global__ __launch_bounds__(256) void k_bwd_carry(ScanArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 xs[kWavesPerGroup][N];
    const int wv = wave_id(), lane = lane_id();
    const int seq = blockIdx.x * kWavesPerGroup + wv;
    if (seq >= a.B * a.H) return;
    const bool act = lane < LANES;
    float2* X = xs[wv];

    CV<SL> u = cv_zero<SL>();
    if (a.dhf && act) u = ld_cv<SL>(a.dhf + (size_t)seq * N, lane);
    const size_t o0 = (size_t)seq * a.C * N;
    IV<SL> pn = {};
    CV<SL> dn = cv_zero<SL>(), vn = cv_zero<SL>();
    if (act) {
        const size_t o = o0 + (size_t)(a.C - 1) * N;
        pn = ld_iv<SL>(a.agg_p + o, lane);
        dn = ld_cv<SL>(a.agg_d + o, lane);
        vn = ld_cv<SL>(a.agg_v + o, lane);
    }
    for (int ch = a.C - 1; ch >= 0; --ch) {
        const size_t o = o0 + (size_t)ch * N;
        if (act) st_cv<SL>(a.U + o, lane, u);
        IV<SL> pc = pn;
        CV<SL> dc = dn, gc = vn;
        if (ch > 0 && act) {
            pn = ld_iv<SL>(a.agg_p + o - N, lane);
            dn = ld_cv<SL>(a.agg_d + o - N, lane);
            vn = ld_cv<SL>(a.agg_v + o - N, lane);
        }
        // u <- gamma_c + conj(d_c) .* u[pi_c]
        wave_sync();
        if (act) st_cv<SL>(X, lane, u);
        wave_sync();
        if (act) {
#pragma unroll
            for (int s = 0; s < SL; ++s) u.v[s] = cadd(gc.v[s], cmulc(dc.v[s], X[pc.v[s]]));
        }
    }
    if (a.dh0 && act) st_cv<SL>(a.dh0 + (size_t)seq * N, lane, u);
}

// One wave per workgroup; dynamic LDS = (tau + 1) states + one exchange row
// of N + 1 entries (the last one the zero row of the source records).
template <int N, int IO>
__global__ __launch_bounds__(64) void k_bwd_emit(ScanArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    extern __shared__ float2 smem[];
    const int lane = lane_id();
    const int task = blockIdx.x;
    const int seq = task / a.C, ch = task - seq * a.C;
    const int bb = seq / a.H, hh = seq - bb * a.H;
    const int s0 = ch * a.tau, len = min(a.tau, a.L - s0);
    const bool act = lane < LANES;
    float2* Hs = smem;                           // Hs[i*N + j] = state before step s0 + i
    float2* X = smem + (size_t)(a.tau + 1) * N;  // exchange row
    if (lane == 0) X[N] = make_float2(0.f, 0.f);

    int kv = 0;
    float dyv = 0.f;
    if (lane < len) {
        const size_t o = ((size_t)bb * a.L + s0 + lane) * a.H + hh;
        kv = a.idx[o];
        kv = (unsigned)kv >= (unsigned)a.K ? 0 : kv;  // reported by k_bwd_agg
        dyv = a.dy[o];
    }
    const size_t stride = (size_t)a.H * N;
    const size_t base = (((size_t)bb * a.L + s0) * a.H + hh) * N;
    const int* pih = a.pi + (size_t)hh * a.K * N;

    // ---- forward recompute of the chunk's states
    CV<SL> h = cv_zero<SL>();
    if (act) {
        h = ld_carry<SL>(a, ((size_t)seq * a.C + ch) * N, lane);
        st_cv<SL>(Hs, lane, h);
    }
    CV<SL> Dn = cv_zero<SL>(), bn = cv_zero<SL>();
    IV<SL> pn = {};
    uint64_t wn[SL];
    int kn = load_entry<N>(a, hh, readlane_i(kv, 0), lane, act, wn);
    if (act) {
        Dn = ld_io<SL, IO>(a.D, base, lane);
        bn = ld_io<SL, IO>(a.b, base, lane);
    }
    for (int t = 0; t < len; ++t) {
        CV<SL> Dt = Dn, bt = bn;
        uint64_t wt[SL];
#pragma unroll
        for (int r = 0; r < SL; ++r) wt[r] = wn[r];
        const int kc = kn;
        if (t + 1 < len) {
            kn = load_entry<N>(a, hh, readlane_i(kv, t + 1), lane, act, wn);
            if (act) {
                Dn = ld_io<SL, IO>(a.D, base + (t + 1) * stride, lane);
                bn = ld_io<SL, IO>(a.b, base + (t + 1) * stride, lane);
            }
        }
        table_step<N>(X, kc, wt, h, Dt, bt, lane, act);
        if (act) st_cv<SL>(Hs + (size_t)(t + 1) * N, lane, h);
    }

    // ---- reverse walk with the true incoming gradient
    CV<SL> g = cv_zero<SL>();
    if (act) g = ld_cv<SL>(a.U + ((size_t)seq * a.C + ch) * N, lane);
    CV<SL> cn = cv_zero<SL>();
    if (act) {
        int k = readlane_i(kv, len - 1);
        const size_t off = base + (len - 1) * stride;
        Dn = ld_io<SL, IO>(a.D, off, lane);
        cn = ld_io<SL, IO>(a.c, off, lane);
        pn = ld_iv<SL>(pih + (size_t)k * N, lane);
    }
    for (int t = len - 1; t >= 0; --t) {
        CV<SL> Dt = Dn, ct = cn;
        IV<SL> pt = pn;
        if (t > 0 && act) {
            int k = readlane_i(kv, t - 1);
            const size_t off = base + (t - 1) * stride;
            Dn = ld_io<SL, IO>(a.D, off, lane);
            cn = ld_io<SL, IO>(a.c, off, lane);
            pn = ld_iv<SL>(pih + (size_t)k * N, lane);
        }
        sanitize_map<N, SL>(pt);
        const float dyt = readlane_f(dyv, t);
        const size_t off = base + t * stride;
        CV<SL> ht = cv_zero<SL>(), hp = cv_zero<SL>(), dct;
        if (act) {
            ht = ld_cv<SL>(Hs + (size_t)(t + 1) * N, lane);
            hp = ld_cv<SL>(Hs + (size_t)t * N, lane);
        }
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            g.v[s].x += dyt * ct.v[s].x;
            g.v[s].y -= dyt * ct.v[s].y;
            dct.v[s] = make_float2(dyt * ht.v[s].x, -dyt * ht.v[s].y);
        }
        wave_sync();
        if (act) {
            st_io<SL, IO>(a.db, off, lane, g);
            st_io<SL, IO>(a.dc, off, lane, dct);
            st_cv<SL>(X, lane, g);
        }
        wave_sync();
        if (act) {
            CV<SL> dDt;
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                float2 gp = X[pt.v[s]];
                dDt.v[s] = cmulc(hp.v[s], gp);
                g.v[s] = cmulc(Dt.v[s], gp);
            }
            st_io<SL, IO>(a.dD, off, lane, dDt);
        }
        if (a.z && act) {
            // the scaled state z_t = D_t .* h_{t-1} for the straight-through gradients
            CV<SL> zt;
#pragma unroll
            for (int s = 0; s < SL; ++s) zt.v[s] = cmul(Dt.v[s], hp.v[s]);
            st_io<SL, (IO == kIoBf16 ? kIoC64 : IO)>(a.z, off, lane, zt);  // bf16 pairs: z complex64
        }
    }
}

// ================================================================== compose
// One wave per (sequence, chunk); any chunk length.
template <int N>
__global__ __launch_bounds__(256) void k_compose(ComposeArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 dsh[kWavesPerGroup][N];
    __shared__ int psh[kWavesPerGroup][N];
    const int wv = wave_id(), lane = lane_id();
    const int nseq = a.B * a.H;
    const int task = blockIdx.x * kWavesPerGroup + wv;
    if (task >= nseq * a.C) return;
    const int seq = task / a.C, ch = task - seq * a.C;
    const int bb = seq / a.H, hh = seq - bb * a.H;
    const int s0 = (int)((long long)ch * a.tau), len = (int)min((long long)a.tau, (long long)a.L - s0);
    const bool act = lane < LANES;
    float2* Ds = dsh[wv];
    int* Ps = psh[wv];
    const size_t stride = (size_t)a.H * N;
    const size_t base = (((size_t)bb * a.L + s0) * a.H + hh) * N;
    const int* pih = a.pi + (size_t)hh * a.K * N;

    bool bad = false;
    IV<SL> pm;
    CV<SL> dm;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        pm.v[s] = lane * SL + s;
        dm.v[s] = make_float2(1.f, 0.f);
    }
    for (int t0 = 0; t0 < len; t0 += kWave) {
        const int n = min(kWave, len - t0);
        int kv = 0;
        if (lane < n) {
            kv = a.idx[((size_t)bb * a.L + s0 + t0 + lane) * a.H + hh];
            bool bk = (unsigned)kv >= (unsigned)a.K;
            bad |= bk;
            kv = bk ? 0 : kv;
        }
        for (int t = 0; t < n; ++t) {
            const int k = readlane_i(kv, t);
            CV<SL> Dt = cv_zero<SL>();
            IV<SL> pt = {};
            if (act) {
                Dt = ld_cv<SL>(a.D + base + (size_t)(t0 + t) * stride, lane);
                pt = ld_iv<SL>(pih + (size_t)k * N, lane);
            }
            bad |= sanitize_map<N, SL>(pt);
            wave_sync();
            if (act) {
                st_cv<SL>(Ds, lane, Dt);
                st_iv<SL>(Ps, lane, pt);
            }
            wave_sync();
            if (act) {
#pragma unroll
                for (int s = 0; s < SL; ++s) {
                    int q = pm.v[s];
                    dm.v[s] = cmul(Ds[q], dm.v[s]);
                    pm.v[s] = Ps[q];
                }
            }
        }
    }
    if (act) {
        const size_t o = ((size_t)seq * a.C + ch) * N;
        st_iv<SL>(a.pi_out + o, lane, pm);
        st_cv<SL>(a.d_out + o, lane, dm);
    }
    if (bad) report_index_error(a.status);
}

inline unsigned groups_for(long long tasks) {
    return (unsigned)((tasks + kWavesPerGroup - 1) / kWavesPerGroup);
}

template <int N, int IO>
hipError_t fwd_chunked_io(const ScanArgs& a, hipStream_t s) {
    const long long tasks = (long long)a.B * a.H * a.C;
    auto agg = k_fwd_agg<N, IO>;
    auto replay = k_fwd_replay<N, IO>;
    hipLaunchKernelGGL(agg, dim3(groups_for(tasks)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_fwd_carry<N>, dim3(groups_for((long long)a.B * a.H)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(replay, dim3(groups_for(tasks)), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int N, int IO>
hipError_t bwd_chunked_io(const ScanArgs& a, hipStream_t s) {
    const long long tasks = (long long)a.B * a.H * a.C;
    auto agg = k_bwd_agg<N, IO>;
    auto emit = k_bwd_emit<N, IO>;
    hipLaunchKernelGGL(agg, dim3(groups_for(tasks)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_bwd_carry<N>, dim3(groups_for((long long)a.B * a.H)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(emit, dim3((unsigned)tasks), dim3(64), bwd_emit_lds_bytes(N, a.tau), s, a);
    return hipGetLastError();
}

// the row format picks the instantiation
template <int N>
hipError_t fwd_chunked_n(const ScanArgs& a, hipStream_t s) {
    switch (a.io) {
        case kIoC64: return fwd_chunked_io<N, kIoC64>(a, s);
        case kIoBf16: return fwd_chunked_io<N, kIoBf16>(a, s);
        case kIoReal: return fwd_chunked_io<N, kIoReal>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <int N>
hipError_t bwd_chunked_n(const ScanArgs& a, hipStream_t s) {
    switch (a.io) {
        case kIoC64: return bwd_chunked_io<N, kIoC64>(a, s);
        case kIoBf16: return bwd_chunked_io<N, kIoBf16>(a, s);
        case kIoReal: return bwd_chunked_io<N, kIoReal>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <int N>
hipError_t compose_n(const ComposeArgs& a, hipStream_t s) {
    const long long tasks = (long long)a.B * a.H * a.C;
    hipLaunchKernelGGL(k_compose<N>, dim3(groups_for(tasks)), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

#define PDSSM_DISPATCH_N(N_, FN, ...)                   \
    switch (N_) {                                       \
        case 8: return FN<8>(__VA_ARGS__);              \
        case 16: return FN<16>(__VA_ARGS__);            \
        case 32: return FN<32>(__VA_ARGS__);            \
        case 64: return FN<64>(__VA_ARGS__);            \
        case 128: return FN<128>(__VA_ARGS__);          \
        case 256: return FN<256>(__VA_ARGS__);          \
        default: return hipErrorInvalidValue;           \
    }

hipError_t launch_fwd_chunked(const ScanArgs& a, hipStream_t s) { PDSSM_DISPATCH_N(a.N, fwd_chunked_n, a, s) }
hipError_t launch_bwd_chunked(const ScanArgs& a, hipStream_t s) { PDSSM_DISPATCH_N(a.N, bwd_chunked_n, a, s) }
hipError_t launch_compose(const ComposeArgs& a, hipStream_t s) { PDSSM_DISPATCH_N(a.N, compose_n, a, s) }

}  // namespace pdssm
