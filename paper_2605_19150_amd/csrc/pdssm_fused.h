// pdssm_fused.h -- launch interface of the fused single-read scan kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "pdssm_io.h"

namespace pdssm {

// Chunk-computing waves per workgroup of the fused kernels (one workgroup per
// sequence; the forward adds one frontier wave).
// Kernels that prefetch the next chunk (two register buffers, when a chunk
// holds <= 8 rows per lane) run fewer, fatter waves.
#ifndef PDSSM_PF_WAVES
#define PDSSM_PF_WAVES 7
#endif
#ifndef PDSSM_PF_MAX_ROWS
#define PDSSM_PF_MAX_ROWS 8
#endif
#ifndef PDSSM_BWD_PF_WAVES
#define PDSSM_BWD_PF_WAVES 8
#endif
constexpr int kFusedWaves = 7;
constexpr bool fused_prefetch(int N, int tau) { return tau * (N > 64 ? N / 64 : 1) <= PDSSM_PF_MAX_ROWS; }
constexpr int fused_waves(int N, int tau) { return fused_prefetch(N, tau) ? PDSSM_PF_WAVES : kFusedWaves; }
constexpr int fused_waves_bwd(int N, int tau) { return fused_prefetch(N, tau) ? PDSSM_BWD_PF_WAVES : kFusedWaves; }
// The prefetching forward also comes with 11 chunk waves (12 with the
// frontier, three per SIMD), used for the 4-byte row formats when the head's
// tables leave LDS room for them: more waves in flight hide the chunk
// passes' LDS round trips (the backward measured faster with 8).
constexpr int kFusedWavesWide = 11;
// Chunk waves a wide forward uses for a head of permutation maps in
// complex64 rows (the rest stay idle).
constexpr int kPermWaves = 7;
// At N = 256 the per-wave LDS buffers (2W published operators of N entries
// and their sorted forms, W staging rows, 2W readout rows) leave room for the
// head's tables only with fewer chunk waves: 5, else 3, in both directions,
// used when 7 do not fit (dictionaries of up to 16, else 32 entries; larger
// ones run the multi-pass kernels).
constexpr int kFusedWavesNarrow = 5;
constexpr int kFusedWavesNarrowest = 3;

// Byte offsets of the fused kernels' dynamic LDS regions.
struct LdsLayout {
    uint32_t rec, dict, mtab, ring, ready, agg, agp, age, agh, agm, aflag, prog, vd, x, cs, pa, sb, total;
};

inline uint32_t align16(size_t x) { return (uint32_t)((x + 15) / 16 * 16); }

// Dictionary tables hold K entries plus one identity entry (index K) that
// pads the last, partial chunk of a sequence with exact no-op steps.  Each
// wave's vd row block has N + 1 rows; row N stays zero.  W is the number of
// chunk-computing waves; one more wave (the frontier wave) carries the state
// from chunk to chunk.  ring: W + 1 carry slots; agg/agp/age/agh/aflag: 2W
// slots of published chunk operators (local state and diagonal; the map, or
// for many-to-one heads its sorted form: position of each source, last
// position of each destination's run, run-start flags; agm: the map itself,
// for the aggregate pass) and their chunk ids; prog: chunks the workgroup's
// waves have finished (the waits' progress measure).
inline LdsLayout fused_lds_layout(int N, int K, int W) {
    LdsLayout l;
    size_t o = 0;
    const size_t KE = (size_t)K + 1;
    l.rec = (uint32_t)o;   o += KE * N * 8;
    l.dict = (uint32_t)o;  o += align16(KE * N);
    l.mtab = (uint32_t)o;  o += align16(KE);
    l.ring = (uint32_t)o;  o += (size_t)(W + 1) * N * 8;
    l.ready = (uint32_t)o; // followed by the 2W operator-slot flags and the progress count
    l.aflag = (uint32_t)(o + 4);
    l.prog = (uint32_t)(o + 4 * (1 + 2 * (size_t)W));
    o += align16((size_t)(2 + 2 * W) * 4);
    l.agg = (uint32_t)o;   o += (size_t)2 * W * N * 16;
    l.agp = (uint32_t)o;   o += align16((size_t)2 * W * N);
    l.age = (uint32_t)o;   o += align16((size_t)2 * W * N * 2);
    l.agh = (uint32_t)o;   o += align16((size_t)2 * W * N);
    l.agm = (uint32_t)o;   o += align16((size_t)2 * W * N);
    l.vd = (uint32_t)o;    o += (size_t)W * (N + 1) * 16;
    l.x = (uint32_t)o;     o += (size_t)(W + 1) * N * 8;
    l.cs = (uint32_t)o;    o += (size_t)2 * W * N * 8;
    l.pa = (uint32_t)o;    o += align16((size_t)W * N);
    l.sb = (uint32_t)o;    // saved-state staging, sized by the caller (fused_lds_add_staging)
    l.total = (uint32_t)o;
    return l;
}

// Adds M saved-state rows of staging to a layout (the forward writes chunk
// states there and flushes them to HBM in bursts of M rows; complex64 rows
// for every row format).
inline LdsLayout fused_lds_add_staging(LdsLayout l, int N, int M) {
    l.total = l.sb + (uint32_t)((size_t)M * N * 8);
    return l;
}

constexpr size_t kMaxLds = 163840;  // gfx950: 160 KiB per workgroup

// Per-call dictionary tables built by the prep kernel (workspace).
struct PrepArgs {
    int H, K, N;
    const int* pi;   // [H][K][N]
    uint8_t* dict;   // [H][K][N] byte copy of pi (sanitised)
    uint64_t* rec;   // [H][K][N] per destination row: 7 source bytes + in-degree byte
                     // (unused source bytes hold N, a zero row, when N <= 128, else 0);
                     // for an entry with a row of more sources, its sorted form (srt_word)
    uint8_t* mtab;   // [H][K] max in-degree of the entry, kFallback (255) = sorted form
    int* status;
};

struct FusedArgs {
    int B, L, H, N, K;
    int tau, C;
    const int* idx;
    const float2* D;
    const float2* b;
    const float2* c;
    const float2* h0;
    const float* dy;
    const float2* dhf;
    float* y;
    float2* hfinal;
    float2* saved;  // [B*H][C][N]: complex64, or float32 entries for the real model (kIoReal)
    float2* dD;
    float2* db;
    float2* dc;
    float2* dh0;
    const uint8_t* dict;
    const uint64_t* rec;
    const uint8_t* mtab;
    int* status;
    LdsLayout lds;
    // Long sequences are cut into S segments of Cs chunks, one workgroup
    // each; an aggregate pass first folds every segment into one PD operator
    // (forward: local state, map, diagonal; backward: local adjoint, map,
    // diagonal), [B*H][S][N] each.  S = 1: one workgroup per sequence.
    int S, Cs;
    int sbM;  // saved-state rows staged in LDS by the forward (0: stored as computed)
    // The forward's layout and staging rows for heads of permutations in a
    // wide complex64 kernel (kPermWaves chunk waves; otherwise equal to lds
    // and sbM).  The tables sit at the same offsets as in lds.
    LdsLayout lds_perm;
    int sbM_perm;
    float2* segA;
    float2* segD;
    int* segP;
    // Chunk waves of this call's kernel: fused_waves / fused_waves_bwd, or
    // kFusedWavesWide (forward), or kFusedWavesNarrow / kFusedWavesNarrowest
    // (N = 256).
    int W;
    // Format of D, b, c and dD, db, dc (kIoC64, kIoBf16 pairs or kIoReal
    // fp32, 4 bytes per entry for the last two: the pointers above are then
    // reinterpreted); everything else keeps its complex64 / fp32 type.
    int io;
    // Backward only, optional: the scaled states z = D_t .* h_{t-1}
    // [B,L,H,N] that the straight-through gradients need (Sec. 3.1 Prop. 2),
    // in the row format of the gradients.
    float2* z;
};

// Per state size N (one translation unit each) ...
template <int N>
hipError_t launch_prep_n(const PrepArgs& p, hipStream_t s);
template <int N>
hipError_t launch_fwd_fused_n(const FusedArgs& a, hipStream_t s);
template <int N>
hipError_t launch_bwd_fused_n(const FusedArgs& a, hipStream_t s);

#define PDSSM_DECLARE_N(N_)                                                    \
    template <>                                                                \
    hipError_t launch_prep_n<N_>(const PrepArgs& p, hipStream_t s);           \
    template <>                                                                \
    hipError_t launch_fwd_fused_n<N_>(const FusedArgs& a, hipStream_t s);     \
    template <>                                                                \
    hipError_t launch_bwd_fused_n<N_>(const FusedArgs& a, hipStream_t s);
PDSSM_DECLARE_N(8)
PDSSM_DECLARE_N(16)
PDSSM_DECLARE_N(32)
PDSSM_DECLARE_N(64)
PDSSM_DECLARE_N(128)
PDSSM_DECLARE_N(256)
#undef PDSSM_DECLARE_N

// ... and the dispatch on N.
#define PDSSM_DISPATCH_N(N_, F_, ARGS_)            \
    switch (N_) {                                  \
        case 8: return F_<8> ARGS_;                \
        case 16: return F_<16> ARGS_;              \
        case 32: return F_<32> ARGS_;              \
        case 64: return F_<64> ARGS_;              \
        case 128: return F_<128> ARGS_;            \
        case 256: return F_<256> ARGS_;            \
        default: return hipErrorInvalidValue;      \
    }
inline hipError_t launch_prep(const PrepArgs& p, hipStream_t s) { PDSSM_DISPATCH_N(p.N, launch_prep_n, (p, s)) }
inline hipError_t launch_fwd_fused(const FusedArgs& a, hipStream_t s) {
    PDSSM_DISPATCH_N(a.N, launch_fwd_fused_n, (a, s))
}
inline hipError_t launch_bwd_fused(const FusedArgs& a, hipStream_t s) {
    PDSSM_DISPATCH_N(a.N, launch_bwd_fused_n, (a, s))
}

}  // namespace pdssm
