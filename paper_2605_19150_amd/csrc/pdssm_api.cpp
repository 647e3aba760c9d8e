// pdssm_api.cpp -- the C ABI of libpdssm.so: argument checks, workspace
// layout and kernel dispatch.  Declarations and the contract are in pdssm.h.
#include "pdssm.h"

#include <hip/hip_runtime.h>

#include <initializer_list>

#include "pdssm_decode.h"
#include "pdssm_select.h"
#include "pdssm_fused.h"
#include "pdssm_internal.h"

namespace {

using pdssm::ScanArgs;

constexpr int kDefaultComposeChunk = 32;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool n_supported(int N) {
    return N == 8 || N == 16 || N == 32 || N == 64 || N == 128 || N == 256;
}

int slots(int N) { return N > 64 ? N / 64 : 1; }

// Scan chunk lengths: 4, 8 or 16 steps with chunk * max(1, N/64) <= 16 (the
// fused kernels keep a chunk's rows in registers).  Default: 8 steps (4 at
// N = 256); 16 steps measured no faster at N <= 64.
bool scan_chunk_ok(int N, int tau) {
    return (tau == 4 || tau == 8 || tau == 16) && tau * slots(N) <= 16;
}

// Dimension checks shared by every op.  Returns PDSSM_OK or a status.
int check_dims(const pdssm_desc* d) {
    if (!d) return PDSSM_ERR_INVALID_ARG;
    if ((d->flags & ~(PDSSM_FLAG_PREPARED | PDSSM_FLAG_BF16_IO | PDSSM_FLAG_REAL_IO)) != 0)
        return PDSSM_ERR_INVALID_ARG;
    // one row format at a time
    if ((d->flags & PDSSM_FLAG_BF16_IO) && (d->flags & PDSSM_FLAG_REAL_IO)) return PDSSM_ERR_INVALID_ARG;
    if (d->B < 1 || d->L < 1 || d->H < 1 || d->N < 1 || d->K < 1 || d->chunk < 0)
        return PDSSM_ERR_INVALID_ARG;
    if (!n_supported(d->N) || d->K > 256) return PDSSM_ERR_UNSUPPORTED;
    const long long elems = (long long)d->B * d->L * d->H * d->N;
    if (elems >= (1LL << 31)) return PDSSM_ERR_UNSUPPORTED;
    if ((long long)d->H * d->K * d->N >= (1LL << 31)) return PDSSM_ERR_UNSUPPORTED;
    return PDSSM_OK;
}

// Bytes per entry of the chunk-entering states (saved): complex64, or fp32
// for the real-valued model.
int state_bytes(const pdssm_desc* d) { return (d->flags & PDSSM_FLAG_REAL_IO) ? 4 : 8; }

// Effective scan chunk (fwd/bwd) or a negative status.
int scan_chunk(const pdssm_desc* d) {
    int st = check_dims(d);
    if (st != PDSSM_OK) return st;
    int tau = d->chunk;
    if (tau == 0) tau = slots(d->N) >= 4 ? 4 : 8;
    if (!scan_chunk_ok(d->N, tau)) return PDSSM_ERR_UNSUPPORTED;
    return tau;
}

struct Range {
    const void* p;
    size_t n;
};

bool overlap(Range a, Range b) {
    if (!a.p || !b.p || a.n == 0 || b.n == 0) return false;
    auto x = reinterpret_cast<uintptr_t>(a.p), y = reinterpret_cast<uintptr_t>(b.p);
    return x < y + b.n && y < x + a.n;
}

// Every output must be disjoint from every input and from every other output.
bool any_overlap(std::initializer_list<Range> outs, std::initializer_list<Range> ins) {
    for (auto o = outs.begin(); o != outs.end(); ++o) {
        for (auto i : ins)
            if (overlap(*o, i)) return true;
        for (auto o2 = o + 1; o2 != outs.end(); ++o2)
            if (overlap(*o, *o2)) return true;
    }
    return false;
}

struct Sizes {
    size_t seqN, stepN, perChunk, idxN, dictN;
};

Sizes sizes_of(const pdssm_desc* d, int C) {
    Sizes s;
    s.seqN = (size_t)d->B * d->H * d->N;
    s.stepN = (size_t)d->B * d->L * d->H * d->N;
    s.perChunk = (size_t)d->B * d->H * C * d->N;
    s.idxN = (size_t)d->B * d->L * d->H;
    s.dictN = (size_t)d->H * d->K * d->N;
    return s;
}

// Saved-state rows the forward stages in LDS before writing them out in one
// burst: stores of chunk states interleaved with the row loads cost far more
// HBM time than the same bytes written together.  As many rows as the free
// LDS holds (up to a whole sequence), at least kMinStaging, else none.
constexpr int kMinStaging = 16;

// N = 256: a narrower wave count when the default one leaves the head's
// tables no room in LDS (compiled for N = 256 only): the wider of the two
// that fits, else the narrowest (the layout check then picks multi-pass).
int narrow_if_needed(const pdssm_desc* d, int W) {
    if (d->N != 256 || pdssm::fused_lds_layout(d->N, d->K, W).total <= pdssm::kMaxLds) return W;
    if (pdssm::fused_lds_layout(d->N, d->K, pdssm::kFusedWavesNarrow).total <= pdssm::kMaxLds)
        return pdssm::kFusedWavesNarrow;
    return pdssm::kFusedWavesNarrowest;
}

int bwd_waves(const pdssm_desc* d, int tau) { return narrow_if_needed(d, pdssm::fused_waves_bwd(d->N, tau)); }

// Chunk waves of the fused forward: the wide count when the prefetching
// kernel runs and its tables leave room for the minimum saved-state staging.
// More waves in flight cover the chunk passes of many-to-one maps (which
// bound their forward) and of the 4-byte row formats; in complex64 a head of
// permutations, bound by HBM, runs kPermWaves of them on a layout of its
// own (measured: markov-manyone 168 -> 154 us, fsa-perm unchanged).
int fwd_waves(const pdssm_desc* d, int tau) {
    if (pdssm::fused_prefetch(d->N, tau) &&
        pdssm::fused_lds_layout(d->N, d->K, pdssm::kFusedWavesWide).total + (size_t)kMinStaging * d->N * 8 <=
            pdssm::kMaxLds)
        return pdssm::kFusedWavesWide;
    return narrow_if_needed(d, pdssm::fused_waves(d->N, tau));
}

// The fused single-read kernels stage one head's dictionary tables in LDS;
// when they do not fit, the chunked three-pass kernels run instead.
pdssm::LdsLayout fused_layout(const pdssm_desc* d, int tau, bool fwd) {
    const int W = fwd ? fwd_waves(d, tau) : bwd_waves(d, tau);
    return pdssm::fused_lds_layout(d->N, d->K, W);
}

int staging_rows(const pdssm_desc* d, const pdssm::LdsLayout& l, int C) {
    if (l.total >= pdssm::kMaxLds) return 0;
    long long m = (long long)(pdssm::kMaxLds - l.total) / ((long long)d->N * 8);
    if (m > C) m = C;
    return m >= kMinStaging ? (int)m : 0;
}

bool use_fused(const pdssm_desc* d) {
    const int tau = scan_chunk(d);
    return fused_layout(d, tau, true).total <= pdssm::kMaxLds && fused_layout(d, tau, false).total <= pdssm::kMaxLds;
}

// Segments per sequence of the fused scans.  One workgroup per sequence
// keeps a CU busy; with fewer sequences than kSegTarget workgroups the
// sequences are cut along L into up to kMaxSeg segments of at least
// kMinSegChunks chunks (so the extra aggregate pass stays short relative to
// the scan).
#ifndef PDSSM_SEG_TARGET
#define PDSSM_SEG_TARGET 256
#endif
constexpr int kSegTarget = PDSSM_SEG_TARGET;
constexpr int kMaxSeg = 8;
constexpr int kMinSegChunks = 32;

struct Segs {
    int S, Cs;
};

Segs segments(const pdssm_desc* d, int C) {
    const long long seqs = (long long)d->B * d->H;
    int S = 1;
    if (seqs < kSegTarget) {
        S = (int)((kSegTarget + seqs - 1) / seqs);
        if (S > kMaxSeg) S = kMaxSeg;
        if (S > C / kMinSegChunks) S = C / kMinSegChunks;
        if (S < 1) S = 1;
    }
    Segs g;
    g.Cs = (C + S - 1) / S;
    g.S = (C + g.Cs - 1) / g.Cs;  // no empty segment
    return g;
}

// Fused workspace: byte dictionary, row records, per-entry max in-degree,
// then the segment aggregates when sequences are cut into segments.
size_t fused_tables_bytes(const Sizes& s, const pdssm_desc* d) {
    return align_up(s.dictN) + align_up(s.dictN * 8) + align_up((size_t)d->H * d->K);
}

size_t fused_ws_bytes(const Sizes& s, const pdssm_desc* d, int C) {
    const Segs g = segments(d, C);
    size_t n = fused_tables_bytes(s, d);
    if (g.S > 1) n += 2 * align_up(s.seqN * g.S * 8) + align_up(s.seqN * g.S * 4);
    return n;
}

// Chunked workspace: the dictionary tables (read from memory by the
// dictionary steps), then int map, complex diag, complex term, complex
// carry/U per chunk.
size_t chunked_ws_bytes(const Sizes& s, const pdssm_desc* d) {
    return fused_tables_bytes(s, d) + align_up(s.perChunk * 4) + 3 * align_up(s.perChunk * 8);
}

size_t ws_bytes_for(const Sizes& s, const pdssm_desc* d, int C) {
    return use_fused(d) ? fused_ws_bytes(s, d, C) : chunked_ws_bytes(s, d);
}

void carve_chunked(ScanArgs& a, void* ws, const Sizes& s, const pdssm_desc* d) {
    char* p = static_cast<char*>(ws) + fused_tables_bytes(s, d);
    a.agg_p = reinterpret_cast<int*>(p);
    p += align_up(s.perChunk * 4);
    a.agg_d = reinterpret_cast<float2*>(p);
    p += align_up(s.perChunk * 8);
    a.agg_v = reinterpret_cast<float2*>(p);
    p += align_up(s.perChunk * 8);
    a.U = reinterpret_cast<float2*>(p);  // fwd: carry when saved == NULL
}

bool narrow_io(const pdssm_desc* d);

// Dictionary tables of the fused kernels at the start of ws.
pdssm::PrepArgs carve_tables(const pdssm_desc* d, const int32_t* pi, void* ws, const Sizes& s, int* status) {
    char* p = static_cast<char*>(ws);
    pdssm::PrepArgs pa;
    pa.H = d->H;
    pa.K = d->K;
    pa.N = d->N;
    pa.pi = pi;
    pa.dict = reinterpret_cast<uint8_t*>(p);
    p += align_up(s.dictN);
    pa.rec = reinterpret_cast<uint64_t*>(p);
    p += align_up(s.dictN * 8);
    pa.mtab = reinterpret_cast<uint8_t*>(p);
    pa.status = status;
    return pa;
}

// Points the fused args at the tables in ws and builds them there unless the
// caller prepared them (PDSSM_FLAG_PREPARED).
hipError_t prep_fused(pdssm::FusedArgs& f, const pdssm_desc* d, const int32_t* pi, void* ws,
                      const Sizes& s, int* status, hipStream_t st, bool fwd) {
    const pdssm::PrepArgs pa = carve_tables(d, pi, ws, s, status);
    f.dict = pa.dict;
    f.rec = pa.rec;
    f.mtab = pa.mtab;
    f.W = fwd ? fwd_waves(d, f.tau) : bwd_waves(d, f.tau);
    f.lds = fused_layout(d, f.tau, fwd);
    f.sbM = fwd ? staging_rows(d, f.lds, f.C) : 0;
    f.lds = pdssm::fused_lds_add_staging(f.lds, d->N, f.sbM);
    // heads of permutations in a wide complex64 forward run kPermWaves
    // chunk waves on their own layout (more rows of staged chunk states)
    f.lds_perm = f.lds;
    f.sbM_perm = f.sbM;
    if (fwd && f.W > pdssm::kPermWaves && !narrow_io(d)) {
        f.lds_perm = pdssm::fused_lds_layout(d->N, d->K, pdssm::kPermWaves);
        f.sbM_perm = staging_rows(d, f.lds_perm, f.C);
        f.lds_perm = pdssm::fused_lds_add_staging(f.lds_perm, d->N, f.sbM_perm);
    }
    const Segs g = segments(d, f.C);
    f.S = g.S;
    f.Cs = g.Cs;
    f.segA = f.segD = nullptr;
    f.segP = nullptr;
    if (g.S > 1) {
        char* p = static_cast<char*>(ws) + fused_tables_bytes(s, d);
        f.segA = reinterpret_cast<float2*>(p);
        p += align_up(s.seqN * g.S * 8);
        f.segD = reinterpret_cast<float2*>(p);
        p += align_up(s.seqN * g.S * 8);
        f.segP = reinterpret_cast<int*>(p);
    }
    if (d->flags & PDSSM_FLAG_PREPARED) return hipSuccess;
    return pdssm::launch_prep(pa, st);
}

// The chunked kernels' per-chunk buffers and dictionary tables in ws; the
// tables are built there unless the caller prepared them.
hipError_t prep_chunked(ScanArgs& a, const pdssm_desc* d, const int32_t* pi, void* ws, const Sizes& s,
                        int* status, hipStream_t st) {
    carve_chunked(a, ws, s, d);
    const pdssm::PrepArgs pa = carve_tables(d, pi, ws, s, status);
    a.rec = pa.rec;
    a.mtab = pa.mtab;
    if (d->flags & PDSSM_FLAG_PREPARED) return hipSuccess;
    return pdssm::launch_prep(pa, st);
}

pdssm::FusedArgs fused_base(const ScanArgs& a) {
    pdssm::FusedArgs f = {};
    f.B = a.B;
    f.L = a.L;
    f.H = a.H;
    f.N = a.N;
    f.K = a.K;
    f.tau = a.tau;
    f.C = a.C;
    f.idx = a.idx;
    f.D = a.D;
    f.b = a.b;
    f.c = a.c;
    f.h0 = a.h0;
    f.dy = a.dy;
    f.dhf = a.dhf;
    f.y = a.y;
    f.hfinal = a.hfinal;
    f.dD = a.dD;
    f.db = a.db;
    f.dc = a.dc;
    f.dh0 = a.dh0;
    f.status = a.status;
    return f;
}

// Row format of D, b, c (and dD, db, dc) selected by the flags.
int io_format(const pdssm_desc* d) {
    if (d->flags & PDSSM_FLAG_REAL_IO) return pdssm::kIoReal;
    if (d->flags & PDSSM_FLAG_BF16_IO) return pdssm::kIoBf16;
    return pdssm::kIoC64;
}

// A 4-byte row format (bf16 pairs or real fp32).
bool narrow_io(const pdssm_desc* d) { return io_format(d) != pdssm::kIoC64; }

// Bytes per entry of D, b, c (and dD, db, dc).
size_t io_bytes(const pdssm_desc* d) { return narrow_io(d) ? 4 : 8; }

ScanArgs base_args(const pdssm_desc* d, int tau) {
    ScanArgs a = {};
    a.B = d->B;
    a.L = d->L;
    a.H = d->H;
    a.N = d->N;
    a.K = d->K;
    a.tau = tau;
    a.C = (d->L + tau - 1) / tau;
    a.io = io_format(d);
    return a;
}

bool misaligned(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) % 16) != 0; }

// int32 / fp32 arrays (idx, y, dy) are read and written as 4-byte words.
bool misaligned4(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) % 4) != 0; }

}  // namespace

extern "C" {

int pdssm_abi_version(void) { return PDSSM_ABI_VERSION; }

int pdssm_chunk_len(const pdssm_desc* d) { return scan_chunk(d); }

int pdssm_num_chunks(const pdssm_desc* d) {
    int tau = scan_chunk(d);
    if (tau < 0) return tau;
    return (d->L + tau - 1) / tau;
}

size_t pdssm_workspace_size(const pdssm_desc* d, int op) {
    if (op == PDSSM_OP_COMPOSE) return check_dims(d) == PDSSM_OK ? 0 : (size_t)-1;
    if (op == PDSSM_OP_STE_GRADS)
        return check_dims(d) == PDSSM_OK ? pdssm::dict_plan(d->B, d->L, d->H, d->N, d->K).bytes : (size_t)-1;
    if (op != PDSSM_OP_FWD && op != PDSSM_OP_BWD) return (size_t)-1;
    int tau = scan_chunk(d);
    if (tau < 0) return (size_t)-1;
    const int C = (d->L + tau - 1) / tau;
    return ws_bytes_for(sizes_of(d, C), d, C);
}

const char* pdssm_status_string(int st) {
    switch (st) {
        case PDSSM_OK: return "PDSSM_OK";
        case PDSSM_ERR_INVALID_ARG: return "PDSSM_ERR_INVALID_ARG: bad pointer, size, flags or overlapping buffers";
        case PDSSM_ERR_UNSUPPORTED: return "PDSSM_ERR_UNSUPPORTED: N, K, chunk or total size outside the supported set";
        case PDSSM_ERR_WORKSPACE: return "PDSSM_ERR_WORKSPACE: workspace missing or smaller than pdssm_workspace_size";
        case PDSSM_ERR_HIP: return "PDSSM_ERR_HIP: a HIP kernel launch failed";
        case PDSSM_ERR_INDEX: return "PDSSM_ERR_INDEX: idx or pi entry out of range";
        default: return "unknown pdssm status";
    }
}

int pdssm_scan_segments(const pdssm_desc* d) {
    const int tau = scan_chunk(d);
    if (tau < 0) return tau;
    if (!use_fused(d)) return 1;
    return segments(d, (d->L + tau - 1) / tau).S;
}

int pdssm_uses_fused(const pdssm_desc* d) {
    const int tau = scan_chunk(d);
    if (tau < 0) return tau;
    return use_fused(d) ? 1 : 0;
}

int pdssm_prepare(const pdssm_desc* d, const int32_t* pi, void* ws, size_t ws_bytes, int* dev_status,
                  void* stream) {
    int tau = scan_chunk(d);
    if (tau < 0) return tau;
    if (!pi || misaligned(pi)) return PDSSM_ERR_INVALID_ARG;
    const int C = (d->L + tau - 1) / tau;
    const Sizes s = sizes_of(d, C);
    const size_t need = ws_bytes_for(s, d, C);
    if (!ws || ws_bytes < need || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0)
        return PDSSM_ERR_WORKSPACE;
    if (overlap({ws, need}, {pi, (size_t)d->H * d->K * d->N * 4})) return PDSSM_ERR_INVALID_ARG;
    const hipError_t e = pdssm::launch_prep(carve_tables(d, pi, ws, s, dev_status), static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

int pdssm_scan_fwd(const pdssm_desc* d, const int32_t* idx, const int32_t* pi,
                   const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                   const pdssm_c64* h0, float* y, pdssm_c64* h_final, pdssm_c64* saved,
                   void* ws, size_t ws_bytes, int* dev_status, void* stream) {
    int tau = scan_chunk(d);
    if (tau < 0) return tau;
    if (!idx || !pi || !D || !b || !c || !y) return PDSSM_ERR_INVALID_ARG;
    for (const void* p : {(const void*)D, (const void*)b, (const void*)c, (const void*)h0,
                          (const void*)h_final, (const void*)saved, (const void*)pi})
        if (misaligned(p)) return PDSSM_ERR_INVALID_ARG;
    if (misaligned4(idx) || misaligned4(y)) return PDSSM_ERR_INVALID_ARG;
    ScanArgs a = base_args(d, tau);
    const Sizes s = sizes_of(d, a.C);
    const size_t need = ws_bytes_for(s, d, a.C);
    if (!ws || ws_bytes < need || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0)
        return PDSSM_ERR_WORKSPACE;
    const size_t nidx = s.idxN * 4, npi = (size_t)d->H * d->K * d->N * 4, nst = s.stepN * io_bytes(d);
    if (any_overlap({{y, s.idxN * 4}, {h_final, s.seqN * 8}, {saved, s.perChunk * state_bytes(d)}, {ws, need}},
                    {{idx, nidx}, {pi, npi}, {D, nst}, {b, nst}, {c, nst}, {h0, s.seqN * 8}}))
        return PDSSM_ERR_INVALID_ARG;
    a.idx = idx;
    a.pi = pi;
    a.D = reinterpret_cast<const float2*>(D);
    a.b = reinterpret_cast<const float2*>(b);
    a.c = reinterpret_cast<const float2*>(c);
    a.h0 = reinterpret_cast<const float2*>(h0);
    a.y = y;
    a.hfinal = reinterpret_cast<float2*>(h_final);
    a.status = dev_status;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (use_fused(d)) {
        pdssm::FusedArgs f = fused_base(a);
        f.saved = reinterpret_cast<float2*>(saved);
        f.io = io_format(d);
        e = prep_fused(f, d, pi, ws, s, dev_status, st, true);
        if (e == hipSuccess) e = pdssm::launch_fwd_fused(f, st);
    } else {
        e = prep_chunked(a, d, pi, ws, s, dev_status, st);
        a.carry = saved ? reinterpret_cast<float2*>(saved) : a.U;
        if (e == hipSuccess) e = pdssm::launch_fwd_chunked(a, st);
    }
    return e == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

namespace {

int scan_bwd_impl(const pdssm_desc* d, const int32_t* idx, const int32_t* pi, const pdssm_c64* D,
                  const pdssm_c64* b, const pdssm_c64* c, const pdssm_c64* saved, const float* dy,
                  const pdssm_c64* dh_final, pdssm_c64* dD, pdssm_c64* db, pdssm_c64* dc, pdssm_c64* dh0,
                  pdssm_c64* z, void* ws, size_t ws_bytes, int* dev_status, void* stream) {
    int tau = scan_chunk(d);
    if (tau < 0) return tau;
    if (!idx || !pi || !D || !b || !c || !saved || !dy || !dD || !db || !dc)
        return PDSSM_ERR_INVALID_ARG;
    for (const void* p : {(const void*)D, (const void*)b, (const void*)c, (const void*)saved,
                          (const void*)dh_final, (const void*)dD, (const void*)db,
                          (const void*)dc, (const void*)dh0, (const void*)pi})
        if (misaligned(p)) return PDSSM_ERR_INVALID_ARG;
    if (misaligned4(idx) || misaligned4(dy)) return PDSSM_ERR_INVALID_ARG;
    ScanArgs a = base_args(d, tau);
    const Sizes s = sizes_of(d, a.C);
    const size_t need = ws_bytes_for(s, d, a.C);
    if (!ws || ws_bytes < need || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0)
        return PDSSM_ERR_WORKSPACE;
    if (misaligned(z)) return PDSSM_ERR_INVALID_ARG;
    const size_t nidx = s.idxN * 4, npi = (size_t)d->H * d->K * d->N * 4, nst = s.stepN * io_bytes(d);
    // z: complex64 with bf16 pairs (rounding it would round the
    // straight-through inputs), else the gradients' row format
    const size_t nz = s.stepN * (io_format(d) == pdssm::kIoBf16 ? 8 : io_bytes(d));
    if (any_overlap({{dD, nst}, {db, nst}, {dc, nst}, {dh0, s.seqN * 8}, {z, nz}, {ws, need}},
                    {{idx, nidx}, {pi, npi}, {D, nst}, {b, nst}, {c, nst}, {saved, s.perChunk * state_bytes(d)},
                     {dy, nidx}, {dh_final, s.seqN * 8}}))
        return PDSSM_ERR_INVALID_ARG;
    a.idx = idx;
    a.pi = pi;
    a.D = reinterpret_cast<const float2*>(D);
    a.b = reinterpret_cast<const float2*>(b);
    a.c = reinterpret_cast<const float2*>(c);
    a.dy = dy;
    a.dhf = reinterpret_cast<const float2*>(dh_final);
    a.dD = reinterpret_cast<float2*>(dD);
    a.db = reinterpret_cast<float2*>(db);
    a.dc = reinterpret_cast<float2*>(dc);
    a.dh0 = reinterpret_cast<float2*>(dh0);
    a.z = reinterpret_cast<float2*>(z);
    a.status = dev_status;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (use_fused(d)) {
        pdssm::FusedArgs f = fused_base(a);
        f.saved = const_cast<float2*>(reinterpret_cast<const float2*>(saved));
        f.z = reinterpret_cast<float2*>(z);
        f.io = io_format(d);
        e = prep_fused(f, d, pi, ws, s, dev_status, st, false);
        if (e == hipSuccess) e = pdssm::launch_bwd_fused(f, st);
    } else {
        e = prep_chunked(a, d, pi, ws, s, dev_status, st);
        a.carry = const_cast<float2*>(reinterpret_cast<const float2*>(saved));
        if (e == hipSuccess) e = pdssm::launch_bwd_chunked(a, st);
    }
    return e == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

}  // namespace

int pdssm_scan_bwd(const pdssm_desc* d, const int32_t* idx, const int32_t* pi,
                   const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                   const pdssm_c64* saved, const float* dy, const pdssm_c64* dh_final,
                   pdssm_c64* dD, pdssm_c64* db, pdssm_c64* dc, pdssm_c64* dh0,
                   void* ws, size_t ws_bytes, int* dev_status, void* stream) {
    return scan_bwd_impl(d, idx, pi, D, b, c, saved, dy, dh_final, dD, db, dc, dh0, nullptr, ws, ws_bytes,
                         dev_status, stream);
}

int pdssm_scan_bwd_ste(const pdssm_desc* d, const int32_t* idx, const int32_t* pi,
                       const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                       const pdssm_c64* saved, const float* dy, const pdssm_c64* dh_final,
                       pdssm_c64* dD, pdssm_c64* db, pdssm_c64* dc, pdssm_c64* dh0,
                       pdssm_c64* z, void* ws, size_t ws_bytes, int* dev_status, void* stream) {
    if (!z) return PDSSM_ERR_INVALID_ARG;
    return scan_bwd_impl(d, idx, pi, D, b, c, saved, dy, dh_final, dD, db, dc, dh0, z, ws, ws_bytes, dev_status,
                         stream);
}

int pdssm_ste_grads(const pdssm_desc* d, const int32_t* idx, const int32_t* pi, const pdssm_c64* g,
                    const pdssm_c64* z, float* q, float* G, void* ws, size_t ws_bytes, int* dev_status,
                    void* stream) {
    const int st = check_dims(d);
    if (st != PDSSM_OK) return st;
    if (!idx || !g || !z || (!q && !G) || (q && !pi)) return PDSSM_ERR_INVALID_ARG;
    if (misaligned4(idx)) return PDSSM_ERR_INVALID_ARG;
    if (misaligned(g) || misaligned(z) || misaligned(pi) || (reinterpret_cast<uintptr_t>(G) & 3) != 0 ||
        (reinterpret_cast<uintptr_t>(q) & 3) != 0)
        return PDSSM_ERR_INVALID_ARG;
    const pdssm::DictPlan plan = pdssm::dict_plan(d->B, d->L, d->H, d->N, d->K);
    if (!ws || ws_bytes < plan.bytes || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0)
        return PDSSM_ERR_WORKSPACE;
    // g in the row format (bf16 pairs, real fp32 or complex64); z complex64
    // with bf16 pairs (as pdssm_scan_bwd_ste writes it), else the same format
    const size_t nidx = (size_t)d->B * d->L * d->H * 4, nst = nidx / 4 * d->N * io_bytes(d);
    const size_t nz = nidx / 4 * d->N * (io_format(d) == pdssm::kIoBf16 ? 8 : io_bytes(d));
    const size_t nG = (size_t)d->H * d->K * d->N * d->N * 4, npi = (size_t)d->H * d->K * d->N * 4;
    if (any_overlap({{G, nG}, {q, nidx * d->K}, {ws, plan.bytes}}, {{idx, nidx}, {g, nst}, {z, nz}, {pi, npi}}))
        return PDSSM_ERR_INVALID_ARG;
    pdssm::SteGradArgs a = {};
    a.B = d->B;
    a.L = d->L;
    a.H = d->H;
    a.N = d->N;
    a.K = d->K;
    a.idx = idx;
    a.pi = pi;
    a.io = io_format(d);
    a.g = reinterpret_cast<const float2*>(g);
    a.z = reinterpret_cast<const float2*>(z);
    a.q = q;
    a.G = G;
    a.plan = plan;
    a.ws = static_cast<unsigned char*>(ws);
    a.status = dev_status;
    return pdssm::launch_ste_grads(a, static_cast<hipStream_t>(stream)) == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

int pdssm_decode_step(const pdssm_desc* d, const int32_t* idx, const int32_t* pi, const pdssm_c64* D,
                      const pdssm_c64* b, const pdssm_c64* c, const pdssm_c64* h_in, pdssm_c64* h_out, float* y,
                      int* dev_status, void* stream) {
    const int st = check_dims(d);
    if (st != PDSSM_OK) return st;
    if (!idx || !pi || !D || !b || !c || !h_out || !y) return PDSSM_ERR_INVALID_ARG;
    for (const void* p : {(const void*)pi, (const void*)D, (const void*)b, (const void*)c, (const void*)h_in,
                          (const void*)h_out})
        if (misaligned(p)) return PDSSM_ERR_INVALID_ARG;
    if (misaligned4(idx) || misaligned4(y)) return PDSSM_ERR_INVALID_ARG;
    const size_t nseq = (size_t)d->B * d->H, nrow = nseq * d->N * 8, nio = nseq * d->N * io_bytes(d);
    const size_t npi = (size_t)d->H * d->K * d->N * 4;
    // the state may be updated in place (h_out == h_in); no other overlap
    if (any_overlap({{h_out, nrow}, {y, nseq * 4}},
                    {{idx, nseq * 4}, {pi, npi}, {D, nio}, {b, nio}, {c, nio}, {h_in == h_out ? nullptr : h_in, nrow}}))
        return PDSSM_ERR_INVALID_ARG;
    pdssm::DecodeArgs a = {};
    a.B = d->B;
    a.H = d->H;
    a.N = d->N;
    a.K = d->K;
    a.idx = idx;
    a.pi = pi;
    a.io = io_format(d);
    a.D = D;
    a.b = b;
    a.c = c;
    a.h_in = reinterpret_cast<const float2*>(h_in);
    a.h_out = reinterpret_cast<float2*>(h_out);
    a.y = y;
    a.status = dev_status;
    return pdssm::launch_decode(a, static_cast<hipStream_t>(stream)) == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

int pdssm_dict_argmax(int32_t H, int32_t K, int32_t N, const float* M, int32_t* pi, void* stream) {
    if (H < 1 || K < 1 || !n_supported(N) || K > 256) return H < 1 || K < 1 ? PDSSM_ERR_INVALID_ARG : PDSSM_ERR_UNSUPPORTED;
    if ((long long)H * K * N * N >= (1LL << 31)) return PDSSM_ERR_UNSUPPORTED;
    if (!M || !pi || (reinterpret_cast<uintptr_t>(M) & 3) || (reinterpret_cast<uintptr_t>(pi) & 3))
        return PDSSM_ERR_INVALID_ARG;
    const size_t nM = (size_t)H * K * N * N * 4, npi = (size_t)H * K * N * 4;
    if (any_overlap({{pi, npi}}, {{M, nM}})) return PDSSM_ERR_INVALID_ARG;
    return pdssm::launch_dict_argmax(M, pi, H * K, N, static_cast<hipStream_t>(stream)) == hipSuccess
               ? PDSSM_OK
               : PDSSM_ERR_HIP;
}

int pdssm_route(int32_t T, int32_t Dm, int32_t H, int32_t K, const uint16_t* u, const uint16_t* S,
                float* logits, int32_t* idx, void* stream) {
    if (T < 1 || Dm < 1 || H < 1 || K < 1) return PDSSM_ERR_INVALID_ARG;
    if (K > 256 || Dm % 8 != 0) return PDSSM_ERR_UNSUPPORTED;
    if ((H + 256 / K - 1) / (256 / K) > 65535) return PDSSM_ERR_UNSUPPORTED;  // head groups (grid y)
    if ((long long)T * Dm >= (1LL << 31) || (long long)T * H * K >= (1LL << 31) ||
        (long long)H * K * Dm >= (1LL << 31))
        return PDSSM_ERR_UNSUPPORTED;
    if (!u || !S || !idx || misaligned(u) || misaligned(S) || (reinterpret_cast<uintptr_t>(logits) & 3) ||
        (reinterpret_cast<uintptr_t>(idx) & 3))
        return PDSSM_ERR_INVALID_ARG;
    const size_t nu = (size_t)T * Dm * 2, nS = (size_t)H * K * Dm * 2;
    if (any_overlap({{logits, (size_t)T * H * K * 4}, {idx, (size_t)T * H * 4}}, {{u, nu}, {S, nS}}))
        return PDSSM_ERR_INVALID_ARG;
    pdssm::RouteArgs a = {};
    a.T = T;
    a.Dm = Dm;
    a.H = H;
    a.K = K;
    a.u = u;
    a.S = S;
    a.logits = logits;
    a.idx = idx;
    return pdssm::launch_route(a, static_cast<hipStream_t>(stream)) == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

int pdssm_project(int32_t T, int32_t Dm, int32_t H, int32_t K, int32_t N, const uint16_t* u,
                  const uint16_t* S, const uint16_t* Wb, const uint16_t* Wc, const uint16_t* Wd, float* logits,
                  int32_t* idx, pdssm_c64* b, pdssm_c64* c, pdssm_c64* D, void* stream) {
    if (T < 1 || Dm < 1 || H < 1 || !u) return PDSSM_ERR_INVALID_ARG;
    if ((!Wb) != (!b) || (!Wc) != (!c) || (!Wd) != (!D)) return PDSSM_ERR_INVALID_ARG;
    if (!S && !Wb && !Wc && !Wd) return PDSSM_ERR_INVALID_ARG;
    if (S && (K < 1 || !idx)) return PDSSM_ERR_INVALID_ARG;
    if ((logits || idx) && !S) return PDSSM_ERR_INVALID_ARG;
    const bool proj = Wb || Wc || Wd;
    if (proj && !n_supported(N)) return PDSSM_ERR_UNSUPPORTED;
    if ((S && K > 256) || Dm % 32 != 0) return PDSSM_ERR_UNSUPPORTED;
    const long long rows = (S ? (long long)H * K : 0) > (proj ? 2LL * H * N : 0) ? (long long)H * K : 2LL * H * N;
    if ((long long)(T + 256) * Dm * 2 >= (1LL << 32) || (rows + 256) * Dm * 2 >= (1LL << 32) ||
        (long long)T * H * (S ? K : 1) >= (1LL << 31) || (proj && 2LL * T * H * N >= (1LL << 31)))
        return PDSSM_ERR_UNSUPPORTED;
    for (const void* p : {(const void*)u, (const void*)S, (const void*)Wb, (const void*)Wc, (const void*)Wd,
                          (const void*)b, (const void*)c, (const void*)D})
        if (misaligned(p)) return PDSSM_ERR_INVALID_ARG;
    if (misaligned4(logits) || misaligned4(idx)) return PDSSM_ERR_INVALID_ARG;
    const size_t nu = (size_t)T * Dm * 2, nS = S ? (size_t)H * K * Dm * 2 : 0, nW = (size_t)H * 2 * N * Dm * 2;
    const size_t nout = (size_t)T * H * N * 8;
    if (any_overlap({{logits, S ? (size_t)T * H * K * 4 : 0}, {idx, S ? (size_t)T * H * 4 : 0}, {b, nout},
                     {c, nout}, {D, nout}},
                    {{u, nu}, {S, nS}, {Wb, nW}, {Wc, nW}, {Wd, nW}}))
        return PDSSM_ERR_INVALID_ARG;
    pdssm::ProjectArgs a = {};
    a.T = T;
    a.Dm = Dm;
    a.H = H;
    a.K = S ? K : 1;
    a.N = proj ? N : 8;
    a.u = u;
    a.S = S;
    a.logits = logits;
    a.idx = idx;
    const uint16_t* W[3] = {Wb, Wc, Wd};
    pdssm_c64* out[3] = {b, c, D};
    for (int i = 0; i < 3; ++i)
        if (W[i]) {
            a.W[a.nproj] = W[i];
            a.out[a.nproj] = reinterpret_cast<float*>(out[i]);
            a.kind[a.nproj] = i == 2 ? pdssm::kProjGen : pdssm::kProjPlain;
            ++a.nproj;
        }
    return pdssm::launch_project(a, static_cast<hipStream_t>(stream)) == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

int pdssm_softmax_vjp(const float* x, const float* gy, float* gx, int64_t outer, int32_t len, int64_t inner,
                      float temp, void* stream) {
    if (!x || !gy || !gx || outer < 0 || len < 1 || inner < 1) return PDSSM_ERR_INVALID_ARG;
    if (!(temp > 0.f) || temp > 3.0e38f) return PDSSM_ERR_INVALID_ARG;
    // up to 64 lanes per (outer, inner) fibre: fewer than 2^31 fibres keeps
    // the grid below 2^29 blocks
    if (outer > (1LL << 40) / len / inner || outer >= (1LL << 31) / inner) return PDSSM_ERR_UNSUPPORTED;
    const size_t n = (size_t)outer * len * inner * 4;
    if (((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(gy) | reinterpret_cast<uintptr_t>(gx)) & 3) != 0)
        return PDSSM_ERR_INVALID_ARG;
    if (any_overlap({{gx, n}}, {{x, n}, {gy, n}})) return PDSSM_ERR_INVALID_ARG;
    return pdssm::launch_softmax_vjp(x, gy, gx, outer, len, inner, 1.f / temp, static_cast<hipStream_t>(stream)) ==
                   hipSuccess
               ? PDSSM_OK
               : PDSSM_ERR_HIP;
}

int pdssm_compose_chunks(const pdssm_desc* d, const int32_t* idx, const int32_t* pi,
                         const pdssm_c64* D, int32_t* pi_out, pdssm_c64* d_out,
                         int* dev_status, void* stream) {
    int st = check_dims(d);
    if (st != PDSSM_OK) return st;
    if (narrow_io(d)) return PDSSM_ERR_UNSUPPORTED;
    if (!idx || !pi || !D || !pi_out || !d_out) return PDSSM_ERR_INVALID_ARG;
    if (misaligned(D) || misaligned(pi) || misaligned(pi_out) || misaligned(d_out) || misaligned4(idx))
        return PDSSM_ERR_INVALID_ARG;
    pdssm::ComposeArgs a = {};
    a.B = d->B;
    a.L = d->L;
    a.H = d->H;
    a.N = d->N;
    a.K = d->K;
    a.tau = d->chunk == 0 ? kDefaultComposeChunk : d->chunk;
    if (a.tau > d->L) a.tau = d->L;
    a.C = (d->L + a.tau - 1) / a.tau;
    const size_t per = (size_t)d->B * d->H * a.C * d->N;
    const size_t nst = (size_t)d->B * d->L * d->H * d->N * 8;
    if (any_overlap({{pi_out, per * 4}, {d_out, per * 8}},
                    {{idx, (size_t)d->B * d->L * d->H * 4}, {pi, (size_t)d->H * d->K * d->N * 4},
                     {D, nst}}))
        return PDSSM_ERR_INVALID_ARG;
    a.idx = idx;
    a.pi = pi;
    a.D = reinterpret_cast<const float2*>(D);
    a.pi_out = pi_out;
    a.d_out = reinterpret_cast<float2*>(d_out);
    a.status = dev_status;
    hipError_t e = pdssm::launch_compose(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PDSSM_OK : PDSSM_ERR_HIP;
}

}  // extern "C"
