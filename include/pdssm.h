/*
 * pdssm.h -- C ABI of the MI355X (gfx950) PD-scan library, libpdssm.so.
 *
 * The library computes the forward and backward pass of the structured sparse
 * linear recurrence of Flash PD-SSM (arXiv 2605.19150):
 *
 *   h_t = P_t D_t h_{t-1} + b_t,      y_t = Re( sum_n c_t[n] h_t[n] ),
 *
 * per (batch b, head h) sequence, t = 0..L-1, state size N.
 *   - P_t is column-one-hot (paper Sec. 2.3 column hardmax; Sec. 3.1 eq. (5);
 *     App. D): it is stored as an int map pi_t of length N, and column j has
 *     its one in row pi_t[j].  Source entry j of the state is scaled by D_t[j]
 *     and moved to entry pi_t[j]; entries mapped to the same row add up.
 *   - pi_t is row k_t = idx[b,t,h] of the per-head dictionary pi[h,:,:]
 *     (Sec. 3.1 eqs. (5)-(8), hard selection; App. E.2.1 index arrays).
 *   - D_t is a per-step complex diagonal, b_t the per-step input term
 *     (App. E.2 recurrence), c_t the readout vector and Re the real readout
 *     (Sec. 2.1 eq. (1) with psi = Re).
 *   - Two PD operators compose in linear time (App. E.2 associative operator,
 *     App. E.3.1 accumulator update): applying (pi1, d1) then (pi2, d2) gives
 *     (pi2[pi1[j]], d2[pi1[j]] * d1[j]).
 *   - The sequence is cut into chunks of `chunk` steps (App. E.1 Algorithm 1,
 *     chunk c = steps [c*chunk, min((c+1)*chunk, L)), last one may be short).
 *     Only the states entering each chunk ("saved") ever reach memory; the
 *     per-step states h_t are never written.
 *
 * Conventions shared by every entry point
 *   - Tensors are dense row-major device memory owned by the caller.  Complex
 *     numbers are interleaved (re, im) float32 pairs (== torch.complex64).
 *       idx [B,L,H] int32 in [0,K)   pi [H,K,N] int32 in [0,N)
 *       D, b, c [B,L,H,N] complex    y, dy [B,L,H] float32
 *       h0, h_final, dh_final, dh0 [B,H,N] complex
 *       saved [B,H,C,N] complex (fp32 for the real model), C = pdssm_num_chunks(desc)
 *   - The library never allocates or frees memory and never synchronises.
 *     Scratch memory comes from the caller as `ws` (at least
 *     pdssm_workspace_size(desc, op) bytes, 256-byte aligned).  All work is
 *     enqueued in order on `stream` (a hipStream_t; NULL = default stream)
 *     and the call returns once it is enqueued.
 *   - Outputs are overwritten, never accumulated.  Outputs must not overlap
 *     inputs or each other.  Optional pointers may be NULL.
 *   - Return value: PDSSM_OK, or a negative pdssm_status detected on the host
 *     (bad pointer or size, unsupported N or chunk, workspace too small, HIP
 *     launch failure).  Nothing is enqueued when a host check fails.
 *   - Index checking is always on: an idx entry outside [0,K) or a pi entry
 *     outside [0,N) is replaced by 0 inside the kernels (so every memory access
 *     stays in bounds) and PDSSM_ERR_INDEX is stored to *dev_status (a device
 *     int the caller zeroes beforehand and reads after synchronising; it is
 *     never cleared by the library).  Results of an affected sequence are then
 *     meaningless.  dev_status may be NULL.
 *   - Complex gradients follow dX = dl/dRe(X) + i*dl/dIm(X) (torch's
 *     convention) for the loss l = sum_t dy_t*y_t + Re(sum conj(dh_final)*h_L).
 *   - Supported sizes: N in {8, 16, 32, 64, 128, 256}; 1 <= K <= 256;
 *     B, L, H >= 1 with B*L*H*N < 2^31.  For scan_fwd / scan_bwd the chunk is
 *     4, 8 or 16 steps with chunk * max(1, N/64) <= 16, or 0 for the default
 *     (8 for N <= 128, 4 for N = 256); pdssm_compose_chunks takes any chunk
 *     >= 1 (0 = 32).  One head's dictionary tables, (K+1)*N*9 bytes plus the
 *     per-wave buffers, are staged in the 160 KiB LDS of a workgroup; larger
 *     dictionaries run slower multi-pass kernels with the same results.
 *   - Calls on different streams may run concurrently if their outputs and
 *     workspaces do not overlap; the library keeps no mutable global state
 *     apart from the device array of pdssm_scan_fwd_noalloc.
 *   - Waits between the waves of a workgroup are bounded: a wait that sees no
 *     progress for a long window (a fault, not a slow input) stores
 *     PDSSM_ERR_HIP to *dev_status and releases every wave, so the kernel
 *     always ends.
 */
#ifndef PDSSM_H
#define PDSSM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PDSSM_ABI_VERSION 1

typedef struct pdssm_c64 {
    float re, im;
} pdssm_c64;

typedef struct pdssm_desc {
    int32_t B, L, H, N, K; /* batch, steps, heads, state size, dictionary size */
    int32_t chunk;         /* steps per chunk; 0 = default; fwd and bwd must agree */
    uint32_t flags;        /* 0 or PDSSM_FLAG_PREPARED | (PDSSM_FLAG_BF16_IO or PDSSM_FLAG_REAL_IO) */
} pdssm_desc;

/* desc->flags bit for pdssm_scan_fwd / pdssm_scan_bwd: the dictionary tables in
 * ws were built by pdssm_prepare for this desc and the current contents of pi;
 * the scan reuses them instead of rebuilding them. */
#define PDSSM_FLAG_PREPARED 1u

/* desc->flags bit for pdssm_scan_fwd / pdssm_scan_bwd / pdssm_decode_step (and
 * pdssm_prepare, which ignores it): D, b, c and dD, db, dc are bf16 (re, im) pairs, 4 bytes
 * per complex entry (real part in the low 16 bits; torch:
 * view_as_real(x).to(bfloat16)), the paper's bf16 input setting (App. E,
 * kernel efficiency: the complex inputs split into two bf16 halves, fp32
 * arithmetic).  Every other tensor (idx, pi, h0, h_final, saved, y, dy,
 * dh_final, dh0) keeps its type.  The arithmetic is fp32 as without the
 * flag: inputs widen exactly, gradients are rounded to nearest (ties to
 * even) when stored.  The straight-through pair keeps z complex64 (a bf16 z
 * would round the straight-through inputs): pdssm_scan_bwd_ste writes it so,
 * and pdssm_ste_grads takes g = db as bf16 pairs with that complex64 z.
 * pdssm_compose_chunks returns PDSSM_ERR_UNSUPPORTED. */
#define PDSSM_FLAG_BF16_IO 2u

/* desc->flags bit for pdssm_scan_fwd / pdssm_scan_bwd / pdssm_decode_step (and
 * pdssm_prepare, which ignores it): the real-valued model (App. B, the MAD and time-series
 * setups use it): D, b, c and dD, db, dc are real fp32 [B,L,H,N], 4 bytes per
 * entry, the recurrence h_t = P_t (D_t .* h_{t-1}) + b_t over the reals and
 * y_t = sum_n c_t[n] h_t[n].  The saved chunk states are real fp32 too:
 * saved holds B*H*C*N floats (4 bytes per entry, [B,H,C,N]; the pointer is
 * reinterpreted like those of D, b, c), which pdssm_scan_bwd reads back the
 * same way.  Every other tensor keeps its type: h0, h_final, dh_final and dh0
 * stay complex64; for the real model h0 and dh_final hold real values (their
 * imaginary parts must be 0; or NULL) and h_final, dh0 come out with
 * imaginary parts 0.  The single-read scan kernels
 * keep the state real (float arithmetic, half the work of complex64); every
 * product that feeds a sum is a fused multiply-add in both settings, so every
 * result still equals, bit for bit, the real part of a complex64 call on the
 * same values (saved: the real parts of the complex64 call's saved states;
 * the multi-pass kernels, for dictionaries beyond LDS, and the decode step
 * compute the complex64 arithmetic on the real rows).  Cannot be
 * combined with
 * PDSSM_FLAG_BF16_IO (PDSSM_ERR_INVALID_ARG).  The scans, pdssm_decode_step
 * and the straight-through pair pdssm_scan_bwd_ste / pdssm_ste_grads support
 * it (z, g real fp32 rows); pdssm_compose_chunks returns
 * PDSSM_ERR_UNSUPPORTED. */
#define PDSSM_FLAG_REAL_IO 4u

typedef enum pdssm_status {
    PDSSM_OK = 0,
    PDSSM_ERR_INVALID_ARG = -1, /* NULL required pointer, bad size, overlap, unknown flags */
    PDSSM_ERR_UNSUPPORTED = -2, /* N, K or chunk outside the supported set */
    PDSSM_ERR_WORKSPACE = -3,   /* ws NULL or smaller than pdssm_workspace_size */
    PDSSM_ERR_HIP = -4,         /* a HIP call reported an error; in *dev_status: a wait gave up */
    PDSSM_ERR_INDEX = -5        /* written to *dev_status by kernels only */
} pdssm_status;

typedef enum pdssm_op {
    PDSSM_OP_FWD = 1,
    PDSSM_OP_BWD = 2,
    PDSSM_OP_COMPOSE = 3,
    PDSSM_OP_STE_GRADS = 4
} pdssm_op;

/* ABI version of the loaded library (PDSSM_ABI_VERSION at build time). */
int pdssm_abi_version(void);

/* Effective chunk length tau of desc (resolves chunk = 0; the chunk of App.
 * E.1 Algorithm 1), or a negative status. */
int pdssm_chunk_len(const pdssm_desc* desc);

/* C = ceil(L / tau), the number of chunks of App. E.1 Algorithm 1 (the last
 * one may be short) for the effective chunk: the third extent of `saved`.
 * Negative status for an invalid desc. */
int pdssm_num_chunks(const pdssm_desc* desc);

/* Workspace bytes the op needs for desc (0 if none): the per-head dictionary
 * tables (App. E.2.1: one dictionary serves every step) and, for few long
 * sequences, the segment aggregates of App. E.1 Algorithm 1 one level up
 * (PDSSM_OP_FWD / PDSSM_OP_BWD), or the map-grouped partial sums of the
 * straight-through gradients (PDSSM_OP_STE_GRADS); (size_t)-1 if desc is
 * invalid. */
size_t pdssm_workspace_size(const pdssm_desc* desc, int op);

/* 1 if the scans of desc run the single-read kernels (one head's dictionary
 * tables fit in LDS), 0 if they run the multi-pass kernels, or a negative
 * status for an invalid desc. */
int pdssm_uses_fused(const pdssm_desc* desc);

/* Number of segments each sequence is cut into along L by the single-read
 * scans (1, or up to 8 when there are fewer than 256 sequences and at least
 * 32 chunks per segment): segment s covers chunks [s*Cs, min((s+1)*Cs, C)),
 * Cs = ceil(C/S), one workgroup each, after a pass that folds every segment
 * into one PD operator (App. E.1 Algorithm 1's aggregate-then-carry
 * structure, one level up).  Negative status for an invalid desc. */
int pdssm_scan_segments(const pdssm_desc* desc);

/* Human-readable name of a status code (static string, never NULL); the
 * codes are this library's, not the paper's. */
const char* pdssm_status_string(int status);

/*
 * Dictionary preparation (App. E.2.1: the per-head transition dictionary is
 * shared by every step of a call, so its per-step tables are built once).
 * Builds, in ws, a byte copy of every map pi[h,k,:], per destination row the
 * list of its sources (the gather form of the column-one-hot map) and each
 * map's largest in-degree.  pdssm_scan_fwd and pdssm_scan_bwd always do this
 * themselves first, unless desc->flags has PDSSM_FLAG_PREPARED: then they use
 * the tables already in ws, which must come from pdssm_prepare with the same
 * desc (flags aside), the same ws and the current contents of pi, enqueued
 * before them on the same stream or ordered before them by the caller.
 * An entry of pi outside [0,N) is reported through *dev_status here.
 * ws: at least pdssm_workspace_size(desc, PDSSM_OP_FWD) bytes (the forward and
 * backward sizes are equal), 256-byte aligned, not overlapping pi.  When the
 * scans of desc run the chunked kernels (dictionaries too large for LDS) no
 * tables are needed and the call enqueues nothing.
 */
int pdssm_prepare(const pdssm_desc* desc, const int32_t* pi, void* ws, size_t ws_bytes,
                  int* dev_status, void* stream);

/*
 * Forward scan (App. E.1 Algorithm 1 / App. E.2 recurrence, readout of
 * Sec. 2.1 eq. (1) fused in).
 * In:  idx, pi, D, b, c (required); h0 (NULL = zero initial state).
 * Out: y (required); h_final = h_{L-1} (optional); saved (optional): the state
 *      entering every chunk, saved[b,h,c,:] = h_{c*chunk-1} (h0 for c = 0),
 *      which pdssm_scan_bwd needs (fp32 entries with PDSSM_FLAG_REAL_IO).
 */
int pdssm_scan_fwd(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                   const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                   const pdssm_c64* h0, float* y, pdssm_c64* h_final, pdssm_c64* saved,
                   void* ws, size_t ws_bytes, int* dev_status, void* stream);

/*
 * pdssm_scan_fwd for callers that cannot allocate device memory or pass a
 * workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments and results as pdssm_scan_fwd
 * without ws / ws_bytes; the workspace is a device array inside the library,
 * PDSSM_NOALLOC_SCRATCH_BYTES bytes per GPU, held from the first call on a
 * GPU until the process ends.  The call uses the array of the current device
 * (hipGetDevice); the stream must belong to that device.  It allocates and
 * frees nothing.
 *   - PDSSM_ERR_WORKSPACE when pdssm_workspace_size(desc, PDSSM_OP_FWD)
 *     exceeds the array (every workload of up to 256 dictionary entries of
 *     N = 128 per head, and segmented long sequences, fit).
 *   - PDSSM_ERR_INVALID_ARG with PDSSM_FLAG_PREPARED (the tables are built
 *     in the array by every call).
 * Every call on one GPU shares that GPU's array, which keeps the last
 * call's contents (each call rebuilds everything it reads there): calls that
 * overlap in time on one GPU (different streams, or host threads) race.
 */
#define PDSSM_NOALLOC_SCRATCH_BYTES (16u << 20)
int pdssm_scan_fwd_noalloc(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                           const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                           const pdssm_c64* h0, float* y, pdssm_c64* h_final, pdssm_c64* saved,
                           int* dev_status, void* stream);

/*
 * Backward scan: the vector-Jacobian product of pdssm_scan_fwd (the paper
 * leaves the adjoint of the scan unstated; this is the exact adjoint of the
 * forward above).  Per sequence, with g_t the gradient reaching h_t:
 *   g_t     = dy_t * conj(c_t) + (conj(D_{t+1}) * g_{t+1}[pi_{t+1}])
 *   dD_t[j] = conj(h_{t-1}[j]) * g_t[pi_t[j]],  db_t = g_t,
 *   dc_t    = dy_t * conj(h_t),  dh0[j] = conj(D_0[j]) * g_0[pi_0[j]],
 * starting from g_{L-1} = dy_{L-1} conj(c_{L-1}) + dh_final.
 * In:  idx, pi, D, b, c, saved (from pdssm_scan_fwd with the same desc and h0),
 *      dy (required); dh_final (NULL = zero).  h0 is not read: the states are
 *      recomputed from saved.
 * Out: dD, db, dc (required); dh0 (optional).
 */
int pdssm_scan_bwd(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                   const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                   const pdssm_c64* saved, const float* dy, const pdssm_c64* dh_final,
                   pdssm_c64* dD, pdssm_c64* db, pdssm_c64* dc, pdssm_c64* dh0,
                   void* ws, size_t ws_bytes, int* dev_status, void* stream);

/*
 * Backward scan for the straight-through surrogate gradients of the hard map
 * selection (Sec. 3.1 Prop. 2 and its derivation in the appendix).  Does
 * everything pdssm_scan_bwd does (same arguments, same results) and also
 * writes z [B,L,H,N] complex (required): z_t = D_t .* h_{t-1} (h_{-1} = h0),
 * the state entering the map of step t, which pdssm_ste_grads needs together
 * with db (the gradient g_t reaching h_t).  Same workspace as pdssm_scan_bwd
 * (PDSSM_OP_BWD).  z must not overlap any other argument.  With
 * PDSSM_FLAG_REAL_IO z is a real fp32 row like db; with PDSSM_FLAG_BF16_IO
 * it stays complex64 (unrounded) while dD, db, dc are bf16 pairs.
 */
int pdssm_scan_bwd_ste(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                       const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                       const pdssm_c64* saved, const float* dy, const pdssm_c64* dh_final,
                       pdssm_c64* dD, pdssm_c64* db, pdssm_c64* dc, pdssm_c64* dh0,
                       pdssm_c64* z, void* ws, size_t ws_bytes, int* dev_status, void* stream);

/*
 * The inputs of the two straight-through surrogate gradients (Sec. 3.1
 * Prop. 2), from g = db and z of pdssm_scan_bwd_ste.  With P_t the real
 * N x N matrix of step t (column j has its one in row pi_t[j]), the loss
 * gradient for P_t is dP_t[i][j] = Re(g_t[i] * conj(z_t[j])), and:
 *   q [B,L,H,K] float32 (optional): q[b,t,h,k] = <dP_t, P_k> =
 *       sum_j Re(g_t[pi[h,k,j]] * conj(z_t[j])), the gradient with respect to
 *       the weight of map k at step t when P_t = sum_k v_t[k] P_k, at the
 *       one-hot v_t of the forward.  pdssm_softmax_vjp over k with the
 *       routing logits turns it into their surrogate gradient.
 *   G [H,K,N,N] float32 (optional): G[h,k,i,j] = sum over the steps (b,t)
 *       with idx[b,t,h] == k of dP_t[i][j], the gradient of dictionary matrix
 *       P_k (row i = destination, column j = source).  pdssm_softmax_vjp down
 *       the columns of the dense dictionary M[h,k] turns it into its surrogate
 *       gradient.  Maps no step chose get zeros.
 * At least one of q, G.  The steps are grouped by map (a stable counting
 * sort) and every sum runs in a fixed order (deterministic results).
 * In:  idx [B,L,H], pi [H,K,N] (needed for q), g, z [B,L,H,N] complex64, or
 *      real fp32 with PDSSM_FLAG_REAL_IO (the real-valued model: Re(g conj z)
 *      is then g z), or with PDSSM_FLAG_BF16_IO g as bf16 (re, im) pairs
 *      (4 bytes per entry, widened exactly) and z complex64, as
 *      pdssm_scan_bwd_ste writes them; desc->chunk is ignored.
 * ws:  at least pdssm_workspace_size(desc, PDSSM_OP_STE_GRADS) bytes, 256-byte
 *      aligned.  An idx entry outside [0,K) counts as map 0 and is reported
 *      through *dev_status; a pi entry outside [0,N) reads row 0.
 */
int pdssm_ste_grads(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                    const pdssm_c64* g, const pdssm_c64* z, float* q, float* G, void* ws,
                    size_t ws_bytes, int* dev_status, void* stream);

/*
 * Selection front end (Sec. 3.1 eqs. (5)-(8), App. E.2.1).  Ties go to the
 * first maximal index.
 *
 * pdssm_dict_argmax: the maps of every dense dictionary matrix,
 *   pi[h,k,j] = argmax_i M[h,k,i,j] (the column argmax; once per step of the
 *   optimizer).  M [H,K,N,N] float32 (row i, column j), pi [H,K,N] int32.
 *   N in {8,...,256}, K <= 256.  Needs no workspace.
 *
 * pdssm_route: the routing scores and choices of every token,
 *   logits[t,h,k] = sum_d u[t,d] * S[h,k,d],  idx[t,h] = argmax_k logits[t,h,k],
 *   t = 0..T-1 (T = B*L; [T,H,K] is [B,L,H,K], [T,H] is [B,L,H]).
 *   u [T,Dm] and S [H,K,Dm] bf16 (row-major, 16-byte aligned, Dm a
 *   multiple of 8), logits [T,H,K] float32 (optional: the straight-through
 *   backward needs them, inference does not), idx [T,H] int32 (required).
 *   The product runs on the matrix cores with fp32 accumulation and the
 *   argmax is taken on the fp32 logits.  Needs no workspace.
 */
int pdssm_dict_argmax(int32_t H, int32_t K, int32_t N, const float* M, int32_t* pi, void* stream);
int pdssm_route(int32_t T, int32_t Dm, int32_t H, int32_t K, const uint16_t* u, const uint16_t* S,
                float* logits, int32_t* idx, void* stream);

/*
 * pdssm_project: everything a layer derives from its tokens u_t in one
 * product on the matrix cores (bf16 operands, fp32 accumulation), u read from
 * memory once:
 *   - the routing of pdssm_route (S non-NULL: logits optional, idx required);
 *   - b[t,h,n] = P_b[t,h,2n] + i P_b[t,h,2n+1], the input term b_t = B(u_t)
 *     u_t of the recurrence (App. E.2; Sec. 2.1 eq. (1)), and likewise
 *     c[t,h,n] from P_c, the readout vector C(u_t);
 *   - D[t,h,n] = sigmoid(P_d[t,h,2n]) * exp(i P_d[t,h,2n+1]), the diagonal
 *     generator D(u_t) (App. E.2.1 computes b and this generator as plain
 *     matrix products; the paper leaves its nonlinearity open: this one keeps
 *     |D| < 1 with a free phase),
 * where P_x[t,h,r] = sum_d u[t,d] W_x[h,r,d].  u [T,Dm] bf16; W_b, W_c, W_d
 * [H,2N,Dm] bf16 (rows 2n and 2n+1 of a head: real and imaginary part, or
 * magnitude logit and phase, of entry n); b, c, D [T,H,N] complex64 = the
 * scans' [B,L,H,N] layout with T = B*L.  Each of W_b, W_c, W_d and its
 * output is given or NULL together; at least one of S, W_b, W_c, W_d.
 * Dm a multiple of 32; N in {8,...,256}; K <= 256; u, S, W and the complex
 * outputs 16-byte aligned, logits and idx 4-byte aligned; row offsets of
 * (T + 256) rows of u and (H*2N + 256) rows of W below 2^32 bytes
 * (else PDSSM_ERR_UNSUPPORTED).  Needs no workspace.
 */
int pdssm_project(int32_t T, int32_t Dm, int32_t H, int32_t K, int32_t N, const uint16_t* u,
                  const uint16_t* S, const uint16_t* Wb, const uint16_t* Wc, const uint16_t* Wd, float* logits,
                  int32_t* idx, pdssm_c64* b, pdssm_c64* c, pdssm_c64* D, void* stream);

/*
 * Vector-Jacobian product of the tempered softmax that stands in for a hard
 * argmax in the backward pass (Sec. 3.1, slope-annealed straight-through
 * estimation; Prop. 2): along the middle axis of x [outer, len, inner]
 * (row-major), with s = softmax(x / temp),
 *   gx = s * (gy - sum(s * gy)) / temp.
 * Routing logits [B,L,H,K] with q: outer = B*L*H, len = K, inner = 1.
 * Dense dictionary M [H,K,N,N] with G: outer = H*K, len = N, inner = N (the
 * softmax runs down each column, where the argmax gives pi[h,k,j]).
 * x, gy, gx float32 device arrays; gx must not overlap x or gy; temp > 0;
 * outer*inner < 2^31 and outer*len*inner <= 2^40 (else PDSSM_ERR_UNSUPPORTED).
 * Needs no workspace.
 */
int pdssm_softmax_vjp(const float* x, const float* gy, float* gx, int64_t outer, int32_t len,
                      int64_t inner, float temp, void* stream);

/*
 * One step of the recurrence for every (batch, head) sequence: the
 * constant-memory recurrent form used for token-by-token inference (App. E.2
 * recurrence with the column-one-hot map of Sec. 3.1 eq. (5), readout of
 * Sec. 2.1 eq. (1)):
 *   h_out[r] = b[r] + sum_{j: pi_t[j] = r} D[j] * h_in[j],  pi_t = pi[h, idx[b,h], :],
 *   y = Re( sum_n c[n] * h_out[n] ).
 * Colliding sources add in ascending source order.  desc: B, H, N, K are
 * used (N and K as for the scans), L and chunk are ignored.
 * In:  idx [B,H] int32, pi [H,K,N] int32, D, b, c [B,H,N] complex,
 *      h_in [B,H,N] complex (NULL = zero state).
 * Out: h_out [B,H,N] complex (may be the same buffer as h_in: in-place
 *      update), y [B,H] float32.  Needs no workspace.
 * With PDSSM_FLAG_BF16_IO or PDSSM_FLAG_REAL_IO in desc->flags, D, b, c are
 * bf16 (re, im) pairs or real fp32 (4 bytes per entry) as for the scans;
 * h_in, h_out stay complex64 and the arithmetic is the same fp32 (the
 * results equal a complex64 call on the widened values bit for bit).
 */
int pdssm_decode_step(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                      const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                      const pdssm_c64* h_in, pdssm_c64* h_out, float* y, int* dev_status,
                      void* stream);

/*
 * Composed operator of every chunk in PD form (App. E.3.1 accumulator update,
 * App. E.2 associative operator): for chunk c of sequence (b,h),
 * A_{e-1} ... A_s with A_t = P_t D_t is returned as pi_out[b,h,c,:] (int32,
 * exact) and d_out[b,h,c,:] (complex), i.e. column j of the product holds
 * d_out[j] in row pi_out[j].  chunk >= L gives one whole-sequence map.
 * Needs no workspace.  Out: pi_out, d_out [B,H,C,N] (required).
 */
int pdssm_compose_chunks(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                         const pdssm_c64* D, int32_t* pi_out, pdssm_c64* d_out,
                         int* dev_status, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PDSSM_H */
