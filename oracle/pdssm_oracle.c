/*
 * pdssm_oracle.c -- CPU reference ("oracle") for the PD scan.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * definition that the GPU library is checked against.  Only the tests, the
 * smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product path never does.  It shares no code with the HIP library.
 *
 * Everything is plain sequential C in double precision (complex numbers are
 * interleaved (re, im) pairs of doubles).  One (batch, head) sequence is
 * independent of every other one.
 *
 * Definitions followed (paper: "Flash PD-SSM", arXiv 2605.19150):
 *
 *  - Recurrence, App. E.2 (the PD-SSM update x_t = P_t D_t x_{t-1} + b_t) with
 *    the column-one-hot reading of P_t (Sec. 2.3 eq. for column_hardmax,
 *    Sec. 3.1 eq. (5), App. D's construction A(sigma) = sum_q enc(delta(q,
 *    sigma)) enc(q)^T): column j of P_t has its single one in row pi_t(j), so
 *    source entry j of the state moves to entry pi_t(j), scaled by D_t[j]
 *    first; entries that land on the same row add up.
 *  - Map selection, Sec. 3.1 eqs. (5)-(8) and App. E.2.1: pi_t is row
 *    idx[b,t,h] of the per-head dictionary pi[h, :, :] (0-based indices).
 *  - Readout, Sec. 2.1 eq. (1) with psi = Re: y_t = Re( sum_n c_t[n] h_t[n] ),
 *    taken on the state after step t, no conjugation.
 *  - Composition of two PD operators, App. E.2 (associative operator) and
 *    App. E.3.1 (accumulator update): applying (pi1, d1) then (pi2, d2) gives
 *    (pi2[pi1[j]], d2[pi1[j]] * d1[j]).
 *  - Chunk boundaries, App. E.1 (Algorithm 1): chunk c covers steps
 *    [c*chunk, min((c+1)*chunk, L)); the last chunk may be partial.
 *  - Backward: the paper does not write out the adjoint of the scan; this is
 *    the vector-Jacobian product of the forward definition above, with the
 *    complex-gradient convention dX = dl/dRe(X) + i*dl/dIm(X) and the loss
 *    l = sum_t dy_t*y_t + Re(sum_n conj(dh_final[n]) * h_L[n]).
 *
 * Index errors (idx outside [0,K), pi outside [0,N)) make the functions
 * return -1 before touching any output.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define RE(p, i) ((p)[2 * (size_t)(i)])
#define IM(p, i) ((p)[2 * (size_t)(i) + 1])

static int check_indices(int B, int L, int H, int N, int K,
                         const int32_t* idx, const int32_t* pi)
{
    size_t nidx = (size_t)B * L * H, npi = (size_t)H * K * N;
    for (size_t i = 0; i < nidx; ++i)
        if (idx[i] < 0 || idx[i] >= K) return -1;
    for (size_t i = 0; i < npi; ++i)
        if (pi[i] < 0 || pi[i] >= N) return -1;
    return 0;
}

static int bad_dims(int B, int L, int H, int N, int K)
{
    return B < 1 || L < 1 || H < 1 || N < 1 || K < 1;
}

/* Offset of element [b, t, h, n] of a [B, L, H, N] tensor. */
static size_t at4(int L, int H, int N, int b, int t, int h, int n)
{
    return (((size_t)b * L + t) * H + h) * N + n;
}

/*
 * One step of the recurrence on a single sequence:
 *   hn[r] = bt[r] + sum over j with p[j] == r of Dt[j] * hp[j].
 */
static void pd_step(int N, const int32_t* p, const double* Dt, const double* bt,
                    const double* hp, double* hn)
{
    for (int r = 0; r < N; ++r) {
        RE(hn, r) = RE(bt, r);
        IM(hn, r) = IM(bt, r);
    }
    for (int j = 0; j < N; ++j) {
        double dr = RE(Dt, j), di = IM(Dt, j);
        double xr = RE(hp, j), xi = IM(hp, j);
        int r = p[j];
        RE(hn, r) += dr * xr - di * xi;
        IM(hn, r) += dr * xi + di * xr;
    }
}

/* Gather the N-vector of a [B,L,H,N] complex tensor at (b, t, h). */
static void load_vec(const double* src, int L, int H, int N, int b, int t, int h,
                     double* dst)
{
    memcpy(dst, src + 2 * at4(L, H, N, b, t, h, 0), sizeof(double) * 2 * N);
}

int pdssm_oracle_num_chunks(int L, int chunk)
{
    if (L < 1 || chunk < 1) return -1;
    return (L + chunk - 1) / chunk;
}

/*
 * Forward scan.
 *   idx [B,L,H] int32, pi [H,K,N] int32
 *   D, b, c [B,L,H,N] complex (interleaved doubles)
 *   h0 [B,H,N] complex or NULL (zero initial state)
 * Outputs (each may be NULL except y):
 *   y [B,L,H] double
 *   h_final [B,H,N] complex: state after the last step
 *   saved [B,H,C,N] complex: state entering chunk c, i.e. after step
 *         c*chunk - 1 (h0 for c = 0); only written when chunk > 0.
 */
int pdssm_oracle_fwd(int B, int L, int H, int N, int K,
                     const int32_t* idx, const int32_t* pi,
                     const double* D, const double* b, const double* c,
                     const double* h0, double* y, double* h_final,
                     int chunk, double* saved)
{
    if (bad_dims(B, L, H, N, K) || !idx || !pi || !D || !b || !c || !y) return -2;
    if (saved && chunk < 1) return -2;
    if (check_indices(B, L, H, N, K, idx, pi)) return -1;
    int C = saved ? pdssm_oracle_num_chunks(L, chunk) : 0;

    double* hp = malloc(sizeof(double) * 2 * N);
    double* hn = malloc(sizeof(double) * 2 * N);
    double* Dt = malloc(sizeof(double) * 2 * N);
    double* bt = malloc(sizeof(double) * 2 * N);
    if (!hp || !hn || !Dt || !bt) { free(hp); free(hn); free(Dt); free(bt); return -3; }

    for (int bb = 0; bb < B; ++bb) {
        for (int h = 0; h < H; ++h) {
            if (h0) memcpy(hp, h0 + 2 * (((size_t)bb * H + h) * N), sizeof(double) * 2 * N);
            else memset(hp, 0, sizeof(double) * 2 * N);
            for (int t = 0; t < L; ++t) {
                if (saved && t % chunk == 0) {
                    size_t o = (((size_t)bb * H + h) * C + t / chunk) * N;
                    memcpy(saved + 2 * o, hp, sizeof(double) * 2 * N);
                }
                const int32_t* p = pi + ((size_t)h * K + idx[((size_t)bb * L + t) * H + h]) * N;
                load_vec(D, L, H, N, bb, t, h, Dt);
                load_vec(b, L, H, N, bb, t, h, bt);
                pd_step(N, p, Dt, bt, hp, hn);
                /* readout on the new state */
                const double* ct = c + 2 * at4(L, H, N, bb, t, h, 0);
                double acc = 0.0;
                for (int n = 0; n < N; ++n)
                    acc += RE(ct, n) * RE(hn, n) - IM(ct, n) * IM(hn, n);
                y[((size_t)bb * L + t) * H + h] = acc;
                double* sw = hp; hp = hn; hn = sw;
            }
            if (h_final)
                memcpy(h_final + 2 * (((size_t)bb * H + h) * N), hp, sizeof(double) * 2 * N);
        }
    }
    free(hp); free(hn); free(Dt); free(bt);
    return 0;
}

/*
 * Backward scan: vector-Jacobian product of pdssm_oracle_fwd.
 *   dy [B,L,H] double, dh_final [B,H,N] complex or NULL (zero)
 * Outputs: dD, db, dc [B,L,H,N] complex; dh0 [B,H,N] complex or NULL.
 * The states h_t of one sequence are recomputed by the plain forward loop and
 * kept whole, then the adjoint runs backwards in time:
 *   g_t   = dy_t * conj(c_t) + (gradient arriving from step t+1)
 *   db_t  = g_t
 *   dc_t  = dy_t * conj(h_t)
 *   dD_t[j] = conj(h_{t-1}[j]) * g_t[pi_t(j)]
 *   (gradient into h_{t-1})[j] = conj(D_t[j]) * g_t[pi_t(j)]
 */
int pdssm_oracle_bwd(int B, int L, int H, int N, int K,
                     const int32_t* idx, const int32_t* pi,
                     const double* D, const double* b, const double* c,
                     const double* h0, const double* dy, const double* dh_final,
                     double* dD, double* db, double* dc, double* dh0)
{
    if (bad_dims(B, L, H, N, K) || !idx || !pi || !D || !b || !c || !dy ||
        !dD || !db || !dc) return -2;
    if (check_indices(B, L, H, N, K, idx, pi)) return -1;

    /* hs[t+1] = state after step t; hs[0] = initial state */
    double* hs = malloc(sizeof(double) * 2 * N * ((size_t)L + 1));
    double* Dt = malloc(sizeof(double) * 2 * N);
    double* bt = malloc(sizeof(double) * 2 * N);
    double* g = malloc(sizeof(double) * 2 * N);
    double* gp = malloc(sizeof(double) * 2 * N);
    if (!hs || !Dt || !bt || !g || !gp) {
        free(hs); free(Dt); free(bt); free(g); free(gp); return -3;
    }

    for (int bb = 0; bb < B; ++bb) {
        for (int h = 0; h < H; ++h) {
            size_t sh = ((size_t)bb * H + h) * N;
            if (h0) memcpy(hs, h0 + 2 * sh, sizeof(double) * 2 * N);
            else memset(hs, 0, sizeof(double) * 2 * N);
            for (int t = 0; t < L; ++t) {
                const int32_t* p = pi + ((size_t)h * K + idx[((size_t)bb * L + t) * H + h]) * N;
                load_vec(D, L, H, N, bb, t, h, Dt);
                load_vec(b, L, H, N, bb, t, h, bt);
                pd_step(N, p, Dt, bt, hs + 2 * (size_t)N * t, hs + 2 * (size_t)N * (t + 1));
            }

            if (dh_final) memcpy(g, dh_final + 2 * sh, sizeof(double) * 2 * N);
            else memset(g, 0, sizeof(double) * 2 * N);
            for (int t = L - 1; t >= 0; --t) {
                double dyt = dy[((size_t)bb * L + t) * H + h];
                const double* ct = c + 2 * at4(L, H, N, bb, t, h, 0);
                const double* ht = hs + 2 * (size_t)N * (t + 1);
                const double* hprev = hs + 2 * (size_t)N * t;
                double* dbt = db + 2 * at4(L, H, N, bb, t, h, 0);
                double* dct = dc + 2 * at4(L, H, N, bb, t, h, 0);
                double* dDt = dD + 2 * at4(L, H, N, bb, t, h, 0);
                for (int n = 0; n < N; ++n) {
                    /* readout term: dy * conj(c) */
                    RE(g, n) += dyt * RE(ct, n);
                    IM(g, n) -= dyt * IM(ct, n);
                    RE(dbt, n) = RE(g, n);
                    IM(dbt, n) = IM(g, n);
                    RE(dct, n) = dyt * RE(ht, n);
                    IM(dct, n) = -dyt * IM(ht, n);
                }
                const int32_t* p = pi + ((size_t)h * K + idx[((size_t)bb * L + t) * H + h]) * N;
                load_vec(D, L, H, N, bb, t, h, Dt);
                for (int j = 0; j < N; ++j) {
                    RE(gp, j) = RE(g, p[j]);
                    IM(gp, j) = IM(g, p[j]);
                }
                for (int j = 0; j < N; ++j) {
                    double gr = RE(gp, j), gi = IM(gp, j);
                    double xr = RE(hprev, j), xi = IM(hprev, j);
                    /* conj(h_{t-1}[j]) * g_t[p[j]] */
                    RE(dDt, j) = xr * gr + xi * gi;
                    IM(dDt, j) = xr * gi - xi * gr;
                    /* conj(D_t[j]) * g_t[p[j]] */
                    double dr = RE(Dt, j), di = IM(Dt, j);
                    RE(g, j) = dr * gr + di * gi;
                    IM(g, j) = dr * gi - di * gr;
                }
            }
            if (dh0) memcpy(dh0 + 2 * sh, g, sizeof(double) * 2 * N);
        }
    }
    free(hs); free(Dt); free(bt); free(g); free(gp);
    return 0;
}

/*
 * Composed map of every chunk: for chunk c of sequence (b, h), the product
 * A_{e-1} ... A_s (A_t = P_t D_t) in PD form (pi_out, d_out), folded from the
 * identity (pi = j, d = 1) one step at a time with the composition rule
 *   pi <- pi_t[pi],  d <- D_t[pi] * d   (D_t indexed by the old pi).
 * Outputs pi_out [B,H,C,N] int32 and d_out [B,H,C,N] complex.
 * chunk >= L gives one whole-sequence map per (b, h).
 */
int pdssm_oracle_compose(int B, int L, int H, int N, int K,
                         const int32_t* idx, const int32_t* pi, const double* D,
                         int chunk, int32_t* pi_out, double* d_out)
{
    if (bad_dims(B, L, H, N, K) || chunk < 1 || !idx || !pi || !D || !pi_out || !d_out)
        return -2;
    if (check_indices(B, L, H, N, K, idx, pi)) return -1;
    int C = pdssm_oracle_num_chunks(L, chunk);
    for (int bb = 0; bb < B; ++bb) {
        for (int h = 0; h < H; ++h) {
            for (int cc = 0; cc < C; ++cc) {
                size_t o = (((size_t)bb * H + h) * C + cc) * N;
                int32_t* pm = pi_out + o;
                double* dm = d_out + 2 * o;
                for (int j = 0; j < N; ++j) {
                    pm[j] = j;
                    RE(dm, j) = 1.0;
                    IM(dm, j) = 0.0;
                }
                int s = cc * chunk, e = s + chunk < L ? s + chunk : L;
                for (int t = s; t < e; ++t) {
                    const int32_t* p = pi + ((size_t)h * K + idx[((size_t)bb * L + t) * H + h]) * N;
                    const double* Dt = D + 2 * at4(L, H, N, bb, t, h, 0);
                    for (int j = 0; j < N; ++j) {
                        int q = pm[j];
                        double ar = RE(Dt, q), ai = IM(Dt, q);
                        double xr = RE(dm, j), xi = IM(dm, j);
                        RE(dm, j) = ar * xr - ai * xi;
                        IM(dm, j) = ar * xi + ai * xr;
                        pm[j] = p[q];
                    }
                }
            }
        }
    }
    return 0;
}

/*
 * Straight-through surrogate gradients of the hard map selection (Sec. 3.1,
 * Prop. 2 "Surrogate Gradients", derived in the appendix section on the
 * surrogate gradient expressions).  The selected matrix P_t is a real N x N
 * matrix in the dense view, with the state scaled before the map:
 *     h_t = P_t z_t + b_t,   z_t = D_t .* h_{t-1}.
 * The loss is linear in each single P_t, and its gradient with respect to the
 * real entries of P_t is, under the convention dX = dl/dRe(X) + i dl/dIm(X),
 *     dP_t[i][j] = Re( g_t[i] * conj(z_t[j]) ),
 * where g_t is the gradient reaching h_t (db_t of the backward).  Two
 * quantities follow:
 *   - the score of every candidate map k at every step (the gradient of the
 *     loss with respect to the weight of map k in P_t = sum_k v_t[k] P_k,
 *     taken at the one-hot v_t of the forward pass):
 *         q[b,t,h,k] = <dP_t, P_k>_F = sum_j Re( g_t[pi[h,k,j]] * conj(z_t[j]) );
 *   - the gradient of every dictionary matrix, summed over the steps that
 *     selected it:
 *         G[h,k,i,j] = sum over (b,t) with idx[b,t,h] == k of dP_t[i][j].
 * Both are the inputs of the tempered-softmax Jacobians of Prop. 2.
 * q [B,L,H,K] double (may be NULL), G [H,K,N,N] double (may be NULL),
 * zout [B,L,H,N] complex (may be NULL): z_t of every step.
 */
int pdssm_oracle_ste(int B, int L, int H, int N, int K,
                     const int32_t* idx, const int32_t* pi,
                     const double* D, const double* b, const double* c,
                     const double* h0, const double* dy, const double* dh_final,
                     double* q, double* G, double* zout)
{
    if (bad_dims(B, L, H, N, K) || !idx || !pi || !D || !b || !c || !dy) return -2;
    if (check_indices(B, L, H, N, K, idx, pi)) return -1;

    double* hs = malloc(sizeof(double) * 2 * N * ((size_t)L + 1));
    double* Dt = malloc(sizeof(double) * 2 * N);
    double* bt = malloc(sizeof(double) * 2 * N);
    double* g = malloc(sizeof(double) * 2 * N);
    double* gn = malloc(sizeof(double) * 2 * N);
    double* z = malloc(sizeof(double) * 2 * N);
    if (!hs || !Dt || !bt || !g || !gn || !z) {
        free(hs); free(Dt); free(bt); free(g); free(gn); free(z); return -3;
    }
    if (G) memset(G, 0, sizeof(double) * (size_t)H * K * N * N);

    for (int bb = 0; bb < B; ++bb) {
        for (int h = 0; h < H; ++h) {
            size_t sh = ((size_t)bb * H + h) * N;
            /* states of the whole sequence: hs[t+1] = h_t, hs[0] = initial state */
            if (h0) memcpy(hs, h0 + 2 * sh, sizeof(double) * 2 * N);
            else memset(hs, 0, sizeof(double) * 2 * N);
            for (int t = 0; t < L; ++t) {
                const int32_t* p = pi + ((size_t)h * K + idx[((size_t)bb * L + t) * H + h]) * N;
                load_vec(D, L, H, N, bb, t, h, Dt);
                load_vec(b, L, H, N, bb, t, h, bt);
                pd_step(N, p, Dt, bt, hs + 2 * (size_t)N * t, hs + 2 * (size_t)N * (t + 1));
            }

            if (dh_final) memcpy(g, dh_final + 2 * sh, sizeof(double) * 2 * N);
            else memset(g, 0, sizeof(double) * 2 * N);
            for (int t = L - 1; t >= 0; --t) {
                double dyt = dy[((size_t)bb * L + t) * H + h];
                const double* ct = c + 2 * at4(L, H, N, bb, t, h, 0);
                for (int n = 0; n < N; ++n) { /* g_t: add the readout term dy_t conj(c_t) */
                    RE(g, n) += dyt * RE(ct, n);
                    IM(g, n) -= dyt * IM(ct, n);
                }
                int kt = idx[((size_t)bb * L + t) * H + h];
                load_vec(D, L, H, N, bb, t, h, Dt);
                const double* hprev = hs + 2 * (size_t)N * t;
                for (int j = 0; j < N; ++j) { /* z_t = D_t .* h_{t-1} */
                    RE(z, j) = RE(Dt, j) * RE(hprev, j) - IM(Dt, j) * IM(hprev, j);
                    IM(z, j) = RE(Dt, j) * IM(hprev, j) + IM(Dt, j) * RE(hprev, j);
                }
                if (zout) memcpy(zout + 2 * at4(L, H, N, bb, t, h, 0), z, sizeof(double) * 2 * N);
                if (q) {
                    double* qt = q + ((size_t)bb * L + t) * H * K + (size_t)h * K;
                    for (int k = 0; k < K; ++k) {
                        const int32_t* pk = pi + ((size_t)h * K + k) * N;
                        double acc = 0.0;
                        for (int j = 0; j < N; ++j) /* Re(g[pk[j]] * conj(z[j])) */
                            acc += RE(g, pk[j]) * RE(z, j) + IM(g, pk[j]) * IM(z, j);
                        qt[k] = acc;
                    }
                }
                if (G) {
                    double* Gk = G + ((size_t)h * K + kt) * N * N;
                    for (int i = 0; i < N; ++i)
                        for (int j = 0; j < N; ++j)
                            Gk[(size_t)i * N + j] += RE(g, i) * RE(z, j) + IM(g, i) * IM(z, j);
                }
                /* gradient reaching h_{t-1}: conj(D_t[j]) * g_t[pi_t(j)] */
                const int32_t* p = pi + ((size_t)h * K + kt) * N;
                for (int j = 0; j < N; ++j) {
                    double gr = RE(g, p[j]), gi = IM(g, p[j]);
                    double dr = RE(Dt, j), di = IM(Dt, j);
                    RE(gn, j) = dr * gr + di * gi;
                    IM(gn, j) = dr * gi - di * gr;
                }
                double* sw = g; g = gn; gn = sw;
            }
        }
    }
    free(hs); free(Dt); free(bt); free(g); free(gn); free(z);
    return 0;
}
