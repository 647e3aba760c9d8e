"""numpy <-> C marshalling for the float64 oracle (test infrastructure only).

Every function takes numpy arrays in the library's layouts:
  idx [B,L,H] int, pi [H,K,N] int, D/b/c [B,L,H,N] complex, h0 [B,H,N]
complex or None, dy [B,L,H] real, dh_final [B,H,N] complex or None.
Inputs are promoted to float64 / complex128 (exact for float32 inputs) and
the results come back as float64 / complex128 arrays.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pdssm_oracle.c")
_LIB = os.path.join(_HERE, "libpdssm_oracle.so")
_lib = None


def oracle_lib_path():
    return _LIB


def build_oracle(force=True):
    """Compile the oracle with gcc (-O2, plain C11).  Returns the .so path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Werror",
             "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build_oracle(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.pdssm_oracle_fwd.argtypes = [I, I, I, I, I, P, P, P, P, P, P, P, P, I, P]
        lib.pdssm_oracle_bwd.argtypes = [I, I, I, I, I, P, P, P, P, P, P, P, P, P, P, P, P]
        lib.pdssm_oracle_compose.argtypes = [I, I, I, I, I, P, P, P, I, P, P]
        lib.pdssm_oracle_num_chunks.argtypes = [I, I]
        lib.pdssm_oracle_ste.argtypes = [I, I, I, I, I, P, P, P, P, P, P, P, P, P, P, P]
        for f in (lib.pdssm_oracle_fwd, lib.pdssm_oracle_bwd, lib.pdssm_oracle_compose,
                  lib.pdssm_oracle_num_chunks, lib.pdssm_oracle_ste):
            f.restype = I
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _cplx(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.complex128)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _dims(idx, pi, D):
    B, L, H = idx.shape
    H2, K, N = pi.shape
    assert H2 == H and D.shape == (B, L, H, N), (idx.shape, pi.shape, D.shape)
    return B, L, H, N, K


def _check(rc, what):
    if rc == -1:
        raise IndexError("%s: idx or pi out of range" % what)
    if rc != 0:
        raise ValueError("%s: oracle returned %d" % (what, rc))


def oracle_num_chunks(L, chunk):
    return _load().pdssm_oracle_num_chunks(int(L), int(chunk))


def oracle_fwd(idx, pi, D, b, c, h0=None, chunk=0):
    """Returns (y [B,L,H] f64, h_final [B,H,N] c128, saved [B,H,C,N] c128 or None)."""
    idx, pi = _i32(idx), _i32(pi)
    D, b, c, h0 = _cplx(D), _cplx(b), _cplx(c), _cplx(h0)
    B, L, H, N, K = _dims(idx, pi, D)
    y = np.empty((B, L, H), np.float64)
    hf = np.empty((B, H, N), np.complex128)
    saved = None
    if chunk > 0:
        C = oracle_num_chunks(L, chunk)
        saved = np.empty((B, H, C, N), np.complex128)
    rc = _load().pdssm_oracle_fwd(B, L, H, N, K, _ptr(idx), _ptr(pi), _ptr(D), _ptr(b),
                                  _ptr(c), _ptr(h0), _ptr(y), _ptr(hf), int(chunk),
                                  _ptr(saved))
    _check(rc, "oracle_fwd")
    return y, hf, saved


def oracle_bwd(idx, pi, D, b, c, dy, h0=None, dh_final=None):
    """Returns (dD, db, dc [B,L,H,N] c128, dh0 [B,H,N] c128)."""
    idx, pi = _i32(idx), _i32(pi)
    D, b, c, h0, dhf = _cplx(D), _cplx(b), _cplx(c), _cplx(h0), _cplx(dh_final)
    dy = np.ascontiguousarray(dy, dtype=np.float64)
    B, L, H, N, K = _dims(idx, pi, D)
    assert dy.shape == (B, L, H)
    dD = np.empty((B, L, H, N), np.complex128)
    db = np.empty_like(dD)
    dc = np.empty_like(dD)
    dh0 = np.empty((B, H, N), np.complex128)
    rc = _load().pdssm_oracle_bwd(B, L, H, N, K, _ptr(idx), _ptr(pi), _ptr(D), _ptr(b),
                                  _ptr(c), _ptr(h0), _ptr(dy), _ptr(dhf), _ptr(dD),
                                  _ptr(db), _ptr(dc), _ptr(dh0))
    _check(rc, "oracle_bwd")
    return dD, db, dc, dh0


def oracle_compose(idx, pi, D, chunk):
    """Returns (pi_out [B,H,C,N] int32, d_out [B,H,C,N] c128) per chunk."""
    idx, pi, D = _i32(idx), _i32(pi), _cplx(D)
    B, L, H, N, K = _dims(idx, pi, D)
    C = oracle_num_chunks(L, chunk)
    if C < 1:
        raise ValueError("bad chunk")
    pm = np.empty((B, H, C, N), np.int32)
    dm = np.empty((B, H, C, N), np.complex128)
    rc = _load().pdssm_oracle_compose(B, L, H, N, K, _ptr(idx), _ptr(pi), _ptr(D),
                                      int(chunk), _ptr(pm), _ptr(dm))
    _check(rc, "oracle_compose")
    return pm, dm


def oracle_ste(idx, pi, D, b, c, dy, h0=None, dh_final=None, want_z=False):
    """Straight-through surrogate inputs (Sec. 3.1 Prop. 2 and its appendix
    derivation): q [B,L,H,K] f64, the score of every candidate map at every
    step, and G [H,K,N,N] f64, the gradient of every dictionary matrix summed
    over the steps that selected it (rows = destination i, columns = source
    j, as in the dense P_k whose column j has its one in row pi[h,k,j]).
    With want_z, also z [B,L,H,N] c128: z_t = D_t .* h_{t-1} of every step."""
    idx, pi = _i32(idx), _i32(pi)
    D, b, c, h0, dhf = _cplx(D), _cplx(b), _cplx(c), _cplx(h0), _cplx(dh_final)
    dy = np.ascontiguousarray(dy, dtype=np.float64)
    B, L, H, N, K = _dims(idx, pi, D)
    assert dy.shape == (B, L, H)
    q = np.empty((B, L, H, K), np.float64)
    G = np.empty((H, K, N, N), np.float64)
    z = np.empty((B, L, H, N), np.complex128) if want_z else None
    rc = _load().pdssm_oracle_ste(B, L, H, N, K, _ptr(idx), _ptr(pi), _ptr(D), _ptr(b),
                                  _ptr(c), _ptr(h0), _ptr(dy), _ptr(dhf), _ptr(q), _ptr(G), _ptr(z))
    _check(rc, "oracle_ste")
    return (q, G, z) if want_z else (q, G)


def oracle_softmax_vjp(x, gy, axis, temp):
    """Vector-Jacobian product of the tempered softmax s = softmax(x / temp)
    along `axis` (the backward stand-in for a hard argmax in Prop. 2):
    gx = s * (gy - sum(s * gy)) / temp, in float64."""
    x = np.asarray(x, np.float64) / float(temp)
    gy = np.asarray(gy, np.float64)
    e = np.exp(x - x.max(axis=axis, keepdims=True))
    s = e / e.sum(axis=axis, keepdims=True)
    return s * (gy - (s * gy).sum(axis=axis, keepdims=True)) / float(temp)


def oracle_surrogate_grads(q, G, logits, M, temp):
    """The two surrogate gradients of Prop. 2 from the oracle_ste outputs:
    d logits [B,L,H,K] (routing scores k(u_t), softmax over k) and
    dM [H,K,N,N] (dense dictionary, softmax over the rows i of every
    column j, the argmax that gives pi[h,k,j])."""
    return oracle_softmax_vjp(logits, q, -1, temp), oracle_softmax_vjp(M, G, 2, temp)


def oracle_dict_argmax(M):
    """Maps of the dense dictionary (Sec. 3.1 eq. (5), App. E.2.1):
    pi[h,k,j] = argmax_i M[h,k,i,j], ties to the first maximal index."""
    M = np.asarray(M, np.float64)
    return np.argmax(M, axis=2).astype(np.int32)


def oracle_route(u, S):
    """Routing scores and choices (Sec. 3.1 eqs. (6)-(7)): u [B,L,Dm],
    S [H,K,Dm] (their exact values, e.g. widened bf16) -> logits [B,L,H,K]
    float64 = sum_d u[b,t,d] S[h,k,d], idx [B,L,H] = first argmax over k."""
    u = np.asarray(u, np.float64)
    S = np.asarray(S, np.float64)
    logits = np.einsum("bld,hkd->blhk", u, S)
    return logits, np.argmax(logits, axis=3).astype(np.int32)


def oracle_project(u, S=None, Wb=None, Wc=None, Wd=None):
    """The per-token projections of one layer, in float64 on the exact input
    values (e.g. widened bf16).  u [B,L,Dm]; per-head weights [H,2N,Dm] whose
    rows 2n and 2n+1 give the real and imaginary part of entry n:
      - b[b,t,h,n] = sum_d u W_b[h,2n,d] + i sum_d u W_b[h,2n+1,d], the input
        term b_t = B(u_t) u_t of the recurrence (App. E.2; Sec. 2.1 eq. (1));
      - c[b,t,h,n] likewise from W_c, the readout vector C(u_t);
      - D[b,t,h,n] = sigmoid(a) * exp(i theta), a = sum_d u W_d[h,2n,d],
        theta = sum_d u W_d[h,2n+1,d]: the diagonal generator D(u_t) (App.
        E.2.1 computes b and this generator as plain matrix products; the
        paper leaves the nonlinearity open: a magnitude in (0, 1) and a free
        phase);
      - with S [H,K,Dm]: the routing logits and choices of oracle_route.
    Returns a dict with the keys of the weights given (logits and idx for S)."""
    u = np.asarray(u, np.float64)
    out = {}
    if S is not None:
        out["logits"], out["idx"] = oracle_route(u, S)

    def proj(W):
        P = np.einsum("bld,hrd->blhr", u, np.asarray(W, np.float64))  # [B,L,H,2N]
        return P[..., 0::2], P[..., 1::2]

    if Wb is not None:
        re, im = proj(Wb)
        out["b"] = re + 1j * im
    if Wc is not None:
        re, im = proj(Wc)
        out["c"] = re + 1j * im
    if Wd is not None:
        a, theta = proj(Wd)
        out["D"] = (1.0 / (1.0 + np.exp(-a))) * np.exp(1j * theta)
    return out
