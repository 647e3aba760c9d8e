"""Seeded synthetic inputs for the PD scan.

This module only draws random numbers; it holds none of the scan's arithmetic.
Both the float64 oracle and the GPU library consume exactly the arrays made
here (the GPU side after a host-to-device copy), so the two never disagree on
inputs.

Layouts (row-major, the library's ABI layouts):
  idx [B,L,H] int32 in [0,K)      per-step dictionary index k_t
  pi  [H,K,N] int32 in [0,N)      per-head dictionary of column-one-hot maps
  D, b, c [B,L,H,N] complex64     diagonal, input term, readout vector
  dy  [B,L,H] float32             upstream gradient of y
  h0, dh_final [B,H,N] complex64  optional initial state / final-state gradient

Draw order for one config: idx, pi, |D|, arg D, b, c, dy, then h0 and
dh_final when asked for.  "Complex normal with variance s2" means real and
imaginary parts are independent N(0, s2/2), so E|z|^2 = s2.

The five named workloads follow the scan's uses in the paper: a tiny
fixed-point case, the state-tracking shape of Fig. 1 (L=2048, hidden 1024 as
16 heads of 64), the long multivariate time-series shape of the UEA tasks
(L=18000), and a hybrid language-model layer (32 heads of 128, L=4096).  The
paper's datasets are not used; these synthetic draws stand in for them.
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    L: int
    H: int
    N: int
    K: int
    pi_kind: str = "uniform"      # "uniform" (many-to-one allowed) | "perm" | "identity"
    dmag: tuple = (0.5, 0.99)     # (lo, hi) uniform magnitude, or ("sigmoid", mu, sd)
    bc_var: float = 1.0           # variance of the complex normal b and c
    idx_kind: str = "uniform"     # "uniform" | "markov"
    fwd_only: bool = False
    note: str = field(default="", compare=False)

    @property
    def state_updates(self):
        return self.B * self.L * self.H * self.N


WORKLOADS = {
    1: Workload("tiny-fwd B1 L64 H1 N8 K4", 1, 64, 1, 8, 4, "uniform", (0.5, 0.99), 1.0,
                "uniform", fwd_only=True),
    2: Workload("fsa-perm B16 L2048 H16 N64 K16", 16, 2048, 16, 64, 16, "perm", (0.9, 1.0),
                1.0 / 64, "uniform"),
    3: Workload("markov-manyone B16 L2048 H16 N64 K16", 16, 2048, 16, 64, 16, "uniform",
                (0.5, 0.999), 1.0 / 64, "markov"),
    4: Workload("timeseries B8 L18000 H8 N128 K32", 8, 18000, 8, 128, 32, "uniform",
                (0.95, 0.9999), 1.0 / 128, "uniform"),
    5: Workload("hybrid-lm B8 L4096 H32 N128 K64", 8, 4096, 32, 128, 64, "uniform",
                ("sigmoid", 2.0, 1.0), 1.0 / 128, "uniform"),
}


def _cnormal(rng, shape, var):
    s = np.float32(np.sqrt(var / 2.0))
    out = np.empty(shape, np.complex64)
    out.real = rng.standard_normal(shape, dtype=np.float32) * s
    out.imag = rng.standard_normal(shape, dtype=np.float32) * s
    return out


def _markov_idx(rng, B, L, H, K):
    """Per head a random row-stochastic K x K transition table softmax(2 g);
    per (b, h) a chain idx_0 ~ U[0,K), idx_{t+1} ~ Cat(T_h[idx_t]) drawn by
    inverse CDF."""
    g = rng.standard_normal((H, K, K))
    w = np.exp(2.0 * g - (2.0 * g).max(axis=2, keepdims=True))
    T = w / w.sum(axis=2, keepdims=True)
    cdf = np.cumsum(T, axis=2)
    cdf[:, :, -1] = 1.0
    u = rng.random((B, L, H))
    idx = np.empty((B, L, H), np.int32)
    cur = rng.integers(0, K, size=(B, H))
    hh = np.arange(H)[None, :]
    idx[:, 0, :] = cur
    for t in range(1, L):
        rows = cdf[hh, cur]                                   # [B,H,K]
        cur = np.minimum((rows < u[:, t, :, None]).sum(axis=2), K - 1)
        idx[:, t, :] = cur
    return idx


def _rnormal_c(rng, shape, var):
    """Real normal values of variance var, as complex64 with imaginary part 0."""
    out = np.zeros(shape, np.complex64)
    out.real = rng.standard_normal(shape, dtype=np.float32) * np.float32(np.sqrt(var))
    return out


def make_inputs(B, L, H, N, K, seed=0, pi_kind="uniform", dmag=(0.5, 0.99), bc_var=1.0,
                idx_kind="uniform", with_h0=False, with_dhf=False, dy=True, real=False):
    """Draw one input set.  Returns a dict of numpy arrays.

    real: the real-valued model's inputs: D = magnitude * random sign (the
    real counterpart of the uniform phase), b and c real normal of variance
    bc_var, all float32; h0 and dh_final real normal values held as complex64
    with imaginary part 0."""
    rng = np.random.default_rng(seed)
    if idx_kind == "uniform":
        idx = rng.integers(0, K, size=(B, L, H), dtype=np.int32)
    elif idx_kind == "markov":
        idx = _markov_idx(rng, B, L, H, K)
    else:
        raise ValueError(idx_kind)
    if pi_kind == "uniform":
        pi = rng.integers(0, N, size=(H, K, N), dtype=np.int32)
    elif pi_kind == "perm":
        pi = np.stack([np.stack([rng.permutation(N) for _ in range(K)]) for _ in range(H)])
        pi = pi.astype(np.int32)
    elif pi_kind == "identity":
        pi = np.broadcast_to(np.arange(N, dtype=np.int32), (H, K, N)).copy()
    else:
        raise ValueError(pi_kind)
    shape = (B, L, H, N)
    if dmag[0] == "sigmoid":
        z = rng.standard_normal(shape, dtype=np.float32) * np.float32(dmag[2]) + np.float32(dmag[1])
        mag = 1.0 / (1.0 + np.exp(-z))
    else:
        lo, hi = dmag
        mag = rng.random(shape, dtype=np.float32) * np.float32(hi - lo) + np.float32(lo)
    if real:
        sign = np.where(rng.random(shape, dtype=np.float32) < 0.5, np.float32(-1.0), np.float32(1.0))
        D = (mag * sign).astype(np.float32)
        del mag, sign
        sd = np.float32(np.sqrt(bc_var))
        b = rng.standard_normal(shape, dtype=np.float32) * sd
        c = rng.standard_normal(shape, dtype=np.float32) * sd
        state = _rnormal_c
    else:
        phase = rng.random(shape, dtype=np.float32) * np.float32(2.0 * np.pi)
        D = np.empty(shape, np.complex64)
        D.real = mag * np.cos(phase)
        D.imag = mag * np.sin(phase)
        del mag, phase
        b = _cnormal(rng, shape, bc_var)
        c = _cnormal(rng, shape, bc_var)
        state = _cnormal
    out = dict(idx=idx, pi=pi, D=D, b=b, c=c)
    if dy:
        out["dy"] = rng.standard_normal((B, L, H), dtype=np.float32)
    if with_h0:
        out["h0"] = state(rng, (B, H, N), 1.0)
    if with_dhf:
        out["dh_final"] = state(rng, (B, H, N), 1.0)
    return out


def workload_inputs(i, seed=0, **kw):
    """Inputs of named workload i (1..5)."""
    w = WORKLOADS[i]
    return make_inputs(w.B, w.L, w.H, w.N, w.K, seed=seed, pi_kind=w.pi_kind, dmag=w.dmag,
                       bc_var=w.bc_var, idx_kind=w.idx_kind, **kw)


def fsa_inputs(B, L, H, N, K, seed=0, perm=False, n_accept=None):
    """Finite-automaton embedding (paper App. D): every D is exactly 1, every b
    is 0, h0 is a one-hot start state and c is the 0/1 indicator of a random
    accepting set.  Transition tables are random maps (permutations if perm)."""
    rng = np.random.default_rng(seed)
    idx = rng.integers(0, K, size=(B, L, H), dtype=np.int32)
    if perm:
        pi = np.stack([np.stack([rng.permutation(N) for _ in range(K)]) for _ in range(H)])
    else:
        pi = rng.integers(0, N, size=(H, K, N))
    pi = pi.astype(np.int32)
    start = rng.integers(0, N, size=(B, H))
    h0 = np.zeros((B, H, N), np.complex64)
    for bb in range(B):
        for hh in range(H):
            h0[bb, hh, start[bb, hh]] = 1.0
    if n_accept is None:
        n_accept = max(1, N // 3)
    acc = np.zeros((H, N), np.float32)
    for hh in range(H):
        acc[hh, rng.choice(N, size=n_accept, replace=False)] = 1.0
    shape = (B, L, H, N)
    D = np.ones(shape, np.complex64)
    b = np.zeros(shape, np.complex64)
    c = np.broadcast_to(acc[None, None, :, :], shape).astype(np.complex64)
    dy = rng.standard_normal((B, L, H), dtype=np.float32)
    return dict(idx=idx, pi=pi, D=D, b=b, c=c, h0=h0, dy=dy, start=start, accept=acc)


def sub_sequence(inp, bb, hh):
    """Inputs of the single sequence (bb, hh) as a B=1, H=1 problem."""
    out = {}
    for k in ("D", "b", "c"):
        out[k] = np.ascontiguousarray(inp[k][bb:bb + 1, :, hh:hh + 1])
    out["idx"] = np.ascontiguousarray(inp["idx"][bb:bb + 1, :, hh:hh + 1])
    out["pi"] = np.ascontiguousarray(inp["pi"][hh:hh + 1])
    if "dy" in inp:
        out["dy"] = np.ascontiguousarray(inp["dy"][bb:bb + 1, :, hh:hh + 1])
    for k in ("h0", "dh_final"):
        if inp.get(k) is not None:
            out[k] = np.ascontiguousarray(inp[k][bb:bb + 1, hh:hh + 1])
    return out


def selection_inputs(idx, pi, seed=0, margin=(0.1, 1.0)):
    """Dense scores behind the hard selections, for the surrogate gradients:
    routing logits [B,L,H,K] float32 whose largest entry at (b,t,h) is
    idx[b,t,h], and a dense dictionary M [H,K,N,N] float32 whose largest entry
    in column j of M[h,k] is row pi[h,k,j].  Entries are N(0,1); the selected
    one is then raised to the column's (row's) maximum plus U(margin)."""
    rng = np.random.default_rng(seed)
    B, L, H = idx.shape
    _, K, N = pi.shape
    logits = rng.standard_normal((B, L, H, K), dtype=np.float32)
    bump = rng.uniform(margin[0], margin[1], size=(B, L, H)).astype(np.float32)
    sel = np.take_along_axis(logits, idx[..., None].astype(np.int64), axis=3)[..., 0]
    top = logits.max(axis=3)
    np.put_along_axis(logits, idx[..., None].astype(np.int64),
                      np.maximum(top, sel)[..., None] + bump[..., None], axis=3)
    M = rng.standard_normal((H, K, N, N), dtype=np.float32)
    bump = rng.uniform(margin[0], margin[1], size=(H, K, N)).astype(np.float32)
    top = M.max(axis=2)                                      # [H,K,N] over rows
    rows = pi[:, :, None, :].astype(np.int64)                # [H,K,1,N]
    np.put_along_axis(M, rows, (top + bump)[:, :, None, :], axis=2)
    return logits, M
