"""Pins for the float64 oracle (CPU only).

Each test checks the oracle against something other than itself: a value
worked out by hand, a dense-matrix brute force, torch.autograd and central
finite differences, closed forms (diagonal maps, automaton simulation),
linearity/adjoint identities, split invariance and norm preservation.  A
dropped term, a flipped conjugate, a gather written instead of a scatter or a
transposed composition each fail at least one of them.
"""
import json
import os

import numpy as np
import pytest

from oracle import oracle_bwd, oracle_compose, oracle_fwd
from paper_2605_19150_amd.inputs import fsa_inputs, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _c(a):
    a = np.asarray(a, dtype=np.float64)
    return a[..., 0] + 1j * a[..., 1]


# ---------------------------------------------------------------- dense brute force
def dense_A(p, Dt):
    """Dense N x N matrix of a column-one-hot PD operator: column j holds Dt[j]
    in row p[j] (paper Sec. 2.3: one nonzero per column)."""
    N = len(p)
    A = np.zeros((N, N), np.complex128)
    for j in range(N):
        A[p[j], j] += Dt[j]
    return A


def dense_fwd(inp):
    idx, pi, D, b, c = inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"]
    B, L, H = idx.shape
    N = pi.shape[2]
    h0 = inp.get("h0")
    y = np.zeros((B, L, H))
    hf = np.zeros((B, H, N), np.complex128)
    states = np.zeros((B, L, H, N), np.complex128)
    for bb in range(B):
        for h in range(H):
            x = np.zeros(N, np.complex128) if h0 is None else h0[bb, h].astype(np.complex128)
            for t in range(L):
                A = dense_A(pi[h, idx[bb, t, h]], D[bb, t, h].astype(np.complex128))
                x = A @ x + b[bb, t, h]
                states[bb, t, h] = x
                y[bb, t, h] = (c[bb, t, h].astype(np.complex128) @ x).real
            hf[bb, h] = x
    return y, hf, states


def small(seed, B=2, L=13, H=2, N=5, K=3, **kw):
    return make_inputs(B, L, H, N, K, seed=seed, **kw)


# ---------------------------------------------------------------- P0: hand example
def test_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "hand_example_n3.json")))
    idx = np.array(g["idx"], np.int32)
    pi = np.array(g["pi"], np.int32)
    D, b, c, h0 = _c(g["D"]), _c(g["b"]), _c(g["c"]), _c(g["h0"])
    dy = np.array(g["dy"], np.float64)
    assert D.shape == (1, 3, 1, 3) and h0.shape == (1, 1, 3)
    e = g["expected"]
    y, hf, saved = oracle_fwd(idx, pi, D, b, c, h0=h0, chunk=2)
    np.testing.assert_array_equal(y, np.array(e["y"], np.float64))
    np.testing.assert_array_equal(hf, _c(e["h_final"]))
    np.testing.assert_array_equal(saved, _c(e["chunk2_saved"]))
    pm, dm = oracle_compose(idx, pi, D, chunk=2)
    np.testing.assert_array_equal(pm, np.array(e["chunk2_pi"], np.int32))
    np.testing.assert_array_equal(dm, _c(e["chunk2_d"]))
    dD, db, dc, dh0 = oracle_bwd(idx, pi, D, b, c, dy, h0=h0)
    np.testing.assert_array_equal(dD, _c(e["dD"]))
    np.testing.assert_array_equal(db, _c(e["db"]))
    np.testing.assert_array_equal(dc, _c(e["dc"]))
    np.testing.assert_array_equal(dh0, _c(e["dh0"]))


# ---------------------------------------------------------------- P1: brute force
@pytest.mark.parametrize("seed,pi_kind", [(0, "uniform"), (1, "perm"), (2, "uniform")])
def test_fwd_matches_dense(seed, pi_kind):
    inp = small(seed, pi_kind=pi_kind, with_h0=True)
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    y2, hf2, _ = dense_fwd(inp)
    np.testing.assert_allclose(y, y2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(hf, hf2, rtol=1e-12, atol=1e-12)


def test_fwd_zero_h0_is_none():
    inp = small(3)
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"])
    z = np.zeros((2, 2, 5), np.complex64)
    y2, hf2, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=z)
    np.testing.assert_array_equal(y, y2)
    np.testing.assert_array_equal(hf, hf2)


def test_bwd_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    inp = small(4, B=1, L=9, H=2, N=6, K=3, with_h0=True, with_dhf=True)
    idx, pi = inp["idx"], inp["pi"]
    B, L, H = idx.shape
    N = pi.shape[2]
    # torch's complex gradient convention is dl/dRe + i dl/dIm: grad of Re(a z) is conj(a)
    z = torch.tensor(0.3 + 0.7j, dtype=torch.complex128, requires_grad=True)
    a = torch.tensor(1.5 - 2.0j, dtype=torch.complex128)
    (a * z).real.backward()
    assert abs(complex(z.grad) - (1.5 + 2.0j)) < 1e-15

    T = lambda a: torch.tensor(np.asarray(a, np.complex128), requires_grad=True)  # noqa: E731
    D, b, c, h0 = T(inp["D"]), T(inp["b"]), T(inp["c"]), T(inp["h0"])
    dy = torch.tensor(inp["dy"], dtype=torch.float64)
    dhf = torch.tensor(inp["dh_final"].astype(np.complex128))
    loss = 0
    for bb in range(B):
        for h in range(H):
            x = h0[bb, h]
            for t in range(L):
                p = pi[h, idx[bb, t, h]]
                A = torch.zeros((N, N), dtype=torch.complex128)
                A = A.index_put((torch.tensor(p, dtype=torch.long), torch.arange(N)), D[bb, t, h],
                                accumulate=True)
                x = A @ x + b[bb, t, h]
                loss = loss + dy[bb, t, h] * (c[bb, t, h] @ x).real
            loss = loss + (torch.conj(dhf[bb, h]) @ x).real
    loss.backward()
    dD, db, dc, dh0 = oracle_bwd(idx, pi, inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                                 dh_final=inp["dh_final"])
    for mine, ref in ((dD, D.grad), (db, b.grad), (dc, c.grad), (dh0, h0.grad)):
        np.testing.assert_allclose(mine, ref.numpy(), rtol=1e-12, atol=1e-12)


def _loss(inp, D, b, c, h0, dy, dhf):
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], D, b, c, h0=h0)
    return float((dy * y).sum() + (np.conj(dhf) * hf).real.sum())


def test_bwd_matches_finite_differences():
    """Central differences on real and imaginary parts: independent of any
    autodiff convention."""
    inp = small(5, B=1, L=7, H=1, N=4, K=2, with_h0=True, with_dhf=True)
    args = {k: inp[k].astype(np.complex128) for k in ("D", "b", "c", "h0")}
    dy, dhf = inp["dy"].astype(np.float64), inp["dh_final"].astype(np.complex128)
    grads = oracle_bwd(inp["idx"], inp["pi"], args["D"], args["b"], args["c"], dy,
                       h0=args["h0"], dh_final=dhf)
    gmap = dict(zip(("D", "b", "c", "h0"), grads))
    rng = np.random.default_rng(0)
    eps = 1e-6
    for name in ("D", "b", "c", "h0"):
        arr = args[name]
        for _ in range(6):
            pos = tuple(rng.integers(0, s) for s in arr.shape)
            for part, unit in (("re", 1.0), ("im", 1j)):
                plus = {k: v.copy() for k, v in args.items()}
                minus = {k: v.copy() for k, v in args.items()}
                plus[name][pos] += eps * unit
                minus[name][pos] -= eps * unit
                fd = (_loss(inp, **plus, dy=dy, dhf=dhf) - _loss(inp, **minus, dy=dy, dhf=dhf)) / (2 * eps)
                an = gmap[name][pos]
                an = an.real if part == "re" else an.imag
                assert abs(fd - an) <= 1e-6 * (1 + abs(an)), (name, pos, part, fd, an)


# ---------------------------------------------------------------- P2: composition
def test_compose_equals_dense_product():
    inp = small(6, B=2, L=11, H=2, N=7, K=4)
    idx, pi, D = inp["idx"], inp["pi"], inp["D"]
    for chunk in (1, 3, 4, 11, 50):
        pm, dm = oracle_compose(idx, pi, D, chunk)
        B, L, H = idx.shape
        C = -(-L // chunk)
        assert pm.shape == (B, H, C, 7)
        for bb in range(B):
            for h in range(H):
                for cc in range(C):
                    P = np.eye(7, dtype=np.complex128)
                    for t in range(cc * chunk, min((cc + 1) * chunk, L)):
                        P = dense_A(pi[h, idx[bb, t, h]], D[bb, t, h].astype(np.complex128)) @ P
                    # every column of the product has exactly one nonzero (|D| >= 0.5)
                    rows = np.argmax(np.abs(P), axis=0)
                    np.testing.assert_array_equal(pm[bb, h, cc], rows)
                    np.testing.assert_allclose(dm[bb, h, cc], P[rows, np.arange(7)], rtol=1e-12)
                    np.testing.assert_allclose(dense_A(pm[bb, h, cc], dm[bb, h, cc]), P,
                                               rtol=1e-12, atol=1e-15)


def test_compose_associative_across_chunks():
    """Whole-sequence map == dense product of the per-chunk maps (any split)."""
    inp = small(7, B=1, L=17, H=1, N=6, K=3)
    idx, pi, D = inp["idx"], inp["pi"], inp["D"]
    pw, dw = oracle_compose(idx, pi, D, chunk=17)
    for chunk in (2, 5, 8):
        pm, dm = oracle_compose(idx, pi, D, chunk)
        P = np.eye(6, dtype=np.complex128)
        for cc in range(pm.shape[2]):
            P = dense_A(pm[0, 0, cc], dm[0, 0, cc]) @ P
        np.testing.assert_allclose(dense_A(pw[0, 0, 0], dw[0, 0, 0]), P, rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------- P3: diagonal closed form
def test_identity_maps_reduce_to_diagonal_closed_form():
    """All maps identity: h_t[n] = prod_{u<=t} D_u[n] * sum_{s<=t} b_s[n] / prod_{u<=s} D_u[n]."""
    inp = small(8, B=1, L=20, H=1, N=6, K=3, pi_kind="identity")
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"])
    D = inp["D"][0, :, 0].astype(np.complex128)
    b = inp["b"][0, :, 0].astype(np.complex128)
    c = inp["c"][0, :, 0].astype(np.complex128)
    P = np.cumprod(D, axis=0)
    h = P * np.cumsum(b / P, axis=0)
    np.testing.assert_allclose(hf[0, 0], h[-1], rtol=1e-10)
    np.testing.assert_allclose(y[0, :, 0], (c * h).sum(axis=1).real, rtol=1e-9, atol=1e-12)


def test_constant_diagonal_is_power():
    """Identity maps, D constant, b only at t=0: h_t = D^t b_0 (complex pow)."""
    N, L = 4, 30
    inp = small(9, B=1, L=L, H=1, N=N, K=2, pi_kind="identity")
    d = inp["D"][0, 0, 0].copy()
    inp["D"][:] = d
    inp["b"][0, 1:] = 0
    _, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"])
    np.testing.assert_allclose(hf[0, 0], np.power(d.astype(np.complex128), L - 1) * inp["b"][0, 0, 0],
                               rtol=1e-12)


# ---------------------------------------------------------------- P4: automaton
@pytest.mark.parametrize("perm", [False, True])
def test_fsa_exact(perm):
    """App. D: D = 1, b = 0, one-hot start: the state stays the one-hot code of
    the automaton state q_t = pi_t(q_{t-1}), and y_t is the accept bit."""
    f = fsa_inputs(B=3, L=40, H=2, N=9, K=4, seed=10, perm=perm)
    y, hf, _ = oracle_fwd(f["idx"], f["pi"], f["D"], f["b"], f["c"], h0=f["h0"])
    for bb in range(3):
        for h in range(2):
            q = f["start"][bb, h]
            for t in range(40):
                q = f["pi"][h, f["idx"][bb, t, h], q]
                assert y[bb, t, h] == f["accept"][h, q]
            onehot = np.zeros(9)
            onehot[q] = 1
            np.testing.assert_array_equal(hf[bb, h], onehot)


# ---------------------------------------------------------------- P5: adjoint identities
def test_adjoint_identities():
    """l = sum dy*y + Re<dh_final, h_L> is linear in (b, h0) and in c, so
    l = Re<db, b> + Re<dh0, h0> and sum dy*y = Re<dc, c> exactly."""
    inp = small(11, B=2, L=15, H=3, N=6, K=4, with_h0=True, with_dhf=True)
    a = {k: inp[k].astype(np.complex128) for k in ("D", "b", "c", "h0", "dh_final")}
    dy = inp["dy"].astype(np.float64)
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], a["D"], a["b"], a["c"], h0=a["h0"])
    dD, db, dc, dh0 = oracle_bwd(inp["idx"], inp["pi"], a["D"], a["b"], a["c"], dy, h0=a["h0"],
                                 dh_final=a["dh_final"])
    lhs = (dy * y).sum() + (np.conj(a["dh_final"]) * hf).real.sum()
    rhs = (np.conj(db) * a["b"]).real.sum() + (np.conj(dh0) * a["h0"]).real.sum()
    assert abs(lhs - rhs) <= 1e-10 * (1 + abs(lhs))
    assert abs((dy * y).sum() - (np.conj(dc) * a["c"]).real.sum()) <= 1e-10 * (1 + abs(lhs))


# ---------------------------------------------------------------- P6: split invariance
def test_split_invariance_and_saved_states():
    inp = small(12, B=2, L=23, H=2, N=5, K=3, with_h0=True)
    idx, pi, D, b, c, h0 = (inp[k] for k in ("idx", "pi", "D", "b", "c", "h0"))
    y, hf, saved = oracle_fwd(idx, pi, D, b, c, h0=h0, chunk=6)
    for L1 in (1, 6, 10, 22):
        y1, h1, _ = oracle_fwd(idx[:, :L1], pi, D[:, :L1], b[:, :L1], c[:, :L1], h0=h0)
        y2, h2, _ = oracle_fwd(idx[:, L1:], pi, D[:, L1:], b[:, L1:], c[:, L1:], h0=h1)
        np.testing.assert_allclose(np.concatenate([y1, y2], axis=1), y, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(h2, hf, rtol=1e-12, atol=1e-13)
    # saved[c] is the state entering chunk c
    np.testing.assert_array_equal(saved[:, :, 0], h0.astype(np.complex128))
    for cc in range(1, saved.shape[2]):
        _, hc, _ = oracle_fwd(idx[:, :6 * cc], pi, D[:, :6 * cc], b[:, :6 * cc], c[:, :6 * cc], h0=h0)
        np.testing.assert_allclose(saved[:, :, cc], hc, rtol=1e-12, atol=1e-13)
    # the backward of a split sequence chains through dh0 -> dh_final
    dy = inp["dy"]
    full = oracle_bwd(idx, pi, D, b, c, dy, h0=h0)
    L1 = 10
    _, h1, _ = oracle_fwd(idx[:, :L1], pi, D[:, :L1], b[:, :L1], c[:, :L1], h0=h0)
    g2 = oracle_bwd(idx[:, L1:], pi, D[:, L1:], b[:, L1:], c[:, L1:], dy[:, L1:], h0=h1)
    g1 = oracle_bwd(idx[:, :L1], pi, D[:, :L1], b[:, :L1], c[:, :L1], dy[:, :L1], h0=h0,
                    dh_final=g2[3])
    for k in range(3):
        np.testing.assert_allclose(np.concatenate([g1[k], g2[k]], axis=1), full[k], rtol=1e-12,
                                   atol=1e-13)
    np.testing.assert_allclose(g1[3], full[3], rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- P7: norms
def test_norm_preserved_by_unitary_permutations():
    inp = small(13, B=2, L=50, H=2, N=8, K=3, pi_kind="perm", with_h0=True)
    D = inp["D"].astype(np.complex128)
    inp["D"] = D / np.abs(D)  # unit modulus in float64 (the oracle takes complex128 as is)
    inp["b"][:] = 0
    _, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    np.testing.assert_allclose(np.linalg.norm(hf, axis=-1),
                               np.linalg.norm(inp["h0"].astype(np.complex128), axis=-1), rtol=1e-12)


def test_norm_non_increasing_for_contractive_permutations():
    inp = small(14, B=1, L=30, H=1, N=8, K=3, pi_kind="perm", with_h0=True)
    inp["b"][:] = 0
    prev = np.linalg.norm(inp["h0"].astype(np.complex128))
    for L1 in range(1, 30):
        _, h1, _ = oracle_fwd(inp["idx"][:, :L1], inp["pi"], inp["D"][:, :L1], inp["b"][:, :L1],
                              inp["c"][:, :L1], h0=inp["h0"])
        n = np.linalg.norm(h1)
        assert n <= prev * (1 + 1e-12)
        prev = n


# ---------------------------------------------------------------- errors
def test_index_errors_rejected():
    inp = small(15)
    bad = inp["idx"].copy()
    bad[0, 0, 0] = 3  # K = 3
    with pytest.raises(IndexError):
        oracle_fwd(bad, inp["pi"], inp["D"], inp["b"], inp["c"])
    badp = inp["pi"].copy()
    badp[0, 0, 0] = -1
    with pytest.raises(IndexError):
        oracle_bwd(inp["idx"], badp, inp["D"], inp["b"], inp["c"], inp["dy"])
