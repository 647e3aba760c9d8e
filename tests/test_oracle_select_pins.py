"""Pins for the selection front end of the oracle (CPU only): the column
argmax that turns a dense dictionary into maps and the routing argmax, with
the first-maximal-index tie rule, against explicit loops; the token
projections (b, c and the diagonal generator) against loops and closed
forms."""
import cmath
import math

import numpy as np

from oracle import oracle_dict_argmax, oracle_project, oracle_route


def test_dict_argmax_is_the_column_argmax_with_first_ties():
    M = np.zeros((1, 2, 3, 3))
    # map 0: column 0 peaks at row 2, column 1 ties rows 0 and 1 (-> 0), column 2 peaks at row 1
    M[0, 0] = [[0, 5, 1], [1, 5, 7], [9, 2, 3]]
    # map 1: a constant column ties everywhere (-> row 0)
    M[0, 1] = [[4, 0, 0], [4, 0, 1], [4, 1, 0]]
    np.testing.assert_array_equal(oracle_dict_argmax(M), [[[2, 0, 1], [0, 2, 1]]])


def test_dict_argmax_matches_loops():
    rng = np.random.default_rng(0)
    M = rng.standard_normal((2, 3, 5, 5))
    pi = oracle_dict_argmax(M)
    for h in range(2):
        for k in range(3):
            for j in range(5):
                col = [M[h, k, i, j] for i in range(5)]
                assert pi[h, k, j] == col.index(max(col))


def test_route_matches_loops_and_ties():
    rng = np.random.default_rng(1)
    u = rng.integers(-3, 4, size=(2, 3, 4)).astype(np.float64)
    S = rng.integers(-2, 3, size=(2, 5, 4)).astype(np.float64)
    S[1, 3] = S[1, 1]  # two identical maps: their scores tie, the first wins
    logits, idx = oracle_route(u, S)
    for b in range(2):
        for t in range(3):
            for h in range(2):
                row = [sum(u[b, t, d] * S[h, k, d] for d in range(4)) for k in range(5)]
                assert list(logits[b, t, h]) == row
                assert idx[b, t, h] == row.index(max(row))


def _proj_inputs(seed, B=2, L=3, H=2, N=3, Dm=8):
    rng = np.random.default_rng(seed)
    u = rng.integers(-3, 4, size=(B, L, Dm)).astype(np.float64)
    W = [rng.integers(-2, 3, size=(H, 2 * N, Dm)).astype(np.float64) * 0.25 for _ in range(3)]
    return u, W


def test_project_matches_loops():
    """b, c: real and imaginary parts from rows 2n and 2n+1; D: sigmoid of
    row 2n times the unit phase of row 2n+1 (written with math/cmath per
    element)."""
    u, (Wb, Wc, Wd) = _proj_inputs(3)
    S = np.random.default_rng(4).integers(-2, 3, size=(2, 5, 8)).astype(np.float64)
    out = oracle_project(u, S, Wb, Wc, Wd)
    B, L, Dm = u.shape
    H, N2, _ = Wb.shape
    for bb in range(B):
        for t in range(L):
            for h in range(H):
                for n in range(N2 // 2):
                    dot = lambda W, r: sum(u[bb, t, d] * W[h, r, d] for d in range(Dm))  # noqa: E731
                    assert out["b"][bb, t, h, n] == complex(dot(Wb, 2 * n), dot(Wb, 2 * n + 1))
                    assert out["c"][bb, t, h, n] == complex(dot(Wc, 2 * n), dot(Wc, 2 * n + 1))
                    a, th = dot(Wd, 2 * n), dot(Wd, 2 * n + 1)
                    ref = cmath.rect(1.0 / (1.0 + math.exp(-a)), th)
                    assert abs(out["D"][bb, t, h, n] - ref) <= 1e-15
    lg, idx = oracle_route(u, S)
    np.testing.assert_array_equal(out["logits"], lg)
    np.testing.assert_array_equal(out["idx"], idx)


def test_project_closed_forms():
    """Zero generator weights give D = 1/2 exactly; a magnitude row that
    picks one feature gives a real D = sigmoid(u[d]); a phase row of pi/2 on
    a unit feature turns D imaginary; weights that pick features give b = u
    entries; |D| < 1 always, and arg D is the phase row's value."""
    B, L, H, N, Dm = 1, 4, 2, 3, 8
    rng = np.random.default_rng(7)
    u = rng.standard_normal((B, L, Dm))
    out = oracle_project(u, Wd=np.zeros((H, 2 * N, Dm)))
    assert np.all(out["D"] == 0.5)
    Wd = np.zeros((H, 2 * N, Dm))
    Wd[1, 2 * 1, 5] = 1.0            # head 1, entry 1: magnitude logit = u[5]
    D = oracle_project(u, Wd=Wd)["D"]
    np.testing.assert_allclose(D[..., 1, 1], 1.0 / (1.0 + np.exp(-u[..., 5])), rtol=0, atol=1e-15)
    assert np.all(D[..., 1, 1].imag == 0)
    u1 = np.zeros((1, 1, Dm))
    u1[0, 0, 2] = 1.0
    Wd = np.zeros((1, 2, Dm))
    Wd[0, 1, 2] = math.pi / 2        # phase pi/2, magnitude logit 0
    D = oracle_project(u1, Wd=Wd)["D"][0, 0, 0, 0]
    assert abs(D - 0.5j) <= 1e-16
    Wb = np.zeros((H, 2 * N, Dm))
    for h in range(H):
        for n in range(N):
            Wb[h, 2 * n, n] = 1.0           # real part = u[n]
            Wb[h, 2 * n + 1, n + N] = 1.0   # imaginary part = u[n + N]
    b = oracle_project(u, Wb=Wb)["b"]
    for h in range(H):
        np.testing.assert_array_equal(b[..., h, :], u[..., :N] + 1j * u[..., N:2 * N])
    _, (_, _, Wd) = _proj_inputs(9, Dm=8)
    uu = rng.standard_normal((2, 3, 8)) * 5
    P = np.einsum("bld,hrd->blhr", uu, Wd)
    D = oracle_project(uu, Wd=Wd)["D"]
    assert np.all(np.abs(D) < 1)
    np.testing.assert_allclose(np.angle(D), np.angle(np.exp(1j * P[..., 1::2])), atol=1e-12)
