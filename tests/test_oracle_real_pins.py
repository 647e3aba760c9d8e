"""Pins of the oracle on the real-valued model (App. B: the MAD and
time-series setups run the model over the reals): real D, b, c and h0.

  - the oracle's forward against a dense real recurrence written out with
    numpy matrices (brute force: A_t[pi_t(j), j] += D_t[j], h_t = A_t h + b_t,
    y_t = c_t . h_t);
  - the oracle's gradients against central finite differences of
    l = sum_t dy_t y_t + dh_final . h_final over real parameters;
  - everything it returns has imaginary part exactly 0 (real inputs stay
    real through every product and sum).
"""
import numpy as np
import pytest

from oracle import oracle_bwd, oracle_fwd
from paper_2605_19150_amd.inputs import make_inputs


def dense_real(idx, pi, D, b, c, h0):
    B, L, H, N = D.shape
    y = np.zeros((B, L, H))
    hf = np.zeros((B, H, N))
    for bb in range(B):
        for hh in range(H):
            h = h0[bb, hh].astype(np.float64).copy()
            for t in range(L):
                A = np.zeros((N, N))
                p = pi[hh, idx[bb, t, hh]]
                for j in range(N):
                    A[p[j], j] += D[bb, t, hh, j]
                h = A @ h + b[bb, t, hh]
                y[bb, t, hh] = c[bb, t, hh] @ h
            hf[bb, hh] = h
    return y, hf


def real_case(seed, N=6, K=3, L=9):
    inp = make_inputs(B=2, L=L, H=2, N=N, K=K, seed=seed, with_h0=True, with_dhf=True, real=True)
    for k in ("D", "b", "c"):
        assert inp[k].dtype == np.float32
    for k in ("h0", "dh_final"):
        assert np.all(inp[k].imag == 0)
    return inp


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_real_fwd_matches_dense(seed):
    inp = real_case(seed)
    h0 = inp["h0"].real.astype(np.float64)
    ry, rhf = dense_real(inp["idx"], inp["pi"], inp["D"].astype(np.float64), inp["b"].astype(np.float64),
                         inp["c"].astype(np.float64), h0)
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    np.testing.assert_allclose(y, ry, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(hf.real, rhf, rtol=1e-12, atol=1e-12)
    assert np.all(hf.imag == 0)


def test_real_many_to_one_collisions():
    # every map sends all sources to row 0: the dense sum must agree
    inp = real_case(7, N=5, K=2, L=6)
    inp["pi"][:] = 0
    y, hf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    ry, rhf = dense_real(inp["idx"], inp["pi"], inp["D"].astype(np.float64), inp["b"].astype(np.float64),
                         inp["c"].astype(np.float64), inp["h0"].real.astype(np.float64))
    np.testing.assert_allclose(y, ry, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(hf.real, rhf, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", [3, 4])
def test_real_grads_match_finite_differences(seed):
    inp = real_case(seed)
    idx, pi, dy = inp["idx"], inp["pi"], inp["dy"].astype(np.float64)
    dhf = inp["dh_final"].real.astype(np.float64)
    P = {k: inp[k].astype(np.float64) for k in ("D", "b", "c")}
    P["h0"] = inp["h0"].real.astype(np.float64)

    def loss(Q):
        y, hf = dense_real(idx, pi, Q["D"], Q["b"], Q["c"], Q["h0"])
        return float((dy * y).sum() + (dhf * hf).sum())

    dD, db, dc, dh0 = oracle_bwd(idx, pi, P["D"], P["b"], P["c"], dy, h0=P["h0"], dh_final=dhf)
    grads = {"D": dD, "b": db, "c": dc, "h0": dh0}
    for g in grads.values():
        assert np.all(g.imag == 0)
    rng = np.random.default_rng(seed)
    eps = 1e-6
    for k, g in grads.items():
        for _ in range(6):
            pos = tuple(int(rng.integers(0, n)) for n in P[k].shape)
            Qp = {kk: v.copy() for kk, v in P.items()}
            Qm = {kk: v.copy() for kk, v in P.items()}
            Qp[k][pos] += eps
            Qm[k][pos] -= eps
            fd = (loss(Qp) - loss(Qm)) / (2 * eps)
            assert abs(g.real[pos] - fd) <= 1e-6 + 1e-6 * abs(fd), (k, pos, g.real[pos], fd)


def test_real_surrogate_inputs_match_real_autograd():
    """Straight-through inputs of the real-valued model: on a dense real
    model (float64 throughout, no complex numbers anywhere) with leaf
    dictionary matrices P_k and one-hot routing weights v_t
    (P_t = sum_k v_t[k] P_k), v.grad is the oracle's q and P.grad its G."""
    torch = pytest.importorskip("torch")
    from oracle import oracle_ste
    inp = real_case(5, N=5, K=3, L=7)
    idx, pi = inp["idx"], inp["pi"]
    B, L, H = idx.shape
    K, N = pi.shape[1], pi.shape[2]
    dense = np.zeros((H, K, N, N))
    for h in range(H):
        for k in range(K):
            dense[h, k, pi[h, k], np.arange(N)] = 1.0
    Pk = torch.tensor(dense, dtype=torch.float64, requires_grad=True)
    v = torch.tensor(np.eye(K)[idx], dtype=torch.float64, requires_grad=True)
    R = lambda a: torch.tensor(np.asarray(a, np.float64))  # noqa: E731
    D, b, c, dy = R(inp["D"]), R(inp["b"]), R(inp["c"]), R(inp["dy"])
    h0, dhf = R(inp["h0"].real), R(inp["dh_final"].real)
    loss = 0
    for bb in range(B):
        for h in range(H):
            x = h0[bb, h]
            for t in range(L):
                P = (v[bb, t, h][:, None, None] * Pk[h]).sum(0)
                x = P @ (D[bb, t, h] * x) + b[bb, t, h]
                loss = loss + dy[bb, t, h] * (c[bb, t, h] @ x)
            loss = loss + dhf[bb, h] @ x
    loss.backward()
    q, G, z = oracle_ste(idx, pi, inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                         dh_final=inp["dh_final"], want_z=True)
    assert np.all(np.asarray(z).imag == 0)
    np.testing.assert_allclose(q, v.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(G, Pk.grad.numpy(), rtol=1e-11, atol=1e-11)
