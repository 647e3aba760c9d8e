"""Pins for the straight-through surrogate gradients of the oracle (CPU only).

The oracle's q (score of every candidate map at every step) and G (gradient of
every dictionary matrix) are checked against:
  - exact differences of a dense recurrence written here: the loss is affine
    in each single step's transition matrix, so replacing P_t by P_t + P_k
    changes the loss by exactly q_t[k];
  - torch.autograd on the dense model with real leaf matrices P_k and
    one-hot routing weights v_t (P_t = sum_k v_t[k] P_k);
  - identities that tie them to the backward scan: q_t[k_t] equals
    sum_j Re(conj(D_t[j]) dD_t[j]), and the q_t[k] of the steps that chose k
    add up to <G_k, P_k>.
The tempered-softmax products are checked against torch.autograd through
torch.softmax and against central differences.
"""
import numpy as np
import pytest

from oracle import oracle_bwd, oracle_softmax_vjp, oracle_ste, oracle_surrogate_grads
from paper_2605_19150_amd.inputs import make_inputs, selection_inputs


def dense_P(p):
    """Real N x N matrix of a column-one-hot map: column j has its one in row p[j]."""
    N = len(p)
    P = np.zeros((N, N))
    P[np.asarray(p), np.arange(N)] = 1.0
    return P


def dense_loss(inp, override=None):
    """l = sum_t dy_t y_t + Re sum conj(dh_final) h_L on a dense recurrence
    h_t = P_t (D_t .* h_{t-1}) + b_t; `override` = ((b, t, h), P) replaces one
    step's matrix."""
    idx, pi, D, b, c, dy = (inp[k] for k in ("idx", "pi", "D", "b", "c", "dy"))
    B, L, H = idx.shape
    N = pi.shape[2]
    loss = 0.0
    for bb in range(B):
        for h in range(H):
            x = inp["h0"][bb, h].astype(np.complex128) if "h0" in inp else np.zeros(N, np.complex128)
            for t in range(L):
                P = dense_P(pi[h, idx[bb, t, h]])
                if override is not None and override[0] == (bb, t, h):
                    P = override[1]
                x = P @ (D[bb, t, h].astype(np.complex128) * x) + b[bb, t, h]
                loss += float(dy[bb, t, h]) * (c[bb, t, h].astype(np.complex128) @ x).real
            if "dh_final" in inp:
                loss += (np.conj(inp["dh_final"][bb, h].astype(np.complex128)) @ x).real
    return loss


def _ste(inp):
    return oracle_ste(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"],
                      h0=inp.get("h0"), dh_final=inp.get("dh_final"))


@pytest.mark.parametrize("seed,pi_kind", [(0, "uniform"), (1, "perm")])
def test_scores_are_exact_affine_differences(seed, pi_kind):
    inp = make_inputs(1, 5, 2, 4, 3, seed=seed, pi_kind=pi_kind, with_h0=True, with_dhf=True)
    q, _ = _ste(inp)
    base = dense_loss(inp)
    idx, pi = inp["idx"], inp["pi"]
    for t in range(5):
        for h in range(2):
            for k in range(3):
                P = dense_P(pi[h, idx[0, t, h]]) + dense_P(pi[h, k])
                diff = dense_loss(inp, ((0, t, h), P)) - base
                assert abs(q[0, t, h, k] - diff) <= 1e-10 * (1 + abs(diff)), (t, h, k, q[0, t, h, k], diff)


def test_scores_and_dictionary_gradient_match_autograd():
    torch = pytest.importorskip("torch")
    inp = make_inputs(2, 7, 2, 5, 3, seed=7, with_h0=True, with_dhf=True)
    idx, pi = inp["idx"], inp["pi"]
    B, L, H = idx.shape
    K, N = pi.shape[1], pi.shape[2]
    Pk = torch.tensor(np.stack([np.stack([dense_P(pi[h, k]) for k in range(K)]) for h in range(H)]),
                      dtype=torch.float64, requires_grad=True)
    v = torch.tensor(np.eye(K)[idx], dtype=torch.float64, requires_grad=True)   # [B,L,H,K]
    T = lambda a: torch.tensor(np.asarray(a, np.complex128))  # noqa: E731
    D, b, c, h0, dhf = T(inp["D"]), T(inp["b"]), T(inp["c"]), T(inp["h0"]), T(inp["dh_final"])
    dy = torch.tensor(inp["dy"], dtype=torch.float64)
    loss = 0
    for bb in range(B):
        for h in range(H):
            x = h0[bb, h]
            for t in range(L):
                P = (v[bb, t, h][:, None, None] * Pk[h]).sum(0).to(torch.complex128)
                x = P @ (D[bb, t, h] * x) + b[bb, t, h]
                loss = loss + dy[bb, t, h] * (c[bb, t, h] @ x).real
            loss = loss + (torch.conj(dhf[bb, h]) @ x).real
    loss.backward()
    q, G = _ste(inp)
    np.testing.assert_allclose(q, v.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(G, Pk.grad.numpy(), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("seed,pi_kind", [(2, "uniform"), (3, "perm")])
def test_identities_with_the_backward_scan(seed, pi_kind):
    inp = make_inputs(2, 11, 3, 6, 4, seed=seed, pi_kind=pi_kind, with_h0=True, with_dhf=True)
    q, G = _ste(inp)
    dD, _, _, _ = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"],
                             h0=inp["h0"], dh_final=inp["dh_final"])
    idx, pi = inp["idx"], inp["pi"]
    # the selected map's score is <dP_t, P_{k_t}> = sum_j Re(conj(D_t[j]) dD_t[j])
    sel = np.take_along_axis(q, idx[..., None].astype(np.int64), axis=3)[..., 0]
    ref = (np.conj(inp["D"].astype(np.complex128)) * dD).real.sum(-1)
    np.testing.assert_allclose(sel, ref, rtol=1e-11, atol=1e-11)
    # summed over the steps that chose k, the scores give <G_k, P_k>
    H, K = pi.shape[:2]
    for h in range(H):
        for k in range(K):
            mask = idx[:, :, h] == k
            lhs = q[:, :, h, k][mask].sum()
            rhs = (G[h, k] * dense_P(pi[h, k])).sum()
            assert abs(lhs - rhs) <= 1e-10 * (1 + abs(rhs)), (h, k, lhs, rhs)
    # a map chosen nowhere has a zero gradient
    for h in range(H):
        for k in range(K):
            if not (idx[:, :, h] == k).any():
                assert not G[h, k].any()


def test_zero_upstream_gradient_gives_zero():
    inp = make_inputs(1, 6, 2, 4, 3, seed=4, with_h0=True)
    inp["dy"] = np.zeros_like(inp["dy"])
    q, G = _ste(inp)
    assert not q.any() and not G.any()


@pytest.mark.parametrize("temp", [0.5, 1.0, 3.0])
def test_softmax_vjp_matches_autograd_and_differences(temp):
    torch = pytest.importorskip("torch")
    inp = make_inputs(2, 5, 2, 6, 4, seed=9)
    logits, M = selection_inputs(inp["idx"], inp["pi"], seed=9)
    q, G = _ste(inp)
    dl, dM = oracle_surrogate_grads(q, G, logits, M, temp)
    for x, gy, axis, mine in ((logits, q, 3, dl), (M, G, 2, dM)):
        xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
        (torch.softmax(xt / temp, dim=axis) * torch.tensor(gy)).sum().backward()
        np.testing.assert_allclose(mine, xt.grad.numpy(), rtol=1e-12, atol=1e-13)
        # the softmax Jacobian annihilates constants: every fibre sums to zero
        np.testing.assert_allclose(mine.sum(axis=axis), 0.0, atol=1e-12)
    # central differences on a few logits
    rng = np.random.default_rng(1)
    def f(x):
        e = np.exp(x / temp - (x / temp).max(-1, keepdims=True))
        return ((e / e.sum(-1, keepdims=True)) * q).sum()
    x = logits.astype(np.float64)
    for _ in range(8):
        pos = tuple(rng.integers(0, s) for s in x.shape)
        xp, xm = x.copy(), x.copy()
        xp[pos] += 1e-6
        xm[pos] -= 1e-6
        fd = (f(xp) - f(xm)) / 2e-6
        assert abs(fd - dl[pos]) <= 1e-6 * (1 + abs(fd)), (pos, fd, dl[pos])


def test_softmax_vjp_axis_and_temperature_conventions():
    # two entries: s = (sigmoid(a), 1 - sigmoid(a)) with a = (x0 - x1)/temp; the
    # product with gy = (1, 0) is s0 (1 - s0) (1, -1) / temp
    x = np.array([[0.3, -0.4]])
    for temp in (0.25, 2.0):
        s0 = 1.0 / (1.0 + np.exp(-(0.7 / temp)))
        got = oracle_softmax_vjp(x, np.array([[1.0, 0.0]]), 1, temp)
        np.testing.assert_allclose(got, [[s0 * (1 - s0) / temp, -s0 * (1 - s0) / temp]], rtol=1e-14)
    # M's softmax runs down the rows of each column, where the argmax gives pi
    inp = make_inputs(1, 3, 1, 5, 2, seed=0)
    _, M = selection_inputs(inp["idx"], inp["pi"], seed=0)
    np.testing.assert_array_equal(M.argmax(axis=2), inp["pi"])


def test_selection_inputs_agree_with_the_hard_choices():
    inp = make_inputs(3, 40, 2, 16, 7, seed=5, idx_kind="markov")
    logits, M = selection_inputs(inp["idx"], inp["pi"], seed=5)
    np.testing.assert_array_equal(logits.argmax(axis=3), inp["idx"])
    np.testing.assert_array_equal(M.argmax(axis=2), inp["pi"])


def test_scaled_states_are_d_times_previous_state():
    from oracle import oracle_fwd
    inp = make_inputs(2, 9, 2, 5, 3, seed=11, with_h0=True)
    _, _, z = oracle_ste(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                         want_z=True)
    # h_{t-1} from prefix runs of the forward: the final state of steps 0..t-1
    for t in range(9):
        if t == 0:
            hp = inp["h0"].astype(np.complex128)
        else:
            sub = {k: np.ascontiguousarray(inp[k][:, :t]) for k in ("idx", "D", "b", "c")}
            _, hp, _ = oracle_fwd(sub["idx"], inp["pi"], sub["D"], sub["b"], sub["c"], h0=inp["h0"])
        np.testing.assert_allclose(z[:, t], inp["D"][:, t].astype(np.complex128) * hp, rtol=1e-13, atol=1e-14)
