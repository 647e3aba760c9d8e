"""GPU parity of the straight-through surrogate gradients (Sec. 3.1 Prop. 2):
the scaled states z written by the backward scan, the candidate-map scores q
and the dictionary gradient G (pdssm_ste_grads) and the tempered-softmax
products, through the C ABI, against the float64 oracle.

Tolerance: z, the plain backward outputs and the softmax products as for the
scan, |gpu - ref| <= 1e-5 + 1e-4*|ref| on every real component.  q and G are
sums of products of g and z, each known to that bar; their bar is
|gpu - ref| <= 1e-5 + 1e-4*S with S the sum of the magnitudes |g||z| of the
summands (S >= |ref|), see helpers.assert_close_sum.
"""
import ctypes

import numpy as np
import pytest

from helpers import assert_close, assert_close_sum, ste_scales, sub_sequence
from oracle import oracle_bwd, oracle_softmax_vjp, oracle_ste
from paper_2605_19150_amd.inputs import make_inputs, selection_inputs, workload_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_19150_amd import pdssm  # noqa: E402

DEV = torch.device("cuda:0")


def to_dev(inp):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(DEV) for k, v in inp.items()
            if isinstance(v, np.ndarray) and k not in ("start", "accept")}


def run_ste(inp, chunk=0):
    B, L, H = inp["idx"].shape
    _, K, N = inp["pi"].shape
    T = to_dev(inp)
    s = pdssm.Scan(B, L, H, N, K, chunk, DEV, ste=True)
    s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T.get("h0"))
    s.bwd_ste(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"], dh_final=T.get("dh_final"))
    s.ste_grads(T["idx"], T["pi"])
    s.check_status()
    out = {k: getattr(s, k).cpu().numpy() for k in ("dD", "db", "dc", "dh0", "q", "z", "G")}
    return s, T, out


def check_ste(inp, got):
    rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"],
                    h0=inp.get("h0"), dh_final=inp.get("dh_final"))
    for k, r in zip(("dD", "db", "dc", "dh0"), rg):
        assert_close(k, got[k], r)
    q, G, z = oracle_ste(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"],
                         h0=inp.get("h0"), dh_final=inp.get("dh_final"), want_z=True)
    assert_close("z", got["z"], z)
    qs, Gs = ste_scales(inp["pi"], inp["idx"], rg[1], z)
    assert_close_sum("q", got["q"], q, qs)
    assert_close_sum("G", got["G"], G, Gs)


# (N, K, B, L, H, chunk, pi_kind, idx_kind)
CASES = [
    (8, 5, 2, 37, 3, 4, "uniform", "uniform"),
    (16, 3, 2, 50, 2, 8, "perm", "uniform"),
    (32, 7, 2, 45, 2, 16, "uniform", "markov"),
    (64, 16, 2, 263, 3, 8, "uniform", "markov"),   # skewed groups: several items per group
    (64, 1, 1, 100, 2, 8, "uniform", "uniform"),   # one map
    (64, 20, 2, 70, 2, 4, "perm", "uniform"),      # two blocks of 16 scores
    (128, 9, 2, 80, 2, 8, "uniform", "uniform"),
    (256, 5, 1, 40, 2, 4, "uniform", "uniform"),
    (128, 128, 1, 30, 1, 8, "uniform", "uniform"),  # multi-pass scan (tables beyond LDS)
    (64, 256, 1, 40, 1, 8, "uniform", "uniform"),   # largest dictionary
    (64, 16, 1, 1100, 1, 8, "perm", "uniform"),     # segmented scan
    (32, 6, 1, 2000, 2, 16, "uniform", "uniform"),  # segmented, N < 64
]


@pytest.mark.parametrize("N,K,B,L,H,chunk,pi_kind,idx_kind", CASES)
def test_ste_matches_oracle(N, K, B, L, H, chunk, pi_kind, idx_kind):
    d = pdssm.desc(B, L, H, N, K, chunk)
    print("ste case N=%d K=%d B=%d L=%d H=%d chunk=%d %s %s fused=%d segments=%d" % (
        N, K, B, L, H, chunk, pi_kind, idx_kind, pdssm.load().pdssm_uses_fused(ctypes.byref(d)),
        pdssm.scan_segments(d)), flush=True)
    inp = make_inputs(B, L, H, N, K, seed=N * 7 + K * 13 + L, pi_kind=pi_kind, idx_kind=idx_kind,
                      with_h0=True, with_dhf=True)
    _, _, got = run_ste(inp, chunk)
    check_ste(inp, got)


def test_unused_maps_get_zero_gradient():
    inp = make_inputs(2, 90, 2, 64, 12, seed=3)
    inp["idx"] = (inp["idx"] % 4).astype(np.int32)       # maps 4..11 never chosen
    _, _, got = run_ste(inp)
    assert not got["G"][:, 4:].any()
    check_ste(inp, got)


def test_ste_outputs_are_optional_and_plain_outputs_unchanged():
    inp = make_inputs(2, 120, 2, 64, 6, seed=5, with_h0=True, with_dhf=True)
    B, L, H = inp["idx"].shape
    s, T, got = run_ste(inp)
    plain = pdssm.Scan(B, L, H, 64, 6, 0, DEV)
    plain.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T["h0"])
    plain.bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"], dh_final=T["dh_final"])
    torch.cuda.synchronize()
    for k in ("dD", "db", "dc", "dh0"):   # same kernels' arithmetic: identical bits
        np.testing.assert_array_equal(got[k], getattr(plain, k).cpu().numpy(), err_msg=k)
    # q alone and G alone equal the joint call bit for bit
    q1, G0 = pdssm.ste_grads(T["idx"], T["pi"], s.db, s.z, q=True, G=False)
    q0, G1 = pdssm.ste_grads(T["idx"], T["pi"], s.db, s.z, q=False, G=True)
    assert q0 is None and G0 is None
    np.testing.assert_array_equal(q1.cpu().numpy(), got["q"])
    np.testing.assert_array_equal(G1.cpu().numpy(), got["G"])


def _dense_ref(idx, pi, g, z):
    """q and G straight from their definitions, float64."""
    B, L, H, N = g.shape
    K = pi.shape[1]
    g, z = g.astype(np.complex128), z.astype(np.complex128)
    q = np.empty((B, L, H, K))
    G = np.zeros((H, K, N, N))
    for h in range(H):
        q[:, :, h, :] = (g[:, :, h, :][:, :, pi[h]] * np.conj(z[:, :, h, None, :])).real.sum(-1)
        for k in range(K):
            m = idx[:, :, h] == k
            G[h, k] = (g[:, :, h][m][:, :, None] * np.conj(z[:, :, h][m][:, None, :])).real.sum(0)
    return q, G


def test_ste_grads_alone_many_items_and_deterministic():
    # long groups: each is cut into many items whose partials are added in order
    rng = np.random.default_rng(9)
    B, L, H, N, K = 4, 3000, 2, 64, 3
    idx = rng.integers(0, K, size=(B, L, H), dtype=np.int32)
    pi = rng.integers(0, N, size=(H, K, N), dtype=np.int32)
    g = (rng.standard_normal((B, L, H, N)) + 1j * rng.standard_normal((B, L, H, N))).astype(np.complex64)
    z = (rng.standard_normal((B, L, H, N)) + 1j * rng.standard_normal((B, L, H, N))).astype(np.complex64)
    dv = [torch.from_numpy(a).to(DEV) for a in (idx, pi, g, z)]
    q1, G1 = (t.cpu().numpy() for t in pdssm.ste_grads(*dv))
    q2, G2 = (t.cpu().numpy() for t in pdssm.ste_grads(*dv))
    np.testing.assert_array_equal(G1, G2)
    np.testing.assert_array_equal(q1, q2)
    rq, rG = _dense_ref(idx, pi, g, z)
    qs, Gs = ste_scales(pi, idx, g.astype(np.complex128), z.astype(np.complex128))
    assert_close_sum("q", q1, rq, qs)
    assert_close_sum("G", G1, rG, Gs)


@pytest.mark.parametrize("N,K", [(8, 3), (16, 17), (32, 40), (128, 9), (256, 4), (64, 256)])
def test_ste_grads_alone_sizes(N, K):
    rng = np.random.default_rng(N + K)
    B, L, H = 2, 300, 3
    idx = rng.integers(0, K, size=(B, L, H), dtype=np.int32)
    pi = rng.integers(0, N, size=(H, K, N), dtype=np.int32)
    g = ((rng.standard_normal((B, L, H, N)) + 1j * rng.standard_normal((B, L, H, N))) / 8).astype(np.complex64)
    z = ((rng.standard_normal((B, L, H, N)) + 1j * rng.standard_normal((B, L, H, N))) / 8).astype(np.complex64)
    q, G = (t.cpu().numpy() for t in pdssm.ste_grads(*(torch.from_numpy(a).to(DEV) for a in (idx, pi, g, z))))
    rq, rG = _dense_ref(idx, pi, g, z)
    qs, Gs = ste_scales(pi, idx, g.astype(np.complex128), z.astype(np.complex128))
    assert_close_sum("q", q, rq, qs)
    assert_close_sum("G", G, rG, Gs)


def test_ste_grads_more_groups_than_the_plan_holds_in_lds():
    """H*K = 66*256 groups exceed the 16384 segment counts the planning
    kernel stages in LDS (it then walks them in global memory); most groups
    are empty and get zeros."""
    rng = np.random.default_rng(66)
    B, L, H, N, K = 1, 40, 66, 8, 256
    idx = rng.integers(0, K, size=(B, L, H), dtype=np.int32)
    pi = rng.integers(0, N, size=(H, K, N), dtype=np.int32)
    g = (rng.standard_normal((B, L, H, N)) + 1j * rng.standard_normal((B, L, H, N))).astype(np.complex64)
    z = (rng.standard_normal((B, L, H, N)) + 1j * rng.standard_normal((B, L, H, N))).astype(np.complex64)
    q, G = (t.cpu().numpy() for t in pdssm.ste_grads(*(torch.from_numpy(a).to(DEV) for a in (idx, pi, g, z))))
    rq, rG = _dense_ref(idx, pi, g, z)
    qs, Gs = ste_scales(pi, idx, g.astype(np.complex128), z.astype(np.complex128))
    assert_close_sum("q", q, rq, qs)
    assert_close_sum("G", G, rG, Gs)
    chosen = np.zeros((H, K), dtype=bool)
    for h in range(H):
        chosen[h, np.unique(idx[:, :, h])] = True
    assert not G[~chosen].any()


def test_ste_grads_reports_bad_index():
    B, L, H, N, K = 1, 50, 1, 64, 4
    idx = torch.zeros((B, L, H), dtype=torch.int32, device=DEV)
    idx[0, 7, 0] = 9
    pi = torch.zeros((H, K, N), dtype=torch.int32, device=DEV)
    g = torch.zeros((B, L, H, N), dtype=torch.complex64, device=DEV)
    with pytest.raises(pdssm.PdssmError):
        pdssm.ste_grads(idx, pi, g, g.clone())


@pytest.mark.parametrize("temp", [0.5, 1.0, 3.0])
def test_softmax_vjp(temp):
    inp = make_inputs(3, 50, 2, 64, 16, seed=21)
    logits, M = selection_inputs(inp["idx"], inp["pi"], seed=21)
    rng = np.random.default_rng(2)
    q = rng.standard_normal(logits.shape).astype(np.float32)
    G = rng.standard_normal(M.shape).astype(np.float32)
    dl, dM = pdssm.surrogate_grads(*(torch.from_numpy(a).to(DEV) for a in (q, G, logits, M)), temp)
    assert_close("dlogits", dl.cpu().numpy(), oracle_softmax_vjp(logits, q, 3, temp))
    assert_close("dM", dM.cpu().numpy(), oracle_softmax_vjp(M, G, 2, temp))
    # any axis, including the last and the first
    x = torch.from_numpy(rng.standard_normal((5, 7, 9)).astype(np.float32)).to(DEV)
    gy = torch.from_numpy(rng.standard_normal((5, 7, 9)).astype(np.float32)).to(DEV)
    for dim in (0, 1, 2):
        assert_close("dim%d" % dim, pdssm.softmax_vjp(x, gy, dim, temp).cpu().numpy(),
                     oracle_softmax_vjp(x.cpu().numpy(), gy.cpu().numpy(), dim, temp))


@pytest.mark.parametrize("length", [1, 3, 4, 8, 12, 20, 64, 100, 256, 300])
def test_softmax_vjp_row_lengths(length):
    """Contiguous axis: the 16-byte path (length % 4 == 0, up to 256, aligned
    rows), the general path, and a row view that starts off a 16-byte boundary."""
    rng = np.random.default_rng(length)
    x = torch.from_numpy(rng.standard_normal((37, length + 1)).astype(np.float32) * 3).to(DEV)
    gy = torch.from_numpy(rng.standard_normal((37, length + 1)).astype(np.float32)).to(DEV)
    for xs, gs in ((x[:, :length].contiguous(), gy[:, :length].contiguous()),
                   (x.reshape(-1)[1:1 + 37 * length].reshape(37, length),
                    gy.reshape(-1)[1:1 + 37 * length].reshape(37, length))):
        got = pdssm.softmax_vjp(xs, gs, 1, 0.7).cpu().numpy()
        assert_close("len%d" % length, got, oracle_softmax_vjp(xs.cpu().numpy(), gs.cpu().numpy(), 1, 0.7))


@pytest.mark.parametrize("shape", [(5, 31, 9), (3, 32, 5), (2, 64, 64), (4, 100, 3), (1, 128, 128),
                                   (2, 301, 7), (3, 33, 70)])
def test_softmax_vjp_column_lengths(shape):
    """Strided axis (the middle one): one thread per column below 32 entries,
    four threads per column (quarters merged in order) from 32 on, with
    lengths that leave a short last quarter and column counts that leave
    a partial block."""
    rng = np.random.default_rng(sum(shape))
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * 3).to(DEV)
    gy = torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(DEV)
    got = pdssm.softmax_vjp(x, gy, 1, 0.8).cpu().numpy()
    assert_close("cols%s" % (shape,), got, oracle_softmax_vjp(x.cpu().numpy(), gy.cpu().numpy(), 1, 0.8))


@pytest.mark.parametrize("wl", [2, 3])
def test_full_size_sampled(wl):
    """Workload sizes (B16 L2048 H16 N64 K16): q and z on sampled sequences,
    G of two heads (all 16 sequences each) against the oracle."""
    inp = workload_inputs(wl, seed=0)
    print("full-size ste workload %d" % wl, flush=True)
    s, T, got = run_ste(inp)
    for bb, hh in ((0, 0), (15, 15), (7, 3)):
        sub = sub_sequence(inp, bb, hh)
        q, _, z = oracle_ste(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"], sub["dy"], want_z=True)
        _, db, _, _ = oracle_bwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"], sub["dy"])
        qs, _ = ste_scales(sub["pi"], sub["idx"], db, z)
        assert_close_sum("q[%d,%d]" % (bb, hh), got["q"][bb:bb + 1, :, hh:hh + 1], q, qs)
        assert_close("z[%d,%d]" % (bb, hh), got["z"][bb:bb + 1, :, hh:hh + 1], z)
    for hh in (0, 15):
        hs = {k: np.ascontiguousarray(inp[k][:, :, hh:hh + 1]) for k in ("idx", "D", "b", "c", "dy")}
        _, G, z = oracle_ste(hs["idx"], inp["pi"][hh:hh + 1], hs["D"], hs["b"], hs["c"], hs["dy"], want_z=True)
        _, db, _, _ = oracle_bwd(hs["idx"], inp["pi"][hh:hh + 1], hs["D"], hs["b"], hs["c"], hs["dy"])
        _, Gs = ste_scales(inp["pi"][hh:hh + 1], hs["idx"], db, z)
        assert_close_sum("G[%d]" % hh, got["G"][hh:hh + 1], G, Gs)
