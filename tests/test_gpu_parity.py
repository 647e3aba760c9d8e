"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Tolerance (fp32 compute, float64 reference): |gpu - ref| <= 1e-5 + 1e-4*|ref|
on every real component of y, h_final, saved states and all gradients; the
composed integer maps and the automaton case are compared bit for bit.
"""
import numpy as np
import pytest

from helpers import assert_close, force_sorted_entries, sub_sequence
from oracle import oracle_bwd, oracle_compose, oracle_fwd
from paper_2605_19150_amd.inputs import WORKLOADS, fsa_inputs, make_inputs, workload_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_19150_amd import pdssm  # noqa: E402

DEV = torch.device("cuda:0")


def to_dev(inp):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(DEV) for k, v in inp.items()
            if isinstance(v, np.ndarray) and k not in ("start", "accept")}


def run_gpu(inp, chunk=0, bwd=True):
    T = to_dev(inp)
    y, hf, saved = pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T.get("h0"),
                                  chunk=chunk)
    out = dict(y=y.cpu().numpy(), h_final=hf.cpu().numpy(), saved=saved.cpu().numpy())
    if bwd:
        g = pdssm.scan_bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], saved, T["dy"],
                           dh_final=T.get("dh_final"), chunk=chunk)
        for k, v in zip(("dD", "db", "dc", "dh0"), g):
            out[k] = v.cpu().numpy()
    return out


def eff_chunk(inp, chunk=0):
    B, L, H = inp["idx"].shape
    _, K, N = inp["pi"].shape
    return pdssm.chunk_len(pdssm.desc(B, L, H, N, K, chunk))


def check_all(inp, got, chunk_eff, bwd=True):
    ry, rhf, rsaved = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"],
                                 h0=inp.get("h0"), chunk=chunk_eff)
    assert_close("y", got["y"], ry)
    assert_close("h_final", got["h_final"], rhf)
    assert_close("saved", got["saved"], rsaved)
    if bwd:
        rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"],
                        h0=inp.get("h0"), dh_final=inp.get("dh_final"))
        for k, r in zip(("dD", "db", "dc", "dh0"), rg):
            assert_close(k, got[k], r)


# ------------------------------------------------------------------ small shapes
CASES = []
for N in (8, 16, 32, 64, 128, 256):
    for chunk in (4, 8, 16):
        if chunk * max(1, N // 64) > 16:
            continue
        # ragged edges, and enough chunks (> 12 waves) to wrap the round-robin
        for L in (1, chunk - 1, chunk, chunk + 1, 3 * chunk + 5, 30 * chunk + 7):
            CASES.append((N, chunk, L))


@pytest.mark.parametrize("N,chunk,L", CASES)
def test_small_shapes(N, chunk, L):
    print("case N=%d chunk=%d L=%d" % (N, chunk, L), flush=True)
    inp = make_inputs(B=2, L=L, H=3, N=N, K=5, seed=N * 1000 + chunk * 10 + L, with_h0=True,
                      with_dhf=True)
    got = run_gpu(inp, chunk=chunk)
    check_all(inp, got, chunk)


@pytest.mark.parametrize("pi_kind", ["uniform", "perm", "identity"])
def test_map_kinds_default_chunk(pi_kind):
    inp = make_inputs(B=3, L=200, H=2, N=64, K=7, seed=7, pi_kind=pi_kind, with_h0=True,
                      with_dhf=True)
    got = run_gpu(inp)
    check_all(inp, got, eff_chunk(inp))


def test_single_dictionary_entry_and_k256():
    for K in (1, 256):
        inp = make_inputs(B=1, L=70, H=2, N=32, K=K, seed=K)
        got = run_gpu(inp)
        check_all(inp, got, eff_chunk(inp))


@pytest.mark.parametrize("N", [64, 128])
def test_all_maps_collapse_to_one_row(N):
    """Degenerate many-to-one maps: every entry maps to row 0 (maximal
    collisions, in-degree N: the atomic-scatter branch)."""
    inp = make_inputs(B=1, L=250, H=1, N=N, K=3, seed=3)
    inp["pi"][:] = 0
    got = run_gpu(inp)
    check_all(inp, got, eff_chunk(inp))


def test_mixed_degenerate_and_regular_entries():
    """Some dictionary entries need the atomic branch (a row of in-degree > 7),
    the others the gather records; steps switch between them."""
    inp = make_inputs(B=2, L=400, H=2, N=64, K=6, seed=31, with_h0=True, with_dhf=True)
    inp["pi"][0, 1, :9] = 5
    inp["pi"][1, 4, :] = 63
    got = run_gpu(inp)
    check_all(inp, got, eff_chunk(inp))


@pytest.mark.parametrize("N,chunk", [(16, 8), (32, 16), (64, 4), (64, 8), (64, 16), (128, 4), (128, 8),
                                     (256, 4)])
def test_sorted_form_entries(N, chunk):
    """Heads whose dictionary has entries of in-degree > 7 next to regular
    ones: those steps sum each row's run by a segmented scan inside the
    pipelined chunk pass (and in the backward's state recompute)."""
    inp = make_inputs(B=2, L=300, H=3, N=N, K=6, seed=N + chunk, with_h0=True, with_dhf=True)
    force_sorted_entries(inp, N)
    got = run_gpu(inp, chunk=chunk)
    check_all(inp, got, chunk)


@pytest.mark.parametrize("N,L", [(64, 1500), (128, 2000)])
def test_segmented_scan_with_sorted_form_entries(N, L):
    """One long sequence cut into segments (aggregate pass, then one
    workgroup per segment) where some dictionary entries are in sorted form:
    the run folds of the aggregate pass and the frontier's composition of
    such runs, forward and backward."""
    K = 5
    d = pdssm.desc(1, L, 1, N, K)
    assert pdssm.scan_segments(d) > 1
    inp = make_inputs(B=1, L=L, H=1, N=N, K=K, seed=L + 3, with_h0=True, with_dhf=True)
    inp["pi"][0, 1, :9] = 5
    inp["pi"][0, 3, :] = 0
    inp["idx"][:, ::4, 0] = 1
    inp["idx"][:, 2::5, 0] = 3
    got = run_gpu(inp)
    check_all(inp, got, eff_chunk(inp))


@pytest.mark.parametrize("N,K", [(128, 128), (256, 64)])
def test_large_dictionary_chunked_path(N, K):
    """A head's dictionary tables too large for LDS: the chunked three-pass
    kernels run instead, with the same saved-state layout.  Some entries have
    a row of more than seven sources (the sorted form), and steps choose them
    often."""
    inp = make_inputs(B=2, L=90, H=2, N=N, K=K, seed=N + K, with_h0=True, with_dhf=True)
    assert pdssm.uses_fused(pdssm.desc(2, 90, 2, N, K)) == 0
    inp["pi"][0, 1, :8] = 3          # in-degree exactly 8
    inp["pi"][1, 2, :] = N - 1       # all to one row
    inp["idx"][:, ::3, 0] = 1
    inp["idx"][:, 1::4, 1] = 2
    got = run_gpu(inp)
    check_all(inp, got, eff_chunk(inp))


@pytest.mark.parametrize("K,fused", [(16, 1), (32, 1), (64, 0)])
def test_state_size_256_wave_counts(K, fused):
    """N = 256: five chunk waves (K <= 16), three (K = 32), multi-pass beyond;
    segmented (one sequence) and many sequences, with h0 and dh_final."""
    for B, L, H in ((1, 900, 1), (3, 61, 4)):
        print("N=256 K=%d B=%d L=%d H=%d" % (K, B, L, H), flush=True)
        assert pdssm.uses_fused(pdssm.desc(B, L, H, 256, K)) == fused
        inp = make_inputs(B=B, L=L, H=H, N=256, K=K, seed=K + L, with_h0=True, with_dhf=True)
        got = run_gpu(inp)
        check_all(inp, got, eff_chunk(inp))


# ------------------------------------------------------------------ automaton: exact
@pytest.mark.parametrize("N,perm", [(8, False), (64, True), (64, False), (128, False), (256, True)])
def test_fsa_bit_exact(N, perm):
    f = fsa_inputs(B=2, L=300, H=3, N=N, K=6, seed=N, perm=perm)
    got = run_gpu(f, bwd=False)
    ry, rhf, _ = oracle_fwd(f["idx"], f["pi"], f["D"], f["b"], f["c"], h0=f["h0"])
    np.testing.assert_array_equal(got["y"].astype(np.float64), ry)
    np.testing.assert_array_equal(got["h_final"].astype(np.complex128), rhf)


# ------------------------------------------------------------------ compose: exact maps
@pytest.mark.parametrize("N,chunk,L", [(8, 5, 64), (64, 32, 100), (128, 7, 50), (256, 1, 9),
                                       (64, 1000, 257)])
def test_compose_chunks(N, chunk, L):
    inp = make_inputs(B=2, L=L, H=2, N=N, K=4, seed=chunk + N)
    T = to_dev(inp)
    pm, dm = pdssm.compose_chunks(T["idx"], T["pi"], T["D"], chunk)
    rp, rd = oracle_compose(inp["idx"], inp["pi"], inp["D"], min(chunk, L))
    np.testing.assert_array_equal(pm.cpu().numpy(), rp)
    assert_close("d_out", dm.cpu().numpy(), rd)


# ------------------------------------------------------------------ split / determinism / errors
def test_split_invariance_through_h0():
    inp = make_inputs(B=2, L=150, H=2, N=64, K=4, seed=21, with_h0=True)
    T = to_dev(inp)
    y, hf, _ = pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T["h0"])
    L1 = 77
    sl = lambda k, a, b: T[k][:, a:b].contiguous()  # noqa: E731
    y1, h1, _ = pdssm.scan_fwd(sl("idx", 0, L1), T["pi"], sl("D", 0, L1), sl("b", 0, L1),
                               sl("c", 0, L1), h0=T["h0"])
    y2, h2, _ = pdssm.scan_fwd(sl("idx", L1, 150), T["pi"], sl("D", L1, 150), sl("b", L1, 150),
                               sl("c", L1, 150), h0=h1.clone())
    ry, rhf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    assert_close("y split", torch.cat([y1, y2], 1).cpu().numpy(), ry)
    assert_close("h_final split", h2.cpu().numpy(), rhf)


@pytest.mark.parametrize("N", [64, 128])
def test_split_invariance_backward_through_dh_final(N):
    """Two calls chained backwards: the second segment's dh0 is the first
    segment's dh_final; the gradients match one backward over the whole
    sequence (the oracle's)."""
    L, L1 = 133, 58
    inp = make_inputs(B=2, L=L, H=2, N=N, K=4, seed=31 + N, with_h0=True, with_dhf=True)
    T = to_dev(inp)
    sl = lambda k, a, b: T[k][:, a:b].contiguous()  # noqa: E731
    parts = [tuple(sl(k, a, b) for k in ("idx", "D", "b", "c", "dy")) for a, b in ((0, L1), (L1, L))]
    _, h1, s1 = pdssm.scan_fwd(parts[0][0], T["pi"], *parts[0][1:4], h0=T["h0"])
    h1, s1 = h1.clone(), s1.clone()
    _, _, s2 = pdssm.scan_fwd(parts[1][0], T["pi"], *parts[1][1:4], h0=h1)
    g2 = [t.clone() for t in pdssm.scan_bwd(parts[1][0], T["pi"], *parts[1][1:4], s2.clone(), parts[1][4],
                                            dh_final=T["dh_final"])]
    g1 = [t.clone() for t in pdssm.scan_bwd(parts[0][0], T["pi"], *parts[0][1:4], s1, parts[0][4],
                                            dh_final=g2[3])]
    rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                    dh_final=inp["dh_final"])
    for i, name in enumerate(("dD", "db", "dc")):
        assert_close(name + " split", torch.cat([g1[i], g2[i]], 1).cpu().numpy(), rg[i])
    assert_close("dh0 split", g1[3].cpu().numpy(), rg[3])


@pytest.mark.parametrize("N,pi_kind", [(64, "perm"), (64, "uniform"), (128, "uniform")])
def test_segment_protocol_from_entry_points(N, pi_kind):
    """The sequence-sharded scan, run on one GPU with three segments as if each
    were another device: a segment's aggregate is pdssm_compose_chunks over the
    whole segment (map, diagonal) plus its scan from zero (local state); an
    aggregate is applied to the incoming state by a one-step scan whose
    dictionary holds each sequence's composed map (idx[b] = b); every segment
    then scans from its composed entering state.  Outputs match the oracle's
    scan of the whole sequence."""
    B, H, K = 3, 2, 5
    cuts = [0, 41, 90, 157]
    inp = make_inputs(B=B, L=cuts[-1], H=H, N=N, K=K, seed=N + len(pi_kind), pi_kind=pi_kind, with_h0=True)
    T = to_dev(inp)
    sl = lambda k, a, b: T[k][:, a:b].contiguous()  # noqa: E731
    seg = [tuple(sl(k, cuts[g], cuts[g + 1]) for k in ("idx", "D", "b", "c")) for g in range(3)]

    def aggregate(g):
        idx, D, b, c = seg[g]
        pm, dm = pdssm.compose_chunks(idx, T["pi"], D, idx.shape[1])
        _, local, _ = pdssm.scan_fwd(idx, T["pi"], D, b, c)
        return pm[:, :, 0], dm[:, :, 0], local.clone()

    def apply(agg, carry):
        pm, dm, local = agg
        idx1 = torch.arange(B, dtype=torch.int32, device=DEV).view(B, 1, 1).expand(B, 1, H).contiguous()
        pi1 = pm.permute(1, 0, 2).contiguous()  # [H, K = B, N]
        zero = torch.zeros((B, 1, H, N), dtype=torch.complex64, device=DEV)
        _, hf, _ = pdssm.scan_fwd(idx1, pi1, dm.unsqueeze(1).contiguous(), local.unsqueeze(1).contiguous(), zero,
                                  h0=carry)
        return hf.clone()

    aggs = [None] + [aggregate(g) for g in (1, 2)]  # computed independently of segment 0
    carry = [T["h0"]]
    run = lambda parts, h0: pdssm.scan_fwd(parts[0], T["pi"], *parts[1:], h0=h0)  # noqa: E731
    _, h1, _ = run(seg[0], T["h0"])
    carry.append(h1.clone())
    carry.append(apply(aggs[1], carry[1]))
    ys, hfin = [], None
    for g in range(3):
        y, hf, _ = run(seg[g], carry[g])
        ys.append(y.clone())
        hfin = hf.clone()
    # the composed entering state of segment 2 equals the state the scan reaches there
    _, h_two, _ = run([torch.cat([seg[0][i], seg[1][i]], 1) for i in range(4)], T["h0"])
    assert_close("carry 2", carry[2].cpu().numpy(), h_two.cpu().numpy())
    ry, rhf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    assert_close("y by segments", torch.cat(ys, 1).cpu().numpy(), ry)
    assert_close("h_final by segments", hfin.cpu().numpy(), rhf)


@pytest.mark.parametrize("N,B,L,H,K,sorted_form", [
    (64, 2, 300, 4, 8, False), (128, 2, 300, 4, 8, False), (256, 2, 300, 4, 8, False),
    (128, 1, 2000, 1, 8, False), (64, 2, 300, 3, 8, True), (128, 1, 2000, 3, 8, True),
    (256, 2, 300, 3, 16, True), (128, 2, 90, 3, 128, True), (256, 2, 90, 3, 64, True)])
def test_deterministic(N, B, L, H, K, sorted_form):
    """Two runs give the same bits: colliding sources are added in an order
    fixed by the map (uniform maps; with sorted_form also entries of
    in-degree > 7; segmented sequences; the multi-pass kernels at K = 128
    (N = 128) and K = 64 (N = 256))."""
    inp = make_inputs(B=B, L=L, H=H, N=N, K=K, seed=5, with_h0=True, with_dhf=True)
    if sorted_form:
        force_sorted_entries(inp, N)
    a = run_gpu(inp)
    b = run_gpu(inp)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_deterministic_full_size_manyone():
    """The many-to-one workload at full size (B16 L2048 H16 N64 K16, Markov
    map choices), whose head 4 has an entry of in-degree 9: two runs give the
    same bits in every output."""
    w = WORKLOADS[3]
    inp = workload(3)
    assert _max_in_degree(inp["pi"]) > 7
    T = to_dev(inp)
    outs = []
    for _ in range(2):
        s = pdssm.Scan(w.B, w.L, w.H, w.N, w.K)
        s.prepare(T["pi"])
        s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"])
        s.bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"])
        s.check_status()
        outs.append({k: getattr(s, k).clone() for k in ("y", "h_final", "saved", "dD", "db", "dc", "dh0")})
        del s
    for k in outs[0]:
        assert torch.equal(outs[0][k], outs[1][k]), k


def _max_in_degree(pi):
    H, K, N = pi.shape
    m = 0
    for h in range(H):
        for k in range(K):
            m = max(m, int(np.bincount(pi[h, k], minlength=N).max()))
    return m


@pytest.mark.parametrize("N,K,pi_kind", [(64, 16, "perm"), (64, 16, "uniform"), (128, 64, "uniform"),
                                         (128, 128, "uniform")])
def test_prepared_tables_match_per_call_build(N, K, pi_kind):
    """Scans on tables from pdssm_prepare give the same bits as scans that
    build them per call; after pi changes, prepare again and the scans follow
    the new dictionary."""
    inp = make_inputs(B=2, L=77, H=3, N=N, K=K, seed=N + K, pi_kind=pi_kind, with_h0=True,
                      with_dhf=True)
    T = to_dev(inp)
    ref = run_gpu(inp)
    s = pdssm.Scan(2, 77, 3, N, K)
    s.prepare(T["pi"])
    for _ in range(2):
        s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T["h0"])
        s.bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"], dh_final=T["dh_final"])
        s.check_status()
        for k in ("y", "h_final", "saved", "dD", "db", "dc", "dh0"):
            np.testing.assert_array_equal(getattr(s, k).cpu().numpy(), ref[k], err_msg=k)
    inp2 = dict(inp)
    inp2["pi"] = np.ascontiguousarray(inp["pi"][:, ::-1])
    T["pi"].copy_(torch.from_numpy(inp2["pi"]))
    s.prepare(T["pi"])
    s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T["h0"])
    s.bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"], dh_final=T["dh_final"])
    s.check_status()
    got = {k: getattr(s, k).cpu().numpy() for k in ("y", "h_final", "saved", "dD", "db", "dc", "dh0")}
    check_all(inp2, got, s.chunk)


@pytest.mark.parametrize("N,chunk,L,B,H,pi_kind", [
    (64, 8, 1000, 1, 2, "perm"), (64, 8, 1003, 1, 2, "uniform"), (128, 4, 701, 1, 3, "uniform"),
    (8, 8, 2100, 1, 1, "uniform"), (128, 8, 1100, 1, 1, "perm"), (32, 16, 1500, 2, 1, "uniform")])
def test_segmented_scan(N, chunk, L, B, H, pi_kind):
    """Few long sequences run cut into segments along L (an aggregate pass,
    then one workgroup per segment); results match the oracle like the
    unsegmented scan, including the saved chunk states, h_final and dh0."""
    d = pdssm.desc(B, L, H, N, 5, chunk)
    assert pdssm.scan_segments(d) > 1
    inp = make_inputs(B=B, L=L, H=H, N=N, K=5, seed=L + N, pi_kind=pi_kind, with_h0=True,
                      with_dhf=True)
    got = run_gpu(inp, chunk=chunk)
    check_all(inp, got, chunk)


def _guarded(shape, dtype, pad=4096):
    """An output tensor inside a larger buffer whose margins hold a marker."""
    n = int(np.prod(shape))
    buf = torch.full((n + 2 * pad,), 7.25, dtype=dtype, device=DEV)
    return buf, buf[pad:pad + n].view(shape), pad


def _margins_intact(buf, pad):
    m = torch.cat([buf[:pad], buf[-pad:]])
    return bool((m == 7.25).all())


@pytest.mark.parametrize("N,K,L,chunk", [(64, 16, 77, 8), (64, 16, 75, 16), (128, 64, 77, 4),
                                         (128, 128, 77, 0), (256, 8, 43, 4), (8, 4, 13, 8)])
def test_outputs_stay_inside_their_tensors(N, K, L, chunk):
    """Every output is written inside its own tensor: with ragged last chunks
    (padded steps) the bytes around each output stay untouched, and the
    values match the oracle."""
    import ctypes
    B, H = 2, 3
    inp = make_inputs(B=B, L=L, H=H, N=N, K=K, seed=L + N, with_h0=True, with_dhf=True)
    T = to_dev(inp)
    lib = pdssm.load()
    d = pdssm.desc(B, L, H, N, K, chunk)
    C = pdssm.num_chunks(d)
    ws = torch.empty(max(pdssm.workspace_size(d, pdssm.OP_FWD), 1), dtype=torch.uint8, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    outs = {"y": _guarded((B, L, H), torch.float32), "h_final": _guarded((B, H, N), torch.complex64),
            "saved": _guarded((B, H, C, N), torch.complex64),
            "dD": _guarded((B, L, H, N), torch.complex64), "db": _guarded((B, L, H, N), torch.complex64),
            "dc": _guarded((B, L, H, N), torch.complex64), "dh0": _guarded((B, H, N), torch.complex64)}
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    o = {k: v[1] for k, v in outs.items()}
    rc = lib.pdssm_scan_fwd(ctypes.byref(d), P(T["idx"]), P(T["pi"]), P(T["D"]), P(T["b"]), P(T["c"]),
                            P(T["h0"]), P(o["y"]), P(o["h_final"]), P(o["saved"]), P(ws), ws.numel(),
                            P(status), st)
    assert rc == 0
    rc = lib.pdssm_scan_bwd(ctypes.byref(d), P(T["idx"]), P(T["pi"]), P(T["D"]), P(T["b"]), P(T["c"]),
                            P(o["saved"]), P(T["dy"]), P(T["dh_final"]), P(o["dD"]), P(o["db"]),
                            P(o["dc"]), P(o["dh0"]), P(ws), ws.numel(), P(status), st)
    assert rc == 0
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for k, (buf, _, pad) in outs.items():
        assert _margins_intact(buf, pad), k
    got = {k: v.cpu().numpy() for k, v in o.items()}
    check_all(inp, got, pdssm.chunk_len(d))


def test_out_of_range_indices_flagged_not_faulting():
    inp = make_inputs(B=1, L=40, H=2, N=64, K=4, seed=9)
    bad = dict(inp)
    bad["idx"] = inp["idx"].copy()
    bad["idx"][0, 5, 1] = 4
    T = to_dev(bad)
    with pytest.raises(pdssm.PdssmError) as e:
        pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"])
    assert e.value.status == pdssm.ERR_INDEX
    bad = dict(inp)
    bad["pi"] = inp["pi"].copy()
    bad["pi"][1, 2, 3] = 64
    T = to_dev(bad)
    with pytest.raises(pdssm.PdssmError):
        pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"])
    # the untouched head is still right
    y, _, _ = pdssm.scan_fwd(*(to_dev(inp)[k] for k in ("idx", "pi", "D", "b", "c")))
    ry, _, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"])
    assert_close("y", y.cpu().numpy(), ry)


# ------------------------------------------------------------------ the named workloads
_cache = {}


def workload(i):
    if i not in _cache:
        _cache.clear()
        _cache[i] = workload_inputs(i, seed=0)
    return _cache[i]


def test_workload1_tiny_full():
    inp = workload(1)
    got = run_gpu(inp, bwd=False)
    ry, rhf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"])
    assert_close("y", got["y"], ry)
    assert_close("h_final", got["h_final"], rhf)


@pytest.mark.parametrize("wi", [2, 3, 4, 5])
def test_workload_full_size_every_sequence(wi):
    """Full-size run in the benchmark's launch configuration (prepared
    tables, the same chunk and segments); every sequence is checked against
    the oracle on its own (a pool of host threads runs the float64 oracle one
    sequence per task): y, h_final, saved states, dD, db, dc and dh0."""
    from concurrent.futures import ThreadPoolExecutor

    w = WORKLOADS[wi]
    print("workload %d: %s" % (wi, w.name), flush=True)
    inp = workload(wi)
    s = pdssm.Scan(w.B, w.L, w.H, w.N, w.K)
    T = to_dev(inp)
    s.prepare(T["pi"])
    s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"])
    s.bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"])
    s.check_status()
    del T
    host = {k: getattr(s, k).cpu().numpy() for k in ("y", "h_final", "saved", "dD", "db", "dc", "dh0")}
    del s
    print("workload %d: outputs on the host, checking %d sequences" % (wi, w.B * w.H), flush=True)

    def one(bh):
        bb, hh = bh
        sub = sub_sequence(inp, bb, hh)
        got = dict(y=host["y"][bb:bb + 1, :, hh:hh + 1], h_final=host["h_final"][bb:bb + 1, hh:hh + 1],
                   saved=host["saved"][bb:bb + 1, hh:hh + 1], dD=host["dD"][bb:bb + 1, :, hh:hh + 1],
                   db=host["db"][bb:bb + 1, :, hh:hh + 1], dc=host["dc"][bb:bb + 1, :, hh:hh + 1],
                   dh0=host["dh0"][bb:bb + 1, hh:hh + 1])
        try:
            check_all(sub, got, pdssm.chunk_len(pdssm.desc(w.B, w.L, w.H, w.N, w.K)))
        except AssertionError as e:
            return "sequence (b=%d, h=%d): %s" % (bb, hh, e)
        return None

    with ThreadPoolExecutor(max_workers=16) as pool:
        errs = [e for e in pool.map(one, [(bb, hh) for bb in range(w.B) for hh in range(w.H)]) if e]
    assert not errs, "%d sequences differ; first: %s" % (len(errs), errs[0])
