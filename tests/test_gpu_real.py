"""GPU parity of the real-valued model (PDSSM_FLAG_REAL_IO): D, b, c and dD,
db, dc as real fp32 rows, h0 / dh_final real values held as complex64.

Two checks per case:
  - against the float64 oracle on the same inputs: y, h_final, the saved
    states and every gradient to the scan's bar |gpu - ref| <= 1e-5 +
    1e-4*|ref| (the real model is the complex one restricted to real rows);
  - against the complex64 path on the same values (imaginary parts 0): bit
    for bit, the real path's saved states (fp32) and gradients equal the
    complex path's real parts and the complex path's imaginary parts are 0.
"""
import ctypes

import numpy as np
import pytest

from helpers import assert_close, assert_close_sum, force_sorted_entries, ste_scales, sub_sequence
from oracle import oracle_bwd, oracle_fwd, oracle_ste
from paper_2605_19150_amd.inputs import make_inputs, workload_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_19150_amd import pdssm  # noqa: E402

DEV = torch.device("cuda:0")


def run_both(inp, chunk=0):
    """The real path and the complex64 path on the same real values."""
    B, L, H = inp["idx"].shape
    _, K, N = inp["pi"].shape
    real = {k: torch.from_numpy(inp[k]).to(DEV) for k in ("D", "b", "c")}
    cplx = {k: v.to(torch.complex64) for k, v in real.items()}
    idx, pi = torch.from_numpy(inp["idx"]).to(DEV), torch.from_numpy(inp["pi"]).to(DEV)
    h0 = torch.from_numpy(inp["h0"]).to(DEV) if "h0" in inp else None
    dy = torch.from_numpy(inp["dy"]).to(DEV)
    dhf = torch.from_numpy(inp["dh_final"]).to(DEV) if "dh_final" in inp else None
    out = {}
    for tag, T, re in (("real", real, True), ("c64", cplx, False)):
        s = pdssm.Scan(B, L, H, N, K, chunk, DEV, real=re)
        s.fwd(idx, pi, T["D"], T["b"], T["c"], h0=h0)
        s.bwd(idx, pi, T["D"], T["b"], T["c"], dy, dh_final=dhf)
        s.check_status()
        out[tag] = {k: getattr(s, k).clone() for k in ("y", "h_final", "saved", "dD", "db", "dc", "dh0")}
        out[tag]["chunk"] = s.chunk
        del s
    return out


def check_bits(out):
    r, c = out["real"], out["c64"]
    for k in ("y", "h_final", "dh0"):
        assert torch.equal(r[k], c[k]), k
    for k in ("h_final", "dh0"):
        assert bool((r[k].imag == 0).all()), k
    for k in ("saved", "dD", "db", "dc"):
        assert r[k].dtype == torch.float32
        assert torch.equal(r[k], c[k].real), k
        assert bool((c[k].imag == 0).all()), k


def check_oracle(inp, out):
    r = out["real"]
    ry, rhf, rsaved = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp.get("h0"),
                                 chunk=r["chunk"])
    assert_close("y", r["y"].cpu().numpy(), ry)
    assert_close("h_final", r["h_final"].cpu().numpy(), rhf)
    assert np.all(rsaved.imag == 0)
    assert_close("saved", r["saved"].cpu().numpy(), rsaved.real)
    rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp.get("h0"),
                    dh_final=inp.get("dh_final"))
    for k, g in zip(("dD", "db", "dc"), rg[:3]):
        assert np.all(g.imag == 0), k
        assert_close(k, r[k].cpu().numpy(), g.real)
    assert_close("dh0", r["dh0"].cpu().numpy(), rg[3])


CASES = []
for N in (8, 16, 32, 64, 128, 256):
    for chunk in (4, 8, 16):
        if chunk * max(1, N // 64) > 16:
            continue
        CASES.append((N, chunk, 3 * chunk + 5))
CASES += [(64, 8, 1), (64, 8, 261), (128, 8, 133)]


@pytest.mark.parametrize("N,chunk,L", CASES)
def test_real_io_small(N, chunk, L):
    print("real case N=%d chunk=%d L=%d" % (N, chunk, L), flush=True)
    inp = make_inputs(B=2, L=L, H=3, N=N, K=5, seed=N * 37 + chunk + L, with_h0=True, with_dhf=True, real=True)
    # (N = 256 runs the multi-pass kernels: tables beyond LDS)
    out = run_both(inp, chunk)
    check_bits(out)
    check_oracle(inp, out)


def test_real_io_collisions():
    # all-to-one maps in one head (the atomic-scatter entries) and random maps in the other
    inp = make_inputs(B=2, L=45, H=2, N=64, K=4, seed=11, with_h0=True, with_dhf=True, real=True)
    inp["pi"][0] = 0
    out = run_both(inp, 8)
    check_bits(out)
    check_oracle(inp, out)


@pytest.mark.parametrize("N,B,L", [(64, 2, 300), (128, 2, 300), (64, 1, 2600), (128, 1, 2600)])
def test_real_io_sorted_form_mixed(N, B, L):
    """Heads with sorted-form entries (rows of more than seven sources) next
    to ordinary ones: with real elements their chunks take the pipelined pass
    when no step uses such an entry and the step-by-step pass otherwise
    (head 2 mixes both), also in the aggregate pass of segmented scans
    (L = 2600).  Bit for bit the complex64 path, and the oracle."""
    print("real sorted form N=%d B=%d L=%d" % (N, B, L), flush=True)
    inp = make_inputs(B=B, L=L, H=3, N=N, K=8, seed=N + L, with_h0=True, with_dhf=True, real=True)
    force_sorted_entries(inp, N)
    out = run_both(inp)
    check_bits(out)
    check_oracle(inp, out)


def test_real_io_segmented():
    inp = make_inputs(B=1, L=2600, H=2, N=64, K=16, seed=5, pi_kind="perm", with_h0=True, with_dhf=True,
                      real=True)
    assert pdssm.scan_segments(pdssm.desc(1, 2600, 2, 64, 16)) > 1
    out = run_both(inp)
    check_bits(out)
    check_oracle(inp, out)


def test_real_io_module_functions():
    # scan_fwd / scan_bwd pick the real format from D's dtype and widen a real h0
    inp = make_inputs(B=2, L=37, H=2, N=32, K=3, seed=9, with_h0=True, with_dhf=True, real=True)
    T = {k: torch.from_numpy(np.ascontiguousarray(inp[k])).to(DEV) for k in ("idx", "pi", "D", "b", "c", "dy")}
    h0r = torch.from_numpy(np.ascontiguousarray(inp["h0"].real)).to(DEV)
    dhfr = torch.from_numpy(np.ascontiguousarray(inp["dh_final"].real)).to(DEV)
    y, hf, saved = pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=h0r)
    dD, db, dc, dh0 = pdssm.scan_bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], saved, T["dy"], dh_final=dhfr)
    assert dD.dtype == torch.float32 and dD.shape == T["D"].shape
    ry, rhf, _ = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"])
    assert_close("y", y.cpu().numpy(), ry)
    assert_close("h_final", hf.cpu().numpy(), rhf)
    rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                    dh_final=inp["dh_final"])
    for k, v, g in zip(("dD", "db", "dc"), (dD, db, dc), rg[:3]):
        assert_close(k, v.cpu().numpy(), g.real)
    assert_close("dh0", dh0.cpu().numpy(), rg[3])


# the head of markov-manyone and hybrid-lm with an entry of in-degree > 7
SORTED_HEAD = {3: 4, 5: 18}


def test_real_io_saved_fp32_through_every_entry():
    """The real model's saved states are fp32 [B,H,C,N]: scan_fwd and
    scan_fwd_noalloc (the library's own workspace) give the same bits, on a
    single-read head mix and on a segmented sequence, and scan_bwd reads them
    back."""
    for B, L, H, N, K, seed in ((3, 150, 2, 64, 9, 21), (1, 2600, 1, 128, 8, 22)):
        print("real saved: B%d L%d H%d N%d K%d" % (B, L, H, N, K), flush=True)
        inp = make_inputs(B=B, L=L, H=H, N=N, K=K, seed=seed, with_h0=True, real=True)
        T = {k: torch.from_numpy(np.ascontiguousarray(inp[k])).to(DEV) for k in ("idx", "pi", "D", "b", "c", "dy")}
        h0r = torch.from_numpy(np.ascontiguousarray(inp["h0"].real)).to(DEV)
        y0, h0, s0 = (x.clone() for x in pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=h0r))
        y1, h1, s1 = pdssm.scan_fwd_noalloc(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=h0r)
        torch.cuda.synchronize()
        assert s0.dtype == torch.float32 and s1.dtype == torch.float32
        assert torch.equal(y0, y1) and torch.equal(h0, h1) and torch.equal(s0, s1)
        tau = pdssm.chunk_len(pdssm.desc(B, L, H, N, K))
        _, _, rsaved = oracle_fwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], h0=inp["h0"], chunk=tau)
        assert_close("saved", s0.cpu().numpy(), rsaved.real)
        g = pdssm.scan_bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], s1, T["dy"])
        rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"])
        for k, v, r in zip(("dD", "db", "dc"), g[:3], rg[:3]):
            assert_close(k, v.cpu().numpy(), r.real)


@pytest.mark.parametrize("wl", [2, 3, 4, 5])
def test_real_io_full_size(wl):
    """Every output of the full-size workload bit for bit against complex64;
    sampled sequences (including the head with a sorted-form entry) against
    the oracle."""
    print("real full size workload %d" % wl, flush=True)
    inp = workload_inputs(wl, seed=0, real=True)
    out = run_both(inp)
    check_bits(out)
    r = out["real"]
    B, L, H = inp["idx"].shape
    samples = [(0, 0), (B - 1, H - 1), (B // 2, H // 3)]
    if wl in SORTED_HEAD:
        samples.append((1, SORTED_HEAD[wl]))
    for bb, hh in samples:
        sub = sub_sequence(inp, bb, hh)
        ry, rhf, _ = oracle_fwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"])
        assert_close("y", r["y"][bb:bb + 1, :, hh:hh + 1].cpu().numpy(), ry)
        assert_close("h_final", r["h_final"][bb:bb + 1, hh:hh + 1].cpu().numpy(), rhf)
        rg = oracle_bwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"], sub["dy"])
        for k, g in zip(("dD", "db", "dc"), rg[:3]):
            assert_close(k, r[k][bb:bb + 1, :, hh:hh + 1].cpu().numpy(), g.real)


# (N, K, B, L, H, chunk)
STE_CASES = [(8, 5, 2, 37, 3, 4), (32, 7, 2, 45, 2, 16), (64, 16, 2, 263, 3, 8), (128, 9, 2, 80, 2, 8),
             (64, 16, 1, 1100, 1, 8),
             (256, 5, 1, 40, 2, 4),      # multi-pass scan (tables beyond LDS)
             (128, 128, 1, 30, 1, 8)]    # multi-pass scan, large dictionary


def test_real_multi_pass_large_dictionary():
    inp = make_inputs(B=2, L=70, H=2, N=128, K=128, seed=3, with_h0=True, with_dhf=True, real=True)
    assert pdssm.load().pdssm_uses_fused(ctypes.byref(pdssm.desc(2, 70, 2, 128, 128))) == 0
    out = run_both(inp)
    check_bits(out)
    check_oracle(inp, out)


@pytest.mark.parametrize("N,K,B,L,H,chunk", STE_CASES)
def test_real_ste(N, K, B, L, H, chunk):
    """Straight-through inputs of the real-valued model (real z and g = db,
    scores q, dictionary gradient G): bit for bit the complex64 path on the
    same values, and the oracle."""
    print("real ste N=%d K=%d L=%d" % (N, K, L), flush=True)
    inp = make_inputs(B, L, H, N, K, seed=N * 3 + K + L, with_h0=True, with_dhf=True, real=True)
    idx, pi = torch.from_numpy(inp["idx"]).to(DEV), torch.from_numpy(inp["pi"]).to(DEV)
    h0, dhf = torch.from_numpy(inp["h0"]).to(DEV), torch.from_numpy(inp["dh_final"]).to(DEV)
    dy = torch.from_numpy(inp["dy"]).to(DEV)
    real = {k: torch.from_numpy(inp[k]).to(DEV) for k in ("D", "b", "c")}
    out = {}
    for tag, re in (("real", True), ("c64", False)):
        T = real if re else {k: v.to(torch.complex64) for k, v in real.items()}
        s = pdssm.Scan(B, L, H, N, K, chunk, DEV, ste=True, real=re)
        s.fwd(idx, pi, T["D"], T["b"], T["c"], h0=h0)
        s.bwd_ste(idx, pi, T["D"], T["b"], T["c"], dy, dh_final=dhf)
        s.ste_grads(idx, pi)
        s.check_status()
        out[tag] = {k: getattr(s, k).clone() for k in ("db", "z", "q", "G")}
        del s
    r, c = out["real"], out["c64"]
    assert r["z"].dtype == torch.float32
    for k in ("db", "z"):
        assert torch.equal(r[k], c[k].real), k
    for k in ("q", "G"):
        assert torch.equal(r[k], c[k]), k
    rg = oracle_bwd(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                    dh_final=inp["dh_final"])
    q, G, z = oracle_ste(inp["idx"], inp["pi"], inp["D"], inp["b"], inp["c"], inp["dy"], h0=inp["h0"],
                         dh_final=inp["dh_final"], want_z=True)
    assert_close("z", r["z"].cpu().numpy(), np.asarray(z).real)
    qs, Gs = ste_scales(inp["pi"], inp["idx"], rg[1], z)
    assert_close_sum("q", r["q"].cpu().numpy(), q, qs)
    assert_close_sum("G", r["G"].cpu().numpy(), G, Gs)
    # the module functions take real g and z
    q2, G2 = pdssm.ste_grads(idx, pi, r["db"], r["z"])
    assert torch.equal(q2, r["q"]) and torch.equal(G2, r["G"])


@pytest.mark.parametrize("wl", [2, 4])
def test_real_ste_full_size_matches_complex(wl):
    """Full-size fsa-perm (N=64) and timeseries (N=128, segmented) with real
    rows: the straight-through outputs (fp32 score tiles, the two-block
    K=1 products) equal the complex64 path's on the same values bit for bit."""
    print("real ste full size workload %d" % wl, flush=True)
    inp = workload_inputs(wl, seed=0, real=True)
    B, L, H = inp["idx"].shape
    _, K, N = inp["pi"].shape
    idx, pi = torch.from_numpy(inp["idx"]).to(DEV), torch.from_numpy(inp["pi"]).to(DEV)
    dy = torch.from_numpy(inp["dy"]).to(DEV)
    real = {k: torch.from_numpy(inp[k]).to(DEV) for k in ("D", "b", "c")}
    out = {}
    for tag, re in (("real", True), ("c64", False)):
        T = real if re else {k: v.to(torch.complex64) for k, v in real.items()}
        s = pdssm.Scan(B, L, H, N, K, 0, DEV, ste=True, real=re)
        s.fwd(idx, pi, T["D"], T["b"], T["c"])
        s.bwd_ste(idx, pi, T["D"], T["b"], T["c"], dy)
        s.ste_grads(idx, pi)
        s.check_status()
        out[tag] = {k: getattr(s, k).clone() for k in ("db", "z", "q", "G")}
        del s
        torch.cuda.empty_cache()
    r, c = out["real"], out["c64"]
    for k in ("db", "z"):
        assert torch.equal(r[k], c[k].real), k
    for k in ("q", "G"):
        assert bool(torch.isfinite(r[k]).all()), k
        assert torch.equal(r[k], c[k]), k
