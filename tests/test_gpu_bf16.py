"""GPU parity of the bf16 input/output setting (PDSSM_FLAG_BF16_IO): D, b, c
and dD, db, dc as bf16 (re, im) pairs, fp32 arithmetic.

Two checks per case:
  - against the float64 oracle on the same (bf16-representable) inputs:
    y, h_final and the saved states to the scan's bar (|gpu - ref| <=
    1e-5 + 1e-4*|ref|; the inputs are exact); the gradients, rounded to bf16
    when stored, to 1e-5 + (2^-8 + 1e-4)*|ref| (round to nearest moves a value
    by at most half a bf16 spacing, 2^-8 of its size);
  - against the fp32 path on the same inputs: bit for bit (same arithmetic;
    the bf16 gradients are the fp32 gradients rounded to nearest even).
"""
import numpy as np
import pytest

from helpers import assert_close, sub_sequence
from oracle import oracle_bwd, oracle_fwd
from paper_2605_19150_amd.inputs import make_inputs, workload_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_19150_amd import pdssm  # noqa: E402

DEV = torch.device("cuda:0")
BF_RTOL = 2.0 ** -8 + 1e-4


def to_bf16_pairs(a):
    """complex64 numpy -> (bf16 pairs [..., 2] on the GPU, the exact complex128 values)."""
    t = torch.view_as_real(torch.from_numpy(np.ascontiguousarray(a, np.complex64))).to(torch.bfloat16)
    exact = t.to(torch.float64).numpy()
    return t.contiguous().to(DEV), exact[..., 0] + 1j * exact[..., 1]


def pairs_to_complex(t):
    f = t.to(torch.float64).cpu().numpy()
    return f[..., 0] + 1j * f[..., 1]


def rne_bf16(t):
    """fp32 complex64 GPU tensor -> bf16 pairs, rounded to nearest even (torch's cast)."""
    return torch.view_as_real(t).to(torch.bfloat16)


def run_both(inp, chunk=0):
    """The bf16 path and the fp32 path on the same bf16-representable inputs."""
    B, L, H = inp["idx"].shape
    _, K, N = inp["pi"].shape
    pairs, exact = {}, {}
    for k in ("D", "b", "c"):
        pairs[k], exact[k] = to_bf16_pairs(inp[k])
    cplx = {k: torch.from_numpy(exact[k].astype(np.complex64)).to(DEV) for k in ("D", "b", "c")}
    idx, pi = torch.from_numpy(inp["idx"]).to(DEV), torch.from_numpy(inp["pi"]).to(DEV)
    h0 = torch.from_numpy(inp["h0"]).to(DEV) if "h0" in inp else None
    dy = torch.from_numpy(inp["dy"]).to(DEV)
    dhf = torch.from_numpy(inp["dh_final"]).to(DEV) if "dh_final" in inp else None
    out = {}
    for tag, T, bf in (("bf", pairs, True), ("f32", cplx, False)):
        s = pdssm.Scan(B, L, H, N, K, chunk, DEV, bf16=bf)
        s.fwd(idx, pi, T["D"], T["b"], T["c"], h0=h0)
        s.bwd(idx, pi, T["D"], T["b"], T["c"], dy, dh_final=dhf)
        s.check_status()
        out[tag] = {k: getattr(s, k).clone() for k in ("y", "h_final", "saved", "dD", "db", "dc", "dh0")}
        out[tag]["chunk"] = s.chunk
    return exact, out


def check(inp, exact, out):
    bf, f32 = out["bf"], out["f32"]
    for k in ("y", "h_final", "saved", "dh0"):
        np.testing.assert_array_equal(bf[k].cpu().numpy(), f32[k].cpu().numpy(), err_msg=k)
    for k in ("dD", "db", "dc"):
        assert torch.equal(bf[k], rne_bf16(f32[k])), k
    ry, rhf, rsaved = oracle_fwd(inp["idx"], inp["pi"], exact["D"], exact["b"], exact["c"], h0=inp.get("h0"),
                                 chunk=bf["chunk"])
    assert_close("y", bf["y"].cpu().numpy(), ry)
    assert_close("h_final", bf["h_final"].cpu().numpy(), rhf)
    assert_close("saved", bf["saved"].cpu().numpy(), rsaved)
    rg = oracle_bwd(inp["idx"], inp["pi"], exact["D"], exact["b"], exact["c"], inp["dy"], h0=inp.get("h0"),
                    dh_final=inp.get("dh_final"))
    for k, r in zip(("dD", "db", "dc"), rg[:3]):
        assert_close(k, pairs_to_complex(bf[k]), r, rtol=BF_RTOL)
    assert_close("dh0", bf["dh0"].cpu().numpy(), rg[3])


CASES = []
for N in (8, 16, 32, 64, 128, 256):
    for chunk in (4, 8, 16):
        if chunk * max(1, N // 64) > 16:
            continue
        CASES.append((N, chunk, 3 * chunk + 5))
CASES += [(64, 8, 1), (64, 8, 261), (128, 8, 133)]


@pytest.mark.parametrize("N,chunk,L", CASES)
def test_bf16_io_small(N, chunk, L):
    print("bf16 case N=%d chunk=%d L=%d" % (N, chunk, L), flush=True)
    inp = make_inputs(B=2, L=L, H=3, N=N, K=5, seed=N * 31 + chunk + L, with_h0=True, with_dhf=True)
    # (N = 256 runs the multi-pass kernels: tables beyond LDS)
    exact, out = run_both(inp, chunk)
    check(inp, exact, out)


def test_bf16_io_segmented():
    inp = make_inputs(B=1, L=2600, H=2, N=64, K=16, seed=5, pi_kind="perm", with_h0=True, with_dhf=True)
    assert pdssm.scan_segments(pdssm.desc(1, 2600, 2, 64, 16)) > 1
    exact, out = run_both(inp)
    check(inp, exact, out)


@pytest.mark.parametrize("wl", [2, 3])
def test_bf16_io_full_size(wl):
    inp = workload_inputs(wl, seed=0)
    print("bf16 full size workload %d" % wl, flush=True)
    exact, out = run_both(inp)
    bf, f32 = out["bf"], out["f32"]
    for k in ("y", "h_final", "saved"):
        assert torch.equal(bf[k], f32[k]), k
    for k in ("dD", "db", "dc"):
        assert torch.equal(bf[k], rne_bf16(f32[k])), k
    for bb, hh in ((0, 0), (15, 15), (9, 4)):
        sub = sub_sequence(inp, bb, hh)
        for k in ("D", "b", "c"):
            sub[k] = np.ascontiguousarray(exact[k][bb:bb + 1, :, hh:hh + 1])
        ry, rhf, _ = oracle_fwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"])
        assert_close("y", bf["y"][bb:bb + 1, :, hh:hh + 1].cpu().numpy(), ry)
        rg = oracle_bwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"], sub["dy"])
        for k, r in zip(("dD", "db", "dc"), rg[:3]):
            assert_close(k, pairs_to_complex(bf[k][bb:bb + 1, :, hh:hh + 1]), r, rtol=BF_RTOL)


def test_bf16_io_multi_pass_large_dictionary():
    inp = make_inputs(B=2, L=70, H=2, N=128, K=128, seed=4, with_h0=True, with_dhf=True)
    import ctypes
    assert pdssm.load().pdssm_uses_fused(ctypes.byref(pdssm.desc(2, 70, 2, 128, 128))) == 0
    exact, out = run_both(inp)
    check(inp, exact, out)


@pytest.mark.parametrize("N,K,L", [(64, 16, 300), (128, 32, 200), (32, 5, 77)])
def test_bf16_ste(N, K, L):
    """The straight-through pair with bf16 pairs: z stays complex64 and equals
    the fp32 path's bit for bit; db is its bf16 rounding; q and G from the
    bf16 db equal the complex64 ste_grads on the widened db bit for bit, and
    the oracle's (from the unrounded gradient) within the bf16 rounding."""
    from helpers import assert_close_sum, ste_scales
    from oracle import oracle_bwd, oracle_ste
    print("bf16 ste N=%d K=%d L=%d" % (N, K, L), flush=True)
    B, H = 2, 3
    inp = make_inputs(B, L, H, N, K, seed=N + K + L, with_h0=True, with_dhf=True)
    pairs, exact = {}, {}
    for k in ("D", "b", "c"):
        pairs[k], exact[k] = to_bf16_pairs(inp[k])
    cplx = {k: torch.from_numpy(exact[k].astype(np.complex64)).to(DEV) for k in ("D", "b", "c")}
    idx, pi = torch.from_numpy(inp["idx"]).to(DEV), torch.from_numpy(inp["pi"]).to(DEV)
    h0, dhf = torch.from_numpy(inp["h0"]).to(DEV), torch.from_numpy(inp["dh_final"]).to(DEV)
    dy = torch.from_numpy(inp["dy"]).to(DEV)
    out = {}
    for tag, T, bf in (("bf", pairs, True), ("f32", cplx, False)):
        s = pdssm.Scan(B, L, H, N, K, 0, DEV, ste=True, bf16=bf)
        s.fwd(idx, pi, T["D"], T["b"], T["c"], h0=h0)
        s.bwd_ste(idx, pi, T["D"], T["b"], T["c"], dy, dh_final=dhf)
        s.ste_grads(idx, pi)
        s.check_status()
        out[tag] = {k: getattr(s, k).clone() for k in ("db", "z", "q", "G")}
        del s
    bf, f32 = out["bf"], out["f32"]
    assert bf["z"].dtype == torch.complex64
    assert torch.equal(bf["z"], f32["z"])
    assert torch.equal(bf["db"], rne_bf16(f32["db"]))
    g_wide = torch.view_as_complex(bf["db"].to(torch.float32).contiguous())
    q2, G2 = pdssm.ste_grads(idx, pi, g_wide, bf["z"])
    assert torch.equal(bf["q"], q2) and torch.equal(bf["G"], G2)
    q3, G3 = pdssm.ste_grads(idx, pi, bf["db"], bf["z"])  # module function, bf16 g
    assert torch.equal(bf["q"], q3) and torch.equal(bf["G"], G3)
    rg = oracle_bwd(inp["idx"], inp["pi"], exact["D"], exact["b"], exact["c"], inp["dy"], h0=inp["h0"],
                    dh_final=inp["dh_final"])
    q, G, z = oracle_ste(inp["idx"], inp["pi"], exact["D"], exact["b"], exact["c"], inp["dy"], h0=inp["h0"],
                         dh_final=inp["dh_final"], want_z=True)
    assert_close("z", bf["z"].cpu().numpy(), np.asarray(z))
    qs, Gs = ste_scales(inp["pi"], inp["idx"], rg[1], z)
    assert_close_sum("q", bf["q"].cpu().numpy(), q, qs, rtol=BF_RTOL)
    assert_close_sum("G", bf["G"].cpu().numpy(), G, Gs, rtol=BF_RTOL)
