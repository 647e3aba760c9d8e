"""GPU: pdssm_scan_fwd_noalloc (the forward with the library's own device
workspace) against pdssm_scan_fwd on the same inputs: the same kernels, so
y, h_final and the saved states agree bit for bit.  Two calls in a row, the
second on a smaller input (the array keeps the first call's contents), a
segmented sequence (segment aggregates in the array), and the host-side
rejections (a workspace beyond the array, prepared tables)."""
import ctypes

import numpy as np
import pytest

from paper_2605_19150_amd.inputs import make_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_19150_amd import pdssm  # noqa: E402

DEV = torch.device("cuda:0")


def _dev(inp):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(DEV) for k, v in inp.items()}


def _noalloc_call(T, chunk=0):
    """pdssm_scan_fwd_noalloc through the C ABI, outputs allocated here."""
    B, L, H = T["idx"].shape
    _, K, N = T["pi"].shape
    d = pdssm.desc(B, L, H, N, K, chunk)
    C = pdssm.num_chunks(d)
    y = torch.full((B, L, H), float("nan"), dtype=torch.float32, device=DEV)
    hf = torch.full((B, H, N), float("nan"), dtype=torch.complex64, device=DEV)
    sv = torch.full((B, H, C, N), float("nan"), dtype=torch.complex64, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    P = pdssm._p
    rc = pdssm.load().pdssm_scan_fwd_noalloc(ctypes.byref(d), P(T["idx"]), P(T["pi"]), P(T["D"]), P(T["b"]),
                                             P(T["c"]), P(T.get("h0")), P(y), P(hf), P(sv), P(status),
                                             pdssm._stream(None))
    assert rc == pdssm.OK, pdssm.status_string(rc)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    return y, hf, sv


def _check_same(T, chunk=0):
    y0, h0, s0 = pdssm.scan_fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], h0=T.get("h0"), chunk=chunk)
    y0, h0, s0 = y0.clone(), h0.clone(), s0.clone()
    y1, h1, s1 = _noalloc_call(T, chunk)
    assert torch.equal(y0, y1)
    assert torch.equal(h0, h1)
    assert torch.equal(s0, s1)


def test_noalloc_matches_scan_fwd_twice_second_smaller():
    print("noalloc: B4 L700 H6 N64 K16 then B2 L90 H3 N64 K5", flush=True)
    big = make_inputs(B=4, L=700, H=6, N=64, K=16, seed=1, with_h0=True)
    big["pi"][2, 3, :10] = 7  # a sorted-form entry
    _check_same(_dev(big))
    small = make_inputs(B=2, L=90, H=3, N=64, K=5, seed=2, pi_kind="perm")
    _check_same(_dev(small))


def test_noalloc_segmented_then_smaller_other_size():
    print("noalloc: segmented B1 L3000 H2 N128 K32 then B3 L50 H2 N32 K7", flush=True)
    d = pdssm.desc(1, 3000, 2, 128, 32)
    assert pdssm.scan_segments(d) > 1
    inp = make_inputs(B=1, L=3000, H=2, N=128, K=32, seed=3, with_h0=True)
    _check_same(_dev(inp))
    inp = make_inputs(B=3, L=50, H=2, N=32, K=7, seed=4)
    _check_same(_dev(inp), chunk=16)


def test_noalloc_host_rejections():
    lib = pdssm.load()
    P = ctypes.c_void_p
    fake = lambda n: P((1 << 40) + n * (1 << 30))  # noqa: E731  (never dereferenced)
    d = pdssm.desc(2, 40, 2, 64, 4)
    d.flags = pdssm.FLAG_PREPARED
    args = [fake(i) for i in range(6)] + [None, fake(7), fake(8), fake(9), None, None]
    assert lib.pdssm_scan_fwd_noalloc(ctypes.byref(d), *args[:6], *args[6:]) == pdssm.ERR_INVALID_ARG
    # tables of 256 entries of N = 256 for 64 heads: beyond the array
    big = pdssm.desc(1, 64, 64, 256, 256)
    assert pdssm.workspace_size(big, pdssm.OP_FWD) > (16 << 20)
    assert lib.pdssm_scan_fwd_noalloc(ctypes.byref(big), *args[:6], *args[6:]) == pdssm.ERR_WORKSPACE
    bad = pdssm.desc(2, 40, 2, 48, 4)
    assert lib.pdssm_scan_fwd_noalloc(ctypes.byref(bad), *args[:6], *args[6:]) == pdssm.ERR_UNSUPPORTED
