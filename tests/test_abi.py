"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/pdssm.h declares, and rejects bad arguments before any
HIP call is made."""
import ctypes
import os
import re

import pytest

from paper_2605_19150_amd import pdssm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "pdssm.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pdssm_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pdssm.lib_path()):
        from paper_2605_19150_amd.build import build_library
        build_library()
    return pdssm.load()


def test_exports_every_declared_function(lib):
    names = header_functions()
    assert "pdssm_scan_fwd" in names and "pdssm_scan_bwd" in names and "pdssm_compose_chunks" in names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) <= set(pdssm.EXPORTS) | set(names)
    assert lib.pdssm_abi_version() == 1


def test_chunk_and_workspace_queries(lib):
    d = pdssm.desc(16, 2048, 16, 64, 16)
    assert pdssm.chunk_len(d) == 8
    assert pdssm.num_chunks(d) == 256
    assert pdssm.num_chunks(pdssm.desc(16, 2048, 16, 64, 16, chunk=16)) == 128
    d = pdssm.desc(8, 18000, 8, 128, 32)
    assert pdssm.chunk_len(d) == 8
    assert pdssm.num_chunks(d) == 2250
    assert pdssm.num_chunks(pdssm.desc(8, 18000, 8, 128, 32, chunk=4)) == 4500
    assert pdssm.num_chunks(pdssm.desc(8, 18000, 8, 128, 32, chunk=16)) == pdssm.ERR_UNSUPPORTED
    assert pdssm.chunk_len(pdssm.desc(1, 10, 1, 256, 4)) == 4
    assert pdssm.chunk_len(pdssm.desc(1, 10, 1, 128, 4)) == 8
    for op in (pdssm.OP_FWD, pdssm.OP_BWD):
        n = pdssm.workspace_size(d, op)
        assert n >= 8 * 32 * 128 * 9  # dictionary tables of the fused path
    assert pdssm.workspace_size(d, pdssm.OP_COMPOSE) == 0
    d = pdssm.desc(1, 1, 1, 8, 1)
    assert pdssm.num_chunks(d) == 1
    # few long sequences are cut into segments; many sequences are not
    assert pdssm.scan_segments(pdssm.desc(8, 18000, 8, 128, 32)) == 4
    assert pdssm.scan_segments(pdssm.desc(16, 2048, 16, 64, 16)) == 1
    assert pdssm.scan_segments(pdssm.desc(1, 1000, 2, 64, 16)) == 3
    assert pdssm.scan_segments(pdssm.desc(1, 100, 2, 64, 16)) == 1


@pytest.mark.parametrize("N,K,flags,fused", [
    (64, 16, 0, 1), (128, 32, 0, 1), (128, 128, 0, 0),
    (256, 8, 0, 1), (256, 16, 0, 1),        # five chunk waves keep small dictionaries single-read,
    (256, 32, 0, 1),                        # three the next size up
    (256, 8, pdssm.FLAG_REAL_IO, 1), (256, 8, pdssm.FLAG_BF16_IO, 1),
    (256, 32, pdssm.FLAG_BF16_IO, 1), (256, 64, 0, 0), (256, 64, pdssm.FLAG_REAL_IO, 0),
])
def test_single_read_or_multi_pass(lib, N, K, flags, fused):
    d = pdssm.desc(8, 4096, 16, N, K)
    d.flags = flags
    assert pdssm.uses_fused(d) == fused


@pytest.mark.parametrize("kw,code", [
    (dict(N=48), pdssm.ERR_UNSUPPORTED),
    (dict(N=512), pdssm.ERR_UNSUPPORTED),
    (dict(K=257), pdssm.ERR_UNSUPPORTED),
    (dict(chunk=24), pdssm.ERR_UNSUPPORTED),
    (dict(chunk=32), pdssm.ERR_UNSUPPORTED),
    (dict(N=128, chunk=16), pdssm.ERR_UNSUPPORTED),
    (dict(L=0), pdssm.ERR_INVALID_ARG),
    (dict(B=-1), pdssm.ERR_INVALID_ARG),
    (dict(chunk=-3), pdssm.ERR_INVALID_ARG),
])
def test_bad_descriptors(lib, kw, code):
    args = dict(B=2, L=10, H=2, N=64, K=4, chunk=0)
    args.update(kw)
    d = pdssm.desc(**args)
    assert pdssm.num_chunks(d) == code
    with pytest.raises(pdssm.PdssmError):
        pdssm.workspace_size(d, pdssm.OP_FWD)


def test_flags_known_bits_only(lib):
    d = pdssm.desc(2, 10, 2, 64, 4)
    for ok in (pdssm.FLAG_PREPARED, pdssm.FLAG_BF16_IO, pdssm.FLAG_PREPARED | pdssm.FLAG_BF16_IO,
               pdssm.FLAG_REAL_IO, pdssm.FLAG_PREPARED | pdssm.FLAG_REAL_IO):
        d.flags = ok
        assert pdssm.num_chunks(d) == 2
    # one row format at a time; no unknown bits
    for bad in (pdssm.FLAG_BF16_IO | pdssm.FLAG_REAL_IO, 8, 1 << 31):
        d.flags = bad
        assert pdssm.num_chunks(d) == pdssm.ERR_INVALID_ARG


@pytest.mark.parametrize("flag", ["FLAG_BF16_IO", "FLAG_REAL_IO"])
def test_narrow_io_only_where_supported(lib, flag):
    f = FakeBufs()
    P = lambda n: f(n)  # noqa: E731
    # composition takes complex64 only (the scans, the decode step and the
    # straight-through pair take both narrow formats)
    d = pdssm.desc(2, 40, 2, 64, 4)
    d.flags = getattr(pdssm, flag)
    st = 2 * 40 * 2 * 64 * 8
    assert lib.pdssm_compose_chunks(ctypes.byref(d), P(640), P(2048), P(st), P(st), P(st), None,
                                    None) == pdssm.ERR_UNSUPPORTED
    if flag == "FLAG_BF16_IO":
        # bf16 pairs: g has 4 bytes per entry and z stays complex64 (8), so an
        # output placed in the second half of z's extent overlaps it
        need = lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_STE_GRADS)
        ws = ctypes.c_void_p(f(need).value // 256 * 256 + 256)
        g, z = f(st // 2), f(2 * st)
        q_in_z = ctypes.c_void_p(z.value + st // 2 + 256)
        assert lib.pdssm_ste_grads(ctypes.byref(d), P(640), P(2048), g, z, q_in_z, None, ws, need, None,
                                   None) == pdssm.ERR_INVALID_ARG


def test_prepare_host_checks(lib):
    d = pdssm.desc(2, 40, 2, 64, 4)
    f = FakeBufs()
    pi = f(2 * 4 * 64 * 4)
    need = lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_FWD)
    assert need == lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_BWD)
    ws = ctypes.c_void_p(f(need).value // 256 * 256 + 256)
    assert lib.pdssm_prepare(ctypes.byref(d), None, ws, need, None, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_prepare(ctypes.byref(d), pi, None, need, None, None) == pdssm.ERR_WORKSPACE
    assert lib.pdssm_prepare(ctypes.byref(d), pi, ws, need - 1, None, None) == pdssm.ERR_WORKSPACE
    assert lib.pdssm_prepare(ctypes.byref(d), pi, ctypes.c_void_p(ws.value + 16), need, None,
                             None) == pdssm.ERR_WORKSPACE
    assert lib.pdssm_prepare(ctypes.byref(d), pi, pi, need, None, None) == pdssm.ERR_INVALID_ARG
    bad = pdssm.desc(2, 40, 2, 48, 4)
    assert lib.pdssm_prepare(ctypes.byref(bad), pi, ws, need, None, None) == pdssm.ERR_UNSUPPORTED


def test_status_strings(lib):
    for st in (0, -1, -2, -3, -4, -5):
        assert pdssm.status_string(st).startswith("PDSSM_")
    assert "unknown" in pdssm.status_string(7)


class FakeBufs:
    """Distinct fake device addresses: the host checks reject the call before
    any pointer could be dereferenced."""

    def __init__(self):
        self.next = 1 << 40

    def __call__(self, nbytes):
        p = self.next
        self.next += (nbytes + 4095) // 4096 * 4096 + 4096
        return ctypes.c_void_p(p)


def _fwd_call(lib, d, override=None, ws_bytes=None):
    B, L, H, N, K = d.B, d.L, d.H, d.N, d.K
    f = FakeBufs()
    st = B * L * H * N * 8
    args = dict(idx=f(B * L * H * 4), pi=f(H * K * N * 4), D=f(st), b=f(st), c=f(st), h0=None,
                y=f(B * L * H * 4), hf=f(B * H * N * 8), saved=f(B * H * 64 * N * 8))
    need = lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_FWD)
    args["ws"] = ctypes.c_void_p(f(need).value // 256 * 256 + 256)
    args.update(override or {})
    return lib.pdssm_scan_fwd(ctypes.byref(d), args["idx"], args["pi"], args["D"], args["b"],
                              args["c"], args["h0"], args["y"], args["hf"], args["saved"],
                              args["ws"], need if ws_bytes is None else ws_bytes, None, None)


def test_fwd_rejects_null_required(lib):
    d = pdssm.desc(2, 40, 2, 64, 4)
    for name in ("idx", "pi", "D", "b", "c", "y"):
        assert _fwd_call(lib, d, {name: None}) == pdssm.ERR_INVALID_ARG, name


def test_fwd_rejects_small_workspace(lib):
    d = pdssm.desc(2, 40, 2, 64, 4)
    assert _fwd_call(lib, d, ws_bytes=16) == pdssm.ERR_WORKSPACE
    assert _fwd_call(lib, d, {"ws": None}) == pdssm.ERR_WORKSPACE


def test_fwd_rejects_aliasing_and_misalignment(lib):
    d = pdssm.desc(2, 40, 2, 64, 4)
    f = FakeBufs()
    shared = f(2 * 40 * 2 * 64 * 8)
    assert _fwd_call(lib, d, {"D": shared, "y": shared}) == pdssm.ERR_INVALID_ARG
    assert _fwd_call(lib, d, {"D": ctypes.c_void_p(shared.value + 4)}) == pdssm.ERR_INVALID_ARG


def test_word_arrays_must_be_4_byte_aligned(lib):
    """idx, y and dy are read and written as 4-byte words: a pointer off a
    4-byte boundary is rejected on the host (forward, backward, decode)."""
    d = pdssm.desc(2, 40, 2, 64, 4)
    f = FakeBufs()
    idx, y = f(2 * 40 * 2 * 4), f(2 * 40 * 2 * 4)
    assert _fwd_call(lib, d, {"idx": ctypes.c_void_p(idx.value + 2)}) == pdssm.ERR_INVALID_ARG
    assert _fwd_call(lib, d, {"y": ctypes.c_void_p(y.value + 1)}) == pdssm.ERR_INVALID_ARG
    st = 2 * 40 * 2 * 64 * 8
    args = [f(2 * 40 * 2 * 4), f(2 * 4 * 64 * 4)] + [f(st) for _ in range(3)] + [f(2 * 2 * 5 * 64 * 8)]
    dy = f(2 * 40 * 2 * 4)
    outs = [f(st) for _ in range(3)] + [None]
    need = lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_BWD)
    ws = ctypes.c_void_p(f(need).value // 256 * 256 + 256)
    assert lib.pdssm_scan_bwd(ctypes.byref(d), *args, ctypes.c_void_p(dy.value + 2), None, *outs, ws, need,
                              None, None) == pdssm.ERR_INVALID_ARG
    a2 = list(args)
    a2[0] = ctypes.c_void_p(args[0].value + 1)
    assert lib.pdssm_scan_bwd(ctypes.byref(d), *a2, dy, None, *outs, ws, need, None, None) == pdssm.ERR_INVALID_ARG
    dd = pdssm.desc(2, 1, 3, 64, 4)
    row = 2 * 3 * 64 * 8
    di, dpi, D, b, c, h, dyy = f(2 * 3 * 4), f(3 * 4 * 64 * 4), f(row), f(row), f(row), f(row), f(2 * 3 * 4)
    assert lib.pdssm_decode_step(ctypes.byref(dd), ctypes.c_void_p(di.value + 2), dpi, D, b, c, None, h, dyy,
                                 None, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_decode_step(ctypes.byref(dd), di, dpi, D, b, c, None, h, ctypes.c_void_p(dyy.value + 2),
                                 None, None) == pdssm.ERR_INVALID_ARG


def test_bwd_and_compose_reject_null(lib):
    d = pdssm.desc(2, 40, 2, 64, 4)
    P = ctypes.c_void_p(1 << 40)
    assert lib.pdssm_scan_bwd(ctypes.byref(d), *([None] * 13), 0, None, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_compose_chunks(ctypes.byref(d), P, P, None, None, None, None, None) == pdssm.ERR_INVALID_ARG


def test_ste_entry_points_host_checks(lib):
    d = pdssm.desc(2, 40, 2, 64, 4)
    f = FakeBufs()
    st = 2 * 40 * 2 * 64 * 8
    # the straight-through backward checks what the plain backward checks ...
    assert lib.pdssm_scan_bwd_ste(ctypes.byref(d), *([None] * 14), 0, None, None) == pdssm.ERR_INVALID_ARG
    args = [f(2 * 40 * 2 * 4), f(2 * 4 * 64 * 4)] + [f(st) for _ in range(3)] + [f(2 * 2 * 5 * 64 * 8),
                                                                                f(2 * 40 * 2 * 4), None]
    outs = [f(st) for _ in range(3)] + [None]
    need = lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_BWD)
    ws = ctypes.c_void_p(f(need).value // 256 * 256 + 256)
    # ... and needs z, disjoint from everything else
    assert lib.pdssm_scan_bwd_ste(ctypes.byref(d), *args, *outs, None, ws, need, None, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_scan_bwd_ste(ctypes.byref(d), *args, *outs, args[2], ws, need, None,
                                  None) == pdssm.ERR_INVALID_ARG   # z over D
    assert lib.pdssm_scan_bwd_ste(ctypes.byref(d), *args, *outs, outs[0], ws, need, None,
                                  None) == pdssm.ERR_INVALID_ARG   # z over dD
    # scores and dictionary gradient: required pointers, workspace size and alignment, overlap
    need = lib.pdssm_workspace_size(ctypes.byref(d), pdssm.OP_STE_GRADS)
    assert need >= 2 * 40 * 2 * 4 and need != ctypes.c_size_t(-1).value
    idx, pi, g, z = f(2 * 40 * 2 * 4), f(2 * 4 * 64 * 4), f(st), f(st)
    q, G = f(2 * 40 * 2 * 4 * 4), f(2 * 4 * 64 * 64 * 4)
    ws = ctypes.c_void_p(f(need).value // 256 * 256 + 256)
    call = lambda *a: lib.pdssm_ste_grads(ctypes.byref(d), *a, None, None)  # noqa: E731
    assert call(None, pi, g, z, q, G, ws, need) == pdssm.ERR_INVALID_ARG
    assert call(idx, pi, g, z, None, None, ws, need) == pdssm.ERR_INVALID_ARG   # nothing asked for
    assert call(idx, None, g, z, q, G, ws, need) == pdssm.ERR_INVALID_ARG    # scores need pi
    assert call(idx, pi, g, None, q, G, ws, need) == pdssm.ERR_INVALID_ARG
    assert call(idx, pi, g, z, q, G, None, need) == pdssm.ERR_WORKSPACE
    assert call(idx, pi, g, z, q, G, ws, need - 1) == pdssm.ERR_WORKSPACE
    assert call(idx, pi, g, z, q, G, ctypes.c_void_p(ws.value + 16), need) == pdssm.ERR_WORKSPACE
    assert call(idx, pi, g, z, q, g, ws, need) == pdssm.ERR_INVALID_ARG    # G over g
    assert call(idx, pi, g, z, pi, G, ws, need) == pdssm.ERR_INVALID_ARG   # q over pi
    assert call(idx, pi, g, z, q, q, ws, need) == pdssm.ERR_INVALID_ARG    # q over G
    assert call(idx, pi, ctypes.c_void_p(g.value + 8), z, q, G, ws, need) == pdssm.ERR_INVALID_ARG
    bad = pdssm.desc(2, 40, 2, 48, 4)
    assert lib.pdssm_ste_grads(ctypes.byref(bad), idx, pi, g, z, q, G, ws, need, None,
                               None) == pdssm.ERR_UNSUPPORTED
    with pytest.raises(pdssm.PdssmError):
        pdssm.workspace_size(bad, pdssm.OP_STE_GRADS)
    # tempered softmax: sizes, temperature, overlap
    x, gy, gx = f(4096), f(4096), f(4096)
    sm = lib.pdssm_softmax_vjp
    assert sm(x, gy, gx, 8, 16, 1, ctypes.c_float(0.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, gx, 8, 16, 1, ctypes.c_float(-1.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, gx, 8, 16, 1, ctypes.c_float(float("nan")), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, gx, 8, 0, 1, ctypes.c_float(1.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, gx, 8, 16, 0, ctypes.c_float(1.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(None, gy, gx, 8, 16, 1, ctypes.c_float(1.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, x, 8, 16, 1, ctypes.c_float(1.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, ctypes.c_void_p(gx.value + 2), 8, 16, 1, ctypes.c_float(1.0), None) == pdssm.ERR_INVALID_ARG
    assert sm(x, gy, gx, 1 << 31, 1, 1, ctypes.c_float(1.0), None) == pdssm.ERR_UNSUPPORTED
    # an empty outer extent enqueues nothing and succeeds
    assert sm(x, gy, gx, 0, 16, 1, ctypes.c_float(1.0), None) == pdssm.OK


def test_ste_grads_workspace_bounds(lib):
    # the partial buffer stays bounded (<= 256 MiB) even for the largest N
    for dims in ((16, 2048, 16, 64, 16), (8, 4096, 32, 128, 64), (1, 32767, 256, 256, 256),
                 (8, 18000, 8, 128, 32), (1, 1, 1, 8, 1)):
        d = pdssm.desc(*dims)
        B, L, H, N, K = dims
        n = pdssm.workspace_size(d, pdssm.OP_STE_GRADS)
        assert n <= B * L * H * 4 + H * K * 64 * 1024 + (1 << 28) + 64 * 256, dims


def test_decode_host_checks(lib):
    d = pdssm.desc(2, 1, 3, 64, 4)
    f = FakeBufs()
    row = 2 * 3 * 64 * 8
    idx, pi, D, b, c, h, y = f(2 * 3 * 4), f(3 * 4 * 64 * 4), f(row), f(row), f(row), f(row), f(2 * 3 * 4)
    call = lambda *a: lib.pdssm_decode_step(ctypes.byref(d), *a, None, None)  # noqa: E731
    for i in (0, 1, 2, 3, 4, 6, 7):   # every pointer but h_in is required
        args = [idx, pi, D, b, c, h, h, y]
        args[i] = None
        assert call(*args) == pdssm.ERR_INVALID_ARG, i
    assert call(idx, pi, D, b, c, h, D, y) == pdssm.ERR_INVALID_ARG            # h_out over D
    assert call(idx, pi, D, b, c, h, ctypes.c_void_p(h.value + 64), y) == pdssm.ERR_INVALID_ARG  # partial overlap
    assert call(idx, pi, D, b, c, h, h, ctypes.c_void_p(h.value + 8)) == pdssm.ERR_INVALID_ARG   # y over h
    assert call(idx, pi, ctypes.c_void_p(D.value + 8), b, c, None, h, y) == pdssm.ERR_INVALID_ARG
    bad = pdssm.desc(2, 1, 3, 48, 4)
    assert lib.pdssm_decode_step(ctypes.byref(bad), idx, pi, D, b, c, None, h, y, None,
                                 None) == pdssm.ERR_UNSUPPORTED


def test_select_host_checks(lib):
    f = FakeBufs()
    M, pi = f(4 * 5 * 64 * 64 * 4), f(4 * 5 * 64 * 4)
    assert lib.pdssm_dict_argmax(4, 5, 48, M, pi, None) == pdssm.ERR_UNSUPPORTED
    assert lib.pdssm_dict_argmax(0, 5, 64, M, pi, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_dict_argmax(4, 5, 64, None, pi, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_dict_argmax(4, 5, 64, M, M, None) == pdssm.ERR_INVALID_ARG     # pi over M
    u, S, lg, idx = f(100 * 64 * 2), f(8 * 4 * 64 * 2), f(100 * 32 * 4), f(100 * 8 * 4)
    assert lib.pdssm_route(100, 60, 8, 4, u, S, lg, idx, None) == pdssm.ERR_UNSUPPORTED   # Dm % 8
    assert lib.pdssm_route(100, 64, 8, 257, u, S, lg, idx, None) == pdssm.ERR_UNSUPPORTED
    assert lib.pdssm_route(0, 64, 8, 4, u, S, lg, idx, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_route(100, 64, 8, 4, u, S, lg, None, None) == pdssm.ERR_INVALID_ARG
    assert lib.pdssm_route(100, 64, 8, 4, u, S, u, idx, None) == pdssm.ERR_INVALID_ARG    # logits over u
    assert lib.pdssm_route(100, 64, 8, 4, ctypes.c_void_p(u.value + 2), S, lg, idx, None) == pdssm.ERR_INVALID_ARG


def test_project_host_checks(lib):
    f = FakeBufs()
    T, Dm, H, K, N = 100, 64, 4, 8, 16
    u, S = f(T * Dm * 2), f(H * K * Dm * 2)
    Wb, Wc, Wd = f(H * 2 * N * Dm * 2), f(H * 2 * N * Dm * 2), f(H * 2 * N * Dm * 2)
    lg, idx = f(T * H * K * 4), f(T * H * 4)
    b, c, D = f(T * H * N * 8), f(T * H * N * 8), f(T * H * N * 8)
    call = lambda *a: lib.pdssm_project(*a, None)  # noqa: E731
    # nothing asked for; routing without idx; logits without S; weights without output and back
    assert call(T, Dm, H, K, N, u, None, None, None, None, None, None, None, None, None) == pdssm.ERR_INVALID_ARG
    assert call(T, Dm, H, K, N, u, S, None, None, None, lg, None, None, None, None) == pdssm.ERR_INVALID_ARG
    assert call(T, Dm, H, K, N, u, None, Wb, None, None, lg, None, b, None, None) == pdssm.ERR_INVALID_ARG
    assert call(T, Dm, H, K, N, u, None, Wb, None, None, None, None, None, None, None) == pdssm.ERR_INVALID_ARG
    assert call(T, Dm, H, K, N, u, None, None, None, None, None, None, None, None, D) == pdssm.ERR_INVALID_ARG
    # sizes: contraction not a multiple of 32, N and K outside the supported set
    assert call(T, 48, H, K, N, u, S, Wb, Wc, Wd, lg, idx, b, c, D) == pdssm.ERR_UNSUPPORTED
    assert call(T, Dm, H, K, 48, u, S, Wb, Wc, Wd, lg, idx, b, c, D) == pdssm.ERR_UNSUPPORTED
    assert call(T, Dm, H, 257, N, u, S, Wb, Wc, Wd, lg, idx, b, c, D) == pdssm.ERR_UNSUPPORTED
    assert call(0, Dm, H, K, N, u, S, Wb, Wc, Wd, lg, idx, b, c, D) == pdssm.ERR_INVALID_ARG
    # alignment and overlap
    assert call(T, Dm, H, K, N, u, S, Wb, Wc, Wd, lg, idx, ctypes.c_void_p(b.value + 8), c, D) == pdssm.ERR_INVALID_ARG
    assert call(T, Dm, H, K, N, u, S, Wb, Wc, Wd, lg, ctypes.c_void_p(idx.value + 2), b, c, D) == pdssm.ERR_INVALID_ARG
    assert call(T, Dm, H, K, N, u, S, Wb, Wc, Wd, lg, idx, b, b, D) == pdssm.ERR_INVALID_ARG        # c over b
    assert call(T, Dm, H, K, N, u, S, Wb, Wc, Wd, lg, idx, b, c, Wd) == pdssm.ERR_INVALID_ARG       # D over its weights
