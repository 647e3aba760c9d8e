"""Thin ctypes binding of libpdssm.so (the C ABI declared in include/pdssm.h).

Only argument marshalling happens here: shape/dtype/device checks, output and
workspace allocation with torch, and passing raw device pointers plus the
current HIP stream to the library.  Every step of the scan runs in the HIP
kernels.  If the library is missing the binding raises; there is no fallback.

Tensor layouts (all contiguous, on one GPU):
  idx [B,L,H] int32, pi [H,K,N] int32, D/b/c [B,L,H,N] complex64,
  h0/h_final/dh_final/dh0 [B,H,N] complex64, y/dy [B,L,H] float32,
  saved [B,H,C,N] complex64 (C = num_chunks).
With bf16 I/O (FLAG_BF16_IO), D, b, c and dD, db, dc are bfloat16 tensors
  [B,L,H,N,2] holding (re, im) (torch.view_as_real(x).to(torch.bfloat16)).
The real-valued model (FLAG_REAL_IO): D, b, c, dD, db, dc and saved are
  float32 ([B,L,H,N], saved [B,H,C,N]: the states are real); h0, dh_final,
  h_final and dh0 stay complex64 (scan_fwd and scan_bwd also take a real
  float32 h0 / dh_final and widen it).
Straight-through surrogate gradients (Sec. 3.1 Prop. 2): q [B,L,H,K] float32,
  z [B,L,H,N] complex64, G [H,K,N,N] float32, routing logits [B,L,H,K] and
  dense dictionary M [H,K,N,N] float32.
"""
import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpdssm.so")
_lib = None

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_INDEX = 0, -1, -2, -3, -4, -5
OP_FWD, OP_BWD, OP_COMPOSE, OP_STE_GRADS = 1, 2, 3, 4
FLAG_PREPARED = 1
FLAG_BF16_IO = 2
FLAG_REAL_IO = 4


class PdssmError(RuntimeError):
    def __init__(self, status, what):
        super().__init__("%s: %s" % (what, status_string(status)))
        self.status = status


class Desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("L", ctypes.c_int32), ("H", ctypes.c_int32),
                ("N", ctypes.c_int32), ("K", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


EXPORTS = ("pdssm_abi_version", "pdssm_chunk_len", "pdssm_num_chunks", "pdssm_workspace_size",
           "pdssm_uses_fused", "pdssm_scan_segments", "pdssm_status_string", "pdssm_prepare", "pdssm_scan_fwd", "pdssm_scan_fwd_noalloc",
           "pdssm_scan_bwd", "pdssm_compose_chunks", "pdssm_scan_bwd_ste", "pdssm_ste_grads",
           "pdssm_softmax_vjp", "pdssm_decode_step", "pdssm_dict_argmax", "pdssm_route", "pdssm_project")


def lib_path():
    return _LIB_PATH


def load():
    """Load libpdssm.so once (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError("libpdssm.so is not built (%s); run __graft_entry__.build()" % _LIB_PATH)
    L = ctypes.CDLL(_LIB_PATH)
    P, I, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    D = ctypes.POINTER(Desc)
    L.pdssm_abi_version.argtypes, L.pdssm_abi_version.restype = [], I
    L.pdssm_chunk_len.argtypes, L.pdssm_chunk_len.restype = [D], I
    L.pdssm_num_chunks.argtypes, L.pdssm_num_chunks.restype = [D], I
    L.pdssm_workspace_size.argtypes, L.pdssm_workspace_size.restype = [D, I], Z
    L.pdssm_status_string.argtypes, L.pdssm_status_string.restype = [I], ctypes.c_char_p
    L.pdssm_uses_fused.argtypes, L.pdssm_uses_fused.restype = [D], I
    L.pdssm_scan_segments.argtypes, L.pdssm_scan_segments.restype = [D], I
    L.pdssm_prepare.argtypes, L.pdssm_prepare.restype = [D, P, P, Z, P, P], I
    L.pdssm_scan_fwd.argtypes = [D] + [P] * 10 + [Z, P, P]
    L.pdssm_scan_fwd.restype = I
    L.pdssm_scan_fwd_noalloc.argtypes = [D] + [P] * 11
    L.pdssm_scan_fwd_noalloc.restype = I
    L.pdssm_scan_bwd.argtypes = [D] + [P] * 13 + [Z, P, P]
    L.pdssm_scan_bwd.restype = I
    L.pdssm_compose_chunks.argtypes = [D] + [P] * 7
    L.pdssm_compose_chunks.restype = I
    L.pdssm_scan_bwd_ste.argtypes = [D] + [P] * 14 + [Z, P, P]
    L.pdssm_scan_bwd_ste.restype = I
    L.pdssm_ste_grads.argtypes = [D] + [P] * 7 + [Z, P, P]
    L.pdssm_ste_grads.restype = I
    L.pdssm_softmax_vjp.argtypes = [P, P, P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_float, P]
    L.pdssm_softmax_vjp.restype = I
    L.pdssm_decode_step.argtypes = [D] + [P] * 10
    L.pdssm_decode_step.restype = I
    I32 = ctypes.c_int32
    L.pdssm_dict_argmax.argtypes = [I32, I32, I32, P, P, P]
    L.pdssm_dict_argmax.restype = I
    L.pdssm_route.argtypes = [I32, I32, I32, I32, P, P, P, P, P]
    L.pdssm_route.restype = I
    L.pdssm_project.argtypes = [I32] * 5 + [P] * 10 + [P]
    L.pdssm_project.restype = I
    if L.pdssm_abi_version() != 1:
        raise ImportError("libpdssm.so ABI version mismatch")
    _lib = L
    return L


def status_string(st):
    return load().pdssm_status_string(int(st)).decode()


def desc(B, L, H, N, K, chunk=0):
    return Desc(int(B), int(L), int(H), int(N), int(K), int(chunk), 0)


def scan_segments(d):
    return load().pdssm_scan_segments(ctypes.byref(d))


def uses_fused(d):
    """1 when the single-read kernels run this descriptor, 0 when the
    multi-pass kernels do (dictionary tables beyond LDS), < 0 on error."""
    return load().pdssm_uses_fused(ctypes.byref(d))


def chunk_len(d):
    return load().pdssm_chunk_len(ctypes.byref(d))


def num_chunks(d):
    return load().pdssm_num_chunks(ctypes.byref(d))


def workspace_size(d, op):
    n = load().pdssm_workspace_size(ctypes.byref(d), int(op))
    if n == ctypes.c_size_t(-1).value:
        raise PdssmError(ERR_INVALID_ARG, "workspace_size")
    return n


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t, name, dtype, shape, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if t.device != device or t.device.type != "cuda":
        raise ValueError("%s must be on %s" % (name, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def dims_of(idx, pi):
    B, L, H = idx.shape
    H2, K, N = pi.shape
    if H2 != H:
        raise ValueError("idx and pi disagree on H")
    return B, L, H, N, K


def is_bf16_io(D):
    """D given as bf16 (re, im) pairs [..., N, 2] rather than complex64."""
    return isinstance(D, torch.Tensor) and D.dtype == torch.bfloat16


def is_real_io(D):
    """D given as real float32 rows (the real-valued model)."""
    return isinstance(D, torch.Tensor) and D.dtype == torch.float32


def _check_inputs(idx, pi, D, b, c):
    B, L, H, N, K = dims_of(idx, pi)
    dev = idx.device
    _need(idx, "idx", torch.int32, (B, L, H), dev)
    _need(pi, "pi", torch.int32, (H, K, N), dev)
    for t, n in ((D, "D"), (b, "b"), (c, "c")):
        if is_bf16_io(D):
            _need(t, n, torch.bfloat16, (B, L, H, N, 2), dev)
        elif is_real_io(D):
            _need(t, n, torch.float32, (B, L, H, N), dev)
        else:
            _need(t, n, torch.complex64, (B, L, H, N), dev)
    return B, L, H, N, K, dev


class Scan:
    """Pre-allocated outputs and one workspace for one problem size; prepare(),
    fwd() and bwd() allocate nothing, so they can be timed in a loop.

    Without prepare() every scan builds the dictionary tables itself.  After
    prepare(pi) the scans reuse the tables in the workspace; call prepare()
    again whenever the contents of pi change."""

    def __init__(self, B, L, H, N, K, chunk=0, device="cuda", ste=False, bf16=False, real=False):
        self.d = desc(B, L, H, N, K, chunk)
        self.dp = desc(B, L, H, N, K, chunk)
        self.bf16 = bf16
        self.real = real
        self.d.flags = (FLAG_BF16_IO if bf16 else 0) | (FLAG_REAL_IO if real else 0)
        self.dp.flags = FLAG_PREPARED | self.d.flags
        self.prepared = False
        self.dims = (B, L, H, N, K)
        self.device = torch.device(device)
        self.C = num_chunks(self.d)
        if self.C < 0:
            raise PdssmError(self.C, "num_chunks")
        self.chunk = chunk_len(self.d)
        self.fused = uses_fused(self.d) == 1
        self.segments = load().pdssm_scan_segments(ctypes.byref(self.d))
        dev = self.device
        nws = max(workspace_size(self.d, OP_FWD), workspace_size(self.d, OP_BWD), 1)
        self.ws = torch.empty(nws, dtype=torch.uint8, device=dev)
        self.y = torch.empty((B, L, H), dtype=torch.float32, device=dev)
        self.h_final = torch.empty((B, H, N), dtype=torch.complex64, device=dev)
        self.saved = torch.empty((B, H, self.C, N), dtype=torch.float32 if real else torch.complex64, device=dev)
        if bf16:
            self.dD = torch.empty((B, L, H, N, 2), dtype=torch.bfloat16, device=dev)
        elif real:
            self.dD = torch.empty((B, L, H, N), dtype=torch.float32, device=dev)
        else:
            self.dD = torch.empty((B, L, H, N), dtype=torch.complex64, device=dev)
        self.db = torch.empty_like(self.dD)
        self.dc = torch.empty_like(self.dD)
        self.dh0 = torch.empty((B, H, N), dtype=torch.complex64, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.ste = ste
        if ste:
            self.q = torch.empty((B, L, H, K), dtype=torch.float32, device=dev)
            self.z = torch.empty((B, L, H, N), dtype=torch.float32 if real else torch.complex64, device=dev)
            self.G = torch.empty((H, K, N, N), dtype=torch.float32, device=dev)
            self.ws_ste = torch.empty(max(workspace_size(self.d, OP_STE_GRADS), 1), dtype=torch.uint8,
                                      device=dev)

    def _desc(self):
        return ctypes.byref(self.dp if self.prepared else self.d)

    def _check(self, idx, pi, D, b, c, h0=None, dy=None, dh_final=None):
        """Every tensor argument has the type, shape, device and layout this
        Scan was built for (the library reads them through raw pointers)."""
        B, L, H, N, K = self.dims
        dev = self.device if self.device.index is not None else idx.device
        _need(idx, "idx", torch.int32, (B, L, H), dev)
        _need(pi, "pi", torch.int32, (H, K, N), dev)
        for t, n in ((D, "D"), (b, "b"), (c, "c")):
            if self.bf16:
                _need(t, n, torch.bfloat16, (B, L, H, N, 2), dev)
            elif self.real:
                _need(t, n, torch.float32, (B, L, H, N), dev)
            else:
                _need(t, n, torch.complex64, (B, L, H, N), dev)
        for t, n in ((h0, "h0"), (dh_final, "dh_final")):
            if t is not None:
                _need(t, n, torch.complex64, (B, H, N), dev)
        if dy is not None:
            _need(dy, "dy", torch.float32, (B, L, H), dev)

    def prepare(self, pi, stream=None):
        B, L, H, N, K = self.dims
        _need(pi, "pi", torch.int32, (H, K, N), pi.device)
        st = load().pdssm_prepare(ctypes.byref(self.d), _p(pi), _p(self.ws), self.ws.numel(),
                                  _p(self.status), _stream(stream))
        if st != OK:
            raise PdssmError(st, "pdssm_prepare")
        self.prepared = True

    def fwd(self, idx, pi, D, b, c, h0=None, stream=None):
        self._check(idx, pi, D, b, c, h0=h0)
        st = load().pdssm_scan_fwd(self._desc(), _p(idx), _p(pi), _p(D), _p(b), _p(c),
                                   _p(h0), _p(self.y), _p(self.h_final), _p(self.saved),
                                   _p(self.ws), self.ws.numel(), _p(self.status), _stream(stream))
        if st != OK:
            raise PdssmError(st, "pdssm_scan_fwd")
        return self.y, self.h_final, self.saved

    def bwd(self, idx, pi, D, b, c, dy, dh_final=None, stream=None):
        self._check(idx, pi, D, b, c, dy=dy, dh_final=dh_final)
        st = load().pdssm_scan_bwd(self._desc(), _p(idx), _p(pi), _p(D), _p(b), _p(c),
                                   _p(self.saved), _p(dy), _p(dh_final), _p(self.dD), _p(self.db),
                                   _p(self.dc), _p(self.dh0), _p(self.ws), self.ws.numel(),
                                   _p(self.status), _stream(stream))
        if st != OK:
            raise PdssmError(st, "pdssm_scan_bwd")
        return self.dD, self.db, self.dc, self.dh0

    def bwd_ste(self, idx, pi, D, b, c, dy, dh_final=None, stream=None):
        """bwd() plus the scaled states z (Scan(..., ste=True))."""
        self._check(idx, pi, D, b, c, dy=dy, dh_final=dh_final)
        st = load().pdssm_scan_bwd_ste(self._desc(), _p(idx), _p(pi), _p(D), _p(b), _p(c),
                                       _p(self.saved), _p(dy), _p(dh_final), _p(self.dD), _p(self.db),
                                       _p(self.dc), _p(self.dh0), _p(self.z), _p(self.ws),
                                       self.ws.numel(), _p(self.status), _stream(stream))
        if st != OK:
            raise PdssmError(st, "pdssm_scan_bwd_ste")
        return self.dD, self.db, self.dc, self.dh0, self.z

    def ste_grads(self, idx, pi, q=True, G=True, stream=None):
        """Scores q [B,L,H,K] and dictionary gradient G [H,K,N,N] from the db
        and z of the last bwd_ste() (each None when not asked for)."""
        qq, GG = (self.q if q else None), (self.G if G else None)
        B, L, H, N, K = self.dims
        _need(idx, "idx", torch.int32, (B, L, H), self.db.device)
        _need(pi, "pi", torch.int32, (H, K, N), self.db.device)
        st = load().pdssm_ste_grads(ctypes.byref(self.d), _p(idx), _p(pi), _p(self.db), _p(self.z), _p(qq),
                                    _p(GG), _p(self.ws_ste), self.ws_ste.numel(), _p(self.status),
                                    _stream(stream))
        if st != OK:
            raise PdssmError(st, "pdssm_ste_grads")
        return qq, GG

    def check_status(self):
        """Synchronise and raise if a kernel flagged an out-of-range index."""
        torch.cuda.synchronize(self.device)
        st = int(self.status.item())
        if st != OK:
            raise PdssmError(st, "kernel index check")


def _state_arg(x, name, real, dims, dev):
    """A [B,H,N] state argument: complex64, or for the real model also float32
    (widened to complex64, imaginary part 0)."""
    if x is None:
        return None
    if real and isinstance(x, torch.Tensor) and x.dtype == torch.float32:
        _need(x, name, torch.float32, dims, dev)
        return x.to(torch.complex64)
    _need(x, name, torch.complex64, dims, dev)
    return x


def scan_fwd(idx, pi, D, b, c, h0=None, chunk=0, stream=None):
    """Returns (y [B,L,H] f32, h_final [B,H,N] c64, saved [B,H,C,N] c64, or
    f32 for real inputs)."""
    B, L, H, N, K, dev = _check_inputs(idx, pi, D, b, c)
    h0 = _state_arg(h0, "h0", is_real_io(D), (B, H, N), dev)
    s = Scan(B, L, H, N, K, chunk, dev, bf16=is_bf16_io(D), real=is_real_io(D))
    s.fwd(idx, pi, D, b, c, h0, stream)
    s.check_status()
    return s.y, s.h_final, s.saved


def scan_fwd_noalloc(idx, pi, D, b, c, h0=None, chunk=0, y=None, h_final=None, saved=None, stream=None):
    """pdssm_scan_fwd_noalloc: the forward with the library's own device
    workspace (no workspace argument).  Outputs may be passed in (y, h_final,
    saved); the call then allocates nothing.  Returns (y, h_final, saved)."""
    B, L, H, N, K, dev = _check_inputs(idx, pi, D, b, c)
    h0 = _state_arg(h0, "h0", is_real_io(D), (B, H, N), dev)
    d = desc(B, L, H, N, K, chunk)
    d.flags = (FLAG_BF16_IO if is_bf16_io(D) else 0) | (FLAG_REAL_IO if is_real_io(D) else 0)
    C = num_chunks(d)
    if C < 0:
        raise PdssmError(C, "num_chunks")
    y = torch.empty((B, L, H), dtype=torch.float32, device=dev) if y is None else y
    h_final = torch.empty((B, H, N), dtype=torch.complex64, device=dev) if h_final is None else h_final
    sdt = saved_dtype(D)
    saved = torch.empty((B, H, C, N), dtype=sdt, device=dev) if saved is None else saved
    _need(y, "y", torch.float32, (B, L, H), dev)
    _need(h_final, "h_final", torch.complex64, (B, H, N), dev)
    _need(saved, "saved", sdt, (B, H, C, N), dev)
    st = load().pdssm_scan_fwd_noalloc(ctypes.byref(d), _p(idx), _p(pi), _p(D), _p(b), _p(c), _p(h0), _p(y),
                                       _p(h_final), _p(saved), None, _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_scan_fwd_noalloc")
    return y, h_final, saved


def saved_dtype(D):
    """dtype of the saved chunk states for inputs D: float32 for the real
    model (its states are real), else complex64."""
    return torch.float32 if is_real_io(D) else torch.complex64


def scan_bwd(idx, pi, D, b, c, saved, dy, dh_final=None, chunk=0, stream=None):
    """Returns (dD, db, dc [B,L,H,N] c64, or [B,L,H,N,2] bf16 for bf16 inputs,
    or [B,L,H,N] f32 for real inputs; dh0 [B,H,N] c64)."""
    B, L, H, N, K, dev = _check_inputs(idx, pi, D, b, c)
    s = Scan(B, L, H, N, K, chunk, dev, bf16=is_bf16_io(D), real=is_real_io(D))
    _need(saved, "saved", saved_dtype(D), (B, H, s.C, N), dev)
    _need(dy, "dy", torch.float32, (B, L, H), dev)
    dh_final = _state_arg(dh_final, "dh_final", is_real_io(D), (B, H, N), dev)
    s.saved = saved
    s.bwd(idx, pi, D, b, c, dy, dh_final, stream)
    s.check_status()
    return s.dD, s.db, s.dc, s.dh0


def compose_chunks(idx, pi, D, chunk, stream=None):
    """Returns (pi_out [B,H,C,N] int32, d_out [B,H,C,N] c64)."""
    B, L, H, N, K = dims_of(idx, pi)
    dev = idx.device
    _need(idx, "idx", torch.int32, (B, L, H), dev)
    _need(pi, "pi", torch.int32, (H, K, N), dev)
    _need(D, "D", torch.complex64, (B, L, H, N), dev)
    if chunk < 1:
        raise ValueError("chunk must be >= 1")
    tau = min(int(chunk), L)
    C = -(-L // tau)
    pi_out = torch.empty((B, H, C, N), dtype=torch.int32, device=dev)
    d_out = torch.empty((B, H, C, N), dtype=torch.complex64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    d = desc(B, L, H, N, K, tau)
    st = load().pdssm_compose_chunks(ctypes.byref(d), _p(idx), _p(pi), _p(D), _p(pi_out),
                                     _p(d_out), _p(status), _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_compose_chunks")
    torch.cuda.synchronize(dev)
    if int(status.item()) != OK:
        raise PdssmError(int(status.item()), "kernel index check")
    return pi_out, d_out


def scan_bwd_ste(idx, pi, D, b, c, saved, dy, dh_final=None, chunk=0, stream=None):
    """Returns (dD, db, dc, dh0, z [B,L,H,N] c64, or f32 for real inputs;
    with bf16 inputs dD, db, dc are bf16 pairs and z stays c64)."""
    B, L, H, N, K, dev = _check_inputs(idx, pi, D, b, c)
    s = Scan(B, L, H, N, K, chunk, dev, ste=True, bf16=is_bf16_io(D), real=is_real_io(D))
    _need(saved, "saved", saved_dtype(D), (B, H, s.C, N), dev)
    _need(dy, "dy", torch.float32, (B, L, H), dev)
    dh_final = _state_arg(dh_final, "dh_final", is_real_io(D), (B, H, N), dev)
    s.saved = saved
    out = s.bwd_ste(idx, pi, D, b, c, dy, dh_final, stream)
    s.check_status()
    return out


def ste_grads(idx, pi, g, z, q=True, G=True, stream=None):
    """(q [B,L,H,K] f32 or None, G [H,K,N,N] f32 or None) from g = db and z
    of scan_bwd_ste: the scores of every map at every step and, per head and
    map, the sum of Re(g_t z_t^H) over the steps that chose the map.  g, z
    complex64; or float32 for the real-valued model; or g as bf16 (re, im)
    pairs [B,L,H,N,2] (the bf16 setting's db) with z complex64."""
    B, L, H = idx.shape
    N = g.shape[3]
    K = pi.shape[1]
    dev = idx.device
    real, bf16 = is_real_io(g), is_bf16_io(g)
    _need(idx, "idx", torch.int32, (B, L, H), dev)
    _need(pi, "pi", torch.int32, (H, K, N), dev)
    if bf16:
        _need(g, "g", torch.bfloat16, (B, L, H, N, 2), dev)
    else:
        _need(g, "g", torch.float32 if real else torch.complex64, (B, L, H, N), dev)
    _need(z, "z", torch.float32 if real else torch.complex64, (B, L, H, N), dev)
    d = desc(B, L, H, N, K)
    d.flags = FLAG_REAL_IO if real else (FLAG_BF16_IO if bf16 else 0)
    ws = torch.empty(max(workspace_size(d, OP_STE_GRADS), 1), dtype=torch.uint8, device=dev)
    qq = torch.empty((B, L, H, K), dtype=torch.float32, device=dev) if q else None
    GG = torch.empty((H, K, N, N), dtype=torch.float32, device=dev) if G else None
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    st = load().pdssm_ste_grads(ctypes.byref(d), _p(idx), _p(pi), _p(g), _p(z), _p(qq), _p(GG), _p(ws),
                                ws.numel(), _p(status), _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_ste_grads")
    torch.cuda.synchronize(dev)
    if int(status.item()) != OK:
        raise PdssmError(int(status.item()), "kernel index check")
    return qq, GG


def softmax_vjp(x, gy, dim, temp, out=None, stream=None):
    """gx = s * (gy - sum(s * gy, dim)) / temp with s = softmax(x / temp, dim)."""
    if x.dtype != torch.float32 or gy.dtype != torch.float32 or x.shape != gy.shape:
        raise TypeError("x and gy must be float32 tensors of one shape")
    if not (x.is_contiguous() and gy.is_contiguous()) or x.device.type != "cuda" or gy.device != x.device:
        raise ValueError("x and gy must be contiguous and on one GPU")
    dim = dim % x.dim()
    outer = 1
    for n in x.shape[:dim]:
        outer *= int(n)
    inner = 1
    for n in x.shape[dim + 1:]:
        inner *= int(n)
    gx = torch.empty_like(x) if out is None else out
    _need(gx, "out", torch.float32, tuple(x.shape), x.device)
    st = load().pdssm_softmax_vjp(_p(x), _p(gy), _p(gx), outer, int(x.shape[dim]), inner, float(temp),
                                  _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_softmax_vjp")
    return gx


def surrogate_grads(q, G, logits, M, temp, stream=None):
    """The two surrogate gradients of Prop. 2: (d logits [B,L,H,K], dM [H,K,N,N])."""
    return softmax_vjp(logits, q, 3, temp, stream=stream), softmax_vjp(M, G, 2, temp, stream=stream)


def decode_step(idx, pi, D, b, c, h=None, out=None, y=None, stream=None, check=True):
    """One recurrence step per sequence: returns (h_new [B,H,N] c64, y [B,H] f32).
    idx [B,H] int32; D, b, c [B,H,N] c64 (or [B,H,N,2] bf16 pairs, or [B,H,N]
    float32 for the real-valued model); h [B,H,N] c64 or None (zero state).
    out may be h itself (in-place update)."""
    B, H = idx.shape
    H2, K, N = pi.shape
    if H2 != H:
        raise ValueError("idx and pi disagree on H")
    dev = idx.device
    _need(idx, "idx", torch.int32, (B, H), dev)
    _need(pi, "pi", torch.int32, (H, K, N), dev)
    for t, n in ((D, "D"), (b, "b"), (c, "c")):
        if is_bf16_io(D):
            _need(t, n, torch.bfloat16, (B, H, N, 2), dev)
        elif is_real_io(D):
            _need(t, n, torch.float32, (B, H, N), dev)
        else:
            _need(t, n, torch.complex64, (B, H, N), dev)
    if h is not None:
        _need(h, "h", torch.complex64, (B, H, N), dev)
    out = torch.empty((B, H, N), dtype=torch.complex64, device=dev) if out is None else out
    y = torch.empty((B, H), dtype=torch.float32, device=dev) if y is None else y
    status = torch.zeros(1, dtype=torch.int32, device=dev) if check else None
    d = desc(B, 1, H, N, K)
    d.flags = (FLAG_BF16_IO if is_bf16_io(D) else 0) | (FLAG_REAL_IO if is_real_io(D) else 0)
    st = load().pdssm_decode_step(ctypes.byref(d), _p(idx), _p(pi), _p(D), _p(b), _p(c), _p(h), _p(out), _p(y),
                                  _p(status), _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_decode_step")
    if check:
        torch.cuda.synchronize(dev)
        if int(status.item()) != OK:
            raise PdssmError(int(status.item()), "kernel index check")
    return out, y


def dict_argmax(M, stream=None):
    """pi [H,K,N] int32 = first argmax over the rows i of every column j of
    the dense dictionary M [H,K,N,N] float32."""
    H, K, N, N2 = M.shape
    if N2 != N:
        raise ValueError("M must be [H,K,N,N]")
    _need(M, "M", torch.float32, (H, K, N, N), M.device)
    pi = torch.empty((H, K, N), dtype=torch.int32, device=M.device)
    st = load().pdssm_dict_argmax(H, K, N, _p(M), _p(pi), _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_dict_argmax")
    return pi


def route(u, S, logits=True, stream=None):
    """Routing scores and choices: u [B,L,Dm] bf16, S [H,K,Dm] bf16 ->
    (logits [B,L,H,K] f32 or None, idx [B,L,H] int32)."""
    B, L, Dm = u.shape
    H, K, Dm2 = S.shape
    if Dm2 != Dm:
        raise ValueError("u and S disagree on the contraction length")
    _need(u, "u", torch.bfloat16, (B, L, Dm), u.device)
    _need(S, "S", torch.bfloat16, (H, K, Dm), u.device)
    lg = torch.empty((B, L, H, K), dtype=torch.float32, device=u.device) if logits else None
    idx = torch.empty((B, L, H), dtype=torch.int32, device=u.device)
    st = load().pdssm_route(B * L, Dm, H, K, _p(u), _p(S), _p(lg), _p(idx), _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_route")
    return lg, idx


def project(u, S=None, Wb=None, Wc=None, Wd=None, logits=True, N=None, stream=None):
    """pdssm_project: the token projections of a layer in one product.
    u [B,L,Dm] bf16; S [H,K,Dm] bf16 (routing); Wb, Wc, Wd [H,2N,Dm] bf16
    (b, c and the diagonal generator).  Returns a dict with logits [B,L,H,K]
    f32 and idx [B,L,H] int32 (with S), and b, c, D [B,L,H,N] complex64 (each
    with its weights)."""
    B, L, Dm = u.shape
    dev = u.device
    _need(u, "u", torch.bfloat16, (B, L, Dm), dev)
    Ws = [w for w in (Wb, Wc, Wd) if w is not None]
    if S is None and not Ws:
        raise ValueError("project: nothing to compute")
    H = S.shape[0] if S is not None else Ws[0].shape[0]
    K = S.shape[1] if S is not None else 1
    if Ws:
        N = Ws[0].shape[1] // 2
    N = N or 8
    if S is not None:
        _need(S, "S", torch.bfloat16, (H, K, Dm), dev)
    for w, n in ((Wb, "Wb"), (Wc, "Wc"), (Wd, "Wd")):
        if w is not None:
            _need(w, n, torch.bfloat16, (H, 2 * N, Dm), dev)
    out = {}
    if S is not None:
        out["logits"] = torch.empty((B, L, H, K), dtype=torch.float32, device=dev) if logits else None
        out["idx"] = torch.empty((B, L, H), dtype=torch.int32, device=dev)
    for w, n in ((Wb, "b"), (Wc, "c"), (Wd, "D")):
        if w is not None:
            out[n] = torch.empty((B, L, H, N), dtype=torch.complex64, device=dev)
    st = load().pdssm_project(B * L, Dm, H, K, N, _p(u), _p(S), _p(Wb), _p(Wc), _p(Wd), _p(out.get("logits")),
                              _p(out.get("idx")), _p(out.get("b")), _p(out.get("c")), _p(out.get("D")),
                              _stream(stream))
    if st != OK:
        raise PdssmError(st, "pdssm_project")
    return out
