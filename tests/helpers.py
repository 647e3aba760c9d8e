"""Shared helpers for the GPU parity tests."""
import numpy as np

from paper_2605_19150_amd.inputs import sub_sequence  # noqa: F401

RTOL = 1e-4
ATOL = 1e-5


def as_parts(a):
    """Complex -> [..., 2] real view; real arrays unchanged."""
    a = np.asarray(a)
    if np.iscomplexobj(a):
        return np.stack([a.real, a.imag], -1).astype(np.float64)
    return a.astype(np.float64)


def assert_close(name, got, ref, rtol=RTOL, atol=ATOL):
    """|got - ref| <= atol + rtol*|ref| on every real component (ref = float64 oracle)."""
    g, r = as_parts(got), as_parts(ref)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    err = np.abs(g - r)
    tol = atol + rtol * np.abs(r)
    bad = ~(err <= tol)
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError("%s: %d/%d components out of tolerance; worst at %s: got %r ref %r"
                             % (name, int(bad.sum()), bad.size, i, g[i], r[i]))
