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


def assert_close_sum(name, got, ref, scale, rtol=RTOL, atol=ATOL):
    """Bar for a quantity that is a sum of products of scan outputs (the
    straight-through scores q and the dictionary gradient G): |got - ref| <=
    atol + rtol*scale, where scale >= |ref| is the sum of the magnitudes of the
    summands.  Each factor is itself only known to the scan's bar (1e-4
    relative), so a sum whose terms cancel inherits an error proportional to
    the size of its terms, not of its result."""
    g, r, s = np.asarray(got, np.float64), np.asarray(ref, np.float64), np.asarray(scale, np.float64)
    assert g.shape == r.shape == s.shape, (name, g.shape, r.shape, s.shape)
    assert (s >= np.abs(r) * (1 - 1e-9) - 1e-300).all(), name + ": scale below |ref|"
    err = np.abs(g - r)
    tol = atol + rtol * s
    bad = ~(err <= tol)
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError("%s: %d/%d components out of tolerance; worst at %s: got %r ref %r scale %r"
                             % (name, int(bad.sum()), bad.size, i, g[i], r[i], s[i]))


def ste_scales(pi, idx, g, z):
    """Magnitude sums for assert_close_sum: qs[b,t,h,k] = sum_j |g_t[pi_k(j)]| |z_t[j]|
    and Gs[h,k,i,j] = sum over the steps that chose k of |g_t[i]| |z_t[j]|."""
    ag, az = np.abs(g), np.abs(z)
    B, L, H, N = ag.shape
    K = pi.shape[1]
    qs = np.empty((B, L, H, K))
    Gs = np.zeros((H, K, N, N))
    for h in range(H):
        qs[:, :, h, :] = np.einsum("blkn,bln->blk", ag[:, :, h, :][:, :, pi[h]], az[:, :, h, :])
        for k in range(K):
            m = idx[:, :, h] == k
            if m.any():
                Gs[h, k] = ag[:, :, h][m].T @ az[:, :, h][m]
    return qs, Gs


def force_sorted_entries(inp, N):
    """Entries with a row of more than seven sources (stored in sorted form):
    in-degree exactly 8 in head 0, all-to-one in head 1, two rows of 12 and
    9 sources in head 2 (if present); steps choose them often, and the other
    entries of those heads keep their maps."""
    H, K = inp["pi"].shape[:2]
    inp["pi"][0, 1, :8] = 5
    inp["pi"][1 % H, 0, :] = N - 1
    if H > 2:
        inp["pi"][2, 3, :12] = 0
        inp["pi"][2, 3, 12:21] = N // 2
    inp["idx"][:, ::2, 0] = 1
    inp["idx"][:, 1::3, 1 % H] = 0
