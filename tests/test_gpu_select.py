"""GPU parity of the selection front end against the float64 oracle.

dict_argmax: bit for bit (no arithmetic; ties to the first maximal index).
route: logits within |gpu - ref| <= 1e-5 + 1e-4*S, S = sum_d |u_d S_d| (an
fp32 sum of Dm bf16 products, see helpers.assert_close_sum); idx is exactly
the first argmax of the GPU's own logits, and equals the oracle's choice
wherever the oracle's two best scores are further apart than that bar (where
they are not, the GPU's choice must score within the bar of the best).
"""
import numpy as np
import pytest

from helpers import assert_close_sum
from oracle import oracle_dict_argmax, oracle_route

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU machines, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2605_19150_amd import pdssm  # noqa: E402

DEV = torch.device("cuda:0")


@pytest.mark.parametrize("N", [8, 16, 32, 64, 128, 256])
def test_dict_argmax(N):
    rng = np.random.default_rng(N)
    H, K = 3, 5
    M = rng.standard_normal((H, K, N, N)).astype(np.float32)
    M[0, 0] = np.round(M[0, 0])          # many exact ties
    M[1, 2, :, :] = 1.0                  # every column ties everywhere
    pi = pdssm.dict_argmax(torch.from_numpy(M).to(DEV)).cpu().numpy()
    np.testing.assert_array_equal(pi, oracle_dict_argmax(M))


def _bf16(a):
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    return t, t.to(torch.float64).numpy()


def check_route(B, L, H, K, Dm, seed):
    rng = np.random.default_rng(seed)
    ut, u = _bf16(rng.standard_normal((B, L, Dm)))
    St, S = _bf16(rng.standard_normal((H, K, Dm)) / np.sqrt(Dm))
    logits, idx = pdssm.route(ut.to(DEV), St.to(DEV))
    lg, ix = logits.cpu().numpy(), idx.cpu().numpy()
    rl, ri = oracle_route(u, S)
    scale = np.einsum("bld,hkd->blhk", np.abs(u), np.abs(S))
    assert_close_sum("logits", lg, rl, scale)
    np.testing.assert_array_equal(ix, np.argmax(lg, axis=3))          # first argmax of its own logits
    tol = 1e-5 + 1e-4 * scale.max(axis=3)
    top2 = np.sort(rl, axis=3)[..., -2:] if K > 1 else np.concatenate([rl, rl - 1], axis=3)
    clear = (top2[..., 1] - top2[..., 0]) > 2 * tol
    np.testing.assert_array_equal(ix[clear], ri[clear])
    chosen = np.take_along_axis(rl, ix[..., None].astype(np.int64), axis=3)[..., 0]
    assert (rl.max(axis=3) - chosen <= 2 * tol).all()
    _, idx2 = pdssm.route(ut.to(DEV), St.to(DEV), logits=False)
    np.testing.assert_array_equal(idx2.cpu().numpy(), ix)
    return clear.mean()


@pytest.mark.parametrize("B,L,H,K,Dm", [
    (2, 100, 16, 16, 1024),   # a fsa-perm-like layer: 16 heads x 16 maps, d = 1024
    (1, 70, 7, 5, 72),        # ragged: tokens, heads per tile, contraction tail
    (1, 65, 32, 64, 256),     # 4 heads per tile
    (2, 33, 2, 256, 64),      # one head per tile
    (1, 1, 1, 1, 8),          # smallest
    (3, 50, 300, 3, 16),      # many head groups
    (8, 2048, 32, 64, 64),    # 256-token tiles, 512 of them, two slices of the contraction
    (1, 18693, 28, 64, 32),   # 256-token tiles, a ragged last one, a tile count not a multiple of 8
])
def test_route(B, L, H, K, Dm):
    print("route B=%d L=%d H=%d K=%d Dm=%d" % (B, L, H, K, Dm), flush=True)
    frac = check_route(B, L, H, K, Dm, seed=B + L + H + K + Dm)
    assert frac > 0.9 or K == 1


def test_route_full_size():
    """fsa-perm routing: B16 L2048, 16 heads x 16 maps, d = 1024."""
    frac = check_route(16, 2048, 16, 16, 1024, seed=0)
    assert frac > 0.99


def test_route_hybrid_full_size_sampled():
    """hybrid-lm routing: B8 L4096 (32768 tokens), 32 heads x 64 maps, d = 4096;
    logits and choices of sampled tokens against the oracle."""
    rng = np.random.default_rng(3)
    B, L, H, K, Dm = 8, 4096, 32, 64, 4096
    ut = torch.from_numpy(rng.standard_normal((B, L, Dm), dtype=np.float32)).to(torch.bfloat16)
    St = torch.from_numpy(rng.standard_normal((H, K, Dm), dtype=np.float32) / np.float32(np.sqrt(Dm))).to(
        torch.bfloat16)
    logits, idx = pdssm.route(ut.to(DEV), St.to(DEV))
    rows = np.sort(rng.choice(B * L, size=96, replace=False))
    u = ut.reshape(B * L, Dm)[rows].to(torch.float64).numpy()[None]
    S = St.to(torch.float64).numpy()
    lg = logits.reshape(B * L, H, K)[rows].cpu().numpy()[None]
    ix = idx.reshape(B * L, H)[rows].cpu().numpy()[None]
    rl, ri = oracle_route(u, S)
    scale = np.einsum("bld,hkd->blhk", np.abs(u), np.abs(S))
    assert_close_sum("logits", lg, rl, scale)
    np.testing.assert_array_equal(ix, np.argmax(lg, axis=3))
    tol = 1e-5 + 1e-4 * scale.max(axis=3)
    top2 = np.sort(rl, axis=3)[..., -2:]
    clear = (top2[..., 1] - top2[..., 0]) > 2 * tol
    np.testing.assert_array_equal(ix[clear], ri[clear])
    assert clear.mean() > 0.9
