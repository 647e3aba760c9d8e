"""Pins for the selection front end of the oracle (CPU only): the column
argmax that turns a dense dictionary into maps and the routing argmax, with
the first-maximal-index tie rule, against explicit loops."""
import numpy as np

from oracle import oracle_dict_argmax, oracle_route


def test_dict_argmax_is_the_column_argmax_with_first_ties():
    M = np.zeros((1, 2, 3, 3))
    # map 0: column 0 peaks at row 2, column 1 ties rows 0 and 1 (-> 0), column 2 peaks at row 1
    M[0, 0] = [[0, 5, 1], [1, 5, 7], [9, 2, 3]]
    # map 1: a constant column ties everywhere (-> row 0)
    M[0, 1] = [[4, 0, 0], [4, 0, 1], [4, 1, 0]]
    np.testing.assert_array_equal(oracle_dict_argmax(M), [[[2, 0, 1], [0, 2, 1]]])


def test_dict_argmax_matches_loops():
    rng = np.random.default_rng(0)
    M = rng.standard_normal((2, 3, 5, 5))
    pi = oracle_dict_argmax(M)
    for h in range(2):
        for k in range(3):
            for j in range(5):
                col = [M[h, k, i, j] for i in range(5)]
                assert pi[h, k, j] == col.index(max(col))


def test_route_matches_loops_and_ties():
    rng = np.random.default_rng(1)
    u = rng.integers(-3, 4, size=(2, 3, 4)).astype(np.float64)
    S = rng.integers(-2, 3, size=(2, 5, 4)).astype(np.float64)
    S[1, 3] = S[1, 1]  # two identical maps: their scores tie, the first wins
    logits, idx = oracle_route(u, S)
    for b in range(2):
        for t in range(3):
            for h in range(2):
                row = [sum(u[b, t, d] * S[h, k, d] for d in range(4)) for k in range(5)]
                assert list(logits[b, t, h]) == row
                assert idx[b, t, h] == row.index(max(row))
