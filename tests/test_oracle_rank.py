"""Pins of the ranking (Eq. 4-5) and of the block counts (Alg. 2)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O


def brute_topk(s, k):
    key = [(-(0.0 if v == 0 else float(v)), i) for i, v in enumerate(s)]
    chosen = sorted(range(len(s)), key=lambda i: key[i])[:k]
    f = np.zeros(len(s), np.uint8)
    f[chosen] = 1
    return f


@pytest.mark.parametrize("seed", range(40))
def test_rank_matches_full_sort_with_ties(seed):
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 13))
    pool = np.array([0.0, -0.0, 1.0, 1.0, 2.5, -3.0, np.inf, -np.inf, 7.0, 1e-45], np.float32)
    s = rng.choice(pool, T).astype(np.float32)
    for k in range(T + 1):
        assert np.array_equal(O.rank_k(s, k), brute_topk(s, k))


def test_rank_invariants_zipf():
    rng = np.random.default_rng(0)
    s = rng.zipf(1.1, 4096).astype(np.float32)
    flag, hi, lo = O.rank(s, 26, 100)
    K = 4096 * 26 // 100
    assert flag.sum() == K == len(hi)
    assert len(hi) + len(lo) == 4096                      # Eq. (9): every token kept
    assert s[flag == 1].min() >= s[flag == 0].max()
    thr = s[flag == 1].min()
    tied = np.flatnonzero(s == thr)
    # equal scores at the threshold are taken by increasing index
    taken = tied[flag[tied] == 1]
    assert np.array_equal(taken, tied[: len(taken)])


def test_rank_all_equal_and_extremes():
    s = np.full(10, 3.0, np.float32)
    assert np.array_equal(np.flatnonzero(O.rank_k(s, 4)), [0, 1, 2, 3])
    assert O.rank_k(s, 0).sum() == 0 and O.rank_k(s, 10).sum() == 10


def test_rank_nan_is_an_error():
    with pytest.raises(O.OracleError):
        O.rank_k(np.array([1.0, np.nan], np.float32), 1)


@pytest.mark.parametrize("T,r,K", [(2048, (26, 100), 532), (32768, (26, 100), 8519),
                                    (16384, (26, 100), 4259), (131072, (40, 100), 52428),
                                    (4096, (25, 100), 1024), (7, (1, 2), 3)])
def test_top_count_floor(T, r, K):
    assert O.top_count(T, *r) == K == (Fraction(*r) * T).__floor__()


def test_block_count_round_half_even():
    assert O.block_count(64, 26, 100) == 17
    assert O.block_count(64, 25, 100) == 16
    assert O.block_count(64, 35, 100) == 22
    for n in range(0, 130):
        for r in [(1, 2), (26, 100), (35, 100), (3, 8), (1, 4)]:
            assert O.block_count(n, *r) == round(Fraction(r[0] * n, r[1]))
