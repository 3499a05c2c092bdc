"""Pins of the oracle's token-importance indicators (Sec. 3.3): delta-norm
(Eq. 3), norm, variance and cosine-delta of the hidden states, key-/value-norm
of the cache tensors.  Closed forms on exactly representable inputs, special
cases that reduce to library routines, and invariances."""
import numpy as np
import pytest
import scipy.spatial.distance as dist

from oracle import oracle as O


def grid_states(rng, m, T, d, lo=-64, hi=65, scale=8):
    """fp16-exact states: integers / scale."""
    return (rng.integers(lo, hi, (m + 1, T, d)) / scale).astype(np.float16)


def test_delta_norm_closed_forms():
    rng = np.random.default_rng(1)
    T, d, m = 9, 256, 4
    h0 = grid_states(rng, 0, T, d)[0].astype(np.float64)
    # constant drift: every layer adds the same delta of norm 0.5 sqrt(d)
    delta = rng.choice([-0.5, 0.5], (T, d))
    H = np.stack([h0 + k * delta for k in range(m + 1)]).astype(np.float16)
    assert np.array_equal(O.score_hidden(O.DELTA_NORM, H), np.full(T, 0.5 * np.sqrt(d)))
    # one channel moving by c_k: the mean of |c_k - c_{k-1}|, not |c_m - c_0| / m
    c = np.array([0.0, 3.0, 1.0, 1.5, 7.0])
    H = np.stack([h0 for _ in range(m + 1)])
    H[:, :, 17] += c[:, None]
    got = O.score_hidden(O.DELTA_NORM, H.astype(np.float16))
    assert np.allclose(got, np.abs(np.diff(c)).mean(), rtol=0, atol=1e-12)


def test_delta_norm_m1_is_euclidean_distance_and_invariances():
    rng = np.random.default_rng(2)
    H = rng.standard_normal((2, 40, 512)).astype(np.float16)
    want = [dist.euclidean(H[1, t].astype(np.float64), H[0, t].astype(np.float64)) for t in range(40)]
    assert np.allclose(O.score_hidden(O.DELTA_NORM, H), want, rtol=1e-13)
    G = grid_states(rng, 3, 20, 128, lo=-16, hi=17)
    base = O.score_hidden(O.DELTA_NORM, G)
    shift = (rng.integers(-16, 17, 128) / 8).astype(np.float16)       # exact: |sum| <= 4
    assert np.array_equal(O.score_hidden(O.DELTA_NORM, (G.astype(np.float32) + shift).astype(np.float16)), base)
    perm = rng.permutation(128)
    assert np.allclose(O.score_hidden(O.DELTA_NORM, G[:, :, perm]), base, rtol=1e-14)
    assert np.array_equal(O.score_hidden(O.DELTA_NORM, G * np.float16(2)), 2 * base)


def test_norm_and_variance():
    rng = np.random.default_rng(3)
    H = rng.standard_normal((3, 30, 300)).astype(np.float16)            # d need not be a power of 2
    last = H[-1].astype(np.float64)
    assert np.allclose(O.score_hidden(O.NORM, H), np.linalg.norm(last, axis=1), rtol=1e-14)
    assert np.allclose(O.score_hidden(O.VARIANCE, H), np.var(last, axis=1), rtol=1e-12)
    # the last state only, not the first
    H2 = H.copy()
    H2[0] = 0
    assert np.array_equal(O.score_hidden(O.NORM, H2), O.score_hidden(O.NORM, H))
    # two values a, b in equal numbers: variance ((a - b) / 2)^2 (population)
    X = np.zeros((1, 4, 64), np.float16)
    X[0, :, :32], X[0, :, 32:] = 3.0, -1.0
    assert np.array_equal(O.score_hidden(O.VARIANCE, X), np.full(4, 4.0))
    assert np.array_equal(O.score_hidden(O.NORM, X), np.full(4, np.sqrt(32 * 9 + 32)))


def test_cosine_delta():
    rng = np.random.default_rng(4)
    H = rng.standard_normal((2, 25, 256)).astype(np.float16)
    want = [dist.cosine(H[1, t].astype(np.float64), H[0, t].astype(np.float64)) for t in range(25)]
    assert np.allclose(O.score_hidden(O.COSINE_DELTA, H), want, rtol=1e-12, atol=1e-15)
    # quarter turns in a plane: 1 - cos(90 deg) = 1 per step; opposite: 2
    X = np.zeros((3, 2, 8), np.float16)
    X[0, :, 0], X[1, :, 1], X[2, :, 1] = 1.0, 2.0, -0.5
    assert np.array_equal(O.score_hidden(O.COSINE_DELTA, X), np.full(2, 1.5))
    # positive scaling of a state leaves it unchanged; a zero state counts as orthogonal
    G = grid_states(rng, 2, 10, 64)
    Gs = G.copy()
    Gs[1] *= np.float16(4)
    assert np.allclose(O.score_hidden(O.COSINE_DELTA, Gs), O.score_hidden(O.COSINE_DELTA, G), rtol=1e-13)
    Z = np.zeros((2, 1, 16), np.float16)
    Z[1, 0, 3] = 1.0
    assert np.array_equal(O.score_hidden(O.COSINE_DELTA, Z), [1.0])


def test_kv_norm():
    rng = np.random.default_rng(5)
    X = rng.standard_normal((6, 50, 128)).astype(np.float16)           # 6 rows = layers x kv heads
    cat = np.transpose(X, (1, 0, 2)).reshape(50, -1).astype(np.float64)
    assert np.allclose(O.score_kv_norm(X), np.linalg.norm(cat, axis=1), rtol=1e-14)
    C = np.full((4, 3, 128), 0.5, np.float16)
    assert np.array_equal(O.score_kv_norm(C), np.full(3, 0.5 * np.sqrt(4 * 128)))


def test_bf16_states_and_errors():
    import torch
    rng = np.random.default_rng(6)
    bits = rng.integers(0, 2**16, (3, 5, 64), dtype=np.uint16)
    bits[(bits & 0x7F80) == 0x7F80] = 0x3F80                              # no inf / NaN
    ref = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).float().numpy()
    assert np.array_equal(O.bf16_bits_to_f32(bits), ref)
    with pytest.raises(O.OracleError):
        O.score_hidden(O.DELTA_NORM, np.zeros((1, 3, 8), np.float16))    # m = 0
    with pytest.raises(O.OracleError):
        O.score_hidden(O.NORM, np.full((1, 2, 8), np.inf, np.float16))
