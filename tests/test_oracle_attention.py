"""Pins of the oracle's decode attention (the consumer of the cache, Sec. 3.1,
Alg. 1): a textbook numpy formula, special cases, and the 16-level reduction
to FP16 attention."""
import numpy as np
import pytest

from oracle import oracle as O


def textbook(q, k, v):
    lg = q @ k.T / np.sqrt(q.shape[1])
    lg -= lg.max(1, keepdims=True)
    p = np.exp(lg)
    return (p / p.sum(1, keepdims=True)) @ v


@pytest.mark.parametrize("n", [1, 2, 7, 300])
def test_attention_textbook(n):
    rng = np.random.default_rng(n)
    q = rng.standard_normal((4, 128))
    k = rng.standard_normal((n, 128)) * 3
    v = rng.standard_normal((n, 128))
    assert np.allclose(O.attention(q, k, v), textbook(q, k, v), atol=1e-12, rtol=1e-12)


def test_special_cases():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((4, 128))
    v = rng.standard_normal((5, 128))
    k1 = rng.standard_normal((1, 128))
    assert np.allclose(O.attention(q, k1, v[:1]), np.repeat(v[:1], 4, 0), atol=1e-14)
    k = np.repeat(k1, 5, 0)
    assert np.allclose(O.attention(q, k, v), np.repeat(v.mean(0, keepdims=True), 4, 0), atol=1e-14)
    perm = rng.permutation(5)
    k = rng.standard_normal((5, 128))
    assert np.allclose(O.attention(q, k, v), O.attention(q, k[perm], v[perm]), atol=1e-13)
    big = np.zeros((2, 128)); big[0, 0] = 1e4      # no overflow: max is subtracted
    assert np.allclose(O.attention(np.eye(1, 128) * 50, big, v[:2]), v[:1], atol=1e-12)


def test_split_merge_identity():
    """The log-sum-exp merge of partial softmaxes over a split of the tokens
    equals the whole (the identity a split-K decode relies on)."""
    rng = np.random.default_rng(2)
    q = rng.standard_normal((4, 128)); k = rng.standard_normal((100, 128)) * 2
    v = rng.standard_normal((100, 128))
    parts = []
    for sl in (slice(0, 13), slice(13, 64), slice(64, 100)):
        lg = q @ k[sl].T / np.sqrt(128)
        m = lg.max(1, keepdims=True); p = np.exp(lg - m)
        parts.append((m, p.sum(1, keepdims=True), p @ v[sl]))
    M = np.max([m for m, _, _ in parts], 0)
    Lsum = sum(l * np.exp(m - M) for m, l, _ in parts)
    O_ = sum(o * np.exp(m - M) for m, _, o in parts) / Lsum
    assert np.allclose(O_, O.attention(q, k, v), atol=1e-12)


def test_sixteen_levels_reduce_to_fp16_attention():
    rng = np.random.default_rng(3)
    T = 512
    K = (rng.standard_normal((T, 128)) * np.where(np.arange(128) < 4, 10, 1)).astype(np.float16)
    V = rng.standard_normal((T, 128)).astype(np.float16)
    q = rng.standard_normal((4, 128)).astype(np.float16).astype(np.float64)
    kc, km = O.quantize_rows(K, 0, 16, 32)
    vc, vm = O.quantize_rows(V, 0, 16, 32)
    kh = O.dequantize_rows(kc, km, 0, 16, 32)
    vh = O.dequantize_rows(vc, vm, 0, 16, 32)
    sK = km[..., 0].view(np.float16).astype(np.float64).max(1)
    sV = vm[..., 0].view(np.float16).astype(np.float64).max()
    eps = np.abs(q).sum(1).max() * sK.max() * (0.5 + 16 * 2.0**-10) / np.sqrt(128)
    bound = (np.exp(2 * eps) - 1) * np.abs(vh).max() + sV * (0.5 + 16 * 2.0**-10)
    d = np.abs(O.attention(q, kh, vh) - O.attention(q, K.astype(np.float64), V.astype(np.float64)))
    assert d.max() <= bound
    # rows that are constant per group quantize exactly: equality with FP16 attention
    Kc = np.repeat(rng.standard_normal((T, 4)), 32, 1).astype(np.float16)
    Vc = np.repeat(rng.standard_normal((T, 4)), 32, 1).astype(np.float16)
    kc, km = O.quantize_rows(Kc, 0, 16, 32)
    vc, vm = O.quantize_rows(Vc, 0, 16, 32)
    a = O.attention(q, O.dequantize_rows(kc, km, 0, 16, 32), O.dequantize_rows(vc, vm, 0, 16, 32))
    assert np.array_equal(a, O.attention(q, Kc.astype(np.float64), Vc.astype(np.float64)))


def test_attention_units_equals_per_unit_attention():
    """The unit-parallel form (timing runs) computes each unit exactly as the
    one-unit call, whatever the unit sizes."""
    rng = np.random.default_rng(11)
    units = [(rng.standard_normal((4, 128)), rng.standard_normal((n, 128)), rng.standard_normal((n, 128)))
             for n in (1, 7, 64, 300, 2049)]
    for (q, k, v), got in zip(units, O.attention_units(units)):
        assert np.array_equal(got, O.attention(q, k, v))
