"""Pins of the oracle's own binary16 conversion against numpy's (an independent
implementation of IEEE round-to-nearest-even)."""
import numpy as np

from oracle import oracle as O


def test_f16_to_f32_exhaustive():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = O.f16_bits_to_f32(h)
    ref = h.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_f32_to_f16_random_and_edges():
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 2**32, 2_000_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    edges = np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, -65520.0, 2.0**-24, 2.0**-25,
                      1.5 * 2.0**-25, 2.0**-14, 2.0**-14 - 2.0**-25, 1.0 + 2.0**-11,
                      1.0 + 3 * 2.0**-11, np.inf, -np.inf, 1e-30, 7.5, 0.1, 1 / 3],
                     dtype=np.float32)
    # every f16 midpoint, exactly representable in f32
    h = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    mids = ((lo[:-1] + lo[1:]) / 2).astype(np.float32)
    for v in (x, edges, mids, -mids):
        got = O.f32_to_f16_bits(v)
        with np.errstate(over="ignore"):
            ref = v.astype(np.float16).view(np.uint16)
        ok = ~np.isnan(v)
        assert np.array_equal(got[ok], ref[ok])
        assert np.all((got[~ok] & 0x7C00) == 0x7C00) and np.all(got[~ok] & 0x3FF)
