"""Exact pins of the oracle's quantizers where a rule, not a tolerance,
decides the result (Sec. 4.1 affine base, Sec. 4.9 TurboQuant-MSE base):

* exact ties of the affine code rounding (round half to even, reading R5),
  on rows whose arithmetic is exact in fp32, expected codes from rational
  arithmetic;
* exact ties of the Lloyd-Max threshold test (strict >, an exact tie goes to
  the lower cell, reading R8), on rows built so that a rotated
  coordinate equals the fp32 product of the stored norm and a threshold;
* fp16 parameters that would overflow (2-level affine scale, rotated-affine
  zero and scale) saturate at +-65504 (reading R18): finite input never
  yields non-finite parameters or reconstructions.

Expected values come from Python Fractions and plain IEEE operations of
numpy, never from the oracle itself."""
from fractions import Fraction

import numpy as np
import pytest
import scipy.linalg

from oracle import oracle as O
from tests.tie_rows import _fwht32_exact, _norm_f16, tq_tie_rows

F16_MAX = 65504.0


def frac(x):
    return Fraction(float(x))


def f16_sat_bits(x32):
    """fp16 rounding (RNE, numpy) of an fp32 value, +-inf replaced by +-65504."""
    with np.errstate(over="ignore"):
        h = np.float16(np.float32(x32))
    if np.isinf(h):
        h = np.float16(np.copysign(F16_MAX, float(h)))
    return np.array([h]).view(np.uint16)[0]


# --------------------------------------------------- affine: exact ties --

@pytest.mark.parametrize("L", [2, 3, 5, 6, 7, 8])
@pytest.mark.parametrize("G", [32, 128])
def test_affine_exact_ties_round_half_to_even(L, G):
    """Rows with min z and max z + (L-1) 2^-k: the stored scale is exactly
    2^-k, its reciprocal 2^k, and (x - z) 2^k is exact in fp32 for x on a
    2^-(k+1) grid, so every half-step value is an exact tie.  The code must be
    the even neighbour, read off with Fraction's round (half to even)."""
    rng = np.random.default_rng(10 * L + G)
    rows = []
    for k in (0, 2, 5):
        for z in (0.0, -3.0, 1.5):
            step = 2.0 ** -k
            row = np.empty(128)
            for g in range(128 // G):
                sl = slice(g * G, (g + 1) * G)
                v = z + rng.integers(0, 2 * (L - 1) + 1, G) * step / 2
                v[0], v[1] = z, z + (L - 1) * step
                row[sl] = v
            rows.append(row)
    X = np.array(rows).astype(np.float16)
    assert np.array_equal(X.astype(np.float64), np.array(rows))           # exact in fp16
    codes, meta = O.quantize_rows(X, O.AFFINE, L, G)
    n_ties = 0
    for i, row in enumerate(rows):
        k = (0, 2, 5)[i // 3]
        z = (0.0, -3.0, 1.5)[i % 3]
        for g in range(128 // G):
            assert meta[i, g, 0] == np.array([np.float16(2.0 ** -k)]).view(np.uint16)[0]
            assert meta[i, g, 1] == np.array([np.float16(z)]).view(np.uint16)[0]
        for j in range(128):
            t = (Fraction(row[j]) - Fraction(z)) * 2 ** k
            want = min(max(round(t), 0), L - 1)                              # half to even
            n_ties += t.denominator == 2
            assert codes[i, j] == want, (i, j, t, codes[i, j], want)
    assert n_ties > 50


def test_affine_tie_examples_by_hand():
    """Scale 1, zero 0, 6 levels: 0.5 -> 0, 1.5 -> 2, 2.5 -> 2, 3.5 -> 4,
    4.5 -> 4 (a round-half-up rule would give 1, 2, 3, 4, 5)."""
    row = np.zeros(128, np.float16)
    row[:7] = [0, 5, 0.5, 1.5, 2.5, 3.5, 4.5]
    codes, _ = O.quantize_rows(row[None], O.AFFINE, 6, 128)
    assert list(codes[0, :7]) == [0, 5, 0, 2, 2, 4, 4]


# ------------------------------------------- tq: exact threshold ties --

@pytest.mark.parametrize("L", [3, 4])
def test_tq_threshold_exact_ties_go_to_the_lower_cell(L):
    """Rows whose rotated coordinate y_j equals fl32(rho * tau_k) exactly, for
    every threshold tau_k (for 4 levels the middle threshold is 0: a zero
    coordinate).  The code must count only thresholds strictly below y_j."""
    mu32, tau32 = O.codebook32(L)
    rows = tq_tie_rows(tau32)
    X = np.array(rows)
    sw = np.zeros(4, np.uint32)
    codes, rho = O.quantize_rows(X, O.TQ, L, sign_words=sw)
    H = scipy.linalg.hadamard(128)
    n_ties = 0
    for i, x in enumerate(X):
        y, exact = _fwht32_exact(x.astype(np.float64))
        assert exact, "row %d: the fp32 transform is not exact" % i
        assert np.array_equal(y, H @ x.astype(np.float64))
        rf = np.float16(np.array([rho[i]], np.uint16).view(np.float16)[0])
        assert rf == _norm_f16(x)
        thr = [np.float32(np.float32(rf) * t) for t in tau32]          # the fp32 products the test compares with
        for j in range(128):
            want = sum(1 for th in thr if Fraction(y[j]) > frac(th))
            n_ties += any(Fraction(y[j]) == frac(th) for th in thr)
            assert codes[i, j] == want, (i, j, y[j], thr, codes[i, j], want)
    assert n_ties >= len(tau32)


# ------------------------------------------------------- saturation -----

def test_affine_two_levels_saturates_the_scale():
    """2 levels over a range above 65504: (max - min) / 1 overflows fp16; the
    scale is stored as 65504 and codes are the nearest of {zero, zero +
    65504} (clamped)."""
    X = np.zeros((3, 128), np.float16)
    X[0, :64], X[0, 64:] = -60000, 60000
    X[1] = np.linspace(-65504, 65504, 128).astype(np.float16)
    X[2, ::2], X[2, 1::2] = -40000, 30000
    codes, meta = O.quantize_rows(X, O.AFFINE, 2, 128)
    for i in range(3):
        mn, mx = X[i].astype(np.float32).min(), X[i].astype(np.float32).max()
        assert meta[i, 0, 0] == f16_sat_bits(np.float32(mx - mn))
        assert meta[i, 0, 1] == np.array([np.float16(mn)]).view(np.uint16)[0]
        s = frac(np.array([meta[i, 0, 0]], np.uint16).view(np.float16)[0])
        for j in range(128):
            t = (frac(X[i, j]) - frac(mn)) / s
            assert codes[i, j] == min(max(round(t), 0), 1)
    assert np.all(meta[:2, 0, 0] == 0x7BFF) and meta[2, 0, 0] == f16_sat_bits(70000.0)
    xh = O.dequantize_rows(codes, meta, O.AFFINE, 2, 128)
    assert np.all(np.isfinite(xh))


@pytest.mark.parametrize("L", [3, 5, 6])
@pytest.mark.parametrize("G", [32, 128])
def test_rotated_affine_saturates_zero_and_scale(L, G):
    """Rows whose rotated coordinates leave the fp16 range (y = H x / 16 of a
    row of -9000 has y_0 = -72000): zero and scale are stored saturated at
    +-65504, codes against the stored pair, reconstruction finite.  Expected
    parameters and codes from the exact rotation (integer rows: every fp32
    sum is exact)."""
    H = scipy.linalg.hadamard(128).astype(np.float64)
    rows = [np.full(128, -9000.0), np.full(128, 9000.0), np.zeros(128)]
    rows[2][:8] = [65504, -65504, 65504, 65504, -65504, 65504, 65504, 65504]
    rng = np.random.default_rng(G + L)
    rows.append(rng.choice([-65504.0, 65504.0, 0.0], 128))
    X = np.array(rows).astype(np.float16)
    sw = np.zeros(4, np.uint32)
    codes, meta = O.quantize_rows(X, O.ROT_AFFINE, L, G, sw)
    Y = X.astype(np.float64) @ H.T / 16
    assert np.abs(Y).max() > F16_MAX
    for i in range(len(rows)):
        for g in range(128 // G):
            y = Y[i, g * G:(g + 1) * G]
            z16 = f16_sat_bits(np.float32(y.min()))
            z16 = 0 if z16 == 0x8000 else z16
            zf = np.float32(np.array([z16], np.uint16).view(np.float16)[0])
            s32 = np.float32(np.float32(y.max()) - zf) / np.float32(L - 1)
            s16 = f16_sat_bits(max(np.float32(s32), np.float32(0)))
            assert meta[i, g, 1] == z16 and meta[i, g, 0] == s16, (i, g)
            sf = np.float32(np.array([s16], np.uint16).view(np.float16)[0])
            inv = np.float32(1) / sf if sf != 0 else np.float32(0)
            for jj, yj in enumerate(y):
                c = np.float32(np.float32(np.float32(yj) - zf) * inv)    # the format's fp32 steps
                want = min(max(round(frac(c)), 0), L - 1)
                assert codes[i, g * G + jj] == want
    assert np.all((meta & 0x7C00) != 0x7C00)                             # no inf / NaN stored
    xh = O.dequantize_rows(codes, meta, O.ROT_AFFINE, L, G, sw)
    assert np.all(np.isfinite(xh))


@pytest.mark.parametrize("base,levels", [(O.AFFINE, (2, 3, 5, 6, 7, 8)), (O.ROT_AFFINE, (3, 4, 5, 6, 7, 8))])
def test_finite_input_gives_finite_parameters(base, levels):
    """Random rows over the whole finite fp16 range (uniform bit patterns,
    extremes, constant rows): every stored parameter is finite and every
    reconstruction is finite."""
    rng = np.random.default_rng(base)
    bits = rng.integers(0, 0x7C00, (400, 128), dtype=np.uint32).astype(np.uint16)
    bits |= (rng.integers(0, 2, (400, 128)) << 15).astype(np.uint16)
    X = bits.view(np.float16).copy()
    X[:50] = rng.choice([-65504, 65504, -1e-7, 0], (50, 128)).astype(np.float16)
    X[50] = 65504
    X[51] = -65504
    sw = rng.integers(0, 2**32, 4, dtype=np.uint64).astype(np.uint32)
    for L in levels:
        for G in (32, 128):
            codes, meta = O.quantize_rows(X, base, L, G, sw)
            assert np.all((meta & 0x7C00) != 0x7C00), (L, G)
            xh = O.dequantize_rows(codes, meta, base, L, G, sw)
            assert np.all(np.isfinite(xh)), (L, G)
