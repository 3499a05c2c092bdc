"""Pins of the oracle's base quantizers: affine (Sec. 4.1) and
TurboQuant-MSE (Sec. 4.9)."""
import os

import numpy as np
import pytest
import scipy.integrate
import scipy.linalg
import scipy.stats

from oracle import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def nearest_grid(x, z, s, L):
    """argmin_k |x - (z + k s)| in exact float64; returns (code, tie_distance)."""
    s = np.broadcast_to(np.asarray(s, np.float64), np.broadcast(x, s).shape)
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(s > 0, (x - z) / np.where(s > 0, s, 1), 0.0)
    k = np.clip(np.floor(t + 0.5), 0, L - 1)
    frac = np.abs(t - np.floor(t) - 0.5)
    return k.astype(np.int64), frac


@pytest.mark.parametrize("L", [3, 5, 6, 16])
@pytest.mark.parametrize("G", [32, 128])
def test_affine_matches_nearest_grid_point(L, G):
    rng = np.random.default_rng(L * 1000 + G)
    X = (rng.standard_normal((500, 128)) * rng.choice([0.01, 1, 30], (500, 1))).astype(np.float16)
    X[0, :] = 1.5                                              # constant row
    X[1, ::2] = -0.0
    codes, meta = O.quantize_rows(X, 0, L, G)
    xf = X.astype(np.float64)
    for g in range(128 // G):
        sl = slice(g * G, (g + 1) * G)
        mn = X[:, sl].astype(np.float32).min(1)
        mx = X[:, sl].astype(np.float32).max(1)
        s16 = ((mx - mn) / np.float32(L - 1)).astype(np.float16)      # numpy's own IEEE ops
        assert np.array_equal(meta[:, g, 0], s16.view(np.uint16))
        assert np.array_equal(meta[:, g, 1], (mn + np.float32(0)).astype(np.float16).view(np.uint16))
        s = s16.astype(np.float64)[:, None]
        z = mn.astype(np.float64)[:, None]
        ref, frac = nearest_grid(xf[:, sl], z, s, L)
        got = codes[:, sl].astype(np.int64)
        # fp32 reciprocal-multiply may flip only points within a hair of a midpoint
        assert np.all((got == ref) | (frac < 1e-5))
        xhat = z + got * s
        err = np.abs(xhat - xf[:, sl])
        assert np.all(err <= s * (0.5 + L * 2.0**-10) + 1e-30)
        nz = s[:, 0] > 0
        amin = np.argmin(xf[:, sl], 1)
        amax = np.argmax(xf[:, sl], 1)
        assert np.all(got[np.arange(500), amin][nz] == 0)
        assert np.all(got[np.arange(500), amax][nz] == L - 1)
    assert np.all(codes[0] == 0) and np.all(meta[0, :, 0] == 0)


@pytest.mark.parametrize("L", [3, 5, 6])
def test_affine_exhaustive_fp16_in_range(L):
    h = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    v = h.view(np.float16)
    v = v[np.isfinite(v) & (np.abs(v.astype(np.float32)) <= 4)]
    n = (len(v) + 125) // 126
    X = np.zeros((n, 128), np.float16)
    X[:, 0], X[:, 1] = -4, 4
    flat = np.concatenate([v, np.zeros(n * 126 - len(v), np.float16)])
    X[:, 2:] = flat.reshape(n, 126)
    codes, meta = O.quantize_rows(X, 0, L, 128)
    s = np.float64(np.float16(np.float32(8) / np.float32(L - 1)))
    ref, frac = nearest_grid(X.astype(np.float64), -4.0, s, L)
    assert np.all((codes == ref) | (frac < 1e-5))


def read_max_table():
    rows = {}
    for line in open(os.path.join(GOLD, "lloyd_max_gaussian.txt")):
        if line.startswith("#") or not line.strip():
            continue
        L, outs, thr, mse = [p.strip() for p in line.split("|")]
        rows[int(L)] = ([float(x) for x in outs.split()], [float(x) for x in thr.split()], float(mse))
    return rows


@pytest.mark.parametrize("L", [2, 3, 4])
def test_lloyd_max_equals_published_table(L):
    outs, thr, mse = read_max_table()[L]
    mu, tau, m = O.lloyd_max(L)
    pos_mu = sorted(x for x in mu if x >= -1e-12)
    pos_tau = sorted(x for x in tau if x >= -1e-12)
    assert np.allclose(pos_mu, outs, atol=6e-4)
    assert np.allclose(pos_tau, thr, atol=6e-4)
    assert abs(m - mse) < 1e-4


@pytest.mark.parametrize("L", [2, 3, 4, 5, 6, 8])
def test_lloyd_max_fixed_point(L):
    mu, tau, mse = O.lloyd_max(L)
    edges = np.concatenate([[-np.inf], tau, [np.inf]])
    for k in range(L):
        a, b = edges[k], edges[k + 1]
        p = scipy.stats.norm.cdf(b) - scipy.stats.norm.cdf(a)
        m = scipy.integrate.quad(lambda x: x * scipy.stats.norm.pdf(x), a, b)[0] / p
        assert abs(m - mu[k]) < 1e-9                  # centroid condition
    assert np.allclose(tau, (mu[:-1] + mu[1:]) / 2)   # nearest-neighbour condition
    rng = np.random.default_rng(L)
    x = rng.standard_normal(1_000_000)
    q = mu[np.searchsorted(tau, x)]
    assert abs(np.mean((x - q) ** 2) - mse) < 3e-3


def test_tq_row_against_dense_hadamard():
    rng = np.random.default_rng(5)
    H = scipy.linalg.hadamard(128).astype(np.float64)
    X = rng.standard_normal((300, 128)).astype(np.float32)
    X[:, [3, 40, 77, 100]] *= 10
    X = X.astype(np.float16)
    sw = rng.integers(0, 2**32, 4, dtype=np.uint64).astype(np.uint32)
    sign = np.array([-1.0 if (sw[i // 32] >> (i % 32)) & 1 else 1.0 for i in range(128)])
    for L in (3, 4):
        mu32, tau32 = O.codebook32(L)
        codes, rho = O.quantize_rows(X, 1, L, 128, sw)
        xf = X.astype(np.float64)
        nrm = np.linalg.norm(xf, axis=1)
        assert np.array_equal(rho, nrm.astype(np.float16).view(np.uint16)) or \
            np.all(np.abs(rho.view(np.float16).astype(np.float64) - nrm) <= nrm * 2.0**-10)
        rf = rho.view(np.float16).astype(np.float64)[:, None]
        y = (xf * sign) @ H.T                                      # H diag(sign) x
        assert np.allclose((y ** 2).sum(1), 128 * nrm ** 2)         # Parseval for H/sqrt(128)
        ref = np.searchsorted(tau32.astype(np.float64), y / rf, side="left")
        near = np.min(np.abs((y / rf)[..., None] - tau32[None, None, :]), -1) < 1e-5
        assert np.all((codes == ref) | near)
        xhat = O.dequantize_rows(codes, rho, 1, L, 128, sw)
        ref_hat = ((rf * mu32.astype(np.float64)[codes]) @ H) * sign / 128
        assert np.allclose(xhat, ref_hat, atol=1e-12)
        rel = np.mean((xhat - xf) ** 2) / np.mean(xf ** 2)
        assert rel < O.lloyd_max(L)[2] * 1.3


def test_nonfinite_input_is_reported():
    X = np.zeros((2, 128), np.float16)
    X[1, 5] = np.inf
    with pytest.raises(O.OracleError):
        O.quantize_rows(X, 0, 5, 128)
    with pytest.raises(O.OracleError):
        O.quantize_rows(X, 1, 3, 128, np.zeros(4, np.uint32))


def test_tq_norm_is_correctly_rounded_at_fp16_edges():
    """rho = RN16(RN32(sqrt(sum of squares))) on rows built to sit within one
    fp32 ulp of an fp16 rounding midpoint (Sec. 4.9: the stored norm)."""
    from tests.norm_edge import correctly_rounded_norm_f16, edge_rows
    X = edge_rows(64)
    sw = np.zeros(4, np.uint32)
    _, rho = O.quantize_rows(X, 1, 4, sign_words=sw)
    assert np.array_equal(np.asarray(rho, np.uint16).reshape(-1), correctly_rounded_norm_f16(X))
