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


@pytest.mark.parametrize("L", [2, 3, 5, 6, 7, 8, 16])
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


@pytest.mark.parametrize("L", [2, 3, 5, 6, 7, 8])
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


def sign_vector(sw):
    return np.array([-1.0 if (int(sw[i // 32]) >> (i % 32)) & 1 else 1.0 for i in range(128)])


@pytest.mark.parametrize("L", [3, 5, 6])
@pytest.mark.parametrize("G", [32, 128])
def test_rotated_affine_is_affine_of_the_library_rotation(L, G):
    """On rows whose rotation is exact in fp32 and fp16 (x on a 1/4 grid in
    [-2, 2], so y = H diag(sign) x / 16 lies on a 1/64 grid within 16), the
    rotated quantizer equals the pinned affine quantizer applied to y computed
    with the library's dense Sylvester matrix (Sec. 4.1: affine codes under a
    Hadamard rotation).  A dropped or misplaced sign, another scaling, another
    Hadamard ordering or groups over the wrong coordinates all change the
    codes or the parameters."""
    rng = np.random.default_rng(100 + L * 10 + G)
    H = scipy.linalg.hadamard(128).astype(np.float64)
    n = 400
    X = rng.integers(-8, 9, (n, 128)).astype(np.float64) / 4
    X[:, [3, 40, 77, 100]] = rng.choice([-2.0, 2.0], (n, 4))
    X[0] = 0.25                                                # one non-zero coordinate after H
    X[1] = 0.0                                                 # all zero: scale 0
    sw = rng.integers(0, 2**32, 4, dtype=np.uint64).astype(np.uint32)
    Y = (X * sign_vector(sw)) @ H.T / 16
    assert np.array_equal(Y.astype(np.float16).astype(np.float64), Y)
    X16 = X.astype(np.float16)
    codes, meta = O.quantize_rows(X16, O.ROT_AFFINE, L, G, sw)
    rcodes, rmeta = O.quantize_rows(Y.astype(np.float16), O.AFFINE, L, G)
    assert np.array_equal(codes, rcodes)
    assert np.array_equal(meta, rmeta)
    assert np.all(codes[1] == 0) and np.all(meta[1] == 0)


def test_rotated_affine_dequantization_and_error_bound():
    """x_hat = diag(sign) H y_hat / 8 with y_hat the affine reconstruction
    (the pinned base-0 dequantization); by orthogonality of H / sqrt(128),
    ||x - x_hat|| = sqrt(128)/8 ||y - y_hat||, and every rotated coordinate
    is within half a step (plus fp16 rounding of the stored zero) of its
    reconstruction."""
    rng = np.random.default_rng(7)
    H = scipy.linalg.hadamard(128).astype(np.float64)
    X = rng.standard_normal((300, 128)).astype(np.float32)
    X[:, [3, 40, 77, 100]] *= 10
    X = X.astype(np.float16)
    xf = X.astype(np.float64)
    sw = rng.integers(0, 2**32, 4, dtype=np.uint64).astype(np.uint32)
    sign = sign_vector(sw)
    y = (xf * sign) @ H.T / 16
    for L, G in ((5, 128), (6, 128), (6, 32), (3, 64)):
        codes, meta = O.quantize_rows(X, O.ROT_AFFINE, L, G, sw)
        yhat = O.dequantize_rows(codes, meta, O.AFFINE, L, G)
        xhat = O.dequantize_rows(codes, meta, O.ROT_AFFINE, L, G, sw)
        assert np.allclose(xhat, sign * (yhat @ H.T) / 8, rtol=0, atol=1e-12)
        s = np.repeat(meta[:, :, 0].view(np.float16).astype(np.float64), G, axis=1)
        z = np.repeat(meta[:, :, 1].view(np.float16).astype(np.float64), G, axis=1)
        # zero is min y rounded to fp16: a value below it may sit up to that
        # rounding under code 0; the top code may round the step down as well
        slack = np.abs(z) * 2.0**-11 + s * L * 2.0**-11 + 1e-6 * np.abs(y)
        assert np.all(np.abs(yhat - y) <= s / 2 + slack + 1e-12)
        lhs = np.linalg.norm(xhat - xf, axis=1)
        rhs = np.sqrt(128) / 8 * np.linalg.norm(yhat - y, axis=1)
        assert np.allclose(lhs, rhs, rtol=1e-9, atol=1e-9)
        # rotation spreads the outlier channels: far below the unrotated error
        if G == 128:
            c0, m0 = O.quantize_rows(X, O.AFFINE, L, G)
            e0 = np.mean((O.dequantize_rows(c0, m0, O.AFFINE, L, G) - xf) ** 2)
            assert np.mean((xhat - xf) ** 2) < 0.5 * e0


def test_rotated_affine_nonfinite_and_sign_words():
    X = np.zeros((2, 128), np.float16)
    X[1, 5] = np.nan
    with pytest.raises(O.OracleError):
        O.quantize_rows(X, O.ROT_AFFINE, 6, 128, np.zeros(4, np.uint32))
    # flipping every sign negates y: zero and scale follow the negated row
    rng = np.random.default_rng(3)
    Xr = (rng.integers(-8, 9, (50, 128)) / 4).astype(np.float16)
    a = O.quantize_rows(Xr, O.ROT_AFFINE, 6, 128, np.zeros(4, np.uint32))
    b = O.quantize_rows(-Xr, O.ROT_AFFINE, 6, 128, np.full(4, 0xFFFFFFFF, np.uint32))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    # the least fp16 subnormal in one channel rotates to +-2^-28 everywhere:
    # the zero rounds to -0 in fp16 and is stored as +0 (Sec. 4.1 parameters)
    Xs = np.zeros((4, 128), np.float16)
    Xs[:, 9] = np.float16(2.0**-24)
    c, m = O.quantize_rows(Xs, O.ROT_AFFINE, 5, 32, np.zeros(4, np.uint32))
    assert np.all(m == 0) and np.all(c == 0)
