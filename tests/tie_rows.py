"""Rows whose TurboQuant-MSE codes sit on exact threshold ties (test input
builder; it holds none of the method's arithmetic beyond what it checks in
numpy): a rotated coordinate y_j equals the fp32 product of the row's stored
fp16 norm and a Lloyd-Max threshold exactly."""
import numpy as np


def _fwht32_exact(u):
    """The unnormalized Sylvester transform in numpy fp32 (stages 1..64), and
    whether every butterfly was exact (compared with the fp64 result)."""
    a = u.astype(np.float32).copy()
    b = u.astype(np.float64).copy()
    h = 1
    while h < 128:
        for i in range(128):
            if not i & h:
                a[i], a[i + h] = a[i] + a[i + h], a[i] - a[i + h]
                b[i], b[i + h] = b[i] + b[i + h], b[i] - b[i + h]
        h <<= 1
    return b, np.array_equal(a.astype(np.float64), b)


def _norm_f16(x):
    """rho as the format fixes it: fp32 squares, the fixed pairwise tree, a
    correctly rounded fp32 square root (numpy's IEEE sqrt), fp16 RNE."""
    a = (x.astype(np.float32) ** 2).astype(np.float32)
    h = 64
    while h >= 1:
        a[:h] = (a[:h] + a[h:2 * h]).astype(np.float32)
        h >>= 1
    return np.float16(np.sqrt(np.float32(a[0])))


def _tie_row(rhof, thr32, j_pad):
    """A row x (fp16, sign mask all +) with y_0 = sum x = fl32(rhof * thr32)
    exactly and ||x|| rounding to rhof, or None.  y_0 = a + b with a, b fp16;
    norm padding w at channels j_pad and j_pad + 64 with opposite signs (it
    cancels in y_0).  w is searched so that the stored norm is rhof."""
    V = np.float32(np.float32(rhof) * thr32)
    a = np.float16(V)
    b = np.float16(np.float32(V) - np.float32(a))
    if np.float32(a) + np.float32(b) != V or not np.isfinite(a) or not np.isfinite(b):
        return None
    need = float(rhof) ** 2 - float(a) ** 2 - float(b) ** 2
    if need <= 0:
        return None
    w0 = np.sqrt(need / 2)
    for cand in np.unique(np.float16(w0 * (1 + np.arange(-40, 41) * 2.0 ** -11))):
        x = np.zeros(128, np.float16)
        x[0], x[1] = a, b
        x[j_pad], x[j_pad + 64] = cand, -cand
        if _norm_f16(x) == rhof:
            return x
    return None


def tq_tie_rows(tau32, per_threshold=3):
    """fp16 rows (sign mask all +) with an exact tie at each threshold of
    tau32: for a zero threshold two equal entries (y_j = 0 for odd j), else
    y_0 = fl32(rho * tau) built from two fp16 pieces plus norm padding."""
    rows = []
    for k, t in enumerate(tau32):
        found = 0
        for e in range(-6, 9):
            if found >= per_threshold:
                break
            for m in (1.0, 1.25, 1.5, 1.75, 1.125, 1.375, 1.625, 1.875):
                rhof = np.float16(m * 2.0 ** e)
                if t == 0:
                    x = np.zeros(128, np.float16)
                    x[0] = np.float16(float(rhof) / np.sqrt(2))
                    x[1] = x[0]
                else:
                    x = _tie_row(rhof, t, 5)
                if x is not None:
                    rows.append(x)
                    found += 1
                    if found >= per_threshold:
                        break
        assert found >= 1, "no tie row found for threshold %d" % k
    return rows
