"""Seeded search for 128-channel fp16 rows whose norm sits at an fp16 rounding
edge: the fp32 sum of squares (fixed pairwise tree) has a square root within
one fp32 ulp of the midpoint between two fp16 values, so a square root that is
off by one ulp would move the stored norm by one fp16 ulp (test input
generator; no quantizer arithmetic)."""
import numpy as np


def tree_sum_squares(X):
    a = (X.astype(np.float32) ** 2).astype(np.float32)
    for h in (64, 32, 16, 8, 4, 2, 1):
        a[:, :h] = (a[:, :h] + a[:, h:2 * h]).astype(np.float32)
    return a[:, 0]


def correctly_rounded_norm_f16(X):
    """fp16 bits of RN16(RN32(sqrt(s))), s the fp32 tree sum, via exact double
    arithmetic: RN32 of a correctly rounded double sqrt is correctly rounded."""
    s = tree_sum_squares(X)
    r32 = np.sqrt(s.astype(np.float64)).astype(np.float32)
    return r32.astype(np.float16).view(np.uint16)


def edge_rows(n, seed=11):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        X = rng.standard_normal((1 << 16, 128), dtype=np.float32).astype(np.float16)
        s = tree_sum_squares(X)
        r32 = np.sqrt(s.astype(np.float64)).astype(np.float32)
        up = np.nextafter(r32, np.float32(np.inf))
        dn = np.nextafter(r32, np.float32(0))
        f = lambda v: v.astype(np.float16).view(np.uint16)
        hit = (f(up) != f(r32)) | (f(dn) != f(r32))
        out.extend(X[hit])
    return np.stack(out[:n])
