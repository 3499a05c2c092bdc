"""Independent reader of the packed tile format, written with Python integers
(test infrastructure; shares nothing with the oracle's C packer or the HIP
kernels).  Format (mixed-radix packing, Sec. 4.1):

* a symbol holds n codes of base L as sum_i c_i L^i and takes the least w bits
  with 2^w >= L^n; n = 5, 4, 3, 5 for L = 3, 4, 5, 6 (and 8, 1, 2 for L = 2, 8, 16);
  a line's last symbol holds the remainder digits;
* a K line is one token row (128 channels), a V line one channel column over
  the 64 slots of a tile; segment j of a line is its symbols p = j, j+4, ...;
* a body is segment 0 of every line, then segment 1, 2, 3, bits LSB-first.
"""
DIGITS = {2: 8, 3: 5, 4: 4, 5: 3, 6: 5, 7: 7, 8: 2, 16: 2}


def sym_bits(L, n):
    w = 0
    while (1 << w) < L ** n:
        w += 1
    return w


def line_symbols(L, nvalues):
    n = DIGITS[L]
    return [(p, min(n, nvalues - n * p)) for p in range((nvalues + n - 1) // n)]


def decode_body(body: bytes, L: int, kind: str):
    """-> codes[slot][channel] (64 x 128 list of lists)."""
    big = int.from_bytes(bytes(body), "little")
    nlines, nvals = (64, 128) if kind == "K" else (128, 64)
    n = DIGITS[L]
    lines = [[0] * nvals for _ in range(nlines)]
    pos = 0
    syms = line_symbols(L, nvals)
    for j in range(4):
        for ln in range(nlines):
            for p, nd in syms:
                if p % 4 != j:
                    continue
                w = sym_bits(L, nd)
                v = (big >> pos) & ((1 << w) - 1)
                pos += w
                for i in range(nd):
                    v, c = divmod(v, L)
                    lines[ln][n * p + i] = c
                assert v == 0, "symbol exceeds L^n"
    assert big >> pos == 0, "bits set beyond the last segment"
    if kind == "K":
        return lines
    return [[lines[c][t] for c in range(128)] for t in range(64)]
