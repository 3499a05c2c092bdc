"""Size arithmetic of the packed format (the same rules as csrc/semkv_fmt.h),
for byte accounting in the benchmark: a symbol packs n codes of base L in the
least number of bits, n = 8, 5, 4, 3, 5, 7, 2 for L = 2 .. 8 (mixed-radix
packing, SemKV Sec. 4.1)."""

DIGITS = {2: 8, 3: 5, 4: 4, 5: 3, 6: 5, 7: 7, 8: 2}


def width(L, nd):
    w = 0
    while (1 << w) < L ** nd:
        w += 1
    return w


def line_bits(L, nvalues):
    """Bits of one line of nvalues codes (a 128-channel token row or a
    64-slot channel column)."""
    n = DIGITS[L]
    bits = (nvalues // n) * width(L, n)
    if nvalues % n:
        bits += width(L, nvalues % n)
    return bits
