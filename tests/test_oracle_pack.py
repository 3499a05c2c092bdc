"""Pins of the mixed-radix packing (Sec. 4.1) and of the storage accounting
(Sec. 4.1, Sec. 4.5, Tab. 5, Tab. 6)."""
import os

import numpy as np
import pytest

from oracle import oracle as O
from tests import formatref as F

GOLD = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("L", [2, 3, 4, 5, 6, 7, 8, 16])
def test_symbol_rates_and_bounds(L):
    n = O.symbol_digits(L)
    assert n == F.DIGITS[L]
    w = O.symbol_bits(L, n)
    assert L ** n <= 2 ** w < 2 * L ** n                      # least width
    assert {5: (3, 7), 6: (5, 13)}.get(L, (n, w)) == (n, w)   # 3 in 7 bits, 5 in 13 bits


@pytest.mark.parametrize("L", [2, 3, 4, 5, 6, 7, 8, 16])
@pytest.mark.parametrize("seed", [0, 1])
def test_pack_roundtrip_bigint(L, seed):
    rng = np.random.default_rng(seed * 100 + L)
    kc = rng.integers(0, L, (64, 128)).astype(np.uint8)
    vc = rng.integers(0, L, (64, 128)).astype(np.uint8)
    if seed:                                     # a partial tile: unused slots are zero
        kc[37:] = 0
        vc[37:] = 0
    kb, vb = O.pack_tile(kc, vc, L)
    assert len(kb) == O.tile_bytes(L) and len(kb) % 16 == 0
    assert np.array_equal(np.array(F.decode_body(kb.tobytes(), L, "K")), kc)
    assert np.array_equal(np.array(F.decode_body(vb.tobytes(), L, "V")), vc)


def test_tile_sizes():
    assert [O.tile_bytes(L) for L in (3, 4, 5, 6)] == [1648, 2048, 2400, 2672]
    # the uniform-grid levels: 8 codes per byte (1 bit), two 8-level codes in
    # 6 bits (3 bits), seven 7-level codes in 20 bits (2.857 bits, 1.8 % over log2 7)
    assert O.line_bits(2, 128) == 128 and O.line_bits(8, 128) == 384
    assert O.line_bits(7, 128) == 18 * 20 + 6 and O.line_bits(7, 64) == 9 * 20 + 3
    assert [O.tile_bytes(L) for L in (2, 7, 8)] == [1024, 2928, 3072]
    assert abs(20 / 7 / np.log2(7) - 1 - 0.0177) < 1e-3
    assert O.line_bits(6, 128) == 25 * 13 + 8 and O.line_bits(5, 128) == 42 * 7 + 5
    assert O.line_bits(4, 128) == 256 and O.line_bits(3, 128) == 25 * 8 + 5


def test_worked_example():
    kc = np.zeros((64, 128), np.uint8)
    kc[0, :4] = [1, 2, 3, 4]
    kb, vb = O.pack_tile(kc, kc, 5)
    for line in open(os.path.join(GOLD, "packing_worked_example.txt")):
        if line.startswith("#") or line.startswith("L |") or not line.strip():
            continue
        L, body, byte, value = [p.strip() for p in line.split("|")]
        assert int(L) == 5
        assert (kb if body == "K" else vb)[int(byte)] == int(value), line


def test_pack_rejects_out_of_range_code():
    kc = np.zeros((64, 128), np.uint8)
    kc[3, 3] = 5
    with pytest.raises(O.OracleError):
        O.pack_tile(kc, kc * 0, 5)


def read_accounting():
    out = {}
    for line in open(os.path.join(GOLD, "paper_accounting.txt")):
        if line.startswith("#") or not line.strip():
            continue
        name, code, eff, ratio, _ = [p.strip() for p in line.split("|")]
        f = lambda s: None if s == "-" else float(s)
        out[name] = (f(code), f(eff), f(ratio))
    return out


def test_paper_accounting():
    A = read_accounting()
    rate = {L: O.symbol_bits(L, O.symbol_digits(L)) / O.symbol_digits(L) for L in (2, 3, 4, 5, 6, 8)}
    assert abs(rate[5] - A["pack_rate_L5"][0]) < 5e-4 and abs(rate[6] - A["pack_rate_L6"][0]) < 5e-4
    aff = {"3.0": 8, "2.585": 6, "2.322": 5, "2.0": 4}
    for b, L in aff.items():
        code, eff, ratio = A["uniform_affine_" + b]
        assert abs(rate[L] - code) < 5e-4 and abs(rate[L] + 0.25 - eff) < 1e-3
        assert abs(16 / (rate[L] + 0.25) - ratio) < 0.05
    tq = {"3.0": 8, "2.585": 6, "2.322": 5, "2.0": 4, "1.585": 3, "1.0": 2}
    for b, L in tq.items():
        code, eff, ratio = A["tq_uniform_" + b]
        assert abs(rate[L] - code) < 5e-4 and abs(rate[L] + 0.125 - eff) < 1e-3
        if ratio:
            assert abs(16 / (rate[L] + 0.125) - ratio) < 0.05
    # SemKV mixes: r = 25 % at 6/5 levels (affine); r = 75 % at 4/3 levels (tq)
    code = 0.25 * rate[6] + 0.75 * rate[5]
    c, e, r = A["semkv_affine_r25"]
    assert abs(code - c) < 0.015 and abs(code + 0.25 - e) < 0.005 and abs(16 / (code + 0.25) - r) < 0.01
    c, e, r = A["tq_semkv_2.0_1.585_r75"]
    code = 0.75 * rate[4] + 0.25 * rate[3]
    assert abs(code - c) < 1e-3 and abs(code + 0.125 - e) < 1e-3 and abs(16 / (code + 0.125) - r) < 0.01
    c, e, _ = A["tq_semkv_2.585_2.322"]
    code = 0.25 * rate[6] + 0.75 * rate[5]
    assert abs(code - c) < 0.015 and abs(code + 0.125 - e) < 0.015
    # absolute storage at 128k tokens (Eq. 1 at b = 16) and the packed cache
    gib = 2 ** 30
    assert abs(O.fp16_bytes(131072) / gib - A["fp16_gib_128k"][0]) < 1e-9
    T = 131072
    K = O.top_count(T, 25, 100)
    _, eff = O.effective_bits(K, T - K, 0, 6, 5, 128)
    assert abs(O.fp16_bytes(T) / gib * eff / 16 - A["semkv_gib_128k"][1]) < 0.01
    # tile-padded allocation vs row-exact accounting, 4k..128k (paper: within 0.9 %)
    for T in (4096, 8192, 32768, 131072):
        K = O.top_count(T, 25, 100)
        _, eff = O.effective_bits(K, T - K, 0, 6, 5, 128)
        alloc = O.allocated_bytes(K, T - K, 0, 6, 5, 128)
        exact = O.fp16_bytes(T) * eff / 16
        assert abs(alloc / exact - 1) < A["alloc_tolerance"][0]
        assert 6.0 <= O.fp16_bytes(T) / alloc <= 6.05


def test_operating_point_averages():
    """Eq. (6): average bit width 2.39 (r = 25 %) and 2.41 (r = 35 %) (Sec. 4.1)."""
    lo, hi = np.log2(5), np.log2(6)
    for r, want in ((0.25, 2.39), (0.35, 2.41)):
        assert abs(r * hi + (1 - r) * lo - want) < 0.005
