"""The C-ABI library loads and exports every entry point include/semkv.h
declares; host-side validation and geometry (no GPU calls)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "include", "semkv.h")


@pytest.fixture(scope="module")
def abi():
    from paper_2608_28911_amd import _abi, build
    if not os.path.exists(_abi.LIB_PATH):
        build.build()
    return _abi


def declared():
    src = open(HDR).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(semkv_\w+)\s*\(", src, re.M)))


def test_every_declared_symbol_is_exported(abi):
    names = declared()
    assert len(names) >= 11
    out = subprocess.check_output(["nm", "-D", "--defined-only", abi.LIB_PATH]).decode()
    exported = set(re.findall(r" T (semkv_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    assert set(names) == set(abi.EXPORTS), set(names) ^ set(abi.EXPORTS)
    lib = abi.lib()
    for n in names:
        assert getattr(lib, n) is not None


def test_tracing_entry_point_only_in_the_tracing_build(abi):
    """include/semkv_timeline.h declares the tracing build's one extra call;
    the product library must not carry it (its stamps compile to nothing)."""
    src = open(os.path.join(ROOT, "include", "semkv_timeline.h")).read()
    names = set(re.findall(r"^\s*\w+\s+(semkv_\w+)\s*\(", src, re.M))
    assert names == {"semkv_timeline_read"}
    out = subprocess.check_output(["nm", "-D", "--defined-only", abi.LIB_PATH]).decode()
    assert not names & set(re.findall(r" T (semkv_\w+)", out))


def cfg_for(abi, **kw):
    from paper_2608_28911_amd import make_config
    d = dict(n_layers=2, n_kv_heads=8, batch=1, base=0, L_hi=6, L_lo=5, group=128, r_num=26, r_den=100,
             max_prompt=2048, max_new=128)
    d.update(kw)
    return make_config(**d)


def test_sizes_match_the_format(abi):
    from paper_2608_28911_amd import cache_sizes
    for base, L_hi, L_lo, G in ((0, 6, 5, 128), (0, 6, 5, 32), (1, 4, 3, 128), (0, 5, 4, 64), (2, 6, 5, 128),
                                (2, 5, 4, 32), (0, 8, 7, 128), (0, 7, 6, 128), (2, 3, 2, 128)):
        s = cache_sizes(cfg_for(abi, base=base, L_hi=L_hi, L_lo=L_lo, group=G))
        assert s.tile_bytes_hi == O.tile_bytes(L_hi) and s.tile_bytes_lo == O.tile_bytes(L_lo)
        assert s.record_bytes_hi == O.record_bytes(base, L_hi, G)
        assert s.record_bytes_lo == O.record_bytes(base, L_lo, G)
        K = 2048 * 26 // 100
        assert s.cap_hi_tiles == -(-(K + 128) // 64) and s.cap_lo_tiles == -(-(2048 - K + 128) // 64)
        assert s.pool_bytes == 2 * 8 * s.unit_stride


@pytest.mark.parametrize("bad,status", [
    (dict(head_dim=64), -2), (dict(n_q_heads=16), -2), (dict(block=32), -2), (dict(L_hi=7), -2),
    (dict(base=1, L_hi=6, L_lo=5), -2), (dict(base=1, L_hi=4, L_lo=3, group=32), -2), (dict(group=16), -2),
    (dict(base=2, L_hi=4, L_lo=3), -2), (dict(base=2, group=16), -2), (dict(base=3), -2),
    (dict(L_hi=8, L_lo=7, group=32), -2), (dict(L_hi=8, L_lo=6), -2), (dict(base=1, L_hi=3, L_lo=2), -2),
    (dict(batch=1024, n_layers=64), -2),
    (dict(r_num=3, r_den=2), -1), (dict(r_den=0), -1), (dict(batch=0), -1), (dict(max_prompt=-1), -1)])
def test_config_validation(abi, bad, status):
    s = abi.Sizes()
    assert abi.lib().semkv_cache_sizes(ctypes.byref(cfg_for(abi, **bad)), ctypes.byref(s)) == status


def test_calls_validate_before_touching_the_device(abi):
    lib = abi.lib()
    c = abi.Cache()
    cfg = cfg_for(abi)
    fake = ctypes.c_void_p(0x1000)
    assert lib.semkv_cache_init(ctypes.byref(c), ctypes.byref(cfg), None, fake, fake, fake, None, fake) == -1
    assert lib.semkv_cache_init(ctypes.byref(c), ctypes.byref(cfg), fake, fake, fake, fake, None, fake) == 0
    assert c.sz.unit_stride > 0 and c.n_hi == 0
    nh, nl = ctypes.c_int64(), ctypes.c_int64()
    for T in (1, 3, 100, 1000):                                                   # Eq. (4) sizes
        assert lib.semkv_rank_sizes(ctypes.byref(c), T, ctypes.byref(nh), ctypes.byref(nl)) == 0
        assert nh.value == O.top_count(T, cfg.r_num, cfg.r_den) and nh.value + nl.value == T
    assert lib.semkv_rank_sizes(ctypes.byref(c), 0, ctypes.byref(nh), ctypes.byref(nl)) == -1
    assert lib.semkv_rank_sizes(ctypes.byref(c), 4096, ctypes.byref(nh), ctypes.byref(nl)) == -3
    assert lib.semkv_rank(ctypes.byref(c), None, 16, fake, fake, None) == -1
    assert lib.semkv_rank(ctypes.byref(c), fake, 4096, fake, fake, None) == -3          # T > max_prompt
    assert lib.semkv_quantize_pack(ctypes.byref(c), 5, fake, fake, 0, 128, 128, 128, 16, fake, fake, None) == -1
    assert lib.semkv_quantize_pack(ctypes.byref(c), 0, fake, fake, 0, 128, 128, 100, 16, fake, fake, None) == -1
    assert lib.semkv_append_commit(ctypes.byref(c), fake, None) == -6                 # no layer appended
    assert lib.semkv_decode_attn(ctypes.byref(c), 0, fake, fake, fake, 1 << 20, None) == -6   # empty cache
    assert lib.semkv_decode_attn(ctypes.byref(c), 9, fake, fake, fake, 1 << 20, None) == -1
    assert lib.semkv_flush(ctypes.byref(c), None) == 0                                # nothing to flush
    assert lib.semkv_strerror(-3) == b"capacity exceeded"
    tq = cfg_for(abi, base=1, L_hi=4, L_lo=3)
    assert lib.semkv_cache_init(ctypes.byref(c), ctypes.byref(tq), fake, fake, fake, fake, None, fake) == -1
    assert lib.semkv_cache_reset(None, None) == -1
    assert lib.semkv_dequant(ctypes.byref(c), 0, None, fake, None) == -1
    assert lib.semkv_dequant(ctypes.byref(c), 7, fake, fake, None) == -1             # layer out of range
    assert lib.semkv_dequant(ctypes.byref(c), 0, ctypes.c_void_p(0x1004), fake, None) == -1   # alignment
    assert lib.semkv_dequant(ctypes.byref(c), 0, fake, fake, None) == 0              # empty cache: nothing to do
    assert lib.semkv_score_kv_norm(ctypes.byref(c), fake, 0, 0, 0, 64, 16, fake, None) == -1   # sT < 128
    assert lib.semkv_score_kv_norm(ctypes.byref(c), None, 0, 0, 0, 128, 16, fake, None) == -1
    assert lib.semkv_score_hidden(0, fake, 0, 4, 1, 0, 64, 64, 64, 64, fake, None) == -1      # T = 0
    assert lib.semkv_score_hidden(0, fake, 0, 4, 4, 1 << 32, 64, 64, 64, 64, fake, None) == -2  # grid too large
    rot = cfg_for(abi, base=2)                                                        # needs sign masks too
    assert lib.semkv_cache_init(ctypes.byref(c), ctypes.byref(rot), fake, fake, fake, fake, None, fake) == -1
    assert lib.semkv_cache_init(ctypes.byref(c), ctypes.byref(rot), fake, fake, fake, fake, fake, fake) == 0


@pytest.mark.parametrize("L", [2, 3, 4])
def test_library_codebook_equals_oracle(abi, L):
    """The library solves the Lloyd-Max conditions by bisection, the oracle by
    Lloyd iteration; both must round to the same fp32 constants."""
    from paper_2608_28911_amd import tq_codebook
    mu, tau = tq_codebook(L)
    omu, otau = O.codebook32(L)
    assert np.array_equal(mu.view(np.uint32), omu.view(np.uint32))
    assert np.array_equal(tau.view(np.uint32), otau.view(np.uint32))
