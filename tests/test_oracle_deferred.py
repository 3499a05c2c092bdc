"""Pins of the oracle's unit model: prefill (Alg. 1) and block-exact deferred
quantization of generated tokens (Sec. 3.7, Alg. 2)."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import formatref as F
from workloads import get_config, synth


def test_prefill_pools_and_records():
    cfg = get_config(0, prompt_len=300)
    K, V = synth.unit_kv(cfg, 0, 0, 3)
    s = synth.scores(cfg, 0)
    flag, hi, lo = O.rank(s, cfg.r_num, cfg.r_den)
    u = O.UnitCache(0, 6, 5, 32, 26, 100)
    u.prefill(K, V, flag)
    assert u.count(O.HI) == 78 == 300 * 26 // 100 and u.count(O.LO) == 222
    for p, idx, L in ((O.HI, hi, 6), (O.LO, lo, 5)):
        kc, km, vc, vm, pos = u.pool(p)
        assert np.array_equal(pos, idx)                            # slot order = token order
        rec = u.records(p)
        rb, tb, mb = O.record_bytes(0, L, 32), O.tile_bytes(L), O.meta_bytes(0, 32)
        for t in range((len(idx) + 63) // 64):
            r = rec[t * rb:(t + 1) * rb]
            n = min(64, len(idx) - 64 * t)
            dk = np.array(F.decode_body(r[:tb].tobytes(), L, "K"))
            dv = np.array(F.decode_body(r[tb:2 * tb].tobytes(), L, "V"))
            assert np.array_equal(dk[:n], kc[64 * t:64 * t + n]) and not dk[n:].any()
            assert np.array_equal(dv[:n], vc[64 * t:64 * t + n]) and not dv[n:].any()
            m = r[2 * tb:2 * tb + mb].view(np.uint16).reshape(4, 64, 2)
            assert np.array_equal(m[:, :n].transpose(1, 0, 2), km[64 * t:64 * t + n])
            assert not m[:, n:].any()


@pytest.mark.parametrize("r", [(26, 100), (25, 100), (35, 100)])
def test_block_exact_deferred(r):
    cfg = get_config(3, prompt_len=100, n_gen=64 * 3 + 5)
    K, V = synth.unit_kv(cfg, 0, 0, 0)
    gk, gv = synth.unit_gen_kv(cfg, 0, 0, 0)
    gs = synth.gen_scores(cfg)[:, 0]
    flag, _, _ = O.rank(synth.scores(cfg, 0), *r)
    u = O.UnitCache(0, 6, 5, 128, *r)
    u.prefill(K, V, flag)
    kb = O.block_count(64, *r)
    h0, l0 = u.count(O.HI), u.count(O.LO)
    for i in range(cfg.n_gen):
        u.append_kv(gk[i], gv[i])
        assert len(u.tail_k) <= 64
        u.commit(gs[i])
        if (i + 1) % 64 == 0:
            b = (i + 1) // 64
            assert u.count(O.HI) == h0 + b * kb and u.count(O.LO) == l0 + b * (64 - kb)
            assert not u.tail_k                                    # closed
            blk = gs[i - 63:i + 1]
            _, _, _, _, pos = u.pool(O.HI)
            top = np.sort(np.argsort(-blk, kind="stable")[:kb]) + 100 + i - 63
            assert np.array_equal(pos[-kb:], top)                  # exactly round(rB) by score
        else:
            assert len(u.tail_k) == (i + 1) % 64                   # partial block stays fp16
    u.flush()
    kr = O.block_count(5, *r)
    assert u.count(O.HI) == h0 + 3 * kb + kr
    pos, kh, _ = u.dequantized()
    assert np.array_equal(np.sort(pos), np.arange(100 + cfg.n_gen))   # Eq. (9): all tokens kept
    # a token's codes do not depend on when it was quantized
    _, _, _, _, posh = u.pool(O.HI)
    kc_h = u.pool(O.HI)[0]
    allk = np.concatenate([K, gk])
    ref, _ = O.quantize_rows(allk[posh], 0, 6, 128)
    assert np.array_equal(kc_h, ref)


def test_tail_attention_uses_fp16_values():
    cfg = get_config(3, prompt_len=64, n_gen=10)
    K, V = synth.unit_kv(cfg, 0, 0, 0)
    gk, gv = synth.unit_gen_kv(cfg, 0, 0, 0)
    u = O.UnitCache(0, 6, 5, 128, 26, 100)
    u.prefill(K, V, O.rank(synth.scores(cfg, 0), 26, 100)[0])
    for i in range(10):
        u.append_kv(gk[i], gv[i]); u.commit(1.0)
    pos, kh, vh = u.dequantized()
    assert np.array_equal(kh[-10:], gk.astype(np.float64)) and np.array_equal(vh[-10:], gv.astype(np.float64))
