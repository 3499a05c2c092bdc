"""semkv_dequant against the oracle's dequantization of the same pools: the
values decode attention reads, for every base.  Affine values are one fmaf in
fp32 on both sides and must agree bit for bit; the rotated bases sum the
128-point transform in fp32 against the oracle's fp64, so they agree within
1e-5 of the row norm (7 radix-2 stages, each within one fp32 rounding of
sqrt(128) times the row norm)."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import gpu_util as U
from workloads import get_config, synth

pytestmark = pytest.mark.gpu


def _want(u, cfgw, l, h):
    outs = []
    for kv in (0, 2):
        rows = []
        for p in (0, 1):
            pool = u.pool(p)
            rows.append(O.dequantize_rows(pool[kv], pool[kv + 1], cfgw.base_id, (cfgw.L_hi, cfgw.L_lo)[p], cfgw.group,
                                          synth.sign_words(cfgw, l, h) if cfgw.rotated else None))
        outs.append(np.concatenate(rows))
    return outs


def _compare(got, want, exact, what):
    if exact:
        assert np.array_equal(got.astype(np.float64), want), what
    else:
        tol = 1e-5 * np.linalg.norm(want, axis=1, keepdims=True) + 1e-30
        assert np.all(np.abs(got - want) <= tol), what


@pytest.mark.parametrize("over", [dict(), dict(group=128), dict(base="rot_affine", group=32),
                                  dict(base="rot_affine", L_hi=8, L_lo=7, group=128), dict(L_hi=3, L_lo=2, group=128),
                                  dict(base="tq", L_hi=4, L_lo=3, group=128, r_num=40, r_den=100)])
def test_dequant_matches_oracle_after_prefill(over):
    cfgw = get_config(0, n_layers=2, batch=2, n_kv_heads=2, n_q_heads=8, **over)
    T = 700
    cache = U.make_cache(cfgw, T, n_layers=2, max_new=0)
    scores, _, _ = U.prefill(cache, cfgw, T)
    for l in range(2):
        kh, vh = (t.cpu().numpy() for t in cache.dequant(l))
        assert kh.shape == (2, 2, T, 128)
        for b in range(2):
            flag = O.rank(scores[b], cfgw.r_num, cfgw.r_den)[0]
            for h in range(2):
                u = U.oracle_unit(cfgw, l, b, h, flag, T)
                wk, wv = _want(u, cfgw, l, h)
                exact = cfgw.base == "affine"
                _compare(kh[b, h], wk, exact, "K unit %s" % ((b, l, h),))
                _compare(vh[b, h], wv, exact, "V unit %s" % ((b, l, h),))


def test_dequant_after_block_closes():
    from tests.test_gpu_deferred import run_generation
    cfgw = get_config(3, n_layers=1, batch=1, n_kv_heads=2, n_q_heads=8)
    cache, oracle, _ = run_generation(cfgw, 100, 64 + 7, check_steps=set(), flush=True)
    kh, vh = (t.cpu().numpy() for t in cache.dequant(0))
    for (b, l, h), u in oracle.items():
        wk, wv = _want(u, cfgw, l, h)
        _compare(kh[b, h], wk, True, "K unit %s" % ((b, l, h),))
        _compare(vh[b, h], wv, True, "V unit %s" % ((b, l, h),))
