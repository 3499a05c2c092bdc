"""semkv_decode_attn_noalloc (for callers that cannot allocate) against
semkv_decode_attn, through the C ABI: two calls in a row, the second on a
smaller cache, one-layer and all-layers launches; results within the parity
bar of the workspace entry point's (and identical, since both run the same
plan), every unit also checked against the oracle; a cache beyond the scratch
array's counter capacity is refused before anything runs."""
import ctypes

import numpy as np
import pytest

from oracle import oracle as O
from tests import gpu_util as U
from workloads import get_config, synth

pytestmark = pytest.mark.gpu


def _run(cfgw, T, n_layers, seed_step):
    import torch
    cache = U.make_cache(cfgw, T, n_layers=n_layers, max_new=0)
    scores, _, _ = U.prefill(cache, cfgw, T)
    q = np.stack([synth.query(cfgw, l, seed_step) for l in range(n_layers)])
    qd = torch.from_numpy(q).cuda()
    ws = torch.zeros((cache.sz.workspace_bytes + 3) // 4, dtype=torch.float32, device="cuda")
    for l in range(n_layers):
        want = cache.decode_attn(l, qd[l], workspace=ws).cpu().numpy()
        got = cache.decode_attn_noalloc(l, qd[l]).cpu().numpy()
        assert np.abs(got - want).max() <= U.TOL and np.array_equal(got, want), "layer %d" % l
    want_all = cache.decode_attn(-1, qd, workspace=ws).cpu().numpy()
    got_all = cache.decode_attn_noalloc(-1, qd).cpu().numpy()
    assert np.abs(got_all - want_all).max() <= U.TOL and np.array_equal(got_all, want_all)
    for b in range(cfgw.batch):
        flag = O.rank(scores[b], cfgw.r_num, cfgw.r_den)[0]
        for l in range(n_layers):
            for h in range(cfgw.n_kv_heads):
                u = U.oracle_unit(cfgw, l, b, h, flag, T)
                U.assert_attention_close(got_all[l, b, 4 * h:4 * h + 4],
                                         u.attend(q[l, b, 4 * h:4 * h + 4].astype(np.float64)),
                                         "unit %s" % ((b, l, h),))
    assert cache.status() == 0


def test_noalloc_matches_workspace_entry_point_twice():
    _run(get_config(0, n_layers=3, batch=3, n_kv_heads=4, n_q_heads=16), 1500, 3, 0)
    _run(get_config(4, n_layers=2, batch=1, n_kv_heads=2, n_q_heads=8), 300, 2, 1)     # smaller, tq


def test_noalloc_refuses_beyond_the_scratch():
    import torch
    import paper_2608_28911_amd as P
    # 32 layers x 128 sequences x 8 kv heads = 32768 counters > 4096
    cfg = P.make_config(n_layers=32, n_kv_heads=8, batch=128, base=P.BASE_AFFINE, L_hi=6, L_lo=5, group=128,
                        r_num=26, r_den=100, max_prompt=64, max_new=0)
    cache = P.SemKVCache(cfg)
    s = torch.rand((128, 64), device="cuda")
    hi, lo = cache.rank(s)
    K = torch.zeros((32, 128, 8, 64, 128), dtype=torch.float16, device="cuda")
    cache.quantize_pack(-1, K, K, hi, lo)
    q = torch.zeros((128, 32, 128), dtype=torch.float16, device="cuda")
    with pytest.raises(P.SemKVError) as e:
        cache.decode_attn_noalloc(0, q)
    assert e.value.status == -3
    torch.cuda.synchronize()
