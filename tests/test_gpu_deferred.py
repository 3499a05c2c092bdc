"""GPU parity of block-exact deferred quantization of generated tokens
(Sec. 3.7, Alg. 2): fp16 tail, block close, residual flush, and decode over
pools + tail, against the oracle's unit model."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import gpu_util as U
from workloads import get_config, synth

pytestmark = pytest.mark.gpu


def run_generation(cfgw, T, n_gen, check_steps, flush=False, units=None):
    import torch
    nl = cfgw.n_layers
    cache = U.make_cache(cfgw, T, n_layers=nl, max_new=n_gen)
    scores, hi, lo = U.prefill(cache, cfgw, T)
    flags = [O.rank(scores[b], cfgw.r_num, cfgw.r_den)[0] for b in range(cfgw.batch)]
    if units is None:
        units = [(b, l, h) for b in range(cfgw.batch) for l in range(nl) for h in range(cfgw.n_kv_heads)]
    oracle = {u: U.oracle_unit(cfgw, u[1], u[0], u[2], flags[u[0]], T) for u in units}
    gen = {(b, l, h): synth.unit_gen_kv(cfgw, l, b, h, n_gen)
           for b in range(cfgw.batch) for l in range(nl) for h in range(cfgw.n_kv_heads)}
    gscore = synth.gen_scores(cfgw, n_gen)
    worst = 0.0
    for i in range(n_gen):
        for l in range(nl):
            k = np.stack([np.stack([gen[(b, l, h)][0][i] for h in range(cfgw.n_kv_heads)]) for b in range(cfgw.batch)])
            v = np.stack([np.stack([gen[(b, l, h)][1][i] for h in range(cfgw.n_kv_heads)]) for b in range(cfgw.batch)])
            cache.append_kv(l, torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda())
            for (b, ll, h), u in oracle.items():
                if ll == l:
                    u.append_kv(gen[(b, l, h)][0][i], gen[(b, l, h)][1][i])
            if i in check_steps:
                q = synth.query(cfgw, l, i)
                out = cache.decode_attn(l, torch.from_numpy(q).cuda()).cpu().numpy()
                for (b, ll, h), u in oracle.items():
                    if ll == l:
                        want = u.attend(q[b, 4 * h:4 * h + 4].astype(np.float64))
                        worst = max(worst, U.assert_attention_close(out[b, 4 * h:4 * h + 4], want,
                                                                    "step %d unit %s" % (i, (b, l, h))))
        cache.append_commit(torch.from_numpy(gscore[i]).cuda())
        for (b, l, h), u in oracle.items():
            u.commit(gscore[i][b])
        assert cache.c.n_scored == len(next(iter(oracle.values())).tail_s)
    if flush:
        cache.flush()
        for u in oracle.values():
            u.flush()
    torch.cuda.synchronize()
    assert cache.status() == 0
    # pools bit-exact, flags of every token
    for (b, l, h), u in oracle.items():
        for p in (0, 1):
            n = u.count(p)
            assert n == (cache.c.n_hi if p == 0 else cache.c.n_lo)
            got = U.gpu_records(cache, b, l, h, p, n)
            want = u.records(p)
            if not np.array_equal(got, want):
                bad = np.flatnonzero(got != want)
                raise AssertionError("unit %s pool %d: %d bytes differ, first at %d" % ((b, l, h), p, bad.size, bad[0]))
    for b in range(cfgw.batch):
        u = oracle[next(x for x in oracle if x[0] == b)]
        pos_hi = u.pool(0)[4]
        want = np.zeros(u.n_tokens - len(u.tail_k), np.uint8)
        want[pos_hi] = 1
        assert np.array_equal(U.flags_bits(cache, b, len(want)), want)
    return cache, oracle, worst


def test_two_blocks_and_partial_tail():
    cfgw = get_config(3, n_layers=2, batch=2, n_kv_heads=2, n_q_heads=8)
    run_generation(cfgw, 300, 64 * 2 + 10, check_steps={0, 1, 62, 63, 64, 65, 127, 128, 137})


@pytest.mark.parametrize("n_res", [1, 2, 3, 63])
def test_flush_residual(n_res):
    cfgw = get_config(3, n_layers=1, batch=1, n_kv_heads=2, n_q_heads=8, r_num=35, r_den=100)
    cache, oracle, _ = run_generation(cfgw, 130, 64 + n_res, check_steps={64 + n_res - 1}, flush=True)
    kb = O.block_count(n_res, 35, 100)
    assert cache.c.n_hi == O.top_count(130, 35, 100) + O.block_count(64, 35, 100) + kb


def test_generation_on_the_turboquant_base():
    cfgw = get_config(4, n_layers=1, batch=1, n_kv_heads=2, n_q_heads=8)
    run_generation(cfgw, 200, 64 + 5, check_steps={0, 63, 64, 68})


def test_generation_on_the_rotated_affine_base():
    cfgw = get_config(3, base="rot_affine", n_layers=1, batch=1, n_kv_heads=2, n_q_heads=8)
    run_generation(cfgw, 200, 64 + 5, check_steps={0, 63, 64, 68})


@pytest.mark.parametrize("levels", [(8, 7), (3, 2)])
def test_generation_on_the_level_grid(levels):
    cfgw = get_config(3, L_hi=levels[0], L_lo=levels[1], n_layers=1, batch=1, n_kv_heads=2, n_q_heads=8)
    run_generation(cfgw, 130, 64 + 3, check_steps={0, 64, 66}, flush=True)


def test_generation_with_a_partial_last_round():
    """8 kv heads and a 1100-token prompt at 26 %: two workgroups per unit
    and a last round of two tiles, one of them in the workgroup that also
    takes the fp16 tail of the generated tokens."""
    cfgw = get_config(3, n_layers=1, batch=1, n_kv_heads=8, n_q_heads=32)
    run_generation(cfgw, 1100, 6, check_steps={0, 5}, units=[(0, 0, 0), (0, 0, 5)])


def test_generation_g32():
    cfgw = get_config(3, n_layers=1, batch=1, n_kv_heads=1, n_q_heads=4, group=32)
    run_generation(cfgw, 64, 64 * 3, check_steps={10, 100, 191})


@pytest.mark.parametrize("wl,base", [(3, None), (4, None), (3, "rot_affine")])
def test_fused_append_decode_matches_separate_calls(wl, base):
    """semkv_append_decode (append and attend in one launch) gives the same
    attention, bit for bit, as semkv_append_kv followed by semkv_decode_attn,
    and leaves the same tail, pools and flags, across a block close."""
    import torch
    from paper_2608_28911_amd import SemKVError
    cfgw = get_config(wl, n_layers=2, batch=2, n_kv_heads=2, n_q_heads=8)
    if base:
        cfgw = get_config(wl, n_layers=2, batch=2, n_kv_heads=2, n_q_heads=8, base=base)
    T, n_gen = 150, 64 + 6
    sep, fus = U.make_cache(cfgw, T, max_new=n_gen), U.make_cache(cfgw, T, max_new=n_gen)
    for c in (sep, fus):
        U.prefill(c, cfgw, T)
    gen = {(b, l, h): synth.unit_gen_kv(cfgw, l, b, h, n_gen)
           for b in range(cfgw.batch) for l in range(cfgw.n_layers) for h in range(cfgw.n_kv_heads)}
    gscore = synth.gen_scores(cfgw, n_gen)
    for i in range(n_gen):
        for l in range(cfgw.n_layers):
            k = torch.from_numpy(np.stack([np.stack([gen[(b, l, h)][0][i] for h in range(cfgw.n_kv_heads)])
                                           for b in range(cfgw.batch)])).cuda()
            v = torch.from_numpy(np.stack([np.stack([gen[(b, l, h)][1][i] for h in range(cfgw.n_kv_heads)])
                                           for b in range(cfgw.batch)])).cuda()
            q = torch.from_numpy(synth.query(cfgw, l, i)).cuda()
            sep.append_kv(l, k, v)
            want = sep.decode_attn(l, q)
            got = fus.append_decode_attn(l, k, v, q)
            assert torch.equal(got, want), "step %d layer %d" % (i, l)
            if i == 0 and l == 0:
                with pytest.raises(SemKVError):          # this layer appended the token already
                    fus.append_decode_attn(l, k, v, q)
        s = torch.from_numpy(gscore[i]).cuda()
        sep.append_commit(s)
        fus.append_commit(s)
    torch.cuda.synchronize()
    assert sep.status() == 0 and fus.status() == 0
    assert (sep.c.n_hi, sep.c.n_lo, sep.c.n_scored) == (fus.c.n_hi, fus.c.n_lo, fus.c.n_scored)
    assert torch.equal(sep.flags, fus.flags)
    for b in range(cfgw.batch):
        for l in range(cfgw.n_layers):
            for h in range(cfgw.n_kv_heads):
                for p, n in ((0, sep.c.n_hi), (1, sep.c.n_lo)):
                    nt = -(-n // 64)
                    assert torch.equal(sep.pool_bytes(b, l, h, p, nt), fus.pool_bytes(b, l, h, p, nt))
    assert torch.equal(sep.tail.view(-1, 2, 64, 128)[:, :, :sep.c.n_scored], fus.tail.view(-1, 2, 64, 128)[:, :, :fus.c.n_scored])
