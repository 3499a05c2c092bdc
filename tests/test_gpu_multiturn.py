"""GPU parity of the multi-turn operating point (Sec. 3.7, Sec. 4.6): every
turn resets the cache, ranks and quantizes the accumulated conversation with
the prompt procedure (Eq. 4-7), generates its answer under block-exact
deferred quantization (Alg. 2) and flushes the residual block at the turn's
end.  Flags, pools and attention are checked against the oracle's unit model
turn by turn, at r = 35 % (2.41 code bits)."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import gpu_util as U
from workloads import get_config, synth

pytestmark = pytest.mark.gpu


def run_dialogue(cfgw, check_steps=(0, -1)):
    import torch
    nl, B, H = cfgw.n_layers, cfgw.batch, cfgw.n_kv_heads
    plan = cfgw.turn_plan()
    n_all = cfgw.conversation_len
    rows = {(b, l, h): synth.conversation_kv(cfgw, l, b, h)
            for b in range(B) for l in range(nl) for h in range(H)}
    K = torch.empty((nl, B, H, n_all, 128), dtype=torch.float16)
    V = torch.empty_like(K)
    for (b, l, h), (k, v) in rows.items():
        K[l, b, h], V[l, b, h] = torch.from_numpy(k), torch.from_numpy(v)
    K, V = K.cuda(), V.cuda()
    cache = U.make_cache(cfgw, max(p for p, _ in plan), n_layers=nl, max_new=max(g for _, g in plan))
    step, worst = 0, 0.0
    for turn, (P, g) in enumerate(plan):
        cache.reset()
        sc = synth.turn_scores(cfgw, turn, P)
        hi, lo = cache.rank(torch.from_numpy(sc).cuda())
        cache.quantize_pack(-1, K[:, :, :, :P], V[:, :, :, :P], hi, lo)
        units = {}
        for (b, l, h), (k, v) in rows.items():
            u = O.UnitCache(cfgw.base_id, cfgw.L_hi, cfgw.L_lo, cfgw.group, cfgw.r_num, cfgw.r_den,
                            sign_words=synth.sign_words(cfgw, l, h) if cfgw.rotated else None)
            u.prefill(k[:P], v[:P], O.rank(sc[b], cfgw.r_num, cfgw.r_den)[0])
            units[(b, l, h)] = u
        gs = synth.turn_gen_scores(cfgw, turn, g)
        checks = {i % g for i in check_steps}
        for i in range(g):
            for l in range(nl):
                q = synth.query(cfgw, l, step)
                out = cache.append_decode_attn(l, K[l, :, :, P + i].contiguous(), V[l, :, :, P + i].contiguous(),
                                               torch.from_numpy(q).cuda())
                for (b, ll, h), u in units.items():
                    if ll == l:
                        u.append_kv(rows[(b, l, h)][0][P + i], rows[(b, l, h)][1][P + i])
                if i in checks:
                    o = out.cpu().numpy()
                    for (b, ll, h), u in units.items():
                        if ll == l:
                            want = u.attend(q[b, 4 * h:4 * h + 4].astype(np.float64))
                            worst = max(worst, U.assert_attention_close(
                                o[b, 4 * h:4 * h + 4], want, "turn %d step %d unit %s" % (turn, i, (b, l, h))))
            cache.append_commit(torch.from_numpy(gs[i]).cuda())
            for (b, _, _), u in units.items():
                u.commit(gs[i][b])
            step += 1
        cache.flush()
        for u in units.values():
            u.flush()
        torch.cuda.synchronize()
        assert cache.status() == 0
        # the turn's whole conversation is quantized: pools bit-exact, flags of every token
        for (b, l, h), u in units.items():
            for p in (0, 1):
                n = u.count(p)
                assert n == (cache.c.n_hi if p == 0 else cache.c.n_lo), "turn %d pool %d rows" % (turn, p)
                got = U.gpu_records(cache, b, l, h, p, n)
                assert np.array_equal(got, u.records(p)), "turn %d unit %s pool %d" % (turn, (b, l, h), p)
        for b in range(B):
            u = units[(b, 0, 0)]
            want = np.zeros(P + g, np.uint8)
            want[u.pool(0)[4]] = 1
            assert np.array_equal(U.flags_bits(cache, b, P + g), want), "turn %d flags" % turn
        # no flag beyond the turn survives from a longer earlier turn
        assert not U.flags_bits(cache, 0, cache.sz.flag_words * 32)[P + g:].any()
    return cache, worst


def test_three_turns_block_closes_and_residual_flush():
    cfgw = get_config("llama8b_kv_b4_multiturn4_r35", n_layers=2, batch=2, n_kv_heads=2, n_q_heads=8,
                      turns=((150, 70), (40, 64), (70, 5)))
    cache, worst = run_dialogue(cfgw, check_steps=(0, 63, 64, -1))
    assert cache.c.n_hi == O.top_count(150 + 70 + 40 + 64 + 70, 35, 100) + O.block_count(5, 35, 100)


def test_turn_shorter_than_the_last_clears_old_flags():
    cfgw = get_config("llama8b_kv_b4_multiturn4_r35", n_layers=1, batch=1, n_kv_heads=1, n_q_heads=4,
                      turns=((300, 10), (5, 3)))
    import torch
    plan = cfgw.turn_plan()
    assert plan == [(300, 10), (315, 3)]
    run_dialogue(cfgw)
    # a fresh, shorter prompt after a long dialogue: reset clears the bitmap
    cache = U.make_cache(cfgw, 400, n_layers=1, max_new=16)
    s = torch.from_numpy(np.arange(400, dtype=np.float32)[None]).cuda()
    cache.rank(s)
    cache.reset()
    s2 = torch.from_numpy(np.arange(40, dtype=np.float32)[None]).cuda()
    cache.rank(s2)
    bits = U.flags_bits(cache, 0, 400)
    assert bits[:40].sum() == O.top_count(40, 35, 100) and not bits[40:].any()
