"""Shared helpers of the GPU parity tests: drive the HIP path through the C ABI
and the oracle on the same seeded inputs (test infrastructure)."""
import numpy as np

from oracle import oracle as O
from workloads import synth

TOL = 2e-3            # max-abs attention tolerance against the oracle


def base_id(cfgw):
    return cfgw.base_id


def make_cache(cfgw, T, n_layers=None, max_new=None):
    import paper_2608_28911_amd as P
    nl = cfgw.n_layers if n_layers is None else n_layers
    cfg = P.make_config(n_layers=nl, n_kv_heads=cfgw.n_kv_heads, batch=cfgw.batch, base=base_id(cfgw),
                        L_hi=cfgw.L_hi, L_lo=cfgw.L_lo, group=cfgw.group, r_num=cfgw.r_num,
                        r_den=cfgw.r_den, max_prompt=T, max_new=cfgw.n_gen if max_new is None else max_new)
    signs = synth.all_sign_words(cfgw)[:nl] if cfgw.rotated else None
    return P.SemKVCache(cfg, sign_words=signs)


def prefill(cache, cfgw, T, scores=None, kv=None):
    """Rank + quantize+pack every layer on the GPU.  Returns (scores, hi, lo)."""
    import torch
    if scores is None:
        scores = synth.all_scores(cfgw, T)
    s = torch.from_numpy(scores).cuda()
    hi, lo = cache.rank(s)
    for l in range(cache.cfg.n_layers):
        K, V = synth.layer_kv(cfgw, l, T) if kv is None else kv(l)
        cache.quantize_pack(l, torch.from_numpy(K).cuda(), torch.from_numpy(V).cuda(), hi, lo)
    torch.cuda.synchronize()
    return scores, hi, lo


def oracle_unit(cfgw, l, b, h, flag, T, kv=None):
    u = O.UnitCache(base_id(cfgw), cfgw.L_hi, cfgw.L_lo, cfgw.group, cfgw.r_num, cfgw.r_den,
                    sign_words=synth.sign_words(cfgw, l, h) if cfgw.rotated else None)
    if kv is None:
        K, V = synth.unit_kv(cfgw, l, b, h, T)
    else:
        K, V = kv(l)
        K, V = K[b, h], V[b, h]
    u.prefill(K, V, flag)
    return u


def gpu_records(cache, b, l, h, pool, n_rows):
    nt = (n_rows + 63) // 64
    return cache.pool_bytes(b, l, h, pool, nt).cpu().numpy()


def flags_bits(cache, b, n_tokens):
    w = cache.flags.view(-1)[b * cache.sz.flag_words:(b + 1) * cache.sz.flag_words].cpu().numpy().view(np.uint32)
    bits = np.unpackbits(w.view(np.uint8), bitorder="little")
    return bits[:n_tokens]


def assert_attention_close(got, want, what=""):
    d = np.abs(np.asarray(got, np.float64) - want)
    assert np.all(np.isfinite(got)), what
    assert d.max() <= TOL, "%s: max abs diff %.3g" % (what, d.max())
    return d.max()
