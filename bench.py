#!/usr/bin/env python
"""Benchmark of the SemKV hot path on one MI355X.

Workload (default): Llama-3.1-8B KV geometry, 32 layers x 8 KV heads x 128,
32 query heads, batch 1, 32768-token prompt; importance scores Zipf(1.1); the
top 26 % of tokens at 6 levels (2.585 b), the rest at 5 levels (2.322 b);
affine base with fp16 scale/zero per 128-channel row.  Inputs are seeded
synthetic tensors generated on the device.

Timed step: one decoded token of every sequence through all 32 layers, i.e.
32 launches of the split-K decode attention kernel over the mixed-precision
cache (pools resident in HBM).  The K timed steps are one HIP graph replay
bracketed by events and device synchronization.  The prefill path (rank,
quantize + pack) is timed separately and reported beside it.

After the headline, the default run measures the other workloads the same way
(batch 16 at 16K, the Mistral-7B geometry with its 2048 generated tokens, the
TurboQuant-MSE base at 131K, the single-layer case, and the headline shape with
32-channel metadata) and reports them under "workloads".

Prints one JSON line.  --gpus N with N > 1 is refused: the library runs on
one GPU.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, AMD published peak
# what decode attention computes in: the query and the softmax weights as
# int8 fixed-point digits into exact int32 MFMA sums, the softmax in fp32
DECODE_DTYPE = "i8 MFMA (fixed-point q and softmax weights, exact i32 sums); f32 softmax"
PROFILE = os.path.join(ROOT, "profiles", "decode_kernel_llama8b_b1_t32768.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_28911_amd", "csrc", f)
                  for f in ("decode.hip", "semkv_internal.h", "semkv_fmt.h")]


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per decode launch from the committed counter runs (FETCH_SIZE +
    WRITE_SIZE, calibrated against a copy of known size), or None when the
    kernel sources changed since they were taken."""
    try:
        with open(PROFILE) as fh:
            for line in fh:
                if line.startswith("traffic_bytes_per_launch:"):
                    f = line.split()
                    if f[3] == kernel_source_hash():
                        return int(f[1])
    except (OSError, IndexError, ValueError):
        pass
    return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=128)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama8b_kv_b1_t32768_affine")
    ap.add_argument("--group", type=int, default=None, help="override the affine metadata group")
    ap.add_argument("--base", default=None, choices=["affine", "rot_affine"],
                    help="override an affine workload's base (rot_affine: the affine quantizer of the "
                         "Hadamard-rotated row)")
    ap.add_argument("--levels", default=None, help="override an affine workload's level pair, e.g. 8,7")
    ap.add_argument("--ratio", default=None, help="override the high-precision fraction r, e.g. 0/1 or 35/100")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-indicators", dest="indicators", action="store_false",
                    help="skip timing the token-importance indicators")
    ap.add_argument("--all-layers", action="store_true",
                    help="also time every layer in one decode launch (labelled, not the headline)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle sample")
    ap.add_argument("--no-generate", dest="generate", action="store_false",
                    help="skip the generation leg of workloads with generated tokens")
    ap.add_argument("--no-others", dest="others", action="store_false",
                    help="measure the headline workload only (by default the other workloads follow it)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run a device fill and copy of this many MiB first (hardware counter calibration)")
    return ap.parse_args()


def algorithmic_decode_bytes(cfgw, n_hi, n_lo):
    """Bytes one decode launch (one layer) must move: the packed K and V codes
    of every cached token (row-exact mixed-radix bits), their metadata, the
    query and the output."""
    from paper_2608_28911_amd.fmt import line_bits
    meta = (128 // cfgw.group) * 4 if cfgw.base != "tq" else 2
    per_hi = 2 * line_bits(cfgw.L_hi, 128) / 8 + 2 * meta
    per_lo = 2 * line_bits(cfgw.L_lo, 128) / 8 + 2 * meta
    units = cfgw.batch * cfgw.n_kv_heads
    qo = cfgw.batch * cfgw.n_q_heads * 128 * (2 + 4)
    return units * (n_hi * per_hi + n_lo * per_lo) + qo


HIDDEN_DIM, LAST_M = 4096, 4      # hidden size of Llama-3.1-8B / Mistral-7B; Eq. (3) over the last 4 layers


def indicators(cache, K, gen, dev, reps=3):
    """Time the Sec. 3.3 indicators that produce the prompt's scores: delta-norm
    (Eq. 3) over synthetic hidden states of the last m+1 layers, and key-norm
    over the prompt's K of every layer.  Both read their input once (HBM)."""
    import torch
    import paper_2608_28911_amd as P
    _, B, _, T, _ = K.shape
    Hs = torch.randn((LAST_M + 1, B, T, HIDDEN_DIM), generator=gen, device=dev, dtype=torch.float32).half()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    sc = P.score_hidden("delta_norm", Hs)
    ev[0].record()
    for _ in range(reps):
        P.score_hidden("delta_norm", Hs, scores=sc)
    ev[1].record()
    cache.score_kv_norm(K, scores=sc)
    ev[2].record()
    for _ in range(reps):
        cache.score_kv_norm(K, scores=sc)
    ev[3].record()
    torch.cuda.synchronize()
    dn_us = ev[0].elapsed_time(ev[1]) / reps * 1e3
    kn_us = ev[2].elapsed_time(ev[3]) / reps * 1e3
    dn_bytes = Hs.numel() * 2 + B * T * 4
    kn_bytes = K.numel() * 2 + B * T * 4
    del Hs
    return {"delta_norm_us": round(dn_us, 1), "delta_norm_gbps": round(dn_bytes / (dn_us * 1e-6) / 1e9, 1),
            "key_norm_us": round(kn_us, 1), "key_norm_gbps": round(kn_bytes / (kn_us * 1e-6) / 1e9, 1),
            "hidden_dim": HIDDEN_DIM, "m": LAST_M}


def cpu_baseline(cfgw, seconds):
    """The oracle, as it stands, on a bounded sample of the headline workload:
    the (layer, kv head) units of sequence 0 at its context length, each
    quantized + packed (OpenMP across rows), dequantized in fp64 (the
    oracle's dequantization runs on one thread), then the decode attention of
    all sampled units at once (OpenMP across units, every host core).  Scaled
    to the units of one decode step; the single-thread figure is one unit's
    dequantization and attention on one thread."""
    from oracle import oracle as O
    from workloads import synth
    T = cfgw.prompt_len
    base = cfgw.base_id
    s = synth.scores(cfgw, 0, T)
    flag, _, _ = O.rank(s, cfgw.r_num, cfgw.r_den)
    threads = O.max_threads()
    units, t_quant, t_deq, q_bytes = [], 0.0, 0.0, 0
    n_max = cfgw.n_layers * cfgw.n_kv_heads
    while len(units) < n_max and (t_quant + t_deq) < 0.5 * seconds:
        l, h = divmod(len(units), cfgw.n_kv_heads)
        K, V = synth.unit_kv(cfgw, l, 0, h, T)
        u = O.UnitCache(base, cfgw.L_hi, cfgw.L_lo, cfgw.group, cfgw.r_num, cfgw.r_den,
                        sign_words=synth.sign_words(cfgw, l, h) if cfgw.rotated else None)
        t0 = time.perf_counter()
        u.prefill(K, V, flag)
        u.records(0)
        u.records(1)
        t_quant += time.perf_counter() - t0
        q_bytes += K.nbytes + V.nbytes
        t0 = time.perf_counter()
        _, kh, vh = u.dequantized()
        t_deq += time.perf_counter() - t0
        q = synth.query(cfgw, l, 0)[0, 4 * h:4 * h + 4].astype(np.float64)
        units.append((q, kh, vh))
    t0 = time.perf_counter()
    O.attention_units(units)
    t_attn = time.perf_counter() - t0
    per_unit = (t_deq + t_attn) / len(units)
    units_per_step = cfgw.n_layers * cfgw.batch * cfgw.n_kv_heads
    # one thread: one unit's dequantization (its share of t_deq, which ran on
    # one thread) and its attention at this context
    O.set_threads(1)
    t0 = time.perf_counter()
    O.attention(*units[0])
    t_one = time.perf_counter() - t0 + t_deq / len(units)
    O.set_threads(threads)
    # the indicators (Sec. 3.3) on 1024 tokens: delta-norm over 5 hidden states
    # of width 4096, key-norm over every layer and kv head (single thread)
    rng = np.random.default_rng(0)
    n_tok = 1024
    Hs = rng.standard_normal((LAST_M + 1, n_tok, HIDDEN_DIM), dtype=np.float32).astype(np.float16)
    t0 = time.perf_counter()
    O.score_hidden(O.DELTA_NORM, Hs)
    t_dn = time.perf_counter() - t0
    Ks = rng.standard_normal((cfgw.n_layers * cfgw.n_kv_heads, n_tok, 128), dtype=np.float32).astype(np.float16)
    t0 = time.perf_counter()
    O.score_kv_norm(Ks)
    t_kn = time.perf_counter() - t0
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = None
    return {
        "value": 1.0 / (per_unit * units_per_step) * cfgw.batch,
        "unit": "tokens/s",
        "cores": threads,
        "nproc": os.cpu_count(),
        "affinity_cpus": affinity,
        "kind": "oracle",
        "sample": "%d (layer, kv head) units of sequence 0 at T=%d: fp64 dequantize, one thread (%.3f s), + "
                  "softmax attention of 4 query heads, all units in one OpenMP region over %d threads (%.3f s); "
                  "scaled to %d units per decoded token" % (len(units), T, t_deq, threads, t_attn, units_per_step),
        "quantize_pack_gbps": q_bytes / t_quant / 1e9,
        "quantize_pack_cores": threads,
        "delta_norm_tokens_per_s": n_tok / t_dn, "key_norm_tokens_per_s": n_tok / t_kn, "indicator_cores": 1,
        "single_thread_tokens_per_s": 1.0 / (t_one * units_per_step) * cfgw.batch,
    }


def generation(cfgw, cache, gen, dev, outlier_ch):
    """Generated tokens under block-wise deferred allocation (Alg. 2): per
    token, every layer appends its fp16 K/V to the tail and attends over the
    pools and the tail (one fused launch per layer); then the token's score is
    committed, and every 64th
    commit closes the block (in-block ranking, quantize + pack of the 64 rows
    onto the pool ends).  Each block is captured as two HIP graphs -- its 64
    tokens without the last commit, and that commit with the close -- and
    both are replayed in order under events, so the close is timed on its own.
    Returns the timing summary and the close's algorithmic bytes."""
    import torch
    B, H, Hq, nL, n = cfgw.batch, cfgw.n_kv_heads, cfgw.n_q_heads, cfgw.n_layers, cfgw.n_gen
    blk = cfgw.block
    assert n % blk == 0, "the generation leg closes whole blocks"
    kn = torch.empty((n, nL, B, H, 128), dtype=torch.float16, device=dev)
    vn = torch.empty_like(kn)
    qg = torch.empty((n, nL, B, Hq, 128), dtype=torch.float16, device=dev)
    for i in range(0, n, blk):
        k = torch.randn((blk, nL, B, H, 128), generator=gen, device=dev)
        for l in range(nL):            # the prompt keys' outlier channels
            for h in range(H):
                k[:, l, :, h, outlier_ch[l][h]] *= cfgw.outlier_scale
        kn[i:i + blk] = k.half()
        vn[i:i + blk] = torch.randn((blk, nL, B, H, 128), generator=gen, device=dev).half()
        qg[i:i + blk] = torch.randn((blk, nL, B, Hq, 128), generator=gen, device=dev).half()
        del k
    from workloads import synth
    sg = torch.from_numpy(synth.gen_scores(cfgw)).to(dev)
    out = torch.empty((nL, B, Hq, 128), dtype=torch.float32, device=dev)
    ws = cache.workspace()
    rows0 = cache.c.n_hi + cache.c.n_lo
    graphs = []
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for b0 in range(0, n, blk):
            g_steps, g_close = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_steps, stream=s):
                for i in range(b0, b0 + blk):
                    for l in range(nL):
                        cache.append_decode_attn(l, kn[i, l], vn[i, l], qg[i, l], out=out[l], workspace=ws)
                    if i + 1 < b0 + blk:
                        cache.append_commit(sg[i])
            with torch.cuda.graph(g_close, stream=s):
                cache.append_commit(sg[b0 + blk - 1])
            graphs.append((g_steps, g_close))
    torch.cuda.synchronize()
    assert cache.c.n_scored == 0 and cache.c.n_hi + cache.c.n_lo == rows0 + n
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in graphs]
    torch.cuda.synchronize()
    for (g_steps, g_close), (e0, e1, e2) in zip(graphs, ev):
        e0.record()
        g_steps.replay()
        e1.record()
        g_close.replay()
        e2.record()
    torch.cuda.synchronize()
    assert cache.status() == 0, "device status word %d" % cache.status()
    t_steps = sum(e0.elapsed_time(e1) for e0, e1, _ in ev)
    closes = [e1.elapsed_time(e2) for _, e1, e2 in ev]
    total_ms = t_steps + sum(closes)
    close_us = sum(closes) / len(closes) * 1e3
    # close traffic: the block's fp16 K/V of every layer and kv head read,
    # its rows written packed (row-exact bits + metadata)
    from paper_2608_28911_amd.fmt import line_bits
    from fractions import Fraction
    kb = round(Fraction(cfgw.r_num * blk, cfgw.r_den))      # round(rB), ties to even
    meta = (128 // cfgw.group) * 4
    units = B * nL * H
    close_in = units * 2 * blk * 128 * 2
    close_out = units * (kb * (2 * line_bits(cfgw.L_hi, 128) / 8 + 2 * meta) +
                         (blk - kb) * (2 * line_bits(cfgw.L_lo, 128) / 8 + 2 * meta))
    del kn, vn, qg
    return {
        "tokens": n, "tokens_per_s": round(B * n / (total_ms * 1e-3), 2),
        "ms_per_token": round(total_ms / n, 4),
        "close_us": round(close_us, 2), "close_gbps": round((close_in + close_out) / (close_us * 1e-6) / 1e9, 1),
        "close_bytes": int(close_in + close_out), "blocks": len(graphs),
        "rows_hi": cache.c.n_hi, "rows_lo": cache.c.n_lo,
        "note": "per token: fused append + decode of every layer, then commit; every 64th commit closes the block",
    }


def all_layers_launch(cache, q, ws, args, nL, B, Hq, alg, dev, per_layer_out):
    """The same decode steps with every layer in one launch (queries of all
    layers known up front, which a model does not allow: layer l's query needs
    layer l-1's output).  Reported beside the per-layer headline, labelled: it
    shows what the kernel sustains once the per-launch latency is amortized.
    The launch shares the per-layer legs' workspace; its output of the last
    step must match the per-layer output of that step (other split counts
    merge in another order: within 2e-3)."""
    import torch
    out_all = torch.empty((nL, B, Hq, 128), dtype=torch.float32, device=dev)
    n_steps = q.shape[0]
    for i in range(min(args.warmup, n_steps)):
        cache.decode_attn(-1, q[i], out=out_all, workspace=ws)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(args.warmup, n_steps):
                cache.decode_attn(-1, q[i], out=out_all, workspace=ws)
    torch.cuda.synchronize()
    g.replay()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    g.replay()
    e1.record()
    torch.cuda.synchronize()
    diff = (out_all - per_layer_out).abs().max().item()
    assert diff <= 2e-3, "all-layers launch differs from the per-layer launches by %g" % diff
    us = e0.elapsed_time(e1) * 1e3 / args.steps
    gbps = alg * nL / (us * 1e-6) / 1e9
    return {"us_per_step": round(us, 2), "us_per_layer": round(us / nL, 3), "effective_hbm_gbps": round(gbps, 1),
            "effective_hbm_frac": round(gbps / HBM_PEAK_GBS, 4), "max_abs_vs_per_layer": diff,
            "note": "all layers in one launch per step (queries given up front); not the headline"}


def multiturn(args, cfgw):
    """A dialogue at the multi-turn operating point (Sec. 3.7, Sec. 4.6): each
    turn resets the cache, ranks and quantizes the accumulated conversation
    (rank + quantize/pack of every layer), then generates its answer (per
    token: fused append + decode of every layer, commit; block closes) and
    flushes the residual block.  The whole dialogue is captured as HIP graphs
    (per turn: the prefill, each 64-token block, the residual + flush) and
    replayed in order under events.  One JSON line: generated tokens/s over
    the dialogue, with each turn's prefill and generation times."""
    import torch
    import paper_2608_28911_amd as P
    from workloads import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, H, Hq, nL, blk = cfgw.batch, cfgw.n_kv_heads, cfgw.n_q_heads, cfgw.n_layers, cfgw.block
    plan = cfgw.turn_plan()
    n_all, n_gen = cfgw.conversation_len, sum(g for _, g in plan)
    cfg = P.make_config(n_layers=nL, n_kv_heads=H, batch=B, base=cfgw.base_id, L_hi=cfgw.L_hi, L_lo=cfgw.L_lo,
                        group=cfgw.group, r_num=cfgw.r_num, r_den=cfgw.r_den,
                        max_prompt=max(p for p, _ in plan), max_new=max(g for _, g in plan))
    cache = P.SemKVCache(cfg, sign_words=synth.all_sign_words(cfgw) if cfgw.rotated else None)
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfgw.seed)
    K = torch.randn((nL, B, H, n_all, 128), generator=gen, device=dev).half()
    V = torch.randn((nL, B, H, n_all, 128), generator=gen, device=dev).half()
    kn = K.permute(3, 0, 1, 2, 4).contiguous()      # [token][layer][b][kvh][128]: one step's rows together
    vn = V.permute(3, 0, 1, 2, 4).contiguous()
    qg = torch.randn((n_gen, nL, B, Hq, 128), generator=gen, device=dev).half()
    out = torch.empty((nL, B, Hq, 128), dtype=torch.float32, device=dev)
    ws = cache.workspace()
    scores = [torch.from_numpy(synth.turn_scores(cfgw, t, p)).to(dev) for t, (p, _) in enumerate(plan)]
    gsc = [torch.from_numpy(synth.turn_gen_scores(cfgw, t, g)).to(dev) for t, (_, g) in enumerate(plan)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    turns, step = [], 0
    with torch.cuda.stream(s):
        for t, (p, g) in enumerate(plan):
            gp = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gp, stream=s):
                cache.reset()
                hi, lo = cache.rank(scores[t])
                cache.quantize_pack(-1, K[:, :, :, :p], V[:, :, :, :p], hi, lo)
            gens = []
            for b0 in range(0, g, blk):
                gg = torch.cuda.CUDAGraph()
                with torch.cuda.graph(gg, stream=s):
                    for i in range(b0, min(g, b0 + blk)):
                        for l in range(nL):
                            cache.append_decode_attn(l, kn[p + i, l], vn[p + i, l], qg[step, l], out=out[l],
                                                     workspace=ws)
                        cache.append_commit(gsc[t][i])
                        step += 1
                    if b0 + blk >= g:
                        cache.flush()
                gens.append(gg)
            turns.append((p, g, gp, gens, hi, lo))
    torch.cuda.synchronize()
    for _ in range(args.warmup and 1):          # one untimed pass of the whole dialogue
        for _, _, gp, gens, _, _ in turns:
            gp.replay()
            for gg in gens:
                gg.replay()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in turns]
    for (_, _, gp, gens, _, _), (e0, e1, e2) in zip(turns, ev):
        e0.record()
        gp.replay()
        e1.record()
        for gg in gens:
            gg.replay()
        e2.record()
    torch.cuda.synchronize()
    assert cache.status() == 0, "device status word %d" % cache.status()
    per = [{"prompt": p, "generated": g, "prefill_ms": round(e0.elapsed_time(e1), 3),
            "gen_ms_per_token": round(e1.elapsed_time(e2) / g, 4)}
           for (p, g, *_), (e0, e1, e2) in zip(turns, ev)]
    total_ms = sum(e0.elapsed_time(e2) for e0, _, e2 in ev)
    gen_ms = sum(e1.elapsed_time(e2) for _, e1, e2 in ev)
    # decode traffic of the dialogue: every generated token reads, per layer,
    # the turn's quantized rows (packed) and its fp16 tail
    from paper_2608_28911_amd.fmt import line_bits
    meta = (128 // cfgw.group) * 4 if cfgw.base != "tq" else 2
    per_hi = 2 * line_bits(cfgw.L_hi, 128) / 8 + 2 * meta
    per_lo = 2 * line_bits(cfgw.L_lo, 128) / 8 + 2 * meta
    dec_bytes = 0.0
    from fractions import Fraction
    for p, g in plan:
        kh = p * cfgw.r_num // cfgw.r_den
        n_hi, n_lo = kh, p - kh
        for i in range(g):
            if i and i % blk == 0:
                kb = round(Fraction(cfgw.r_num * blk, cfgw.r_den))
                n_hi, n_lo = n_hi + kb, n_lo + blk - kb
            dec_bytes += nL * B * H * (n_hi * per_hi + n_lo * per_lo + (i % blk + 1) * 512)
    achieved = dec_bytes / (gen_ms * 1e-3) / 1e9
    tokens_per_s = B * n_gen / (total_ms * 1e-3)
    line = {
        "metric": "multi-turn dialogue: generated tokens/s incl. each turn's re-prefill (rank + quantize/pack)",
        "value": round(tokens_per_s, 2), "unit": "tokens/s", "n_gpus": 1, "steps": n_gen, "warmup": 1,
        "ms_per_step": round(total_ms / n_gen, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": DECODE_DTYPE, "data": "synthetic",
        "config": {"workload": cfgw.name, "layers": nL, "batch": B, "kv_heads": H, "q_heads": Hq,
                   "head_dim": 128, "base": cfgw.base, "levels": [cfgw.L_hi, cfgw.L_lo],
                   "r": cfgw.r_num / cfgw.r_den, "group": cfgw.group, "turns": [list(x) for x in cfgw.turns]},
        "turns": per, "dialogue_ms": round(total_ms, 3),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "decode_kernel",
                     "note": "decode bytes of every generated token over the generation replays (commits and "
                             "closes included in the time)"},
    }
    print(json.dumps(line), flush=True)


def run_workload(args, cfgw, headline):
    """Prefill (rank, quantize + pack) and the timed decode steps of one
    workload, inputs generated on the device.  The headline also times the
    indicators and, on request, the all-layers launch.  Returns the measured
    figures."""
    import torch
    import paper_2608_28911_amd as P
    from workloads import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, H, Hq, T, nL = cfgw.batch, cfgw.n_kv_heads, cfgw.n_q_heads, cfgw.prompt_len, cfgw.n_layers
    gen_leg = args.generate and cfgw.n_gen > 0
    cfg = P.make_config(n_layers=nL, n_kv_heads=H, batch=B, base=cfgw.base_id, L_hi=cfgw.L_hi, L_lo=cfgw.L_lo,
                        group=cfgw.group, r_num=cfgw.r_num, r_den=cfgw.r_den, max_prompt=T,
                        max_new=cfgw.n_gen if gen_leg else 0)
    signs = synth.all_sign_words(cfgw) if cfgw.rotated else None
    cache = P.SemKVCache(cfg, sign_words=signs)

    # ---- synthetic inputs, resident in HBM
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfgw.seed)
    K = torch.empty((nL, B, H, T, 128), dtype=torch.float16, device=dev)
    V = torch.empty_like(K)
    outlier_ch = []
    for l in range(nL):
        k = torch.randn((B, H, T, 128), generator=gen, device=dev, dtype=torch.float32)
        ch = torch.randperm(128, generator=gen, device=dev)[:cfgw.outliers * H].view(H, cfgw.outliers)
        outlier_ch.append(ch)
        for h in range(H):
            k[:, h, :, ch[h]] *= cfgw.outlier_scale
        K[l] = k.half()
        V[l] = torch.randn((B, H, T, 128), generator=gen, device=dev, dtype=torch.float32).half()
        del k
    scores = torch.from_numpy(synth.all_scores(cfgw, T)).to(dev)
    n_steps = args.warmup + args.steps
    q = (torch.randn((n_steps, nL, B, Hq, 128), generator=gen, device=dev, dtype=torch.float32)).half()
    out = torch.empty((nL, B, Hq, 128), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()

    # ---- prefill: rank + quantize/pack, timed with events
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    hi, lo = cache.rank(scores)
    n_rank = 20                              # back to back, outputs preallocated
    ev[0].record()
    for _ in range(n_rank):
        cache.rank(scores, out=(hi, lo))
    ev[1].record()
    cache.quantize_pack(-1, K, V, hi, lo)
    torch.cuda.synchronize()
    ev[2].record()
    reps = 3
    for _ in range(reps):
        cache.quantize_pack(-1, K, V, hi, lo)
    ev[3].record()
    torch.cuda.synchronize()
    assert cache.status() == 0, "device status word %d" % cache.status()
    rank_us = ev[0].elapsed_time(ev[1]) / n_rank * 1e3
    quant_ms = ev[2].elapsed_time(ev[3]) / reps
    n_hi, n_lo = cache.c.n_hi, cache.c.n_lo
    t_hi, t_lo = -(-n_hi // 64), -(-n_lo // 64)
    quant_bytes = 2 * K.numel() * 2 + nL * B * H * (t_hi * cache.sz.record_bytes_hi + t_lo * cache.sz.record_bytes_lo)
    ind = indicators(cache, K, gen, dev) if headline and args.indicators else None
    del K, V, hi, lo
    torch.cuda.empty_cache()

    if headline and args.copy_probe_mib > 0:      # known traffic for counter calibration
        nb = args.copy_probe_mib << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---- decode: all timed steps captured in one graph
    ws = cache.workspace()

    def step(i):
        for l in range(nL):
            cache.decode_attn(l, q[i, l], out=out[l], workspace=ws)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(args.warmup):
            step(i)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    # eager reference of the last timed step, to check the graph replays
    step(n_steps - 1)
    torch.cuda.synchronize()
    eager_last = out.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(args.warmup, n_steps):
            step(i)
    torch.cuda.synchronize()
    graph.replay()                           # warm replay (also a correctness check below)
    torch.cuda.synchronize()
    assert torch.equal(out, eager_last), "graph replay differs from eager decode"
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    assert torch.equal(out, eager_last), "graph replay differs from eager decode"
    ms = e0.elapsed_time(e1)
    del graph
    avg_launch_us = ms * 1e3 / (args.steps * nL)
    alg = algorithmic_decode_bytes(cfgw, n_hi, n_lo)
    achieved = alg / (avg_launch_us * 1e-6) / 1e9
    r = {"cfgw": cfgw, "ms_per_step": ms / args.steps, "tokens_per_s": B * args.steps / (ms * 1e-3),
         "decode_us_per_layer": avg_launch_us, "achieved_gbps": achieved, "bytes_per_launch": alg,
         "quantize_pack_gbps": quant_bytes / (quant_ms * 1e-3) / 1e9, "quantize_pack_ms": quant_ms,
         "rank_us": rank_us, "rows_hi": n_hi, "rows_lo": n_lo, "indicators": ind}
    if headline and args.all_layers:
        r["all_layers_launch"] = all_layers_launch(cache, q, ws, args, nL, B, Hq, alg, dev, eager_last)
    del q
    if gen_leg:
        r["generation"] = generation(cfgw, cache, gen, dev, outlier_ch)
    del cache
    torch.cuda.empty_cache()
    return r


def config_of(cfgw, r):
    return {"workload": cfgw.name, "layers": cfgw.n_layers, "batch": cfgw.batch, "context": cfgw.prompt_len,
            "kv_heads": cfgw.n_kv_heads, "q_heads": cfgw.n_q_heads, "head_dim": 128, "base": cfgw.base,
            "levels": [cfgw.L_hi, cfgw.L_lo], "r": cfgw.r_num / cfgw.r_den, "group": cfgw.group,
            "rows_hi": r["rows_hi"], "rows_lo": r["rows_lo"]}


def summary(r):
    """The per-workload figures of a secondary workload."""
    cfgw = r["cfgw"]
    d = {"config": config_of(cfgw, r),
         "decode_us_per_layer": round(r["decode_us_per_layer"], 3),
         "tokens_per_s": round(r["tokens_per_s"], 2),
         "effective_hbm_gbps": round(r["achieved_gbps"], 1),
         "effective_hbm_frac": round(r["achieved_gbps"] / HBM_PEAK_GBS, 4),
         "bytes_per_launch": int(r["bytes_per_launch"]),
         "quantize_pack_gbps": round(r["quantize_pack_gbps"], 1),
         "quantize_pack_ms": round(r["quantize_pack_ms"], 3),
         "rank_us": round(r["rank_us"], 1)}
    if cfgw.n_layers * cfgw.batch * cfgw.n_kv_heads * (r["rows_hi"] + r["rows_lo"]) * 90 < 256 << 20:
        d["note"] = "the packed cache fits the 256 MB last-level cache: not an HBM measurement"
    if "generation" in r:
        d["generation"] = r["generation"]
    return d


# the other workloads the default run measures beside the headline (name,
# label, overrides): every workload of the suite, and the headline shape with
# fp16 scale/zero per 32 channels
SECONDARY = [
    ("llama8b_kv_b1_t32768_affine", "llama8b_kv_b1_t32768_affine_g32", {"group": 32}),
    ("single_layer_t2048_affine_g32", "single_layer_t2048_affine_g32", {}),
    ("llama8b_kv_b16_t16384_affine_dirichlet", "llama8b_kv_b16_t16384_affine_dirichlet", {}),
    ("mistral7b_kv_b4_t32768_gen2048_deferred", "mistral7b_kv_b4_t32768_gen2048_deferred", {}),
    ("llama8b_kv_b1_t131072_tq", "llama8b_kv_b1_t131072_tq", {}),
]


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU; --gpus %d is not supported "
              "(how the path would shard over GPUs is described with the design notes)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    from workloads import get_config

    cfgw = get_config(args.workload)
    if cfgw.turns:
        return multiturn(args, cfgw)
    custom = bool(args.group or args.base or args.levels or args.ratio)
    if custom:
        from dataclasses import replace
        if (args.base or args.levels) and cfgw.base == "tq":
            sys.exit("--base and --levels apply to the affine workloads")
        cfgw = replace(cfgw, group=args.group or cfgw.group, base=args.base or cfgw.base)
        if cfgw.base == "rot_affine":
            cfgw = replace(cfgw, name=cfgw.name.replace("_affine", "_rot_affine"))
        if args.group:
            cfgw = replace(cfgw, name=cfgw.name + "_g%d" % args.group)
        if args.levels:
            lh, ll = (int(x) for x in args.levels.split(","))
            cfgw = replace(cfgw, L_hi=lh, L_lo=ll, name=cfgw.name + "_L%d%d" % (lh, ll))
        if args.ratio:
            rn, rd = (int(x) for x in args.ratio.split("/"))
            cfgw = replace(cfgw, r_num=rn, r_den=rd, name=cfgw.name + "_r%d_%d" % (rn, rd))
    r = run_workload(args, cfgw, headline=True)
    ind = r["indicators"]
    # streaming-read reference: the key-norm kernel of the indicator leg reads
    # the prompt's K once with trivial arithmetic
    stream_gbps = ind["key_norm_gbps"] if ind is not None else None
    achieved = r["achieved_gbps"]
    line = {
        "metric": "mixed-prec decode attn tokens/s + effective HBM GB/s (% peak); quantize+pack GB/s",
        "value": round(r["tokens_per_s"], 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DECODE_DTYPE,
        "data": "synthetic",
        "config": config_of(cfgw, r),
        "effective_hbm_gbps": round(achieved, 1),
        "effective_hbm_frac": round(achieved / HBM_PEAK_GBS, 4),
        "decode_us_per_layer": round(r["decode_us_per_layer"], 3),
        "quantize_pack_gbps": round(r["quantize_pack_gbps"], 1),
        "quantize_pack_ms": round(r["quantize_pack_ms"], 3),
        "rank_us": round(r["rank_us"], 1),
        "stream_read_gbps": stream_gbps,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "frac_of_stream_read": round(achieved / stream_gbps, 4) if stream_gbps else None,
                     "traffic": measured_traffic() if cfgw.name == "llama8b_kv_b1_t32768_affine" else None,
                     "kernel": "decode_kernel", "bytes_per_launch": int(r["bytes_per_launch"])},
    }
    if ind is not None:
        line["indicators"] = ind
    if "all_layers_launch" in r:
        line["all_layers_launch"] = r["all_layers_launch"]
    if "generation" in r:
        line["generation"] = r["generation"]
    if not custom and args.workload == "llama8b_kv_b1_t32768_affine" and args.others:
        line["workloads"] = {}
        for name, label, over in SECONDARY:
            print("bench.py: workload %s" % label, file=sys.stderr, flush=True)
            line["workloads"][label] = summary(run_workload(args, get_config(name, **over), headline=False))
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfgw, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
