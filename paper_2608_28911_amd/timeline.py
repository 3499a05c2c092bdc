"""Per-phase timeline of one decode launch, from the tracing build of the
library (libsemkv_timeline.so: `python paper_2608_28911_amd/build.py
--timeline`, or `--timeline-fine` for the stamps inside the prologue and the
first record; include/semkv_timeline.h).

    python -m paper_2608_28911_amd.timeline [--workload NAME] [--launches N]

Builds the workload's cache on cuda:0 (synthetic rows and scores), runs N
decode launches per layer, and prints, for the last launch, the distribution
over waves of the time (us, from the launch's first wave start) at which each
phase ended, then the merging workgroups and the spread within each unit.
The stamps come from the constant 100 MHz clock (10 ns resolution)."""
import argparse
import ctypes
import os
import sys

import numpy as np

from . import _abi as A
from .build import LIB_TIMELINE

WGS, WAVES, EVENTS = 4096, 16, 32
NAMES = {0: "start", 1: "tables + query operands", 2: "first record in LDS",
         8: "record 1 arithmetic done", 3: "record 1 done (next record in LDS)",
         4: "record 2 done", 5: "record 3 done", 6: "record 4 done", 7: "record 5+ done",
         9: "wave's records done", 10: "workgroup partial merged",
         11: "partial stored", 12: "split counter taken", 13: "last workgroup's merge done",
         16: "record 1: next record's loads issued", 17: "record 1: scores done",
         18: "record 1: softmax and flush done", 19: "prologue: tables written",
         20: "prologue: query value in hand", 21: "prologue: query runs done"}
ORDER = [0, 19, 20, 21, 1, 2, 16, 17, 18, 8, 3, 4, 5, 6, 7, 9, 10, 11, 12, 13]


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="llama8b_kv_b1_t32768_affine")
    ap.add_argument("--launches", type=int, default=5, help="decode launches per layer (the last is shown)")
    ap.add_argument("--save", default=None, help="also save the raw stamps (uint64 [4096][16][32]) to this .npy file")
    args = ap.parse_args(argv)
    if not os.path.exists(LIB_TIMELINE):
        raise SystemExit("libsemkv_timeline.so is not built: python paper_2608_28911_amd/build.py --timeline")
    if A._lib is not None:
        raise SystemExit("the product library is already loaded in this process")
    A.LIB_PATH = LIB_TIMELINE
    lib = A.lib()
    lib.semkv_timeline_read.restype, lib.semkv_timeline_read.argtypes = ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t]

    import torch
    import paper_2608_28911_amd as P
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from workloads import get_config, synth

    cfgw = get_config(args.workload)
    dev = torch.device("cuda:0")
    B, H, Hq, T, nL = cfgw.batch, cfgw.n_kv_heads, cfgw.n_q_heads, cfgw.prompt_len, cfgw.n_layers
    cfg = P.make_config(n_layers=nL, n_kv_heads=H, batch=B, base=cfgw.base_id, L_hi=cfgw.L_hi, L_lo=cfgw.L_lo,
                        group=cfgw.group, r_num=cfgw.r_num, r_den=cfgw.r_den, max_prompt=T, max_new=0)
    cache = P.SemKVCache(cfg, sign_words=synth.all_sign_words(cfgw) if cfgw.rotated else None)
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    hi, lo = cache.rank(torch.from_numpy(synth.all_scores(cfgw, T)).to(dev))
    for l in range(nL):
        K = torch.randn((B, H, T, 128), generator=g, device=dev).half()
        V = torch.randn((B, H, T, 128), generator=g, device=dev).half()
        cache.quantize_pack(l, K, V, hi, lo)
    del K, V
    q = torch.randn((nL, B, Hq, 128), generator=g, device=dev).half()
    out = torch.empty((nL, B, Hq, 128), dtype=torch.float32, device=dev)
    ws = cache.workspace()
    for _ in range(args.launches):
        for l in range(nL):
            cache.decode_attn(l, q[l], out=out[l], workspace=ws)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()

    buf = np.zeros(WGS * WAVES * EVENTS, np.uint64)
    A.check(lib.semkv_timeline_read(buf.ctypes.data_as(ctypes.c_void_p), buf.nbytes), "semkv_timeline_read")
    if args.save:
        np.save(args.save, buf.reshape(WGS, WAVES, EVENTS))
    nsplit = cache.decode_splits() if hasattr(cache, "decode_splits") else None
    d = buf.reshape(WGS, WAVES, EVENTS).astype(np.int64)
    used = np.flatnonzero(d[:, 0, 0] > 0)
    nwg = int(used.max()) + 1
    d = d[:nwg]
    start = d[:, :, 0]
    t0 = start[start > 0].min()
    rel = np.where(d > 0, (d - t0) * 10, -1) / 1e3                     # us
    rel[:, :, 14:16] = -1                                                # counts, not stamps
    print("workload %s: %d workgroups, %d waves stamped (last of %d launches per layer, layer %d)"
          % (args.workload, nwg, int((start > 0).sum()), args.launches, nL - 1))
    print()
    print("| phase end | waves | min | median | p90 | max |")
    print("|---|---:|---:|---:|---:|---:|")
    for ev in ORDER:
        v = rel[:, :, ev]
        v = v[v >= 0]
        if v.size:
            print("| %s | %d | %.2f | %.2f | %.2f | %.2f |" % (NAMES[ev], v.size, v.min(), np.median(v),
                                                              np.percentile(v, 90), v.max()))
    counts = buf.reshape(WGS, WAVES, EVENTS)[:nwg, :, 14:16].astype(np.int64)   # not stamps
    live = start > 0
    fl, rc = counts[:, :, 0][live], counts[:, :, 1][live]
    print()
    print("value-sum flushes: %d of %d records (%.1f %%); per wave: mean %.2f, max %d"
          % (fl.sum(), rc.sum(), 100.0 * fl.sum() / max(1, rc.sum()), fl.mean(), fl.max()))
    # the first record's arithmetic by its pool: wave w of the workgroup of
    # split s takes tile w * nsplit + s first (high-pool tiles lead)
    ns_ = nsplit if nsplit is not None else nwg // max(1, B * H)
    nt0 = (cache.c.n_hi + 63) // 64
    wg_idx = np.arange(nwg)[:, None]
    first = np.arange(WAVES)[None, :] * ns_ + (wg_idx % ns_)
    dur = rel[:, :, 8] - rel[:, :, 2]
    ok = (rel[:, :, 8] >= 0) & (rel[:, :, 2] >= 0)
    for name, sel in (("high-pool (L_hi)", first < nt0), ("low-pool (L_lo)", first >= nt0)):
        v = dur[ok & sel]
        if v.size:
            print("first record's arithmetic, %s first: %d waves, median %.2f us, p90 %.2f" % (name, v.size, np.median(v), np.percentile(v, 90)))
    d2 = rel[:, :, 4] - rel[:, :, 3]
    ok2 = (rel[:, :, 4] >= 0) & (rel[:, :, 3] >= 0)
    if ok2.any():
        print("second record: %d waves, median %.2f us" % (int(ok2.sum()), np.median(d2[ok2])))
    m = np.flatnonzero(rel[:, 0, 13] >= 0)
    print()
    print("merging workgroups (wave 0): %d" % len(m))
    for w in m[:8]:
        row = rel[w, 0]
        print("  wg %4d: " % w + " ".join("%s %.2f" % (NAMES[e].split()[0], row[e])
                                          for e in (0, 1, 2, 9, 10, 11, 12, 13) if row[e] >= 0))
    if nsplit is None:
        nsplit = nwg // max(1, B * H)
    units = nwg // nsplit
    print()
    print("per unit (%d splits each; workgroup = split + %d x unit):" % (nsplit, nsplit))
    for u in range(min(units, 16)):
        wgs = np.arange(u * nsplit, (u + 1) * nsplit)
        rd = rel[wgs, :, 9].max(1)
        ps = rel[wgs, 0, 11]
        print("  unit %2d: records done min %.2f med %.2f max %.2f | partial stored min %.2f max %.2f"
              % (u, rd.min(), np.median(rd), rd.max(), ps.min(), ps.max()))


if __name__ == "__main__":
    main()
