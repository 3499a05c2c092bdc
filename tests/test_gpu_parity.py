"""GPU parity of the HIP path (through the C ABI) against the oracle at sizes
the oracle finishes in seconds: bit-exact flags, slot lists, packed bytes and
metadata; decode attention within 2e-3 max-abs."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import gpu_util as U
from workloads import get_config, synth

pytestmark = pytest.mark.gpu


def _check_prefill(cfgw, T, n_layers=1, units=None, scores=None):
    import torch
    cache = U.make_cache(cfgw, T, n_layers=n_layers, max_new=0)
    scores, hi, lo = U.prefill(cache, cfgw, T, scores=scores)
    assert cache.status() == 0
    hi, lo = hi.cpu().numpy(), lo.cpu().numpy()
    K = O.top_count(T, cfgw.r_num, cfgw.r_den)
    flags = []
    for b in range(cfgw.batch):
        f, ohi, olo = O.rank(scores[b], cfgw.r_num, cfgw.r_den)
        assert np.array_equal(hi[b], ohi) and np.array_equal(lo[b], olo), "slot lists, seq %d" % b
        assert np.array_equal(U.flags_bits(cache, b, T), f), "flags, seq %d" % b
        flags.append(f)
    if units is None:
        units = [(b, l, h) for b in range(cfgw.batch) for l in range(n_layers) for h in range(cfgw.n_kv_heads)]
    for (b, l, h) in units:
        u = U.oracle_unit(cfgw, l, b, h, flags[b], T)
        for p, n in ((0, K), (1, T - K)):
            if n == 0:
                continue
            got = U.gpu_records(cache, b, l, h, p, n)
            want = u.records(p)
            assert got.shape == want.shape
            if not np.array_equal(got, want):
                bad = np.flatnonzero(got != want)
                raise AssertionError("unit %s pool %d: %d bytes differ, first at %d" % ((b, l, h), p, bad.size, bad[0]))
    return cache, flags


def _check_decode(cache, cfgw, T, flags, layers, units=None, step=0):
    import torch
    for l in layers:
        q = synth.query(cfgw, l, step)
        out = cache.decode_attn(l, torch.from_numpy(q).cuda()).cpu().numpy()
        out2 = cache.decode_attn(l, torch.from_numpy(q).cuda()).cpu().numpy()
        assert np.array_equal(out, out2), "decode is not deterministic"
        for b in range(cfgw.batch):
            for h in range(cfgw.n_kv_heads):
                if units is not None and (b, l, h) not in units:
                    continue
                u = U.oracle_unit(cfgw, l, b, h, flags[b], T)
                want = u.attend(q[b, 4 * h:4 * h + 4].astype(np.float64))
                U.assert_attention_close(out[b, 4 * h:4 * h + 4], want, "unit %s" % ((b, l, h),))


def test_single_layer_t2048_g32_full_parity():
    cfgw = get_config(0)
    cache, flags = _check_prefill(cfgw, 2048)
    _check_decode(cache, cfgw, 2048, flags, [0])


@pytest.mark.parametrize("T", [1, 37, 64, 65, 1000])
@pytest.mark.parametrize("G", [32, 64, 128])
def test_ragged_lengths_and_groups(T, G):
    cfgw = get_config(0, group=G, batch=2, n_kv_heads=2, n_q_heads=8)
    cache, flags = _check_prefill(cfgw, T)
    _check_decode(cache, cfgw, T, flags, [0])


@pytest.mark.parametrize("base,lh,ll,G", [("affine", 6, 5, 128), ("affine", 6, 5, 32), ("tq", 4, 3, 128),
                                          ("rot_affine", 6, 5, 64), ("affine", 8, 7, 128), ("affine", 3, 2, 128)])
def test_every_fill_of_a_pools_last_record(base, lh, ll, G):
    """T = 2 (64 + n), r = 1/2: both pools hold 64 + n rows, so each ends in a
    record with n valid slots; n runs over 1..64, so the decode mask covers
    every fill of each 16-token block of a last record, in both pools."""
    for n in range(1, 65):
        T = 2 * (64 + n)
        kw = dict(L_hi=lh, L_lo=ll) if base != "tq" else {}
        cfgw = get_config(0 if base != "tq" else 4, base=base, group=G, r_num=1, r_den=2, batch=1,
                          n_kv_heads=1, n_q_heads=4, n_layers=1, **kw)
        assert O.top_count(T, 1, 2) == T - O.top_count(T, 1, 2) == 64 + n
        try:
            cache, flags = _check_prefill(cfgw, T)
            _check_decode(cache, cfgw, T, flags, [0])
        except AssertionError as e:
            raise AssertionError("last record with %d valid slots: %s" % (n, e)) from None


@pytest.mark.parametrize("base,lh,ll,G", [("affine", 6, 5, 128), ("affine", 6, 5, 32), ("tq", 4, 3, 128),
                                          ("rot_affine", 6, 5, 128), ("affine", 8, 7, 128), ("affine", 3, 2, 128)])
@pytest.mark.parametrize("T,r", [(1100, (26, 100)), (576, (1, 1)), (2200, (1, 1)), (1100, (0, 1)),
                                 (2200, (1, 2)), (6400, (26, 100))])
def test_partial_last_round(base, lh, ll, G, T, r):
    """8 kv heads, so up to 32 workgroups per unit: with the split count
    the host picks (at most a unit's tiles / 8), these prompts leave a last
    round of 1 to nsplit tiles after whole rounds of the 8 waves of every
    workgroup -- its tiles in the low pool (1100 at 26 % and 0 %, 2200 at
    1/2, 6400) or in the high pool (r = 1: 576, 2200) -- so a few waves hold
    one record more than the rest."""
    kw = dict(L_hi=lh, L_lo=ll) if base != "tq" else {}
    cfgw = get_config(0 if base != "tq" else 4, base=base, group=G, r_num=r[0], r_den=r[1], batch=1,
                      n_kv_heads=8, n_q_heads=32, n_layers=1, **kw)
    cache, flags = _check_prefill(cfgw, T, units=[(0, 0, 0), (0, 0, 7)])
    _check_decode(cache, cfgw, T, flags, [0])


def _multi_chunk_scores(T, seed):
    """Three sequences: integer scores 0..3 (ties across every chunk
    boundary), all equal, and normal draws with +0, -0, +inf and -inf."""
    rng = np.random.default_rng(seed)
    s = np.empty((3, T), np.float32)
    s[0] = rng.integers(0, 4, T)
    s[1] = 1.0
    s[2] = rng.standard_normal(T)
    s[2, ::3] = 0.0
    s[2, 1::7] = -0.0
    s[2, 5], s[2, 6] = np.inf, -np.inf
    return s


@pytest.mark.parametrize("r", [(0, 1), (1, 2), (26, 100), (1, 1)])
def test_multi_chunk_ranker(r):
    """Sequences longer than a 4096-token chunk are ranked by one workgroup
    per chunk over five launches (histograms in scratch after the flag
    bitmaps, cleared again by each call).  Two calls in a row on one cache,
    the second shorter, so the second starts from the scratch the first left:
    flags and slot lists bit-exact against the oracle for both."""
    import torch
    cfgw = get_config(0, batch=3, n_kv_heads=1, n_q_heads=4, n_layers=1, r_num=r[0], r_den=r[1])
    cache = U.make_cache(cfgw, 40000, n_layers=1, max_new=0)
    for T, seed in ((40000, 1), (8193, 2), (4097, 3), (12288, 4)):
        s = _multi_chunk_scores(T, seed)
        hi, lo = cache.rank(torch.from_numpy(s).cuda())
        torch.cuda.synchronize()
        hi, lo = hi.cpu().numpy(), lo.cpu().numpy()
        for b in range(3):
            f, ohi, olo = O.rank(s[b], r[0], r[1])
            assert np.array_equal(hi[b], ohi) and np.array_equal(lo[b], olo), "slot lists, T %d seq %d" % (T, b)
            assert np.array_equal(U.flags_bits(cache, b, T), f), "flags, T %d seq %d" % (T, b)
        assert cache.status() == 0
    # per sequence, after the flag bitmaps (rounded up to 64 words): the three
    # histograms (5120 words) must be zero again; the selection state and
    # chunk counts that follow them are rewritten before every read
    words = cache.flags.view(-1).cpu().numpy()
    off = (3 * cache.sz.flag_words + 63) // 64 * 64
    stride = (5136 + 2 * ((40000 + 4095) // 4096) + 63) // 64 * 64
    assert len(words) == off + 3 * stride
    for b in range(3):
        assert not words[off + b * stride:off + b * stride + 5120].any(), "histograms of seq %d not cleared" % b


def test_multi_chunk_ranker_reports_nan():
    import torch
    cfgw = get_config(0, batch=1, n_kv_heads=1, n_q_heads=4, n_layers=1)
    cache = U.make_cache(cfgw, 9000, n_layers=1, max_new=0)
    s = np.random.default_rng(5).standard_normal((1, 9000)).astype(np.float32)
    s[0, 8500] = np.nan
    cache.rank(torch.from_numpy(s).cuda())
    torch.cuda.synchronize()
    assert cache.status() & 1


@pytest.mark.parametrize("r", [(0, 1), (1, 1), (1, 2)])
def test_all_low_all_high_half(r):
    cfgw = get_config(0, r_num=r[0], r_den=r[1], n_kv_heads=2, n_q_heads=8)
    cache, flags = _check_prefill(cfgw, 300)
    _check_decode(cache, cfgw, 300, flags, [0])


def test_tied_scores_and_signed_zero():
    cfgw = get_config(0, batch=3, n_kv_heads=1, n_q_heads=4)
    T = 777
    s = np.zeros((3, T), np.float32)
    s[0] = 1.0                                            # all equal: lowest indices win
    s[1] = np.where(np.arange(T) % 2, 0.0, -0.0)          # +0 and -0 tie
    s[2] = np.random.default_rng(3).integers(0, 3, T).astype(np.float32)
    s[2, 5] = np.inf
    s[2, 6] = -np.inf
    cache, flags = _check_prefill(cfgw, T, scores=s)
    _check_decode(cache, cfgw, T, flags, [0])


@pytest.mark.parametrize("levels", [(6, 4), (4, 3), (5, 3)])
def test_other_affine_level_pairs(levels):
    cfgw = get_config(0, L_hi=levels[0], L_lo=levels[1], n_kv_heads=2, n_q_heads=8, group=64)
    cache, flags = _check_prefill(cfgw, 500)
    _check_decode(cache, cfgw, 500, flags, [0])


def test_turboquant_base_small():
    cfgw = get_config(4, n_layers=2, n_kv_heads=2, n_q_heads=8)
    cache, flags = _check_prefill(cfgw, 1500, n_layers=2)
    _check_decode(cache, cfgw, 1500, flags, [0, 1])


@pytest.mark.parametrize("G", [32, 128])
@pytest.mark.parametrize("levels", [(6, 5), (5, 4)])
def test_rotated_affine_base(levels, G):
    """The affine quantizer of the Hadamard-rotated rows (Sec. 4.1): records
    bit-exact, attention over two layers (two sign masks) within tolerance."""
    cfgw = get_config(0, base="rot_affine", L_hi=levels[0], L_lo=levels[1], group=G, n_layers=2, batch=2,
                      n_kv_heads=2, n_q_heads=8)
    cache, flags = _check_prefill(cfgw, 1000, n_layers=2)
    _check_decode(cache, cfgw, 1000, flags, [0, 1])


@pytest.mark.parametrize("T", [1, 65])
def test_rotated_affine_ragged(T):
    cfgw = get_config(0, base="rot_affine", group=64, n_kv_heads=2, n_q_heads=8)
    cache, flags = _check_prefill(cfgw, T)
    _check_decode(cache, cfgw, T, flags, [0])


@pytest.mark.parametrize("base", ["affine", "rot_affine"])
@pytest.mark.parametrize("r", [(0, 1), (1, 1), (35, 100)])
@pytest.mark.parametrize("levels", [(8, 7), (7, 6), (3, 2)])
def test_level_grid_pairs(levels, r, base):
    """The rest of the integer-level grid (Sec. 4.2): 8, 7 and 2 levels (7
    codes in 20 bits, 2 in 6 bits, 8 in a byte); r = 0 and 1 are the uniform
    grid points of the cliff sweep, 35 % a mix."""
    cfgw = get_config(0, base=base, L_hi=levels[0], L_lo=levels[1], group=128, r_num=r[0], r_den=r[1],
                      n_kv_heads=2, n_q_heads=8)
    cache, flags = _check_prefill(cfgw, 700)
    _check_decode(cache, cfgw, 700, flags, [0])


def test_constant_rows_quantize_exactly():
    import torch
    cfgw = get_config(0, n_kv_heads=1, n_q_heads=4, group=32)
    T = 200
    rng = np.random.default_rng(9)
    K = np.repeat(rng.standard_normal((1, 1, T, 4)), 32, -1).astype(np.float16)
    V = np.repeat(rng.standard_normal((1, 1, T, 4)), 32, -1).astype(np.float16)
    cache = U.make_cache(cfgw, T, max_new=0)
    s = synth.all_scores(cfgw, T)
    U.prefill(cache, cfgw, T, scores=s, kv=lambda l: (K, V))
    q = synth.query(cfgw, 0, 0)
    out = cache.decode_attn(0, torch.from_numpy(q).cuda()).cpu().numpy()
    want = O.attention(q[0, :4].astype(np.float64), K[0, 0].astype(np.float64), V[0, 0].astype(np.float64))
    U.assert_attention_close(out[0, :4], want, "constant rows")


@pytest.mark.parametrize("G", [32, 128])
def test_affine_code_ties_round_to_even(G):
    """Rows built so that every group's scale is exactly 1 (range L-1, L the
    level count the token's rank gives) and half the values sit exactly
    halfway between two codes: the codes round half to even, bit-exact
    against the oracle, in both pools."""
    cfgw = get_config(0, n_kv_heads=1, n_q_heads=4, group=G)
    T = 256
    s = synth.all_scores(cfgw, T)
    f, _, _ = O.rank(s[0], cfgw.r_num, cfgw.r_den)
    rng = np.random.default_rng(31 + G)
    X = np.zeros((2, T, 128), np.float32)
    for kv in range(2):
        for t in range(T):
            L = cfgw.L_hi if f[t] else cfgw.L_lo
            for g in range(128 // G):
                lo = float(rng.choice([-3.0, -1.5, 0.0, 2.0]))
                row = lo + rng.integers(0, 2 * (L - 1) + 1, G) / 2.0
                row[0], row[1] = lo, lo + (L - 1)
                X[kv, t, g * G:(g + 1) * G] = row
    assert np.mean(np.abs(X - np.round(X)) == 0.5) > 0.3          # ties are really there
    K, V = X[0].astype(np.float16)[None, None], X[1].astype(np.float16)[None, None]
    cache = U.make_cache(cfgw, T, max_new=0)
    U.prefill(cache, cfgw, T, scores=s, kv=lambda l: (K, V))
    assert cache.status() == 0
    u = U.oracle_unit(cfgw, 0, 0, 0, f, T, kv=lambda l: (K, V))
    for p in (0, 1):
        assert np.array_equal(U.gpu_records(cache, 0, 0, 0, p, u.count(p)), u.records(p)), "pool %d" % p


def test_status_word_reports_nan_and_inf():
    import torch
    cfgw = get_config(0, n_kv_heads=1, n_q_heads=4)
    T = 100
    s = synth.all_scores(cfgw, T)
    s[0, 7] = np.nan
    cache = U.make_cache(cfgw, T, max_new=0)
    cache.rank(torch.from_numpy(s).cuda())
    torch.cuda.synchronize()
    assert cache.status() & 1
    K, V = synth.layer_kv(cfgw, 0, T)
    K[0, 0, 3, 9] = np.inf
    cache2 = U.make_cache(cfgw, T, max_new=0)
    s2 = synth.all_scores(cfgw, T)
    U.prefill(cache2, cfgw, T, scores=s2, kv=lambda l: (K, V))
    assert cache2.status() & 2


def test_tq_norm_rounding_edge_rows():
    """Rows whose norm sits at an fp16 rounding edge (a square root one ulp off
    would store a different norm): packed records bit-exact."""
    import torch
    from tests.norm_edge import edge_rows
    cfgw = get_config(4, n_layers=1, n_kv_heads=1, n_q_heads=4)
    T = 256
    X = edge_rows(2 * T).reshape(2, T, 128)
    K, V = X[0][None, None], X[1][None, None]
    cache = U.make_cache(cfgw, T, max_new=0)
    s = synth.all_scores(cfgw, T)
    U.prefill(cache, cfgw, T, scores=s, kv=lambda l: (K, V))
    f, _, _ = O.rank(s[0], cfgw.r_num, cfgw.r_den)
    u = U.oracle_unit(cfgw, 0, 0, 0, f, T, kv=lambda l: (K, V))
    for p in (0, 1):
        assert np.array_equal(U.gpu_records(cache, 0, 0, 0, p, u.count(p)), u.records(p)), "pool %d" % p


def test_max_batch():
    """1024 sequences (the most semkv_append_commit takes): rank, quantize,
    decode, a generated token and a residual flush, sampled sequences checked."""
    import torch
    cfgw = get_config(0, batch=1024, n_kv_heads=1, n_q_heads=4, n_gen=2)
    T = 100
    cache = U.make_cache(cfgw, T, n_layers=1, max_new=2)
    scores, hi, lo = U.prefill(cache, cfgw, T)
    hi, lo = hi.cpu().numpy(), lo.cpu().numpy()
    q = synth.query(cfgw, 0, 0)
    k = torch.from_numpy(np.stack([synth.unit_gen_kv(cfgw, 0, b, 0, 1)[0] for b in range(1024)])[:, None, 0]).cuda()
    v = torch.from_numpy(np.stack([synth.unit_gen_kv(cfgw, 0, b, 0, 1)[1] for b in range(1024)])[:, None, 0]).cuda()
    out = cache.append_decode_attn(0, k, v, torch.from_numpy(q).cuda()).cpu().numpy()
    cache.append_commit(torch.arange(1024, dtype=torch.float32).cuda())
    cache.flush()
    torch.cuda.synchronize()
    assert cache.status() == 0 and cache.c.n_hi + cache.c.n_lo == T + 1
    for b in (0, 1, 511, 1023):
        flag, ohi, olo = O.rank(scores[b], cfgw.r_num, cfgw.r_den)
        assert np.array_equal(hi[b], ohi) and np.array_equal(lo[b], olo)
        u = U.oracle_unit(cfgw, 0, b, 0, flag, T)
        u.append_kv(k[b, 0].cpu().numpy(), v[b, 0].cpu().numpy())
        U.assert_attention_close(out[b], u.attend(q[b].astype(np.float64)), "sequence %d" % b)
        u.commit(float(b))
        u.flush()
        for p in (0, 1):
            n = u.count(p)
            assert np.array_equal(U.gpu_records(cache, b, 0, 0, p, n), u.records(p)), "sequence %d pool %d" % (b, p)


@pytest.mark.parametrize("wl", [0, 4])
def test_all_layers_launch(wl):
    """semkv_decode_attn with layer -1 attends over every layer in one launch
    (queries of all layers given up front); each layer's output is checked
    against the oracle, before and after the current token is appended to
    every layer (then read from the fp16 tail)."""
    import torch
    from paper_2608_28911_amd import SemKVError
    cfgw = get_config(wl, n_layers=3, batch=2, n_kv_heads=2, n_q_heads=8)
    T = 900
    cache = U.make_cache(cfgw, T, n_layers=3, max_new=4)
    scores, _, _ = U.prefill(cache, cfgw, T)
    q = np.stack([synth.query(cfgw, l, 0) for l in range(3)])
    units = {}
    for l in range(3):
        for b in range(2):
            flag = O.rank(scores[b], cfgw.r_num, cfgw.r_den)[0]
            for h in range(2):
                units[(b, l, h)] = U.oracle_unit(cfgw, l, b, h, flag, T)
    gen = {key: synth.unit_gen_kv(cfgw, key[1], key[0], key[2], 1) for key in units}
    for step in range(2):
        out = cache.decode_attn(-1, torch.from_numpy(q).cuda()).cpu().numpy()
        for (b, l, h), u in units.items():
            U.assert_attention_close(out[l, b, 4 * h:4 * h + 4], u.attend(q[l, b, 4 * h:4 * h + 4].astype(np.float64)),
                                     "step %d unit %s" % (step, (b, l, h)))
        if step == 1:
            break
        for l in range(3):
            k = np.stack([np.stack([gen[(b, l, h)][0][0] for h in range(2)]) for b in range(2)])
            v = np.stack([np.stack([gen[(b, l, h)][1][0] for h in range(2)]) for b in range(2)])
            cache.append_kv(l, torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda())
            for (b, ll, h), u in units.items():
                if ll == l:
                    u.append_kv(gen[(b, l, h)][0][0], gen[(b, l, h)][1][0])
            if l == 0:
                with pytest.raises(SemKVError):              # layers disagree on the tail length
                    cache.decode_attn(-1, torch.from_numpy(q).cuda())


def test_one_workspace_serves_both_launch_kinds():
    """One workspace serves one-layer and all-layers launches in any order: the
    counter prefix covers every layer (here 4 x 3 x 8 counters, 384 bytes, more
    than one 256-byte block), so the partials of a one-layer launch never land
    on counters an all-layers launch reads.  Every unit of every launch is
    checked against the oracle."""
    import torch
    cfgw = get_config(0, n_layers=4, batch=3, n_kv_heads=8, n_q_heads=32)
    T = 300
    cache = U.make_cache(cfgw, T, n_layers=4, max_new=0)
    scores, _, _ = U.prefill(cache, cfgw, T)
    ws = torch.zeros((cache.sz.workspace_bytes + 3) // 4, dtype=torch.float32, device="cuda")
    q = np.stack([synth.query(cfgw, l, 0) for l in range(4)])
    want = {}
    for b in range(3):
        flag = O.rank(scores[b], cfgw.r_num, cfgw.r_den)[0]
        for l in range(4):
            for h in range(8):
                u = U.oracle_unit(cfgw, l, b, h, flag, T)
                want[(b, l, h)] = u.attend(q[l, b, 4 * h:4 * h + 4].astype(np.float64))
    qd = torch.from_numpy(q).cuda()
    for kind in ("layer", "all", "layer", "all", "all"):
        if kind == "layer":
            out = np.stack([cache.decode_attn(l, qd[l], workspace=ws).cpu().numpy() for l in range(4)])
        else:
            out = cache.decode_attn(-1, qd, workspace=ws).cpu().numpy()
        for (b, l, h), w in want.items():
            U.assert_attention_close(out[l, b, 4 * h:4 * h + 4], w, "%s launch, unit %s" % (kind, (b, l, h)))
    nctr = 4 * 3 * 8
    assert np.all(ws[:nctr].view(torch.int32).cpu().numpy() == 0), "counters left non-zero"


def _huge_rows(rng, n):
    """fp16 rows over the whole finite range: halves at -+60000 (a range above
    65504), constant rows of +-9000 (rotated coordinate +-72000), random bit
    patterns, and unit-scale rows."""
    X = rng.standard_normal((n, 128)).astype(np.float32)
    q = n // 4
    X[:q, :64], X[:q, 64:] = -60000, 60000
    X[q:2 * q] = rng.choice([-9000.0, 9000.0], (q, 1))
    bits = rng.integers(0, 0x7C00, (q, 128), dtype=np.uint32).astype(np.uint16)
    bits |= (rng.integers(0, 2, (q, 128)) << 15).astype(np.uint16)
    X[2 * q:3 * q] = bits.view(np.float16).astype(np.float32)
    X = X.astype(np.float16)
    return X[rng.permutation(n)]


@pytest.mark.parametrize("base,lh,ll,G", [("affine", 3, 2, 128), ("rot_affine", 3, 2, 128),
                                          ("rot_affine", 6, 5, 32), ("rot_affine", 6, 5, 128)])
def test_huge_rows_saturate_the_parameters(base, lh, ll, G):
    """Rows whose 2-level affine scale or rotated-affine zero/scale would
    overflow fp16 (Sec. 4.1's two fp16 parameters, saturated at +-65504):
    records of both pools bit-exact with the oracle, no inf/NaN stored, and
    attention finite and close to the oracle's.  Values reach 6e4 here, so
    the max-abs bar is taken relative to the largest reconstructed value
    (scaling V scales the output and its error alike)."""
    import torch
    cfgw = get_config(0, n_layers=1, n_kv_heads=1, n_q_heads=4, base=base, L_hi=lh, L_lo=ll, group=G)
    T = 300
    rng = np.random.default_rng([lh, ll, G, len(base)])
    K = _huge_rows(rng, T)[None, None]
    V = _huge_rows(rng, T)[None, None]
    s = synth.all_scores(cfgw, T)
    cache = U.make_cache(cfgw, T, max_new=0)
    U.prefill(cache, cfgw, T, scores=s, kv=lambda l: (K, V))
    assert cache.status() == 0
    f = O.rank(s[0], cfgw.r_num, cfgw.r_den)[0]
    u = U.oracle_unit(cfgw, 0, 0, 0, f, T, kv=lambda l: (K, V))
    for p in (0, 1):
        got = U.gpu_records(cache, 0, 0, 0, p, u.count(p))
        assert np.array_equal(got, u.records(p)), "pool %d" % p
        kc, km, vc, vm, _ = u.pool(p)
        assert np.all((km & 0x7C00) != 0x7C00) and np.all((vm & 0x7C00) != 0x7C00)
    q = (synth.query(cfgw, 0, 0).astype(np.float32) * 1e-3).astype(np.float16)
    out = cache.decode_attn(0, torch.from_numpy(q).cuda()).cpu().numpy()
    _, kh, vh = u.dequantized()
    assert np.all(np.isfinite(kh)) and np.all(np.isfinite(vh))
    want = u.attend(q[0].astype(np.float64))
    assert np.all(np.isfinite(out))
    d = np.abs(out[0] - want).max()
    assert d <= U.TOL * max(1.0, np.abs(vh).max()), d


@pytest.mark.parametrize("pool", [0, 1])
def test_tq_threshold_ties_bit_exact(pool):
    """Rows with a rotated coordinate exactly on fl32(rho * tau) for every
    Lloyd-Max threshold of the pool's level count (and on the zero threshold
    of 4 levels): strict >, the tie goes to the lower cell, as in the pinned
    oracle.  All rows go to one pool (r = 1 or r = 0)."""
    from tests.tie_rows import tq_tie_rows
    cfgw = get_config(4, n_layers=1, n_kv_heads=1, n_q_heads=4, r_num=1 - pool, r_den=1)
    mu32, tau32 = O.codebook32(cfgw.L_hi if pool == 0 else cfgw.L_lo)
    rows = tq_tie_rows(tau32, per_threshold=4)
    T = 2 * len(rows) + 70
    X = np.zeros((2, T, 128), np.float16)
    X[0, :len(rows)] = rows
    X[1, len(rows):2 * len(rows)] = rows
    X[:, 2 * len(rows):] = synth.unit_kv(cfgw, 0, 0, 0, 70)[0]
    K, V = X[0][None, None], X[1][None, None]
    s = synth.all_scores(cfgw, T)
    cache = U.make_cache(cfgw, T, max_new=0)
    # the workload's sign masks would move the ties: use all-positive signs
    cache.signs.zero_()
    U.prefill(cache, cfgw, T, scores=s, kv=lambda l: (K, V))
    assert cache.status() == 0
    f = O.rank(s[0], cfgw.r_num, cfgw.r_den)[0]
    u = O.UnitCache(O.TQ, cfgw.L_hi, cfgw.L_lo, 128, cfgw.r_num, cfgw.r_den, sign_words=np.zeros(4, np.uint32))
    u.prefill(X[0], X[1], f)
    assert u.count(pool) == T
    assert np.array_equal(U.gpu_records(cache, 0, 0, 0, pool, T), u.records(pool))
