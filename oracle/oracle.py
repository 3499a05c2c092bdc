"""Python face of the CPU oracle (TEST INFRASTRUCTURE ONLY).

Only tests/, ``__graft_entry__.smoke()`` and the cpu_baseline leg of
``bench.py`` may import this module.  It loads ``liboracle.so`` (plain C, built
from ``semkv_oracle.c`` with gcc) and composes its per-row primitives into the
storage the hot path produces: for one (sequence, layer, kv head) unit, a high-
and a low-precision pool of 64-slot records.  It shares no code with the HIP
library and never imports the product package.

Record format (one 64-slot tile of a pool), bytes in order:
  K body  TB(L)   packed codes, a line = one token row of 128 channels
  V body  TB(L)   packed codes, a line = one channel column over the 64 slots
  K meta  MB      affine and rotated affine:
                          [128/G groups][64 slots] x (fp16 scale, fp16 zero)
                  tq:     [64 slots] x fp16 rho
  V meta  MB      same
"""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "semkv_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

SLOTS = 64
D = 128


# OQ_SANITIZE=1 selects a separate build instrumented with AddressSanitizer
# and UndefinedBehaviorSanitizer (any finding aborts the process); the Python
# process must then start with libasan preloaded (tests/test_oracle_sanitized.py
# runs the CPU oracle tests that way).
SANITIZE = os.environ.get("OQ_SANITIZE") == "1"
if SANITIZE:
    LIB = os.path.join(HERE, "liboracle_san.so")


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (IEEE single precision, no contraction)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < max(
            os.path.getmtime(SRC), os.path.getmtime(os.path.join(HERE, "semkv_oracle.h"))):
        tmp = LIB + ".tmp%d" % os.getpid()
        san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               "-fno-omit-frame-pointer", "-g"] if SANITIZE else []
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                               "-Wall", "-shared", "-fPIC"] + san + ["-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int
        sig = {
            "oq_f32_to_f16": (ctypes.c_uint16, [ctypes.c_float]),
            "oq_f16_to_f32": (ctypes.c_float, [ctypes.c_uint16]),
            "oq_top_count": (i64, [i64, i64, i64]),
            "oq_block_count": (i64, [i64, i64, i64]),
            "oq_rank_k": (i32, [P, i64, i64, P]),
            "oq_affine_row": (i32, [P, i32, i32, P, P]),
            "oq_lloyd_max": (i32, [i32, P, P, P]),
            "oq_tq_row": (i32, [P, P, i32, P, P, P]),
            "oq_rotaffine_row": (i32, [P, P, i32, i32, P, P]),
            "oq_quantize_rows": (i32, [P, i64, i32, i32, i32, P, P, P, P]),
            "oq_symbol_digits": (i32, [i32]),
            "oq_symbol_bits": (i32, [i32, i32]),
            "oq_line_bits": (i64, [i32, i32]),
            "oq_tile_bytes": (i64, [i32]),
            "oq_pack_tile": (i32, [P, P, i32, P, P]),
            "oq_affine_dequant_rows": (None, [P, P, i64, i32, P]),
            "oq_tq_dequant_rows": (None, [P, P, i64, P, P, P]),
            "oq_rotaffine_dequant_rows": (None, [P, P, i64, i32, P, P]),
            "oq_attention": (None, [P, i32, P, P, i64, i32, P]),
            "oq_score_hidden": (i32, [i32, P, i32, i64, i32, P]),
            "oq_score_kv_norm": (i32, [P, i32, i64, P]),
            "oq_bf16_to_f32_n": (None, [P, i64, P]),
            "oq_set_threads": (None, [i32]),
            "oq_max_threads": (i32, []),
            "oq_attention_units": (None, [i32, P, i32, P, P, P, i32, P]),
            "oq_f32_to_f16_n": (None, [P, i64, P]),
            "oq_f16_to_f32_n": (None, [P, i64, P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(_lib, name)
            f.restype, f.argtypes = res, args
    return _lib


def set_threads(n: int) -> None:
    """OpenMP threads of the row-parallel oracle calls (timing runs only)."""
    lib().oq_set_threads(int(n))


def max_threads() -> int:
    """Threads an OpenMP region of the oracle uses."""
    return lib().oq_max_threads()


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


class OracleError(RuntimeError):
    pass


def _check(st):
    if st == -4:
        raise OracleError("non-finite input (NaN/inf)")
    if st != 0:
        raise OracleError("invalid argument (status %d)" % st)


# ------------------------------------------------------------- fp16 -------

def f32_to_f16_bits(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().oq_f32_to_f16_n(_p(x), x.size, _p(out))
    return out


def f16_bits_to_f32(h) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, np.float32)
    lib().oq_f16_to_f32_n(_p(h), h.size, _p(out))
    return out


# ----------------------------------------------------------- ranking ------

def top_count(T, r_num, r_den) -> int:
    """Eq. (4): K = floor(r T)."""
    return lib().oq_top_count(T, r_num, r_den)


def block_count(n, r_num, r_den) -> int:
    """Alg. 2: round(r n), ties to even."""
    return lib().oq_block_count(n, r_num, r_den)


def rank_k(s, k) -> np.ndarray:
    s = np.ascontiguousarray(s, dtype=np.float32)
    flag = np.zeros(s.shape[0], np.uint8)
    _check(lib().oq_rank_k(_p(s), s.shape[0], int(k), _p(flag)))
    return flag


def rank(s, r_num, r_den):
    """Eq. (4)-(5) on one sequence: returns (flag uint8[T], hi_idx, lo_idx)."""
    s = np.asarray(s, dtype=np.float32)
    flag = rank_k(s, top_count(s.shape[0], r_num, r_den))
    return flag, np.flatnonzero(flag).astype(np.int32), np.flatnonzero(flag == 0).astype(np.int32)


def flag_words(flag: np.ndarray, n_words: int | None = None) -> np.ndarray:
    """Precision flags as a bitmap: bit i%32 of word i/32."""
    T = flag.shape[0]
    n_words = (T + 31) // 32 if n_words is None else n_words
    w = np.zeros(n_words, np.uint32)
    for i in np.flatnonzero(flag):
        w[i // 32] |= np.uint32(1 << (int(i) % 32))
    return w


# ---------------------------------------------------------- quantizers ----

def lloyd_max(L):
    """Lloyd-Max codebook of N(0,1): (mu fp64[L], tau fp64[L-1], mse)."""
    mu = np.zeros(L, np.float64)
    tau = np.zeros(max(L - 1, 1), np.float64)
    mse = np.zeros(1, np.float64)
    _check(lib().oq_lloyd_max(L, _p(mu), _p(tau), _p(mse)))
    return mu, tau[: L - 1], float(mse[0])


def codebook32(L):
    mu, tau, _ = lloyd_max(L)
    return mu.astype(np.float32), tau.astype(np.float32)


AFFINE, TQ, ROT_AFFINE = 0, 1, 2


def quantize_rows(X, base, L, G=128, sign_words=None):
    """Rows of fp16 [n, 128] -> (codes uint8 [n,128], meta uint16).
    base 0 affine, 1 TurboQuant-MSE, 2 affine of the rotated row.
    meta: affine / rotated affine [n, 128/G, 2] (scale, zero bits); tq [n] (rho bits)."""
    X = np.ascontiguousarray(X, dtype=np.float16).view(np.uint16)
    n = X.shape[0]
    codes = np.zeros((n, D), np.uint8)
    if base != TQ:
        meta = np.zeros((n, D // G, 2), np.uint16)
        sw = np.zeros(4, np.uint32) if base == AFFINE else np.ascontiguousarray(sign_words, dtype=np.uint32)
        tau = np.zeros(1, np.float32)
    else:
        meta = np.zeros(n, np.uint16)
        sw = np.ascontiguousarray(sign_words, dtype=np.uint32)
        tau = np.ascontiguousarray(codebook32(L)[1])
    if n:
        _check(lib().oq_quantize_rows(_p(X), n, base, L, G, _p(sw), _p(tau), _p(codes), _p(meta)))
    return codes, meta


def dequantize_rows(codes, meta, base, L, G=128, sign_words=None) -> np.ndarray:
    """Fake-quantized values (float64 [n,128]); affine values are fp32 exact."""
    codes = np.ascontiguousarray(codes, np.uint8)
    n = codes.shape[0]
    if base == AFFINE:
        out = np.zeros((n, D), np.float32)
        if n:
            lib().oq_affine_dequant_rows(_p(codes), _p(np.ascontiguousarray(meta, np.uint16)), n, G, _p(out))
        return out.astype(np.float64)
    out = np.zeros((n, D), np.float64)
    if base == ROT_AFFINE:
        if n:
            lib().oq_rotaffine_dequant_rows(_p(codes), _p(np.ascontiguousarray(meta, np.uint16)), n, G,
                                            _p(np.ascontiguousarray(sign_words, np.uint32)), _p(out))
        return out
    mu32 = np.ascontiguousarray(codebook32(L)[0])
    if n:
        lib().oq_tq_dequant_rows(_p(codes), _p(np.ascontiguousarray(meta, np.uint16)), n,
                                 _p(np.ascontiguousarray(sign_words, np.uint32)), _p(mu32), _p(out))
    return out


# ------------------------------------------------------------- packing ----

def symbol_digits(L) -> int:
    return lib().oq_symbol_digits(L)


def symbol_bits(L, nd) -> int:
    return lib().oq_symbol_bits(L, nd)


def line_bits(L, nvalues) -> int:
    return lib().oq_line_bits(L, nvalues)


def tile_bytes(L) -> int:
    return lib().oq_tile_bytes(L)


def meta_bytes(base, G=128) -> int:
    return (D // G) * SLOTS * 4 if base != TQ else SLOTS * 2


def record_bytes(base, L, G=128) -> int:
    return 2 * tile_bytes(L) + 2 * meta_bytes(base, G)


def pack_tile(kcodes, vcodes, L):
    """kcodes, vcodes: uint8 [64 slots, 128] -> (K body, V body) bytes."""
    tb = tile_bytes(L)
    kb = np.zeros(tb, np.uint8)
    vb = np.zeros(tb, np.uint8)
    _check(lib().oq_pack_tile(_p(np.ascontiguousarray(kcodes, np.uint8)),
                              _p(np.ascontiguousarray(vcodes, np.uint8)), L, _p(kb), _p(vb)))
    return kb, vb


def _meta_tile(meta, base, G, lo, hi):
    """Metadata of slots [lo, hi) in record order; unused slots are zero."""
    if base != TQ:
        m = np.zeros((D // G, SLOTS, 2), np.uint16)
        m[:, : hi - lo, :] = np.transpose(meta[lo:hi], (1, 0, 2))
    else:
        m = np.zeros(SLOTS, np.uint16)
        m[: hi - lo] = meta[lo:hi]
    return m.view(np.uint8).reshape(-1)


def build_pool(kcodes, kmeta, vcodes, vmeta, base, L, G=128, cap_tiles=None) -> np.ndarray:
    """Slots 0..n-1 of a pool (codes/meta per slot, slot order) -> record bytes
    of cap_tiles records (default: just enough for n slots)."""
    n = kcodes.shape[0]
    ntile = (n + SLOTS - 1) // SLOTS
    cap = ntile if cap_tiles is None else cap_tiles
    assert cap >= ntile
    rb = record_bytes(base, L, G)
    tb = tile_bytes(L)
    out = np.zeros(cap * rb, np.uint8)
    for t in range(ntile):
        lo, hi = t * SLOTS, min(n, (t + 1) * SLOTS)
        kc = np.zeros((SLOTS, D), np.uint8)
        vc = np.zeros((SLOTS, D), np.uint8)
        kc[: hi - lo] = kcodes[lo:hi]
        vc[: hi - lo] = vcodes[lo:hi]
        kb, vb = pack_tile(kc, vc, L)
        r = out[t * rb:(t + 1) * rb]
        r[:tb] = kb
        r[tb:2 * tb] = vb
        mb = meta_bytes(base, G)
        r[2 * tb:2 * tb + mb] = _meta_tile(kmeta, base, G, lo, hi)
        r[2 * tb + mb:] = _meta_tile(vmeta, base, G, lo, hi)
    return out


# ----------------------------------------------------------- attention ----

def attention(q, khat, vhat) -> np.ndarray:
    """softmax(q K^T / sqrt(D)) V in float64. q [nq, D]; khat, vhat [n, D]."""
    q = np.ascontiguousarray(q, np.float64)
    k = np.ascontiguousarray(khat, np.float64)
    v = np.ascontiguousarray(vhat, np.float64)
    out = np.zeros(q.shape, np.float64)
    assert k.shape[0] >= 1
    lib().oq_attention(_p(q), q.shape[0], _p(k), _p(v), k.shape[0], q.shape[1], _p(out))
    return out


def attention_units(units) -> list:
    """attention(q, khat, vhat) of many independent units at once, OpenMP
    across the units (timing runs).  units: list of (q, khat, vhat)."""
    qs = [np.ascontiguousarray(q, np.float64) for q, _, _ in units]
    ks = [np.ascontiguousarray(k, np.float64) for _, k, _ in units]
    vs = [np.ascontiguousarray(v, np.float64) for _, _, v in units]
    outs = [np.zeros(q.shape, np.float64) for q in qs]
    nq, d = qs[0].shape
    assert all(q.shape == (nq, d) for q in qs) and all(k.shape[0] >= 1 for k in ks)
    ptrs = lambda xs: (ctypes.c_void_p * len(xs))(*[x.ctypes.data for x in xs])
    n = np.array([k.shape[0] for k in ks], np.int64)
    lib().oq_attention_units(len(units), ptrs(qs), nq, ptrs(ks), ptrs(vs), _p(n), d, ptrs(outs))
    return outs


# ---------------------------------------------------------- indicators ----

DELTA_NORM, NORM, VARIANCE, COSINE_DELTA = 0, 1, 2, 3


def bf16_bits_to_f32(h) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, np.float32)
    lib().oq_bf16_to_f32_n(_p(h), h.size, _p(out))
    return out


def score_hidden(indicator, H, bf16=False) -> np.ndarray:
    """Sec. 3.3 hidden-state indicators of one sequence.  H: [m+1, T, d] fp16
    values (or bf16 bits as uint16 with bf16=True), state k = layer L-m+k.
    Returns float64 [T]."""
    Hf = bf16_bits_to_f32(H) if bf16 else np.ascontiguousarray(H, np.float16).astype(np.float32)
    n, T, d = Hf.shape
    s = np.zeros(T, np.float64)
    _check(lib().oq_score_hidden(indicator, _p(Hf), n - 1, T, d, _p(s)))
    return s


def score_kv_norm(X) -> np.ndarray:
    """KV-norm indicator of one sequence: X fp16 [R rows (layer x kv head), T, 128]
    -> sqrt of the sum of squares over every row of each token, float64 [T]."""
    Xf = np.ascontiguousarray(X, np.float16).astype(np.float32)
    R, T, _ = Xf.shape
    s = np.zeros(T, np.float64)
    _check(lib().oq_score_kv_norm(_p(Xf), R, T, _p(s)))
    return s


# ------------------------------------------------ one unit of the cache ----

HI, LO = 0, 1


class UnitCache:
    """The oracle's model of one (sequence, layer, kv head) unit.

    Prompt tokens are ranked once (Eq. 4-5) and quantized into the high or
    low pool (Eq. 7, Alg. 1).  Generated tokens follow Alg. 2: they are kept
    at fp16 in a tail of at most ``block`` rows; when ``block`` scores have
    been committed the block closes, exactly round(r B) of its tokens go to
    the high pool and the rest to the low pool.  ``flush`` closes a partial
    block with round(r n).  Pools keep slot order: increasing token position
    within each pool, prompt first, then blocks in close order.
    """

    def __init__(self, base, L_hi, L_lo, G, r_num, r_den, block=64, sign_words=None):
        self.base, self.L = base, (L_hi, L_lo)
        self.G, self.r_num, self.r_den, self.block = G, r_num, r_den, block
        self.sign_words = sign_words
        self.codes = [{"k": [], "km": [], "v": [], "vm": [], "pos": []} for _ in range(2)]
        self.tail_k, self.tail_v, self.tail_s, self.tail_pos = [], [], [], []
        self.n_tokens = 0

    def _add(self, p, K, V, pos):
        kc, km = quantize_rows(K, self.base, self.L[p], self.G, self.sign_words)
        vc, vm = quantize_rows(V, self.base, self.L[p], self.G, self.sign_words)
        d = self.codes[p]
        d["k"].append(kc); d["km"].append(km); d["v"].append(vc); d["vm"].append(vm)
        d["pos"].append(np.asarray(pos, np.int64))

    def prefill(self, K, V, flag):
        assert self.n_tokens == 0
        T = K.shape[0]
        pos = np.arange(T)
        for p, sel in ((HI, flag == 1), (LO, flag == 0)):
            self._add(p, K[sel], V[sel], pos[sel])
        self.n_tokens = T

    def append_kv(self, k, v):
        assert len(self.tail_k) == len(self.tail_s) and len(self.tail_k) < self.block
        self.tail_k.append(np.asarray(k, np.float16))
        self.tail_v.append(np.asarray(v, np.float16))
        self.tail_pos.append(self.n_tokens)
        self.n_tokens += 1

    def commit(self, score):
        assert len(self.tail_s) + 1 == len(self.tail_k)
        self.tail_s.append(np.float32(score))
        if len(self.tail_s) == self.block:
            self._close()

    def flush(self):
        assert len(self.tail_s) == len(self.tail_k)
        if self.tail_s:
            self._close()

    def _close(self):
        n = len(self.tail_s)
        flag = rank_k(np.array(self.tail_s, np.float32), block_count(n, self.r_num, self.r_den))
        K, V = np.stack(self.tail_k), np.stack(self.tail_v)
        pos = np.array(self.tail_pos)
        for p, sel in ((HI, flag == 1), (LO, flag == 0)):
            self._add(p, K[sel], V[sel], pos[sel])
        self.tail_k, self.tail_v, self.tail_s, self.tail_pos = [], [], [], []

    # views ------------------------------------------------------------
    def pool(self, p):
        d = self.codes[p]
        cat = lambda xs, shape, dt: np.concatenate(xs) if xs else np.zeros(shape, dt)
        mshape = (0, D // self.G, 2) if self.base != TQ else (0,)
        return (cat(d["k"], (0, D), np.uint8), cat(d["km"], mshape, np.uint16),
                cat(d["v"], (0, D), np.uint8), cat(d["vm"], mshape, np.uint16),
                cat(d["pos"], (0,), np.int64))

    def count(self, p) -> int:
        return self.pool(p)[0].shape[0]

    def records(self, p, cap_tiles=None) -> np.ndarray:
        kc, km, vc, vm, _ = self.pool(p)
        return build_pool(kc, km, vc, vm, self.base, self.L[p], self.G, cap_tiles)

    def dequantized(self):
        """(positions, K_hat, V_hat) over every token: pools then fp16 tail."""
        ks, vs, ps = [], [], []
        for p in (HI, LO):
            kc, km, vc, vm, pos = self.pool(p)
            ks.append(dequantize_rows(kc, km, self.base, self.L[p], self.G, self.sign_words))
            vs.append(dequantize_rows(vc, vm, self.base, self.L[p], self.G, self.sign_words))
            ps.append(pos)
        if self.tail_k:
            ks.append(np.stack(self.tail_k).astype(np.float64))
            vs.append(np.stack(self.tail_v).astype(np.float64))
            ps.append(np.array(self.tail_pos))
        return np.concatenate(ps), np.concatenate(ks), np.concatenate(vs)

    def attend(self, q):
        """Decode attention of the GQA query heads q [g, D] over the unit."""
        _, kh, vh = self.dequantized()
        return attention(np.asarray(q, np.float64), kh, vh)


# ------------------------------------------------------------ accounting --

def code_bits_per_value(L) -> float:
    """Row-exact packed code bits per value of one 128-dim token row."""
    return line_bits(L, D) / D


def effective_bits(n_hi, n_lo, base, L_hi, L_lo, G=128, n_layers=32, n_kv_heads=8):
    """Sec. 4.1 accounting, row exact: packed code bits + per-row metadata
    (affine: 2 fp16 per G channels; tq: 1 fp16 per row) + the 1-bit
    per-token precision flag spread over all layers, heads, K and V."""
    n = n_hi + n_lo
    code = (n_hi * line_bits(L_hi, D) + n_lo * line_bits(L_lo, D)) / (n * D)
    meta = 32.0 / G if base != TQ else 16.0 / D
    flag = 1.0 / (n_layers * n_kv_heads * 2 * D)
    return code, code + meta + flag


def allocated_bytes(n_hi, n_lo, base, L_hi, L_lo, G=128, n_layers=32, n_kv_heads=8, batch=1):
    """Bytes of the tile-padded pools for the whole cache (all units)."""
    t_hi = (n_hi + SLOTS - 1) // SLOTS
    t_lo = (n_lo + SLOTS - 1) // SLOTS
    per_unit = t_hi * record_bytes(base, L_hi, G) + t_lo * record_bytes(base, L_lo, G)
    flags = ((n_hi + n_lo + 31) // 32) * 4
    return batch * (n_layers * n_kv_heads * per_unit + flags)


def fp16_bytes(T, n_layers=32, n_kv_heads=8, batch=1):
    """Eq. (1) at b = 16: 2 L H_kv T D * 16 bits."""
    return batch * 2 * n_layers * n_kv_heads * T * D * 2
