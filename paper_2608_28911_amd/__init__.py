"""SemKV hot path on MI355X: Python binding of libsemkv.so.

The binding only marshals arguments: torch supplies device memory and the
current HIP stream, every step of the path (ranking, quantize + pack, deferred
append and close, decode attention) runs in the library's gfx950 kernels.
"""
import ctypes

import numpy as np

from . import _abi
from ._abi import BASE_AFFINE, BASE_ROT_AFFINE, BASE_TQ, SemKVError, check, lib

__all__ = ["SemKVCache", "SemKVError", "BASE_AFFINE", "BASE_TQ", "BASE_ROT_AFFINE", "tq_codebook", "cache_sizes",
           "score_hidden", "INDICATORS"]

INDICATORS = {"delta_norm": _abi.IND_DELTA_NORM, "norm": _abi.IND_NORM, "variance": _abi.IND_VARIANCE,
              "cosine_delta": _abi.IND_COSINE_DELTA}


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def make_config(n_layers, n_kv_heads, batch, base, L_hi, L_lo, group, r_num, r_den,
                max_prompt, max_new, head_dim=128, n_q_heads=None, block=64) -> _abi.Config:
    return _abi.Config(n_layers=n_layers, n_kv_heads=n_kv_heads,
                       n_q_heads=4 * n_kv_heads if n_q_heads is None else n_q_heads,
                       head_dim=head_dim, batch=batch, base=base, L_hi=L_hi, L_lo=L_lo, group=group,
                       r_num=r_num, r_den=r_den, block=block, max_prompt=max_prompt, max_new=max_new)


def cache_sizes(cfg: _abi.Config) -> _abi.Sizes:
    s = _abi.Sizes()
    check(lib().semkv_cache_sizes(ctypes.byref(cfg), ctypes.byref(s)), "semkv_cache_sizes")
    return s


def tq_codebook(L):
    mu = np.zeros(16, np.float32)
    tau = np.zeros(16, np.float32)
    check(lib().semkv_tq_codebook(L, mu.ctypes.data, tau.ctypes.data), "semkv_tq_codebook")
    return mu[:L].copy(), tau[:L - 1].copy()


def score_hidden(indicator, hidden, scores=None):
    """Sec. 3.3 hidden-state indicator on the device.  hidden: fp16 or bf16
    [m+1, B, T, d] (any strides with a unit channel stride), state k = layer
    L-m+k; indicator: a name of INDICATORS or its code.  Returns fp32 [B, T]."""
    import torch
    code = INDICATORS[indicator] if isinstance(indicator, str) else int(indicator)
    assert hidden.dim() == 4 and hidden.stride(3) == 1
    dt = {torch.float16: _abi.DTYPE_F16, torch.bfloat16: _abi.DTYPE_BF16}[hidden.dtype]
    n, B, T, d = hidden.shape
    if scores is None:
        scores = torch.empty((B, T), dtype=torch.float32, device=hidden.device)
    st = hidden.stride()
    check(lib().semkv_score_hidden(code, _ptr(hidden), dt, n - 1, B, T, d, st[0], st[1], st[2], _ptr(scores),
                                   _stream()), "semkv_score_hidden")
    return scores


class SemKVCache:
    """One mixed-precision KV cache on the current GPU (buffers are torch tensors)."""

    def __init__(self, cfg: _abi.Config, sign_words=None, device="cuda"):
        import torch
        self.cfg = cfg
        self.sz = cache_sizes(cfg)
        dev = torch.device(device)
        self.pools = torch.empty(self.sz.pool_bytes, dtype=torch.uint8, device=dev)
        self.tail = torch.empty(self.sz.tail_bytes // 2, dtype=torch.float16, device=dev)
        self.tail_scores = torch.zeros(self.sz.tail_score_bytes // 4, dtype=torch.float32, device=dev)
        self.flags = torch.zeros(self.sz.flag_bytes // 4, dtype=torch.int32, device=dev)
        self.status_word = torch.zeros(4, dtype=torch.int32, device=dev)
        self.signs = None
        if cfg.base != BASE_AFFINE:
            sw = np.ascontiguousarray(sign_words, dtype=np.uint32).reshape(cfg.n_layers, cfg.n_kv_heads, 4)
            self.signs = torch.from_numpy(sw.view(np.int32)).to(dev)
        self.c = _abi.Cache()
        check(lib().semkv_cache_init(ctypes.byref(self.c), ctypes.byref(cfg), _ptr(self.pools),
                                     _ptr(self.tail), _ptr(self.tail_scores), _ptr(self.flags),
                                     _ptr(self.signs) if self.signs is not None else None,
                                     _ptr(self.status_word)), "semkv_cache_init")
        self._ws = None

    # -- the hot path ------------------------------------------------------
    def rank_sizes(self, T):
        """(n_hi, n_lo): the slot-list lengths semkv_rank writes for T tokens."""
        n_hi, n_lo = ctypes.c_int64(), ctypes.c_int64()
        check(lib().semkv_rank_sizes(ctypes.byref(self.c), T, ctypes.byref(n_hi), ctypes.byref(n_lo)),
              "semkv_rank_sizes")
        return n_hi.value, n_lo.value

    def rank(self, scores, out=None):
        """scores: fp32 [B, T] on the device -> (hi_idx [B, K], lo_idx [B, T-K]) int32
        (written into out = (hi_idx, lo_idx) when given)."""
        import torch
        scores = scores.contiguous()
        B, T = scores.shape
        n_hi, n_lo = self.rank_sizes(T)
        if out is None:
            hi = torch.empty((B, n_hi), dtype=torch.int32, device=scores.device)
            lo = torch.empty((B, n_lo), dtype=torch.int32, device=scores.device)
        else:
            hi, lo = out
            assert hi.shape == (B, n_hi) and lo.shape == (B, n_lo) and hi.dtype == lo.dtype == torch.int32
            assert hi.is_contiguous() and lo.is_contiguous()
        check(lib().semkv_rank(ctypes.byref(self.c), _ptr(scores), T, _ptr(hi), _ptr(lo), _stream()),
              "semkv_rank")
        return hi, lo

    def quantize_pack(self, layer, K, V, hi_idx, lo_idx):
        """K, V: fp16 [B, H_kv, T, 128] (layer >= 0) or [n_layers, B, H_kv, T, 128] (layer = -1)."""
        assert K.dtype == V.dtype and K.dtype.itemsize == 2 and K.stride() == V.stride()
        st = K.stride()
        if layer < 0:
            sL, sB, sH, sT = st[0], st[1], st[2], st[3]
        else:
            sL, (sB, sH, sT) = 0, st[:3]
        T = K.shape[-2]
        check(lib().semkv_quantize_pack(ctypes.byref(self.c), layer, _ptr(K), _ptr(V), sL, sB, sH, sT, T,
                                        _ptr(hi_idx), _ptr(lo_idx), _stream()), "semkv_quantize_pack")

    def dequant(self, layer):
        """fp32 (K_hat, V_hat) [B, H_kv, n_hi + n_lo, 128] of `layer`: the high
        pool's slots, then the low pool's, as decode attention reads them."""
        import torch
        n = self.c.n_hi + self.c.n_lo
        shape = (self.cfg.batch, self.cfg.n_kv_heads, n, 128)
        k = torch.empty(shape, dtype=torch.float32, device=self.pools.device)
        v = torch.empty_like(k)
        if n == 0:
            return k, v
        check(lib().semkv_dequant(ctypes.byref(self.c), layer, _ptr(k), _ptr(v), _stream()), "semkv_dequant")
        return k, v

    def score_kv_norm(self, X, scores=None):
        """Key-norm (X = K) or value-norm (X = V) of every token: X fp16
        [n_layers, B, H_kv, T, 128] -> fp32 [B, T] (Sec. 3.3)."""
        import torch
        assert X.dtype == torch.float16 and X.dim() == 5 and X.stride(4) == 1
        T = X.shape[3]
        if scores is None:
            scores = torch.empty((self.cfg.batch, T), dtype=torch.float32, device=X.device)
        st = X.stride()
        check(lib().semkv_score_kv_norm(ctypes.byref(self.c), _ptr(X), st[0], st[1], st[2], st[3], T,
                                        _ptr(scores), _stream()), "semkv_score_kv_norm")
        return scores

    def append_kv(self, layer, k, v):
        check(lib().semkv_append_kv(ctypes.byref(self.c), layer, _ptr(k.contiguous()), _ptr(v.contiguous()),
                                    _stream()), "semkv_append_kv")

    def append_commit(self, score):
        check(lib().semkv_append_commit(ctypes.byref(self.c), _ptr(score.contiguous()), _stream()),
              "semkv_append_commit")

    def flush(self):
        check(lib().semkv_flush(ctypes.byref(self.c), _stream()), "semkv_flush")

    def reset(self):
        """Empty the cache for a new prompt (a multi-turn dialogue's next turn)."""
        check(lib().semkv_cache_reset(ctypes.byref(self.c), _stream()), "semkv_cache_reset")

    def workspace_bytes(self):
        n = ctypes.c_size_t()
        check(lib().semkv_workspace_bytes(ctypes.byref(self.c), ctypes.byref(n)), "semkv_workspace_bytes")
        return n.value

    def workspace(self):
        import torch
        need = max(self.workspace_bytes(), 16)
        if self._ws is None or self._ws.numel() * 4 < need:
            self._ws = torch.zeros((max(need, self.sz.workspace_bytes) + 3) // 4, dtype=torch.float32,
                                   device=self.pools.device)
        return self._ws

    def decode_attn(self, layer, q, out=None, workspace=None):
        """q: fp16 [B, H_q, 128] -> fp32 [B, H_q, 128]; layer = -1: every layer
        in one launch, q fp16 [n_layers, B, H_q, 128] -> fp32 of that shape."""
        import torch
        q = q.contiguous()
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        ws = self.workspace() if workspace is None else workspace
        check(lib().semkv_decode_attn(ctypes.byref(self.c), layer, _ptr(q), _ptr(out), _ptr(ws),
                                      ws.numel() * ws.element_size(), _stream()), "semkv_decode_attn")
        return out

    def decode_attn_noalloc(self, layer, q, out=None):
        """decode_attn with the library's own device scratch instead of a
        workspace (semkv_decode_attn_noalloc: the call allocates nothing)."""
        import torch
        q = q.contiguous()
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        check(lib().semkv_decode_attn_noalloc(ctypes.byref(self.c), layer, _ptr(q), _ptr(out), _stream()),
              "semkv_decode_attn_noalloc")
        return out

    def append_decode_attn(self, layer, k, v, q, out=None, workspace=None):
        """Fused append + decode of one layer: k, v fp16 [B, H_kv, 128] (this
        layer's new token), q fp16 [B, H_q, 128] -> fp32 [B, H_q, 128]."""
        import torch
        q = q.contiguous()
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        ws = self.workspace() if workspace is None else workspace
        check(lib().semkv_append_decode(ctypes.byref(self.c), layer, _ptr(k.contiguous()), _ptr(v.contiguous()),
                                        _ptr(q), _ptr(out), _ptr(ws), ws.numel() * ws.element_size(), _stream()),
              "semkv_append_decode")
        return out

    # -- state -------------------------------------------------------------
    @property
    def counts(self):
        return dict(n_prompt=self.c.n_prompt, n_hi=self.c.n_hi, n_lo=self.c.n_lo, n_scored=self.c.n_scored)

    def status(self) -> int:
        return int(self.status_word[0].item())

    def unit_offset(self, b, layer, kvh) -> int:
        return ((b * self.cfg.n_layers + layer) * self.cfg.n_kv_heads + kvh) * self.sz.unit_stride

    def pool_bytes(self, b, layer, kvh, pool, n_tiles=None):
        """Device bytes of the records of one pool of one unit (a torch view)."""
        off = self.unit_offset(b, layer, kvh)
        rb = self.sz.record_bytes_hi if pool == 0 else self.sz.record_bytes_lo
        if pool == 1:
            off += self.sz.cap_hi_tiles * self.sz.record_bytes_hi
        n = (self.sz.cap_hi_tiles if pool == 0 else self.sz.cap_lo_tiles) if n_tiles is None else n_tiles
        return self.pools[off:off + n * rb]
