"""ctypes declarations of the C ABI in include/semkv.h (argument marshalling only)."""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsemkv.so")

i32, i64, u32, f32, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_float, ctypes.c_size_t
vp = ctypes.c_void_p

SEMKV_OK, SEMKV_EINVAL, SEMKV_EUNSUPPORTED, SEMKV_ECAPACITY, SEMKV_ENAN, SEMKV_EHIP, SEMKV_ESTATE = \
    0, -1, -2, -3, -4, -5, -6
BASE_AFFINE, BASE_TQ, BASE_ROT_AFFINE = 0, 1, 2
STATUS_NAN_SCORE, STATUS_NONFINITE_KV = 1, 2
IND_DELTA_NORM, IND_NORM, IND_VARIANCE, IND_COSINE_DELTA = 0, 1, 2, 3
DTYPE_F16, DTYPE_BF16 = 0, 1


class Config(ctypes.Structure):
    _fields_ = [(n, i32) for n in ("n_layers", "n_kv_heads", "n_q_heads", "head_dim", "batch", "base",
                                   "L_hi", "L_lo", "group", "r_num", "r_den", "block")] + \
               [("max_prompt", i64), ("max_new", i64)]


class Sizes(ctypes.Structure):
    _fields_ = [(n, sz) for n in ("pool_bytes", "tail_bytes", "tail_score_bytes", "flag_bytes",
                                  "workspace_bytes")] + \
               [(n, i64) for n in ("flag_words", "cap_hi_tiles", "cap_lo_tiles", "unit_stride",
                                   "tile_bytes_hi", "tile_bytes_lo", "meta_bytes", "record_bytes_hi",
                                   "record_bytes_lo")]


class Cache(ctypes.Structure):
    _fields_ = [("cfg", Config), ("sz", Sizes),
                ("pools", vp), ("tail", vp), ("tail_scores", vp), ("flags", vp), ("signs", vp),
                ("status", vp),
                ("mu_hi", f32 * 16), ("tau_hi", f32 * 16), ("mu_lo", f32 * 16), ("tau_lo", f32 * 16),
                ("n_prompt", i64), ("n_hi", i64), ("n_lo", i64), ("n_scored", i32), ("appended", u32 * 4)]


EXPORTS = {
    "semkv_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "semkv_cache_sizes": (ctypes.c_int, [ctypes.POINTER(Config), ctypes.POINTER(Sizes)]),
    "semkv_tq_codebook": (ctypes.c_int, [ctypes.c_int, vp, vp]),
    "semkv_cache_init": (ctypes.c_int, [ctypes.POINTER(Cache), ctypes.POINTER(Config), vp, vp, vp, vp,
                                        vp, vp]),
    "semkv_rank_sizes": (ctypes.c_int, [ctypes.POINTER(Cache), i64, ctypes.POINTER(i64), ctypes.POINTER(i64)]),
    "semkv_rank": (ctypes.c_int, [ctypes.POINTER(Cache), vp, i64, vp, vp, vp]),
    "semkv_quantize_pack": (ctypes.c_int, [ctypes.POINTER(Cache), i32, vp, vp, i64, i64, i64, i64, i64,
                                           vp, vp, vp]),
    "semkv_append_kv": (ctypes.c_int, [ctypes.POINTER(Cache), i32, vp, vp, vp]),
    "semkv_append_commit": (ctypes.c_int, [ctypes.POINTER(Cache), vp, vp]),
    "semkv_flush": (ctypes.c_int, [ctypes.POINTER(Cache), vp]),
    "semkv_cache_reset": (ctypes.c_int, [ctypes.POINTER(Cache), vp]),
    "semkv_workspace_bytes": (ctypes.c_int, [ctypes.POINTER(Cache), ctypes.POINTER(sz)]),
    "semkv_decode_attn": (ctypes.c_int, [ctypes.POINTER(Cache), i32, vp, vp, vp, sz, vp]),
    "semkv_decode_attn_noalloc": (ctypes.c_int, [ctypes.POINTER(Cache), i32, vp, vp, vp]),
    "semkv_append_decode": (ctypes.c_int, [ctypes.POINTER(Cache), i32, vp, vp, vp, vp, vp, sz, vp]),
    "semkv_dequant": (ctypes.c_int, [ctypes.POINTER(Cache), i32, vp, vp, vp]),
    "semkv_score_hidden": (ctypes.c_int, [i32, vp, i32, i32, i32, i64, i32, i64, i64, i64, vp, vp]),
    "semkv_score_kv_norm": (ctypes.c_int, [ctypes.POINTER(Cache), vp, i64, i64, i64, i64, i64, vp, vp]),
}

_lib = None


def lib():
    """Load libsemkv.so.  There is no fallback: a missing library is an error."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libsemkv.so is not built; run paper_2608_28911_amd/build.py "
                               "(or __graft_entry__.build())")
        # torch ships its own copy of the HIP runtime (same soname): loaded
        # first, it is the one the library binds to.  Loaded the other way
        # round, the process maps two runtimes and the library's launches do
        # not see torch's streams and allocations.
        import torch  # noqa: F401
        _lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            f = getattr(_lib, name)
            f.restype, f.argtypes = res, args
    return _lib


class SemKVError(RuntimeError):
    def __init__(self, status, what=""):
        msg = lib().semkv_strerror(status).decode()
        super().__init__("%s: %s (%d)" % (what, msg, status))
        self.status = status


def check(status, what=""):
    if status != SEMKV_OK:
        raise SemKVError(status, what)
