"""Seeded generators.  Every array comes from ``numpy.random.default_rng`` keyed
by ``[seed, stream, ...coordinates]`` so that one (layer, sequence, kv head)
unit can be regenerated alone, without drawing the whole cache.

K/V rows are float32 N(0,1) draws cast to float16 (round-to-nearest-even);
keys get ``outliers`` distinct channels per (layer, kv head) scaled by
``outlier_scale`` before the cast.
"""
import numpy as np

from .configs import WorkloadConfig

# stream identifiers (part of the seed key)
S_K, S_V, S_OUTLIER, S_SCORE, S_Q, S_SIGN, S_GEN_K, S_GEN_V, S_GEN_SCORE, S_TURN_SCORE, S_TURN_GEN = range(1, 12)


def _rng(*key):
    return np.random.default_rng([int(k) for k in key])


def outlier_channels(cfg: WorkloadConfig, layer: int, kvh: int) -> np.ndarray:
    if cfg.outliers <= 0:
        return np.zeros(0, dtype=np.int64)
    return np.sort(_rng(cfg.seed, S_OUTLIER, layer, kvh).choice(cfg.head_dim, cfg.outliers, replace=False))


def _rows(cfg, stream, layer, b, kvh, n, outlier):
    x = _rng(cfg.seed, stream, layer, b, kvh).standard_normal((n, cfg.head_dim), dtype=np.float32)
    if outlier:
        ch = outlier_channels(cfg, layer, kvh)
        x[:, ch] *= np.float32(cfg.outlier_scale)
    return x.astype(np.float16)


def unit_kv(cfg: WorkloadConfig, layer: int, b: int, kvh: int, T: int | None = None):
    """Prompt K and V of one (layer, sequence, kv head) unit: two fp16 [T, D]."""
    T = cfg.prompt_len if T is None else T
    return (_rows(cfg, S_K, layer, b, kvh, T, True),
            _rows(cfg, S_V, layer, b, kvh, T, False))


def layer_kv(cfg: WorkloadConfig, layer: int, T: int | None = None):
    """Prompt K and V of one layer: two fp16 [B, H_kv, T, D]."""
    T = cfg.prompt_len if T is None else T
    K = np.empty((cfg.batch, cfg.n_kv_heads, T, cfg.head_dim), np.float16)
    V = np.empty_like(K)
    for b in range(cfg.batch):
        for h in range(cfg.n_kv_heads):
            K[b, h], V[b, h] = unit_kv(cfg, layer, b, h, T)
    return K, V


def scores(cfg: WorkloadConfig, b: int, T: int | None = None) -> np.ndarray:
    """Per-token importance scores of sequence b, float32 [T].

    zipf: integer Zipf(1.1) draws cast to float32 (heavy ties).
    dirichlet: Dirichlet(0.1) weights, a stand-in for accumulated attention.
    """
    T = cfg.prompt_len if T is None else T
    rng = _rng(cfg.seed, S_SCORE, b)
    if cfg.score_dist == "zipf":
        return rng.zipf(1.1, T).astype(np.float32)
    if cfg.score_dist == "dirichlet":
        return rng.dirichlet(np.full(T, 0.1)).astype(np.float32)
    raise ValueError(cfg.score_dist)


def all_scores(cfg: WorkloadConfig, T: int | None = None) -> np.ndarray:
    return np.stack([scores(cfg, b, T) for b in range(cfg.batch)])


def query(cfg: WorkloadConfig, layer: int, step: int) -> np.ndarray:
    """Decode query of one (layer, step): fp16 [B, H_q, D], N(0,1)."""
    x = _rng(cfg.seed, S_Q, layer, step).standard_normal(
        (cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=np.float32)
    return x.astype(np.float16)


def sign_words(cfg: WorkloadConfig, layer: int, kvh: int) -> np.ndarray:
    """Random-sign mask of one (layer, kv head) as 4 uint32 words; bit i set
    means sign -1 on channel i."""
    bits = _rng(cfg.seed, S_SIGN, layer, kvh).integers(0, 2, cfg.head_dim).astype(np.uint64)
    words = np.zeros(cfg.head_dim // 32, np.uint32)
    for i, v in enumerate(bits):
        if v:
            words[i // 32] |= np.uint32(1 << (i % 32))
    return words


def all_sign_words(cfg: WorkloadConfig) -> np.ndarray:
    """uint32 [n_layers, H_kv, D/32]."""
    return np.stack([np.stack([sign_words(cfg, l, h) for h in range(cfg.n_kv_heads)])
                     for l in range(cfg.n_layers)])


def unit_gen_kv(cfg: WorkloadConfig, layer: int, b: int, kvh: int, n: int | None = None):
    """Generated-token K and V of one unit: two fp16 [n_gen, D] (same outlier
    channels as the prompt keys)."""
    n = cfg.n_gen if n is None else n
    return (_rows(cfg, S_GEN_K, layer, b, kvh, n, True),
            _rows(cfg, S_GEN_V, layer, b, kvh, n, False))


def gen_scores(cfg: WorkloadConfig, n: int | None = None) -> np.ndarray:
    """Scores of generated tokens: float32 [n_gen, B]."""
    n = cfg.n_gen if n is None else n
    out = np.empty((n, cfg.batch), np.float32)
    for b in range(cfg.batch):
        rng = _rng(cfg.seed, S_GEN_SCORE, b)
        if cfg.score_dist == "zipf":
            out[:, b] = rng.zipf(1.1, n).astype(np.float32)
        else:
            out[:, b] = rng.random(n, dtype=np.float32)
    return out


# -------------------------------------------------------- multi-turn dialogue

def conversation_kv(cfg: WorkloadConfig, layer: int, b: int, kvh: int):
    """K and V rows of a whole dialogue (every turn's user tokens and answers,
    in order) of one unit: two fp16 [conversation_len, D]; a turn's prompt is
    a prefix, its answer the rows after it."""
    return unit_kv(cfg, layer, b, kvh, cfg.conversation_len)


def turn_scores(cfg: WorkloadConfig, turn: int, T: int) -> np.ndarray:
    """Scores of the accumulated prompt of a turn (re-scored every turn, as a
    fresh prefill would): float32 [B, T], integer Zipf(1.1) draws."""
    return np.stack([_rng(cfg.seed, S_TURN_SCORE, turn, b).zipf(1.1, T).astype(np.float32)
                     for b in range(cfg.batch)])


def turn_gen_scores(cfg: WorkloadConfig, turn: int, n: int) -> np.ndarray:
    """Scores of a turn's generated tokens: float32 [n, B]."""
    return np.stack([_rng(cfg.seed, S_TURN_GEN, turn, b).zipf(1.1, n).astype(np.float32)
                     for b in range(cfg.batch)], axis=1)
