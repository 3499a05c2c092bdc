"""The five synthetic workloads the hot path is tested and measured on.

Shapes follow the KV geometry the paper measures storage on (32 layers x 8 KV
heads x head_dim 128, shared by Llama-3.1-8B and Mistral-7B-v0.3; Sec. 4.5)
and its operating points (Sec. 4.1, Sec. 4.9).  Datasets and model weights are
absent, so every tensor is drawn from a seeded generator (``workloads.synth``).
"""
from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    seed: int
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    batch: int
    prompt_len: int          # T, tokens quantized at prefill (Alg. 1)
    n_gen: int               # generated tokens under deferred blocks (Alg. 2)
    decode_steps: int        # decode steps measured
    base: str                # "affine" | "tq" | "rot_affine"
    L_hi: int                # levels of the high precision (6 -> 2.585 b)
    L_lo: int                # levels of the low precision  (5 -> 2.322 b)
    group: int               # affine metadata group (channels); 128 for tq
    r_num: int               # high-precision fraction r = r_num / r_den
    r_den: int
    block: int = 64          # deferred block size B (Tab. 2)
    score_dist: str = "zipf" # "zipf" | "dirichlet"
    outliers: int = 4        # key channels scaled x10 per (layer, kv head)
    outlier_scale: float = 10.0
    turns: tuple = ()        # multi-turn dialogue: ((user tokens, generated tokens), ...)
    note: str = ""

    @property
    def gqa(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def turn_plan(self):
        """Per turn of a dialogue: (accumulated prompt length P_k, generated
        tokens g_k).  Turn k's prompt is the conversation so far plus the new
        user tokens; its answer follows it."""
        plan, n = [], 0
        for user, gen in self.turns:
            n += user
            plan.append((n, gen))
            n += gen
        return plan

    @property
    def conversation_len(self) -> int:
        return sum(u + g for u, g in self.turns)

    @property
    def base_id(self) -> int:
        """0 affine, 1 TurboQuant-MSE, 2 affine of the Hadamard-rotated row."""
        return BASES[self.base]

    @property
    def rotated(self) -> bool:
        """The base rotates rows by a random-sign Hadamard transform."""
        return self.base != "affine"


BASES = {"affine": 0, "tq": 1, "rot_affine": 2}


CONFIGS = [
    WorkloadConfig(
        name="single_layer_t2048_affine_g32", seed=0, n_layers=1, n_kv_heads=8,
        n_q_heads=32, head_dim=128, batch=1, prompt_len=2048, n_gen=0,
        decode_steps=1, base="affine", L_hi=6, L_lo=5, group=32, r_num=26,
        r_den=100, note="correctness case: 1 layer, one quantize+pack, one decode"),
    WorkloadConfig(
        name="llama8b_kv_b1_t32768_affine", seed=1, n_layers=32, n_kv_heads=8,
        n_q_heads=32, head_dim=128, batch=1, prompt_len=32768, n_gen=0,
        decode_steps=128, base="affine", L_hi=6, L_lo=5, group=128, r_num=26,
        r_den=100, note="headline: 128 decode steps over 32 layers"),
    WorkloadConfig(
        name="llama8b_kv_b16_t16384_affine_dirichlet", seed=2, n_layers=32,
        n_kv_heads=8, n_q_heads=32, head_dim=128, batch=16, prompt_len=16384,
        n_gen=0, decode_steps=64, base="affine", L_hi=6, L_lo=5, group=128,
        r_num=26, r_den=100, score_dist="dirichlet",
        note="batched serving; accumulated-attention-like Dirichlet(0.1) scores"),
    WorkloadConfig(
        name="mistral7b_kv_b4_t32768_gen2048_deferred", seed=3, n_layers=32,
        n_kv_heads=8, n_q_heads=32, head_dim=128, batch=4, prompt_len=32768,
        n_gen=2048, decode_steps=2048, base="affine", L_hi=6, L_lo=5, group=128,
        r_num=26, r_den=100, note="block-exact deferred quantization of 2048 generated tokens"),
    WorkloadConfig(
        name="llama8b_kv_b1_t131072_tq", seed=4, n_layers=32, n_kv_heads=8,
        n_q_heads=32, head_dim=128, batch=1, prompt_len=131072, n_gen=0,
        decode_steps=64, base="tq", L_hi=4, L_lo=3, group=128, r_num=40,
        r_den=100, note="TurboQuant-MSE base, 4/3 Lloyd-Max levels"),
    WorkloadConfig(
        name="llama8b_kv_b4_multiturn4_r35", seed=5, n_layers=32, n_kv_heads=8,
        n_q_heads=32, head_dim=128, batch=4, prompt_len=4352, n_gen=256,
        decode_steps=1024, base="affine", L_hi=6, L_lo=5, group=128, r_num=35,
        r_den=100, turns=((2048, 256), (512, 256), (512, 256), (512, 256)),
        note="multi-turn operating point (2.41 code bits): each turn re-ranks and quantizes the "
             "accumulated conversation, generates block-exactly and flushes its residual block"),
]


def get_config(i_or_name, **overrides) -> WorkloadConfig:
    """Return a workload by index or name, optionally with fields replaced
    (tests shrink layers / tokens this way)."""
    if isinstance(i_or_name, int):
        cfg = CONFIGS[i_or_name]
    else:
        cfg = next(c for c in CONFIGS if c.name == i_or_name)
    return replace(cfg, **overrides) if overrides else cfg
