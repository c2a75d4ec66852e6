"""Seeded synthetic inputs for the MBP decode path: model shapes, weights and prompts.

This package holds no arithmetic of the method itself. It only draws the random
numbers that both the CPU oracle and the HIP library consume, so that the two sides
see bit-identical inputs:

* ``ModelConfig`` / ``WORKLOADS`` -- the architectures and run shapes.  The layer
  split (encoder 2, LM module 16, NT decoder 2, MB head 2 LCA layers or 3 MLP heads)
  is the paper's architecture table (appendix A, hyperparameter table); d_model,
  d_inner = 4 d, RMSNorm eps 1e-6, RoPE base 1e5 and attention scaling 1.0 are from
  the model-architecture paragraph of the experimental setup.
* ``manifest`` -- the fixed name / shape / order list of parameter tensors.
* ``make_weights`` -- N(0, 0.02^2) i.i.d. tensors from NumPy ``PCG64`` streams,
  rounded to bfloat16 (round to nearest even) for bf16 models.
* ``make_prompt`` / ``make_bytes`` -- byte strings in which each byte is a space
  (0x20) with probability 1/6 and otherwise a Zipf(1.1)-ranked non-space byte.
  They stand in for the paper's evaluation text (CNN/DailyMail, Opus-100), which is
  not available; space-delimited patches then have a geometric length, mean 6.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "ModelConfig",
    "Workload",
    "WORKLOADS",
    "SMALL_F32",
    "TINY_FXT",
    "D1024_FXT",
    "manifest",
    "head_manifest_start",
    "make_weights",
    "make_prompt",
    "make_bytes",
    "round_bf16",
]


@dataclass(frozen=True)
class ModelConfig:
    d_model: int
    n_heads: int
    n_enc: int
    n_lm: int
    n_nb: int
    n_mb: int            # LCA: MB transformer layers; MLP: number of MLP heads
    head: str = "lca"    # "lca" | "mlp"
    dtype: str = "bf16"  # "f32" | "bf16"  (storage of weights and KV caches)
    d_ff: int = 0        # 0 -> 4 * d_model
    rope_base: float = 1e5
    rms_eps: float = 1e-6
    attn_scale: float = 1.0
    max_patch: int = 16  # length cap of a segment; 0 = pure space rule
    window_mode: int = 0  # 0: MB layers see only the previous+current group window
    boundary: str = "space"  # "space": 0x20 rule; "learned": boundary predictor on h_e
    # bias of the synthetic boundary probe (learned boundaries); with bp.w ~ N(0, 1/d)
    # the probe w . h / RMS(h) is N(0, 1) over random directions, so -0.43 ends about
    # one segment in three bytes when the encoder states vary freely (the tiny models)
    bp_bias: float = -0.43
    bp_scale: float = 1.0  # bp.w ~ N(0, bp_scale^2 / d)

    def __post_init__(self):
        if self.d_ff == 0:
            object.__setattr__(self, "d_ff", 4 * self.d_model)
        assert self.head in ("lca", "mlp")
        assert self.dtype in ("f32", "bf16")
        assert self.boundary in ("space", "learned")
        assert self.d_model % self.n_heads == 0

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    prompt_len: int
    gen_len: int
    n: int
    tau: float
    mode: str = "threshold"  # "threshold" | "verify" | "external" | "forward" (full-sequence)
    verifier: "ModelConfig" = None  # mode "external": the next-byte model checking the drafts
    temperature: float = 0.0  # > 0: sampled decoding at this temperature (0: greedy)
    top_p: float = 1.0        # nucleus of sampled decoding
    sweep_n: tuple = ()
    sweep_tau: tuple = ()
    note: str = ""


_TINY = ModelConfig(d_model=128, n_heads=4, n_enc=1, n_lm=2, n_nb=1, n_mb=1, head="lca", dtype="f32")
_D1024_LCA = ModelConfig(d_model=1024, n_heads=16, n_enc=2, n_lm=16, n_nb=2, n_mb=2, head="lca", dtype="bf16")
_D1024_MLP = _D1024_LCA.replace(head="mlp", n_mb=3)
_D2048 = ModelConfig(d_model=2048, n_heads=32, n_enc=2, n_lm=16, n_nb=2, n_mb=2, head="lca", dtype="bf16")
# float32 model at the smallest width the persistent engine's register tiles take
# (d_model 256, head size 64): parity of that path at the float32 tolerance
SMALL_F32 = ModelConfig(d_model=256, n_heads=4, n_enc=2, n_lm=2, n_nb=2, n_mb=2, head="lca", dtype="f32")
# next-byte models without an MB head (the FxT baseline the paper verifies MBP drafts
# with: encoder, LM module, next-byte decoder) -- a tiny float32 one and the
# parameter-matched d=1024 one with the 2/16/4 layer split
TINY_FXT = ModelConfig(d_model=128, n_heads=4, n_enc=1, n_lm=2, n_nb=2, n_mb=0, head="lca", dtype="f32")
D1024_FXT = ModelConfig(d_model=1024, n_heads=16, n_enc=2, n_lm=16, n_nb=4, n_mb=0, head="lca", dtype="bf16")

WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", _TINY, batch=1, prompt_len=256, gen_len=128, n=3, tau=0.75),
    "lca_d1024_b1": Workload("lca_d1024_b1", _D1024_LCA, batch=1, prompt_len=4096, gen_len=1024, n=3,
                             tau=0.75, sweep_n=(3, 4, 5, 6, 7)),
    "mlp_d1024_b1": Workload("mlp_d1024_b1", _D1024_MLP, batch=1, prompt_len=4096, gen_len=1024, n=3, tau=0.75),
    "lca_d1024_b64": Workload("lca_d1024_b64", _D1024_LCA, batch=64, prompt_len=2048, gen_len=512, n=5,
                              tau=0.75, sweep_tau=(0.5, 0.75, 0.9)),
    "verify_d2048_b16": Workload("verify_d2048_b16", _D2048, batch=16, prompt_len=8192, gen_len=512, n=7,
                                 tau=0.75, mode="verify"),
    # sampled decoding at the paper's settings for its instruction-following task
    "sampled_d1024_b1": Workload("sampled_d1024_b1", _D1024_LCA, batch=1, prompt_len=4096, gen_len=1024, n=3,
                                 tau=0.75, temperature=0.7, top_p=0.9),
    # the MBP d=1024 model drafts n = 7 candidates, the FxT d=1024 model verifies them
    "extverify_d1024_b1": Workload("extverify_d1024_b1", _D1024_LCA, batch=1, prompt_len=4096, gen_len=1024, n=7,
                                   tau=0.75, mode="external", verifier=D1024_FXT),
    # the training-form forward over one whole 4096-byte sequence (both heads at every
    # position, the MB layers under the full LCA mask, the losses)
    "forward_d1024_t4096": Workload("forward_d1024_t4096", _D1024_LCA, batch=1, prompt_len=4096, gen_len=0, n=0,
                                    tau=0.0, mode="forward"),
    # segments from the learned boundary predictor instead of the space rule; the probe
    # is scaled to confident logits (std about 1 on this model's encoder states) and
    # biased so that about one byte in three ends a segment where decoding runs (the
    # last 1024 prompt bytes: the states drift with position, and about 45% of the
    # whole prompt's bytes end one), the paper's 3x compression
    "learned_d1024_b1": Workload("learned_d1024_b1",
                                 _D1024_LCA.replace(boundary="learned", bp_scale=4.0, bp_bias=0.84), batch=1,
                                 prompt_len=4096, gen_len=1024, n=3, tau=0.75),
}

_BLOCK_PARTS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def _block_shapes(prefix: str, d: int, dff: int):
    shp = {
        "attn_norm": (d,), "wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
        "ffn_norm": (d,), "w_gate": (dff, d), "w_up": (dff, d), "w_down": (d, dff),
    }
    return [(f"{prefix}.{p}", shp[p]) for p in _BLOCK_PARTS]


def manifest(cfg: ModelConfig):
    """Ordered (name, shape) list of every parameter tensor.

    Matrices are stored [out_features, in_features] (y = W x).  The trunk tensors
    come first; the head-specific tensors (LCA MB blocks + MB final norm, or the MLP
    heads) follow, starting at ``head_manifest_start(cfg)``.
    """
    d, dff = cfg.d_model, cfg.d_ff
    out = [("emb", (256, d)), ("bos", (d,))]
    for i in range(cfg.n_enc):
        out += _block_shapes(f"enc.{i}", d, dff)
    for i in range(cfg.n_lm):
        out += _block_shapes(f"lm.{i}", d, dff)
    for i in range(cfg.n_nb):
        out += _block_shapes(f"nt.{i}", d, dff)
    out += [("nt_norm", (d,)), ("unembed", (256, d))]
    if cfg.head == "lca":
        for i in range(cfg.n_mb):
            out += _block_shapes(f"mb.{i}", d, dff)
        out += [("mb_norm", (d,))]
    else:
        for i in range(cfg.n_mb):
            out += [(f"mlp.{i}.norm", (d,)), (f"mlp.{i}.w_gate", (dff, d)),
                    (f"mlp.{i}.w_up", (dff, d)), (f"mlp.{i}.w_down", (d, dff))]
    if cfg.boundary == "learned":
        out += [("bp.w", (d,)), ("bp.b", (1,))]  # boundary predictor: logit = w . h_e / RMS(h_e) + b
    return out


def head_manifest_start(cfg: ModelConfig) -> int:
    return 4 + 9 * (cfg.n_enc + cfg.n_lm + cfg.n_nb)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # finite inputs: u + 0x8000 stays below 2**32, so uint32 arithmetic is exact
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32).reshape(a.shape)


def _is_gain(name: str) -> bool:
    return name.endswith("norm")


def make_weights(cfg: ModelConfig, seed: int = 0, gain_jitter: float = 0.0, logit_gain: float = 1.0,
                 std: float = 0.02) -> dict:
    """Draw every parameter tensor, in manifest order.

    * matrices, the embedding, ``bos`` and ``unembed``: N(0, std^2), trunk tensors from
      ``PCG64(seed)``, head tensors from ``PCG64(seed + 1)`` (so two models that differ
      only in the head share identical trunk weights);
    * norm gains: 1, or 1 + U(-gain_jitter, gain_jitter) from ``PCG64(seed + 2)``;
    * ``logit_gain`` multiplies the two final head norms (``nt_norm``, ``mb_norm``),
      which scales every logit and so raises the top-1 probabilities of a random model;
    * boundary predictor (learned boundaries): ``bp.w`` ~ N(0, cfg.bp_scale^2 / d) from
      the head stream and ``bp.b`` = ``cfg.bp_bias``.
    bf16 models get every tensor rounded to bfloat16.
    """
    rng_trunk = np.random.Generator(np.random.PCG64(seed))
    rng_head = np.random.Generator(np.random.PCG64(seed + 1))
    rng_gain = np.random.Generator(np.random.PCG64(seed + 2))
    start = head_manifest_start(cfg)
    out = {}
    for idx, (name, shape) in enumerate(manifest(cfg)):
        rng = rng_trunk if idx < start else rng_head
        if _is_gain(name):
            if gain_jitter > 0:
                a = 1.0 + rng_gain.uniform(-gain_jitter, gain_jitter, size=shape)
            else:
                a = np.ones(shape)
            if name in ("nt_norm", "mb_norm"):
                a = a * logit_gain
            a = a.astype(np.float32)
        elif name == "bp.w":
            a = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(cfg.bp_scale / np.sqrt(cfg.d_model))
        elif name == "bp.b":
            a = np.full(shape, cfg.bp_bias, dtype=np.float32)
        else:
            a = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)
        if cfg.dtype == "bf16":
            a = round_bf16(a)
        out[name] = np.ascontiguousarray(a, dtype=np.float32)
    return out


_ZIPF_S = 1.1
_PERM_SEED = 77


def _zipf_table():
    ranks = np.arange(1, 256, dtype=np.float64)
    p = ranks ** (-_ZIPF_S)
    p /= p.sum()
    non_space = np.array([b for b in range(256) if b != 0x20], dtype=np.uint8)
    perm = np.random.Generator(np.random.PCG64(_PERM_SEED)).permutation(non_space)
    return p, perm


def make_bytes(seed: int, length: int, space_prob: float = 1.0 / 6.0) -> np.ndarray:
    """``length`` bytes: 0x20 with probability ``space_prob``, else Zipf(1.1) over the
    255 non-space byte values (rank order fixed by a seeded permutation)."""
    p, perm = _zipf_table()
    rng = np.random.Generator(np.random.PCG64(seed))
    is_space = rng.random(length) < space_prob
    ranks = rng.choice(255, size=length, p=p)
    out = perm[ranks]
    out[is_space] = 0x20
    return out.astype(np.uint8)


def make_prompt(row: int, length: int) -> np.ndarray:
    """Prompt of batch row ``row``: seed 1000 + row."""
    return make_bytes(1000 + row, length)
