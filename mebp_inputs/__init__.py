"""Seeded synthetic inputs for the checkpointed LoRA training step.

This module is shared by the CPU oracle (``oracle/``) and by the HIP path's tests and
benchmark. It holds model shapes, a seeded generator and the offline int4 compression
that turns drawn fp32 weights into the compressed input format the step consumes
(the paper's first step, "Base model weights compression", Sec. 3: 4-bit symmetric
INT4 of every non-LoRA parameter including the embeddings). It computes nothing of the
training step itself: no dequantisation, no layer, no loss, no gradient.

Recipe (identical for every consumer):
  * ``numpy.random.default_rng(seed)``; draw order: for each layer the seven base
    projections q, k, v, o, gate, up, down as fp32 ``[out][in]`` ~ N(0, 0.02) (std),
    then the tied embedding ``[V][d]`` ~ N(0, 0.02), then for each layer and each
    adapted module LoRA ``A`` ``[r][in]`` ~ N(0, 1/r) and ``B`` ``[out][r]`` ~ N(0, 0.02),
    then the step input: ``x`` ``[B*T][d]`` ~ N(0, 1) and ``dy`` ~ N(0, 1) for the
    single-block case, or token ids uniform in ``[0, V)`` as int32 ``[B][T]``.
  * Int4 compression: groups of ``group`` consecutive input columns (the last group of a
    row may be shorter); fp16 scale ``s = fp16_RNE(max|w| / 7)`` (max over the fp32
    group, division in fp64); code ``q = clamp(rint_half_even(w / s), -7, 7)`` (0 where
    ``s == 0``); two's-complement nibbles, element ``2j`` of a row in the low nibble of
    byte ``j``.
  * RMSNorm weights are fp32 ones (``norm="ones"``) or ``1 + 0.1*N(0,1)`` drawn from a
    second generator seeded ``seed + 1`` (``norm="random"``, used by tests so that a
    dropped norm weight cannot pass), so the main draw order never changes.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional, Tuple

import numpy as np

PROJ = ("q", "k", "v", "o", "gate", "up", "down")
PROJ_INDEX = {p: i for i, p in enumerate(PROJ)}


@dataclass(frozen=True)
class Config:
    """Shape of a decoder-only transformer and of one training batch."""

    name: str
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int  # 0: no embedding / LM head (single-block case)
    act: str = "silu"  # "silu" (SwiGLU) or "gelu_tanh" (GeGLU)
    rms_eps: float = 1e-6
    rope_theta_global: float = 1e6
    rope_theta_local: float = 1e4
    window: int = 0  # sliding window of local layers, 0 = none
    global_every: int = 0  # 0: every layer global; k: layer l global iff (l+1) % k == 0
    group: int = 32
    lora_rank: int = 8
    lora_alpha: float = 16.0
    lora_modules: Tuple[str, ...] = ("q", "v")
    batch: int = 1
    seq: int = 128
    # architecture details beyond the shapes (all off: the "-shaped" models)
    qkv_bias: bool = False  # Qwen2.5: biases on the q, k, v projections
    qk_norm: bool = False  # Gemma3: RMSNorm over each head of q and k before RoPE
    sandwich_norm: bool = False  # Gemma3: RMSNorm on the attention and MLP outputs before the residual
    embed_scale: bool = False  # Gemma3: embedding output times sqrt(hidden)

    @property
    def arch_flags(self) -> int:
        return (1 if self.qkv_bias else 0) | (2 if self.qk_norm else 0) | (4 if self.sandwich_norm else 0) | \
            (8 if self.embed_scale else 0)

    @property
    def n_tokens(self) -> int:
        return self.batch * self.seq

    @property
    def lora_scale(self) -> float:
        return self.lora_alpha / self.lora_rank

    def proj_shape(self, p: str) -> Tuple[int, int]:
        """(out, in) of base projection ``p``."""
        d, qd, kvd, f = self.hidden, self.n_heads * self.head_dim, self.n_kv_heads * self.head_dim, self.ffn
        return {
            "q": (qd, d), "k": (kvd, d), "v": (kvd, d), "o": (d, qd),
            "gate": (f, d), "up": (f, d), "down": (d, f),
        }[p]

    def is_global(self, layer: int) -> bool:
        return self.global_every == 0 or (layer + 1) % self.global_every == 0

    def layer_window(self, layer: int) -> int:
        return 0 if self.is_global(layer) else self.window

    def layer_theta(self, layer: int) -> float:
        return self.rope_theta_global if self.is_global(layer) else self.rope_theta_local

    def lora_mask(self) -> int:
        m = 0
        for p in self.lora_modules:
            m |= 1 << PROJ_INDEX[p]
        return m

    def lora_param_count(self) -> int:
        tot = 0
        for p in self.lora_modules:
            o, i = self.proj_shape(p)
            tot += self.lora_rank * (o + i)
        return tot * self.n_layers

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


ALL7 = PROJ
QKVO = ("q", "k", "v", "o")

# The five workloads: a single Llama-style block and four model-shaped full steps.
CONFIGS: Dict[str, Config] = {
    "block": Config(
        name="block", n_layers=1, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=688,
        vocab=0, act="silu", rope_theta_global=1e4, rope_theta_local=1e4, lora_rank=8,
        lora_alpha=16.0, lora_modules=("q", "v"), batch=1, seq=128),
    "qwen2.5-0.5b": Config(
        name="qwen2.5-0.5b", n_layers=24, hidden=896, n_heads=14, n_kv_heads=2, head_dim=64,
        ffn=4864, vocab=151936, act="silu", rope_theta_global=1e6, rope_theta_local=1e6,
        lora_rank=8, lora_alpha=16.0, lora_modules=QKVO, batch=1, seq=256),
    "gemma3-1b": Config(
        name="gemma3-1b", n_layers=26, hidden=1152, n_heads=4, n_kv_heads=1, head_dim=256,
        ffn=6912, vocab=262144, act="gelu_tanh", rope_theta_global=1e6, rope_theta_local=1e4,
        window=512, global_every=6, lora_rank=16, lora_alpha=32.0, lora_modules=QKVO,
        batch=1, seq=512),
    "qwen2.5-1.5b": Config(
        name="qwen2.5-1.5b", n_layers=28, hidden=1536, n_heads=12, n_kv_heads=2, head_dim=128,
        ffn=8960, vocab=151936, act="silu", rope_theta_global=1e6, rope_theta_local=1e6,
        lora_rank=16, lora_alpha=32.0, lora_modules=ALL7, batch=4, seq=1024),
    "gemma3-4b": Config(
        name="gemma3-4b", n_layers=34, hidden=2560, n_heads=8, n_kv_heads=4, head_dim=256,
        ffn=10240, vocab=262144, act="gelu_tanh", rope_theta_global=1e6, rope_theta_local=1e4,
        window=1024, global_every=6, lora_rank=16, lora_alpha=32.0, lora_modules=ALL7,
        batch=8, seq=2048),
}
CONFIG_ORDER = ["block", "qwen2.5-0.5b", "gemma3-1b", "qwen2.5-1.5b", "gemma3-4b"]


# ----------------------------------------------------------------------------------------
# Offline int4 compression (produces the compressed input format; not part of the step)
# ----------------------------------------------------------------------------------------
def _quantize_rows(w: np.ndarray, group: int) -> Tuple[np.ndarray, np.ndarray]:
    out, inn = w.shape
    ng = -(-inn // group)
    pad = ng * group - inn
    wp = (np.pad(w, ((0, 0), (0, pad))) if pad else w).reshape(out, ng, group)
    amax = np.abs(wp).max(axis=-1).astype(np.float64)
    s16 = (amax / 7.0).astype(np.float16)
    s = s16.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(s[..., None] > 0, np.rint(wp.astype(np.float64) / s[..., None]), 0.0)
    q = np.clip(q, -7, 7).astype(np.int8).reshape(out, ng * group)[:, :inn]
    u = (q.astype(np.int16) & 0xF).astype(np.uint8)
    q4 = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    return q4, s16.view(np.uint16)


_POOL = None


def quantize_q4(w: np.ndarray, group: int = 32) -> Tuple[np.ndarray, np.ndarray]:
    """Symmetric int4 group quantisation of ``w`` fp32 ``[out][in]``.

    Returns ``(q4, scale_bits)``: packed codes uint8 ``[out][in/2]`` and raw fp16 scale
    bits uint16 ``[out][ceil(in/group)]``. Rows are independent; large matrices are
    processed in row blocks on a thread pool (same result as one block).
    """
    global _POOL
    w = np.asarray(w, dtype=np.float32)
    out, inn = w.shape
    if inn % 2:
        raise ValueError("input dimension must be even to pack two codes per byte")
    rows = max(1, (1 << 18) // max(inn, 1))
    if out <= rows:
        q4, sb = _quantize_rows(w, group)
        return np.ascontiguousarray(q4), np.ascontiguousarray(sb)
    if _POOL is None:
        import os
        from concurrent.futures import ThreadPoolExecutor
        _POOL = ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1)))
    q4 = np.empty((out, inn // 2), np.uint8)
    sb = np.empty((out, -(-inn // group)), np.uint16)

    def job(r0):
        a, b = _quantize_rows(w[r0:r0 + rows], group)
        q4[r0:r0 + rows] = a
        sb[r0:r0 + rows] = b

    list(_POOL.map(job, range(0, out, rows)))
    return q4, sb


# ----------------------------------------------------------------------------------------
# Seeded generator
# ----------------------------------------------------------------------------------------
@dataclass
class Inputs:
    cfg: Config
    base: List[Dict[str, Tuple[np.ndarray, np.ndarray]]]  # per layer: proj -> (q4, scale_bits)
    norm_attn: List[np.ndarray]
    norm_mlp: List[np.ndarray]
    norm_final: Optional[np.ndarray]
    emb: Optional[Tuple[np.ndarray, np.ndarray]]  # (q4 [V][d/2], scale bits [V][d/32])
    lora: List[Dict[str, Tuple[np.ndarray, np.ndarray]]]  # per layer: proj -> (A [r][in], B [out][r])
    x: Optional[np.ndarray] = None  # single-block input [N][d] fp32
    dy: Optional[np.ndarray] = None  # single-block upstream gradient [N][d] fp32
    ids: Optional[np.ndarray] = None  # token ids int32 [B][T]
    extra: dict = field(default_factory=dict)


def _normal(rng, shape, std) -> np.ndarray:
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)


def make_inputs(cfg: Config, seed: int = 0, norm: str = "ones", lora_b_zero: bool = False,
                n_layers: Optional[int] = None) -> Inputs:
    """Draw every input of one training step of ``cfg`` from ``seed``.

    ``n_layers`` (optional) draws only the first layers (the draw order of those layers is
    unchanged; embedding and LoRA are drawn after them, so a truncated model is a
    different, smaller input set). ``lora_b_zero`` sets every LoRA ``B`` to zero after the
    draw (the adapter-is-identity case).
    """
    L = cfg.n_layers if n_layers is None else n_layers
    rng = np.random.default_rng(seed)
    base = []
    for _ in range(L):
        layer = {}
        for p in PROJ:
            o, i = cfg.proj_shape(p)
            layer[p] = quantize_q4(_normal(rng, (o, i), 0.02), cfg.group)
        base.append(layer)
    emb = None
    if cfg.vocab:
        emb = quantize_q4(_normal(rng, (cfg.vocab, cfg.hidden), 0.02), cfg.group)
    lora = []
    r = cfg.lora_rank
    for _ in range(L):
        mods = {}
        for p in PROJ:
            if p not in cfg.lora_modules:
                continue
            o, i = cfg.proj_shape(p)
            A = _normal(rng, (r, i), 1.0 / r)
            B = _normal(rng, (o, r), 0.02)
            if lora_b_zero:
                B[:] = 0
            mods[p] = (A, B)
        lora.append(mods)
    inp = Inputs(cfg=cfg, base=base, norm_attn=[], norm_mlp=[], norm_final=None, emb=emb, lora=lora)
    N, d = cfg.n_tokens, cfg.hidden
    if cfg.vocab:
        inp.ids = rng.integers(0, cfg.vocab, size=(cfg.batch, cfg.seq)).astype(np.int32)
    else:
        inp.x = rng.standard_normal((N, d), dtype=np.float32)
        inp.dy = rng.standard_normal((N, d), dtype=np.float32)
    nrng = np.random.default_rng(seed + 1)

    def nw():
        if norm == "ones":
            return np.ones(d, np.float32)
        if norm == "random":
            return (1.0 + 0.1 * nrng.standard_normal(d)).astype(np.float32)
        raise ValueError(norm)

    inp.norm_attn = [nw() for _ in range(L)]
    inp.norm_mlp = [nw() for _ in range(L)]
    inp.norm_final = nw() if cfg.vocab else None
    # architecture extras, from their own stream (the draws above are unchanged): frozen
    # fp32 vectors, like the norm weights
    arng = np.random.default_rng(seed + 2)
    qd, kvd, dh = cfg.n_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim, cfg.head_dim
    inp.extra["bias"] = [{"q": _normal(arng, (qd,), 0.1), "k": _normal(arng, (kvd,), 0.1),
                          "v": _normal(arng, (kvd,), 0.1)} if cfg.qkv_bias else None for _ in range(L)]

    def vw(n):
        return (1.0 + 0.1 * arng.standard_normal(n)).astype(np.float32) if norm == "random" else np.ones(n, np.float32)
    inp.extra["qk_norm"] = [(vw(dh), vw(dh)) if cfg.qk_norm else None for _ in range(L)]
    inp.extra["post_norm"] = [(vw(d), vw(d)) if cfg.sandwich_norm else None for _ in range(L)]
    return inp


def layer_input(cfg: Config, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """A stand-alone (x, dy) pair ``[N][d]`` fp32 ~ N(0,1) for per-layer tests."""
    rng = np.random.default_rng(seed)
    N, d = cfg.n_tokens, cfg.hidden
    return (rng.standard_normal((N, d), dtype=np.float32),
            rng.standard_normal((N, d), dtype=np.float32))


# Tiny shapes for finite-difference and brute-force checks on the CPU.
TINY = Config(name="tiny", n_layers=2, hidden=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn=96,
              vocab=97, act="silu", rope_theta_global=1e4, rope_theta_local=1e4, window=3,
              global_every=2, lora_rank=2, lora_alpha=4.0, lora_modules=ALL7, batch=2, seq=7)

# Small GPU-compatible shape (head_dim 64, ragged tiles everywhere: T = 160, ffn = 352,
# vocab = 1056, a sliding-window layer and a global layer, all seven projections adapted).
MINI = Config(name="mini", n_layers=2, hidden=128, n_heads=4, n_kv_heads=2, head_dim=64, ffn=352,
              vocab=1056, act="gelu_tanh", rope_theta_global=1e6, rope_theta_local=1e4, window=96,
              global_every=2, lora_rank=16, lora_alpha=32.0, lora_modules=ALL7, batch=2, seq=160)


def make_optimizer_inputs(cfg: Config, seed: int = 0, n_layers: Optional[int] = None):
    """Seeded LoRA-shaped tensors for the optimizer step, per layer and adapted projection:
    gradients ``(gA, gB)``, first moments ``(mA, mB)`` and second moments ``(vA, vB)``
    (non-negative), all fp32. The parameters themselves are the LoRA ``A``, ``B`` of
    ``make_inputs``."""
    L = cfg.n_layers if n_layers is None else n_layers
    rng = np.random.default_rng(seed)
    r = cfg.lora_rank
    out = []
    for _ in range(L):
        mods = {}
        for p in PROJ:
            if p not in cfg.lora_modules:
                continue
            o, i = cfg.proj_shape(p)
            g = (_normal(rng, (r, i), 1e-2), _normal(rng, (o, r), 1e-2))
            m = (_normal(rng, (r, i), 1e-3), _normal(rng, (o, r), 1e-3))
            v = (np.abs(_normal(rng, (r, i), 1e-4)), np.abs(_normal(rng, (o, r), 1e-4)))
            mods[p] = {"g": g, "m": m, "v": v}
        out.append(mods)
    return out
