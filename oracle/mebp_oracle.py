"""CPU fp64 oracle of the MeBP checkpointed LoRA training step.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or execute this
module: it exists so that tests, the smoke check and the benchmark's CPU-baseline leg
can compare the HIP path against a plain, slow, obviously correct computation.

What it computes. MeBP (Sec. 3, Algorithm 1) is gradient checkpointing at every block
boundary: a forward loop stores the boundary activations, then a reverse loop recomputes
each block's forward from its stored input and backpropagates through it. Checkpointing
only reorders work, so the result is exactly ordinary LoRA backpropagation through the
dequantised model (Sec. 5 calls it exact gradient computation). This file therefore
writes that definition out directly in float64 numpy:

  * decompression of the int4 base weights (Sec. 3, "Base model weights compression";
    Algorithm 1, LazyLoadAndDecompressWeights), done lazily per block as in Algorithm 1;
  * each transformer block ``y = F_i(x, w)`` (RMSNorm, q/k/v with LoRA, RoPE, causal GQA
    attention with optional sliding window, o with LoRA and residual, RMSNorm, gated MLP
    with LoRA and residual);
  * its backward graph ``(dE/dx, dE/dw) = B_i(x, dE/dy, w)`` (Sec. 3, display equation:
    the gradient of the scalar ``s = sum(dE/dy * y)``), with hand-derived formulas;
  * the final block: final RMSNorm, tied int4 LM head and next-token cross-entropy
    (blocks are every transformer layer plus the final linear and loss layers, Sec. 4.2);
  * Algorithm 1 itself: forward loop storing checkpoints, reverse loop recomputing.

Numerics: float64 throughout; no blocking, fusion or reordering beyond the definitions.
Readings where the paper is silent (quantiser, packing, RoPE pairing, window mask, loss
normalisation, LoRA form) follow the same conventions as the input generator and are
listed with the design notes. Every function here is pinned by CPU tests against
closed forms, invariants, brute force or finite differences; none is "parity unpinned".
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------------------------------
# Decompression (Sec. 3 "Base model weights compression"; Algorithm 1, decompress)
# ----------------------------------------------------------------------------------------
def unpack_q4(q4: np.ndarray, n_in: int) -> np.ndarray:
    """Signed int4 codes int8 ``[out][n_in]`` from packed bytes ``[out][n_in/2]``.

    Element ``i`` of a row sits in byte ``i // 2``: low nibble for even ``i``, high nibble
    for odd ``i``; a nibble is a two's-complement 4-bit integer.
    """
    q4 = np.asarray(q4, dtype=np.uint8)
    idx = np.arange(n_in)
    byte = q4[:, idx // 2].astype(np.int16)
    nib = (byte >> (4 * (idx & 1))) & 0xF
    return (nib - 16 * (nib >= 8)).astype(np.int8)


def fp16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Value of raw IEEE binary16 bit patterns, decoded from sign/exponent/mantissa."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.int64)
    sign = np.where(b >> 15, -1.0, 1.0)
    e = (b >> 10) & 0x1F
    m = (b & 0x3FF).astype(F64)
    normal = sign * (1.0 + m / 1024.0) * np.exp2(e.astype(F64) - 15.0)
    sub = sign * (m / 1024.0) * 2.0 ** -14
    if np.any(e == 31):
        raise ValueError("inf/nan scale")
    return np.where(e == 0, sub, normal)


def dequant(q4: np.ndarray, scale_bits: np.ndarray, n_in: int, group: int = 32) -> np.ndarray:
    """Decompressed weight ``W_hat[o, i] = q[o, i] * s[o, i // group]`` in fp64 ``[out][in]``."""
    q = unpack_q4(q4, n_in).astype(F64)
    s = fp16_bits_to_f64(scale_bits)
    return q * s[:, np.arange(n_in) // group]


def bf16_rne_bits(x32: np.ndarray) -> np.ndarray:
    """bfloat16 bit pattern of float32 values, round to nearest even (no NaN inputs)."""
    u = np.asarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def dequant_bf16_bits(q4: np.ndarray, scale_bits: np.ndarray, n_in: int, group: int = 32) -> np.ndarray:
    """bf16 bits of ``float32(q*s)`` (the product is exact in float32: <= 14 significant bits)."""
    return bf16_rne_bits(dequant(q4, scale_bits, n_in, group).astype(np.float32))


def fp16_rne_bits(x) -> np.ndarray:
    """IEEE binary16 bit pattern of finite values, rounded to nearest, ties to even.

    Written from the format's definition in exact fp64 arithmetic: magnitudes below
    2^-14 are subnormal multiples of 2^-24; a normal value ``f * 2^e`` (``1 <= f < 2``)
    keeps 10 fraction bits; a rounded magnitude of 2^16 or more is infinity.
    """
    x = np.asarray(x, dtype=F64)
    if not np.all(np.isfinite(x)):
        raise ValueError("fp16_rne_bits takes finite values")
    sign = np.where(np.signbit(x), 0x8000, 0).astype(np.int64)
    a = np.abs(x)
    out = np.zeros(a.shape, np.int64)
    sub = a < 2.0 ** -14
    # subnormal (and zero): the integer number of 2^-24 units, ties to even
    out[sub] = np.rint(a[sub] * 2.0 ** 24).astype(np.int64)
    nrm = ~sub
    if np.any(nrm):
        f, e = np.frexp(a[nrm])  # a = f * 2^e with 0.5 <= f < 1
        e = e.astype(np.int64) - 1  # a = (2 f) * 2^e, 1 <= 2 f < 2
        m = np.rint((2.0 * f - 1.0) * 1024.0).astype(np.int64)  # 10 fraction bits, ties to even
        carry = m == 1024
        e = e + carry
        m = np.where(carry, 0, m)
        bits = (e + 15) * 1024 + m
        out[nrm] = np.where(e + 15 >= 31, 0x7C00, bits)
    return (out | sign).astype(np.uint16)


def dequant_fp16_bits(q4: np.ndarray, scale_bits: np.ndarray, n_in: int, group: int = 32) -> np.ndarray:
    """fp16 bits of ``q*s`` rounded to nearest even (the forward GEMMs' operand type)."""
    return fp16_rne_bits(dequant(q4, scale_bits, n_in, group))


# ----------------------------------------------------------------------------------------
# Elementary blocks
# ----------------------------------------------------------------------------------------
def rmsnorm(x: np.ndarray, w: np.ndarray, eps: float) -> Tuple[np.ndarray, np.ndarray]:
    """``y = x * w / sqrt(mean(x^2) + eps)`` row-wise; returns (y, rstd)."""
    x = np.asarray(x, F64)
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * rstd * np.asarray(w, F64), rstd


def rmsnorm_bwd(x: np.ndarray, w: np.ndarray, rstd: np.ndarray, dy: np.ndarray) -> np.ndarray:
    """Gradient of ``sum(dy * rmsnorm(x))`` w.r.t. x (weight frozen):
    ``dx = rstd * (w*dy - xhat * mean(xhat * w * dy))`` with ``xhat = x * rstd``."""
    x = np.asarray(x, F64)
    wdy = np.asarray(w, F64) * dy
    xhat = x * rstd
    return rstd * (wdy - xhat * np.mean(xhat * wdy, axis=-1, keepdims=True))


def rope_angles(T: int, dh: int, theta: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos, sin ``[T][dh/2]`` of angle ``t * theta**(-2i/dh)`` (position t from 0)."""
    inv = theta ** (-(2.0 * np.arange(dh // 2, dtype=F64)) / dh)
    ang = np.arange(T, dtype=F64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray, inverse: bool = False) -> np.ndarray:
    """Rotate-half RoPE on ``x`` ``[B][T][H][dh]``: pairs (i, i + dh/2) rotate by the angle
    of (t, i); ``inverse`` rotates by minus the angle (this is also the backward map,
    since the rotation is orthogonal)."""
    dh = x.shape[-1]
    x1, x2 = x[..., : dh // 2], x[..., dh // 2:]
    c = cos[None, :, None, :]
    s = sin[None, :, None, :] * (-1.0 if inverse else 1.0)
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attn_mask(T: int, window: int) -> np.ndarray:
    """Key j visible to query i iff ``j <= i`` and (``window == 0`` or ``i - j < window``)."""
    i = np.arange(T)[:, None]
    j = np.arange(T)[None, :]
    m = j <= i
    if window:
        m &= (i - j) < window
    return m


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, window: int) -> Tuple[np.ndarray, np.ndarray]:
    """Causal grouped-query attention. q ``[B][T][Hq][dh]``, k/v ``[B][T][Hkv][dh]``;
    query head h reads KV head ``h // (Hq/Hkv)``; scores ``q.k / sqrt(dh)``; softmax over
    visible keys. Returns (O ``[B][T][Hq][dh]``, P ``[B][Hq][T][T]``)."""
    B, T, Hq, dh = q.shape
    Hkv = k.shape[2]
    grp = Hq // Hkv
    mask = attn_mask(T, window)
    O = np.zeros_like(q, dtype=F64)
    P = np.zeros((B, Hq, T, T), F64)
    for b in range(B):
        for h in range(Hq):
            kh = h // grp
            S = q[b, :, h, :] @ k[b, :, kh, :].T / math.sqrt(dh)
            S = np.where(mask, S, -np.inf)
            S = S - S.max(axis=-1, keepdims=True)
            E = np.exp(S)
            Pm = E / E.sum(axis=-1, keepdims=True)
            P[b, h] = Pm
            O[b, :, h, :] = Pm @ v[b, :, kh, :]
    return O, P


def attention_bwd(q, k, v, P, dO) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Backward of :func:`attention`: ``dP = dO v^T``, ``dS = P (dP - rowsum(dP P))``,
    ``dq = dS k / sqrt(dh)``, ``dk = dS^T q / sqrt(dh)``, ``dv = P^T dO``; dk/dv summed
    over the query heads of a KV group."""
    B, T, Hq, dh = q.shape
    Hkv = k.shape[2]
    grp = Hq // Hkv
    dq = np.zeros_like(q, dtype=F64)
    dk = np.zeros_like(k, dtype=F64)
    dv = np.zeros_like(v, dtype=F64)
    sc = 1.0 / math.sqrt(dh)
    for b in range(B):
        for h in range(Hq):
            kh = h // grp
            Pm = P[b, h]
            dPm = dO[b, :, h, :] @ v[b, :, kh, :].T
            dS = Pm * (dPm - np.sum(dPm * Pm, axis=-1, keepdims=True))
            dq[b, :, h, :] = dS @ k[b, :, kh, :] * sc
            dk[b, :, kh, :] += dS.T @ q[b, :, h, :] * sc
            dv[b, :, kh, :] += Pm.T @ dO[b, :, h, :]
    return dq, dk, dv


_GC = math.sqrt(2.0 / math.pi)


def act(g: np.ndarray, kind: str) -> np.ndarray:
    """SiLU ``g*sigmoid(g)`` or tanh-approximated GELU ``g/2 (1 + tanh(c (g + 0.044715 g^3)))``."""
    if kind == "silu":
        return g / (1.0 + np.exp(-g))
    if kind == "gelu_tanh":
        return 0.5 * g * (1.0 + np.tanh(_GC * (g + 0.044715 * g ** 3)))
    raise ValueError(kind)


def act_grad(g: np.ndarray, kind: str) -> np.ndarray:
    """Derivative of :func:`act`."""
    if kind == "silu":
        sg = 1.0 / (1.0 + np.exp(-g))
        return sg * (1.0 + g * (1.0 - sg))
    if kind == "gelu_tanh":
        t = np.tanh(_GC * (g + 0.044715 * g ** 3))
        return 0.5 * (1.0 + t) + 0.5 * g * (1.0 - t * t) * _GC * (1.0 + 3.0 * 0.044715 * g * g)
    raise ValueError(kind)


# ----------------------------------------------------------------------------------------
# LoRA linear: y = x W^T + s (x A^T) B^T   (LoRA adapters, Sec. 2 / Sec. 3)
# ----------------------------------------------------------------------------------------
def lora_linear(x, W, A=None, B=None, s=1.0):
    """Returns (y, u) with ``u = x A^T`` (None when the projection is not adapted)."""
    y = x @ W.T
    if A is None:
        return y, None
    u = x @ A.T
    return y + s * (u @ B.T), u


def lora_linear_bwd(x, W, u, A, B, s, dy):
    """Backward of :func:`lora_linear` with W frozen. Returns (dx, dA, dB):
    ``du = s dy B``, ``dB = s dy^T u``, ``dA = du^T x``, ``dx = dy W + du A``."""
    dx = dy @ W
    if A is None:
        return dx, None, None
    du = s * (dy @ B)
    dB = s * (dy.T @ u)
    dA = du.T @ x
    return dx + du @ A, dA, dB


# ----------------------------------------------------------------------------------------
# Model state (decompressed lazily per block, Algorithm 1)
# ----------------------------------------------------------------------------------------
@dataclass
class LayerParams:
    W: Dict[str, np.ndarray]  # proj -> W_hat fp64 [out][in]
    norm_attn: np.ndarray
    norm_mlp: np.ndarray
    lora: Dict[str, Tuple[np.ndarray, np.ndarray]]  # proj -> (A, B) fp64
    bias: Optional[Dict[str, np.ndarray]] = None  # q, k, v biases (Qwen2.5)
    q_norm: Optional[np.ndarray] = None  # [dh] per-head RMSNorm weights of q and k (Gemma3)
    k_norm: Optional[np.ndarray] = None
    post_attn_norm: Optional[np.ndarray] = None  # [d] sandwich norms (Gemma3)
    post_mlp_norm: Optional[np.ndarray] = None


def decompress_layer(cfg, inp, l: int) -> LayerParams:
    """LazyLoadAndDecompressWeights(l) of Algorithm 1, in fp64."""
    W = {}
    for p, (q4, sb) in inp.base[l].items():
        W[p] = dequant(q4, sb, cfg.proj_shape(p)[1], cfg.group)
    lora = {p: (np.asarray(A, F64), np.asarray(B, F64)) for p, (A, B) in inp.lora[l].items()}
    P = LayerParams(W, np.asarray(inp.norm_attn[l], F64), np.asarray(inp.norm_mlp[l], F64), lora)
    ex = inp.extra
    if getattr(cfg, "qkv_bias", False):
        P.bias = {p: np.asarray(b, F64) for p, b in ex["bias"][l].items()}
    if getattr(cfg, "qk_norm", False):
        P.q_norm, P.k_norm = (np.asarray(w, F64) for w in ex["qk_norm"][l])
    if getattr(cfg, "sandwich_norm", False):
        P.post_attn_norm, P.post_mlp_norm = (np.asarray(w, F64) for w in ex["post_norm"][l])
    return P


def _lin(P: LayerParams, p: str, x, s):
    A, B = P.lora.get(p, (None, None))
    return lora_linear(x, P.W[p], A, B, s)


# ----------------------------------------------------------------------------------------
# Transformer block forward_i / backward_i (Algorithm 1; Sec. 3 backward graph B_i)
# ----------------------------------------------------------------------------------------
def layer_forward(cfg, l: int, P: LayerParams, x: np.ndarray, keep: bool = False):
    """``y = F_l(x)``; ``x`` fp64 ``[B*T][d]`` (row ``b*T + t``). With ``keep`` also
    returns every intermediate the backward graph needs."""
    Bsz, T = cfg.batch, cfg.seq
    Hq, Hkv, dh = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    s = cfg.lora_scale
    x = np.asarray(x, F64)
    a, rstd1 = rmsnorm(x, P.norm_attn, cfg.rms_eps)
    q, uq = _lin(P, "q", a, s)
    k, uk = _lin(P, "k", a, s)
    v, uv = _lin(P, "v", a, s)
    if P.bias is not None:  # Qwen2.5: q, k, v projections with bias
        q, k, v = q + P.bias["q"], k + P.bias["k"], v + P.bias["v"]
    q_pre, k_pre = q.reshape(Bsz, T, Hq, dh), k.reshape(Bsz, T, Hkv, dh)
    rq = rk = None
    if P.q_norm is not None:  # Gemma3: RMSNorm over each head of q and k, before RoPE
        qn, rq = rmsnorm(q_pre, P.q_norm, cfg.rms_eps)
        kn, rk = rmsnorm(k_pre, P.k_norm, cfg.rms_eps)
    else:
        qn, kn = q_pre, k_pre
    cos, sin = rope_angles(T, dh, cfg.layer_theta(l))
    q4d = rope(qn, cos, sin)
    k4d = rope(kn, cos, sin)
    v4d = v.reshape(Bsz, T, Hkv, dh)
    O4d, Pm = attention(q4d, k4d, v4d, cfg.layer_window(l))
    O = O4d.reshape(Bsz * T, Hq * dh)
    ao, uo = _lin(P, "o", O, s)
    rpa = rpm = None
    if P.post_attn_norm is not None:  # Gemma3 sandwich: norm the branch output, then add
        ao_n, rpa = rmsnorm(ao, P.post_attn_norm, cfg.rms_eps)
        h = x + ao_n
    else:
        h = x + ao
    c, rstd2 = rmsnorm(h, P.norm_mlp, cfg.rms_eps)
    g, ug = _lin(P, "gate", c, s)
    u, uu = _lin(P, "up", c, s)
    z = act(g, cfg.act) * u
    dn, ud = _lin(P, "down", z, s)
    if P.post_mlp_norm is not None:
        dn_n, rpm = rmsnorm(dn, P.post_mlp_norm, cfg.rms_eps)
        y = h + dn_n
    else:
        y = h + dn
    if not keep:
        return y
    cache = dict(x=x, a=a, rstd1=rstd1, q4d=q4d, k4d=k4d, v4d=v4d, P=Pm, O=O, h=h, c=c,
                 rstd2=rstd2, g=g, u=u, z=z, cos=cos, sin=sin, q_pre=q_pre, k_pre=k_pre, rq=rq, rk=rk,
                 ao=ao, rpa=rpa, dn=dn, rpm=rpm,
                 lu=dict(q=uq, k=uk, v=uv, o=uo, gate=ug, up=uu, down=ud))
    return y, cache


def layer_backward(cfg, l: int, P: LayerParams, x: np.ndarray, dy: np.ndarray, cache=None):
    """backward_l of Algorithm 1: recompute the block's forward from its checkpoint ``x``
    (unless ``cache`` is given), then return ``(dx, grads)`` where grads maps each adapted
    projection to ``(dA, dB)``."""
    if cache is None:
        _, cache = layer_forward(cfg, l, P, x, keep=True)
    Bsz, T = cfg.batch, cfg.seq
    Hq, Hkv, dh = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    s = cfg.lora_scale
    lu = cache["lu"]
    grads = {}
    dy = np.asarray(dy, F64)

    def lin_bwd(p, inp, dout):
        A, B = P.lora.get(p, (None, None))
        dxx, dA, dB = lora_linear_bwd(inp, P.W[p], lu[p], A, B, s, dout)
        if A is not None:
            grads[p] = (dA, dB)
        return dxx

    # y = h + down(z)   (sandwich: y = h + RMSNorm(down(z)))
    d_dn = dy if P.post_mlp_norm is None else rmsnorm_bwd(cache["dn"], P.post_mlp_norm, cache["rpm"], dy)
    dz = lin_bwd("down", cache["z"], d_dn)
    g, u = cache["g"], cache["u"]
    dg = dz * u * act_grad(g, cfg.act)
    du = dz * act(g, cfg.act)
    dc = lin_bwd("gate", cache["c"], dg) + lin_bwd("up", cache["c"], du)
    d_h = dy + rmsnorm_bwd(cache["h"], P.norm_mlp, cache["rstd2"], dc)
    # h = x + o(O)   (sandwich: h = x + RMSNorm(o(O)))
    d_ao = d_h if P.post_attn_norm is None else rmsnorm_bwd(cache["ao"], P.post_attn_norm, cache["rpa"], d_h)
    dO = lin_bwd("o", cache["O"], d_ao)
    dq4, dk4, dv4 = attention_bwd(cache["q4d"], cache["k4d"], cache["v4d"], cache["P"],
                                  dO.reshape(Bsz, T, Hq, dh))
    dq4 = rope(dq4, cache["cos"], cache["sin"], inverse=True)
    dk4 = rope(dk4, cache["cos"], cache["sin"], inverse=True)
    if P.q_norm is not None:  # through the per-head norms (biases are frozen: no gradient)
        dq4 = rmsnorm_bwd(cache["q_pre"], P.q_norm, cache["rq"], dq4)
        dk4 = rmsnorm_bwd(cache["k_pre"], P.k_norm, cache["rk"], dk4)
    a = cache["a"]
    da = (lin_bwd("q", a, dq4.reshape(Bsz * T, Hq * dh))
          + lin_bwd("k", a, dk4.reshape(Bsz * T, Hkv * dh))
          + lin_bwd("v", a, dv4.reshape(Bsz * T, Hkv * dh)))
    dx = d_h + rmsnorm_bwd(cache["x"], P.norm_attn, cache["rstd1"], da)
    return dx, grads


# ----------------------------------------------------------------------------------------
# Embedding, final linear + cross-entropy block
# ----------------------------------------------------------------------------------------
def decompress_embedding(cfg, inp) -> np.ndarray:
    q4, sb = inp.emb
    return dequant(q4, sb, cfg.hidden, cfg.group)


def embed(E_hat: np.ndarray, ids: np.ndarray, scale: float = 1.0) -> np.ndarray:
    """``x0[b*T + t] = scale * E_hat[ids[b, t]]`` (tied int4 table, decompressed; Gemma3
    scales the embedding output by sqrt(hidden), the LM head uses the table unscaled)."""
    return scale * E_hat[np.asarray(ids).reshape(-1)]


def embed_scale(cfg) -> float:
    return math.sqrt(cfg.hidden) if getattr(cfg, "embed_scale", False) else 1.0


def lm_head_ce(cfg, E_hat: np.ndarray, norm_final: np.ndarray, xL: np.ndarray, ids: np.ndarray,
               row_chunk: int = 512):
    """Final RMSNorm, logits ``hf E_hat^T``, next-token cross-entropy averaged over the
    ``B*(T-1)`` positions that have a target, and its gradient w.r.t. ``xL``.
    Rows are processed in chunks only to bound memory. Returns (loss, dxL)."""
    Bsz, T = cfg.batch, cfg.seq
    xL = np.asarray(xL, F64)
    hf, rstd = rmsnorm(xL, norm_final, cfg.rms_eps)
    N = Bsz * T
    n = Bsz * (T - 1)
    ids = np.asarray(ids).reshape(Bsz, T)
    tgt = np.full(N, -1, np.int64)
    tgt.reshape(Bsz, T)[:, :-1] = ids[:, 1:]
    dhf = np.zeros_like(hf)
    total = 0.0
    for r0 in range(0, N, row_chunk):
        r1 = min(N, r0 + row_chunk)
        rows = np.arange(r0, r1)
        rows = rows[tgt[rows] >= 0]
        if rows.size == 0:
            continue
        z = hf[rows] @ E_hat.T
        m = z.max(axis=-1, keepdims=True)
        e = np.exp(z - m)
        ssum = e.sum(axis=-1, keepdims=True)
        lse = (m + np.log(ssum))[:, 0]
        t = tgt[rows]
        total += float(np.sum(lse - z[np.arange(rows.size), t]))
        dz = e / ssum
        dz[np.arange(rows.size), t] -= 1.0
        dhf[rows] = (dz / n) @ E_hat
    loss = total / n
    dxL = rmsnorm_bwd(xL, norm_final, rstd, dhf)
    return loss, dxL


def lm_head_ce_rows(cfg, E_hat: np.ndarray, norm_final: np.ndarray, x_rows: np.ndarray, tgt: np.ndarray,
                    n: int):
    """The LM head's per-row terms for selected rows only. Every row's share of the loss
    and of dL/dx_L depends on that row alone (RMSNorm, logits and softmax are row-wise):
    ``row_loss = lse(z) - z[tgt]`` and ``dx = rmsnorm_bwd((softmax(z) - onehot(tgt)) E_hat / n)``
    with ``z = RMSNorm(x) E_hat^T``. ``tgt < 0`` marks a row without a target (zero term,
    zero gradient); ``n`` is the full problem's number of target positions. Used to check
    sampled rows of shapes whose full logits the CPU cannot afford. Returns
    (row_loss [k], dx_rows [k][d])."""
    x_rows = np.asarray(x_rows, F64)
    tgt = np.asarray(tgt, np.int64)
    hf, rstd = rmsnorm(x_rows, norm_final, cfg.rms_eps)
    row_loss = np.zeros(len(tgt))
    dhf = np.zeros_like(hf)
    rows = np.nonzero(tgt >= 0)[0]
    if rows.size:
        z = hf[rows] @ E_hat.T
        m = z.max(axis=-1, keepdims=True)
        e = np.exp(z - m)
        ssum = e.sum(axis=-1, keepdims=True)
        t = tgt[rows]
        row_loss[rows] = (m + np.log(ssum))[:, 0] - z[np.arange(rows.size), t]
        dz = e / ssum
        dz[np.arange(rows.size), t] -= 1.0
        dhf[rows] = (dz / n) @ E_hat
    return row_loss, rmsnorm_bwd(x_rows, norm_final, rstd, dhf)


def lm_head_logits(cfg, E_hat, norm_final, xL):
    """Full logits ``[B*T][V]`` (small shapes only; used by pins)."""
    hf, _ = rmsnorm(np.asarray(xL, F64), norm_final, cfg.rms_eps)
    return hf @ E_hat.T


# ----------------------------------------------------------------------------------------
# Algorithm 1: Backpropagation(x) with a checkpoint at every block boundary
# ----------------------------------------------------------------------------------------
@dataclass
class StepResult:
    loss: float
    grads: List[Dict[str, Tuple[np.ndarray, np.ndarray]]]  # per layer
    ckpts: List[np.ndarray]  # x_0 .. x_L (fp64)
    dx0: np.ndarray  # gradient w.r.t. the embedding output (the frozen table gets none)


def train_step(cfg, inp, keep_ckpts: bool = True) -> StepResult:
    """Backpropagation(x) of Algorithm 1 for one batch of token ids.

    Forward loop: ckpts_i = forward_i(ckpts_{i-1}) with the block's weights decompressed
    just before use. Loss block. Reverse loop: decompress block i again, recompute its
    forward from ckpts_{i-1}, backpropagate the upstream gradient, collect the LoRA
    gradients, drop the checkpoint.
    """
    L = len(inp.base)
    E_hat = decompress_embedding(cfg, inp)
    ckpts = [embed(E_hat, inp.ids, embed_scale(cfg))]
    for l in range(L):
        P = decompress_layer(cfg, inp, l)
        ckpts.append(layer_forward(cfg, l, P, ckpts[l]))
        del P
    loss, g = lm_head_ce(cfg, E_hat, inp.norm_final, ckpts[L], inp.ids)
    grads: List[Optional[dict]] = [None] * L
    kept = list(ckpts) if keep_ckpts else None
    for l in reversed(range(L)):
        P = decompress_layer(cfg, inp, l)
        g, grads[l] = layer_backward(cfg, l, P, ckpts[l], g)
        ckpts[l + 1] = None
        del P
    return StepResult(loss=loss, grads=grads, ckpts=kept if kept is not None else [], dx0=g)


def train_step_stored(cfg, inp) -> StepResult:
    """The same gradients without checkpointing: one forward pass keeps every
    intermediate of every block, then backward uses them (no recomputation)."""
    L = len(inp.base)
    E_hat = decompress_embedding(cfg, inp)
    x = [embed(E_hat, inp.ids, embed_scale(cfg))]
    caches, params = [], []
    for l in range(L):
        P = decompress_layer(cfg, inp, l)
        y, cache = layer_forward(cfg, l, P, x[l], keep=True)
        x.append(y)
        caches.append(cache)
        params.append(P)
    loss, g = lm_head_ce(cfg, E_hat, inp.norm_final, x[L], inp.ids)
    grads: List[Optional[dict]] = [None] * L
    for l in reversed(range(L)):
        g, grads[l] = layer_backward(cfg, l, params[l], x[l], g, cache=caches[l])
    return StepResult(loss=loss, grads=grads, ckpts=x, dx0=g)


def block_forward_backward(cfg, inp, l: int = 0, x=None, dy=None):
    """Single block (no embedding / head): ``(y, dx, grads)`` for input ``x`` and upstream
    gradient ``dy`` (default: the generator's ``x`` / ``dy``)."""
    P = decompress_layer(cfg, inp, l)
    x = inp.x if x is None else x
    dy = inp.dy if dy is None else dy
    y = layer_forward(cfg, l, P, x)
    dx, grads = layer_backward(cfg, l, P, x, dy)
    return y, dx, grads


# ----------------------------------------------------------------------------------------
# Optimizer on the LoRA parameters (Sec. 3, "Runtime implementation": gradients of a batch
# by gradient accumulation, and only the LoRA weights, their gradients and the optimizer
# state kept for the optimizer; Sec. 4.1: the optimizer is AdamW)
# ----------------------------------------------------------------------------------------
def grad_accumulate(acc: Optional[np.ndarray], g: np.ndarray, scale: float) -> np.ndarray:
    """``acc + scale * g``; ``acc = None`` starts a new accumulation (``scale * g``).

    With ``scale = 1/k`` over k micro-batches of equal size this is the gradient of the
    mean loss of their union (the batch relation of the loss normalisation)."""
    g = np.asarray(g, F64)
    return scale * g if acc is None else np.asarray(acc, F64) + scale * g


def adamw_step(p: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray, t: int, lr: float,
               beta1: float, beta2: float, eps: float, weight_decay: float, grad_scale: float = 1.0):
    """One AdamW update (Adam with decoupled weight decay, Loshchilov & Hutter) of one tensor.

    ``t >= 1`` is the index of this update; returns the new ``(p, m, v)``:
        g' = grad_scale * g
        m  = beta1 m + (1 - beta1) g'            v = beta2 v + (1 - beta2) g'^2
        p  = p - lr (weight_decay p + m_hat / (sqrt(v_hat) + eps)),
    with the bias-corrected moments m_hat = m / (1 - beta1^t), v_hat = v / (1 - beta2^t).
    """
    p, g, m, v = (np.asarray(a, F64) for a in (p, g, m, v))
    g = grad_scale * g
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    p = p - lr * (weight_decay * p + m_hat / (np.sqrt(v_hat) + eps))
    return p, m, v
