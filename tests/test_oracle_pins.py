"""Pins of the CPU fp64 oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: exhaustive enumeration,
bit-level IEEE definitions, closed forms, special cases that reduce to a textbook result,
brute-force loops on tiny inputs, finite differences of the backward graph's defining
scalar (Sec. 3, display equation), invariants of LoRA (Sec. 2/3) and of Algorithm 1,
and the trainable-parameter counts printed in Table 1.
"""
import math
import os

import numpy as np
import pytest

import oracle as O
from mebp_inputs import ALL7, CONFIGS, PROJ, TINY, Config, make_inputs, quantize_q4

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------------------
# P1: int4 unpack / dequant (Sec. 3 "Base model weights compression")
# ---------------------------------------------------------------------------------------
def test_unpack_exhaustive_all_nibbles_both_positions():
    # every code -8..7 in the even and the odd position of a byte, packed by hand
    codes = np.arange(-8, 8)
    rows = []
    for lo in codes:
        for hi in codes:
            rows.append([(int(lo) & 0xF) | ((int(hi) & 0xF) << 4)])
    q4 = np.array(rows, np.uint8)
    q = O.unpack_q4(q4, 2)
    exp = np.array([[lo, hi] for lo in codes for hi in codes], np.int8)
    np.testing.assert_array_equal(q, exp)


def test_packer_roundtrip_through_unpack():
    rng = np.random.default_rng(3)
    w = rng.standard_normal((5, 96)).astype(np.float32)
    q4, sb = quantize_q4(w, 32)
    q = O.unpack_q4(q4, 96).astype(np.int64)
    # repack by hand with the documented layout and compare bytes
    u = q & 0xF
    np.testing.assert_array_equal(q4, (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8))
    assert q.min() >= -7 and q.max() <= 7


def test_fp16_decode_matches_ieee_via_numpy_half():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = ((bits >> 10) & 0x1F) != 31
    bits = bits[finite]
    np.testing.assert_array_equal(O.fp16_bits_to_f64(bits), bits.view(np.float16).astype(np.float64))


def test_bf16_rne_known_patterns():
    cases = {
        1.0: 0x3F80, -2.0: 0xC000, 0.0: 0x0000,
        # 1 + 2^-8 is a tie between 1.0 and 1+2^-7: even mantissa wins -> 1.0
        1.0 + 2.0 ** -8: 0x3F80,
        # 1 + 3*2^-8 is a tie between 1+2^-7 (odd) and 1+2^-6 (even) -> 1+2^-6
        1.0 + 3 * 2.0 ** -8: 0x3F82,
        # just above the tie rounds up
        1.0 + 2.0 ** -8 + 2.0 ** -20: 0x3F81,
    }
    for v, b in cases.items():
        assert int(O.bf16_rne_bits(np.float32(v))) == b, v


def test_dequant_value_exact_in_fp32_and_bf16_bits():
    cfg = CONFIGS["block"]
    inp = make_inputs(cfg)
    q4, sb = inp.base[0]["down"]  # in = 688: the last group of each row has 16 elements
    Wd = O.dequant(q4, sb, 688, 32)
    # q*s is exactly representable in float32
    assert np.array_equal(Wd.astype(np.float32).astype(np.float64), Wd)
    bits = O.dequant_bf16_bits(q4, sb, 688, 32)
    # reference: IEEE round-to-nearest-even to 8 significand bits, computed from the
    # exact value by frexp / rint (a different route than the bit trick)
    m, e = np.frexp(Wd)
    ref = np.ldexp(np.rint(m * 256.0) / 256.0, e)
    got = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    np.testing.assert_array_equal(got, ref)


def test_dequant_hand_set_codes_and_scales_one_by_one():
    # a ragged row length (688 = 21 full groups of 32 and one of 16), every group with its
    # own scale (subnormal, small, ordinary and large fp16 values), codes chosen by hand and
    # packed here; each decompressed value is checked against code * scale in Python floats
    n_out, n_in = 3, 688
    ng = (n_in + 31) // 32
    # (the largest, times 1.5 and 7, stays below the fp16 maximum 65504)
    scale_vals = [2.0 ** -24 * 3, 2.0 ** -20, 1.5e-3, 0.0078125, 0.01, 0.02, 1.0, 3.25, 2.0 ** 10, 6000.0]
    s16 = np.empty((n_out, ng), np.float16)
    for o in range(n_out):
        for g in range(ng):
            s16[o, g] = np.float16(scale_vals[(o * ng + g) % len(scale_vals)] * (1 + (g % 5) / 8))
    codes = [[((7 * o + 3 * i + (i // 32)) % 15) - 7 for i in range(n_in)] for o in range(n_out)]
    codes[0][0], codes[0][1], codes[1][687], codes[2][686] = -8, 7, -8, -7  # both nibble positions
    q4 = np.zeros((n_out, n_in // 2), np.uint8)
    for o in range(n_out):
        for i in range(n_in):
            q4[o, i // 2] |= (codes[o][i] & 0xF) << (4 * (i % 2))
    W = O.dequant(q4, s16.view(np.uint16), n_in, 32)
    for o in range(n_out):
        for i in range(n_in):
            assert W[o, i] == codes[o][i] * float(s16[o, i // 32]), (o, i)
    # the same values rounded to the forward GEMMs' fp16 operand
    f16 = O.dequant_fp16_bits(q4, s16.view(np.uint16), n_in, 32)
    for o in range(n_out):
        for i in range(n_in):
            assert f16[o, i] == np.float16(codes[o][i] * float(s16[o, i // 32])).view(np.uint16), (o, i)


def test_dequant_of_quantizer_output_within_half_a_step_ragged_row():
    # the decompressed weight of the offline quantiser's output is within half a
    # quantisation step of the original weight, group by group, including the 16-wide last
    # group of a 688-wide row; the step is the fp16 scale decoded by numpy
    rng = np.random.default_rng(11)
    w = (rng.standard_normal((48, 688)) * 0.02).astype(np.float32)
    w[5, 672:] *= 50.0  # a last group with a much larger scale than its row
    w[7, :32] = 0.0  # an all-zero group
    q4, sb = quantize_q4(w, 32)
    W = O.dequant(q4, sb, 688, 32)
    s = sb.view(np.float16).astype(np.float64)
    for g in range(22):
        cols = slice(32 * g, min(688, 32 * g + 32))
        err = np.abs(W[:, cols] - w[:, cols].astype(np.float64))
        assert np.all(err <= 0.5 * s[:, g:g + 1] * (1 + 2.0 ** -20)), g
    assert np.all(W[7, :32] == 0.0)
    # max |q| = 7 in each nonzero group: the group's largest weight maps to +-7 steps
    for g in range(22):
        cols = slice(32 * g, min(688, 32 * g + 32))
        nz = s[:, g] > 0
        ratio = np.max(np.abs(W[nz, cols]), axis=1) / s[nz, g]
        np.testing.assert_array_equal(ratio, 7.0)


def test_fp16_rne_matches_numpy_half_conversion():
    # every float32 value that lies on the fp16 grid or halfway between two neighbours
    # (ties), plus random values across the whole range including subnormals and overflow
    rng = np.random.default_rng(12)
    h = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    mids = (h[:-1] + h[1:]) / 2.0
    vals = np.concatenate([h, mids, mids * (1 + 2.0 ** -30), mids * (1 - 2.0 ** -30),
                           np.exp(rng.uniform(np.log(2.0 ** -26), np.log(7e4), 200000)), [65519.0, 65520.0, 1e6]])
    vals = np.concatenate([vals, -vals]).astype(np.float32)
    with np.errstate(over="ignore"):  # 65520 and above overflow to infinity on purpose
        ref = vals.astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(O.fp16_rne_bits(vals), ref)


# ---------------------------------------------------------------------------------------
# P2: quantiser bounds (the compressed input format)
# ---------------------------------------------------------------------------------------
def test_quantizer_error_bound_and_full_range():
    rng = np.random.default_rng(1)
    w = (rng.standard_normal((64, 688)) * 0.02).astype(np.float32)
    q4, sb = quantize_q4(w, 32)
    q = O.unpack_q4(q4, 688).astype(np.float64)
    s = O.fp16_bits_to_f64(sb)
    s_full = s[:, np.arange(688) // 32]
    err = np.abs(w.astype(np.float64) - q * s_full)
    # half a step, plus the fp16 rounding of the scale propagated through |q| <= 7
    assert np.all(err <= 0.5 * s_full + 7 * s_full * 2.0 ** -11 + 1e-12)
    qg = np.abs(np.pad(q, ((0, 0), (0, 16))).reshape(64, 22, 32)).max(-1)
    assert np.all(qg == 7)
    # an all-zero group gives a zero scale and zero codes
    w2 = w.copy()
    w2[0, :32] = 0
    q4b, sbb = quantize_q4(w2, 32)
    assert sbb[0, 0] == 0 and np.all(O.unpack_q4(q4b, 688)[0, :32] == 0)


# ---------------------------------------------------------------------------------------
# Elementary blocks: closed forms and special cases
# ---------------------------------------------------------------------------------------
def test_rmsnorm_closed_form():
    d = 32
    x = np.full((3, d), 2.0)
    w = np.linspace(0.5, 1.5, d)
    y, rstd = O.rmsnorm(x, w, 1e-6)
    np.testing.assert_allclose(y, np.broadcast_to(w[None] * 2.0 / math.sqrt(4.0 + 1e-6), y.shape), rtol=1e-15)
    # scale invariance (eps -> 0): rmsnorm(c x) == rmsnorm(x)
    x = np.random.default_rng(0).standard_normal((4, d))
    np.testing.assert_allclose(O.rmsnorm(5 * x, w, 0.0)[0], O.rmsnorm(x, w, 0.0)[0], rtol=1e-13)
    # output rms equals 1 for unit weights, eps = 0
    y, _ = O.rmsnorm(x, np.ones(d), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, -1)), 1.0, rtol=1e-14)


def test_rope_properties():
    rng = np.random.default_rng(0)
    T, dh = 9, 16
    cos, sin = O.rope_angles(T, dh, 1e4)
    x = rng.standard_normal((1, T, 2, dh))
    r = O.rope(x, cos, sin)
    np.testing.assert_allclose(r[:, 0], x[:, 0], rtol=0, atol=0)  # position 0: identity
    pn = lambda z: z[..., : dh // 2] ** 2 + z[..., dh // 2:] ** 2
    np.testing.assert_allclose(pn(r), pn(x), rtol=1e-13)  # each pair keeps its norm
    np.testing.assert_allclose(O.rope(r, cos, sin, inverse=True), x, atol=1e-14)
    # <rope(q, m), rope(k, n)> depends only on m - n
    q = rng.standard_normal(dh)
    k = rng.standard_normal(dh)
    Q = O.rope(np.broadcast_to(q, (1, T, 1, dh)).copy(), cos, sin)[0, :, 0]
    K = O.rope(np.broadcast_to(k, (1, T, 1, dh)).copy(), cos, sin)[0, :, 0]
    for delta in range(0, 4):
        vals = [Q[m] @ K[m - delta] for m in range(delta, T)]
        np.testing.assert_allclose(vals, vals[0], rtol=1e-12, atol=1e-12)
    # the first pair rotates by exactly t radians (theta^0 = 1)
    np.testing.assert_allclose(np.arctan2(sin[:, 0], cos[:, 0]), np.angle(np.exp(1j * np.arange(T))))


def _attn_loops(q, k, v, window):
    """Brute force: explicit loops over batch, head, query, key."""
    B, T, Hq, dh = q.shape
    Hkv = k.shape[2]
    out = np.zeros_like(q)
    for b in range(B):
        for h in range(Hq):
            kh = h * Hkv // Hq
            for i in range(T):
                sc = []
                for j in range(T):
                    vis = j <= i and (window == 0 or i - j < window)
                    sc.append(sum(q[b, i, h, e] * k[b, j, kh, e] for e in range(dh)) / math.sqrt(dh)
                              if vis else None)
                mx = max(s for s in sc if s is not None)
                w = [math.exp(s - mx) if s is not None else 0.0 for s in sc]
                z = sum(w)
                for e in range(dh):
                    out[b, i, h, e] = sum(w[j] * v[b, j, kh, e] for j in range(T)) / z
    return out


@pytest.mark.parametrize("window", [0, 3])
def test_attention_brute_force(window):
    rng = np.random.default_rng(5)
    q = rng.standard_normal((2, 6, 4, 4))
    k = rng.standard_normal((2, 6, 2, 4))
    v = rng.standard_normal((2, 6, 2, 4))
    O_, _ = O.attention(q, k, v, window)
    np.testing.assert_allclose(O_, _attn_loops(q, k, v, window), rtol=1e-12, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(6)
    B, T, H, dh = 1, 8, 2, 4
    k = rng.standard_normal((B, T, H, dh))
    v = rng.standard_normal((B, T, H, dh))
    # T = 1: the only visible key is itself -> O = v
    q1 = rng.standard_normal((B, 1, H, dh))
    np.testing.assert_allclose(O.attention(q1, k[:, :1], v[:, :1], 0)[0], v[:, :1], rtol=1e-15)
    # q = 0: uniform weights over visible keys -> running mean of v
    q0 = np.zeros((B, T, H, dh))
    cm = np.cumsum(v, axis=1) / np.arange(1, T + 1)[None, :, None, None]
    np.testing.assert_allclose(O.attention(q0, k, v, 0)[0], cm, rtol=1e-13)
    # q = 0 with window W: mean over the last W positions
    W = 3
    win = np.stack([v[:, max(0, i - W + 1): i + 1].mean(axis=1) for i in range(T)], axis=1)
    np.testing.assert_allclose(O.attention(q0, k, v, W)[0], win, rtol=1e-13)
    # window >= T equals plain causal
    q = rng.standard_normal((B, T, H, dh))
    np.testing.assert_allclose(O.attention(q, k, v, T)[0], O.attention(q, k, v, 0)[0], rtol=1e-15)
    # GQA with a KV head repeated equals MHA with the repeated heads
    q4 = rng.standard_normal((B, T, 4, dh))
    Og, _ = O.attention(q4, k, v, 0)
    Om, _ = O.attention(q4, np.repeat(k, 2, axis=2), np.repeat(v, 2, axis=2), 0)
    np.testing.assert_allclose(Og, Om, rtol=1e-15)


def test_activation_closed_forms():
    g = np.array([-30.0, -1.0, 0.0, 1.0, 30.0])
    silu = O.act(g, "silu")
    np.testing.assert_allclose(silu, [-30.0 / (1 + math.exp(30)), -1 / (1 + math.e), 0.0,
                                      1 / (1 + math.exp(-1)), 30.0 / (1 + math.exp(-30))], rtol=1e-14)
    ge = O.act(g, "gelu_tanh")
    assert ge[2] == 0.0 and abs(ge[4] - 30.0) < 1e-12 and abs(ge[0]) < 1e-12
    # GELU-tanh is within 1e-3 of the exact erf GELU on [-4, 4]
    xs = np.linspace(-4, 4, 81)
    exact = np.array([0.5 * t * (1 + math.erf(t / math.sqrt(2))) for t in xs])
    assert np.max(np.abs(O.act(xs, "gelu_tanh") - exact)) < 1e-3
    # derivatives at 0: silu' = 1/2, gelu' = 1/2
    np.testing.assert_allclose(O.act_grad(np.zeros(1), "silu"), 0.5)
    np.testing.assert_allclose(O.act_grad(np.zeros(1), "gelu_tanh"), 0.5)


def test_cross_entropy_uniform_logits():
    # zero embedding -> all logits 0 -> loss = ln V exactly; gradient zero (E_hat = 0)
    cfg = TINY
    V, d = cfg.vocab, cfg.hidden
    rng = np.random.default_rng(0)
    ids = rng.integers(0, V, (cfg.batch, cfg.seq))
    xL = rng.standard_normal((cfg.n_tokens, d))
    loss, dx = O.lm_head_ce(cfg, np.zeros((V, d)), np.ones(d), xL, ids)
    assert abs(loss - math.log(V)) < 1e-14
    assert np.all(dx == 0)


def test_cross_entropy_matches_per_row_definition():
    cfg = TINY
    inp = make_inputs(cfg, seed=2, norm="random")
    E = O.decompress_embedding(cfg, inp)
    rng = np.random.default_rng(1)
    xL = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    loss, _ = O.lm_head_ce(cfg, E, inp.norm_final, xL, inp.ids, row_chunk=3)
    z = O.lm_head_logits(cfg, E, inp.norm_final, xL)
    tot = 0.0
    for b in range(cfg.batch):
        for t in range(cfg.seq - 1):
            row = z[b * cfg.seq + t]
            p = np.exp(row - row.max())
            p /= p.sum()
            tot += -math.log(p[inp.ids[b, t + 1]])
    assert abs(loss - tot / (cfg.batch * (cfg.seq - 1))) < 1e-12


# ---------------------------------------------------------------------------------------
# Brute-force loops for a whole tiny block (catches transposed operands / wrong indices)
# ---------------------------------------------------------------------------------------
def _block_loops(cfg, l, P, x):
    N, d = x.shape
    Bsz, T = cfg.batch, cfg.seq
    Hq, Hkv, dh = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    s = cfg.lora_scale

    def norm(z, w):
        out = np.zeros_like(z)
        for n in range(N):
            ms = sum(z[n, i] ** 2 for i in range(z.shape[1])) / z.shape[1]
            for i in range(z.shape[1]):
                out[n, i] = z[n, i] * w[i] / math.sqrt(ms + cfg.rms_eps)
        return out

    def lin(p, z):
        W = P.W[p]
        o_, i_ = W.shape
        out = np.zeros((N, o_))
        A, B = P.lora.get(p, (None, None))
        for n in range(N):
            if A is not None:
                u = [sum(z[n, i] * A[j, i] for i in range(i_)) for j in range(A.shape[0])]
            for o in range(o_):
                acc = sum(z[n, i] * W[o, i] for i in range(i_))
                if A is not None:
                    acc += s * sum(u[j] * B[o, j] for j in range(A.shape[0]))
                out[n, o] = acc
        return out

    a = norm(x, P.norm_attn)
    q, k, v = lin("q", a), lin("k", a), lin("v", a)
    theta = cfg.layer_theta(l)

    def rot(z, H):
        out = z.copy()
        for n in range(N):
            t = n % T
            for h in range(H):
                for i in range(dh // 2):
                    ang = t * theta ** (-2.0 * i / dh)
                    x1, x2 = z[n, h * dh + i], z[n, h * dh + i + dh // 2]
                    out[n, h * dh + i] = x1 * math.cos(ang) - x2 * math.sin(ang)
                    out[n, h * dh + i + dh // 2] = x2 * math.cos(ang) + x1 * math.sin(ang)
        return out

    q, k = rot(q, Hq), rot(k, Hkv)
    att = _attn_loops(q.reshape(Bsz, T, Hq, dh), k.reshape(Bsz, T, Hkv, dh),
                      v.reshape(Bsz, T, Hkv, dh), cfg.layer_window(l)).reshape(N, Hq * dh)
    h = x + lin("o", att)
    c = norm(h, P.norm_mlp)
    g, u = lin("gate", c), lin("up", c)
    z = np.zeros_like(g)
    for n in range(N):
        for f in range(g.shape[1]):
            z[n, f] = float(O.act(np.array(g[n, f]), cfg.act)) * u[n, f]
    return h + lin("down", z)


@pytest.mark.parametrize("layer,act", [(0, "silu"), (1, "gelu_tanh")])
def test_block_forward_brute_force(layer, act):
    cfg = TINY.with_(batch=1, seq=5, hidden=32, ffn=64, n_heads=2, n_kv_heads=1, act=act)
    inp = make_inputs(cfg, seed=4, norm="random")
    P = O.decompress_layer(cfg, inp, layer)
    x = np.random.default_rng(9).standard_normal((cfg.n_tokens, cfg.hidden))
    y = O.layer_forward(cfg, layer, P, x)
    np.testing.assert_allclose(y, _block_loops(cfg, layer, P, x), rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------------------------------
# P3: finite differences of s = sum(dE/dy * F(x)) (Sec. 3 display equation)
# ---------------------------------------------------------------------------------------
def _fd_dir(f, x, v, h=1e-6):
    return (f(x + h * v) - f(x - h * v)) / (2 * h)


def _assert_fd(f, x, grad, n_dirs=4, seed=0, tol=1e-6):
    rng = np.random.default_rng(seed)
    for _ in range(n_dirs):
        v = rng.standard_normal(x.shape)
        fd = _fd_dir(f, x, v)
        an = float(np.sum(grad * v))
        assert abs(fd - an) <= tol * max(1.0, abs(an)), (fd, an)


@pytest.mark.parametrize("layer", [0, 1])
@pytest.mark.parametrize("act", ["silu", "gelu_tanh"])
def test_block_backward_finite_differences(layer, act):
    cfg = TINY.with_(act=act)
    inp = make_inputs(cfg, seed=7, norm="random")
    P = O.decompress_layer(cfg, inp, layer)
    rng = np.random.default_rng(11)
    x = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dy = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dx, grads = O.layer_backward(cfg, layer, P, x, dy)

    def s_of_x(xx):
        return float(np.sum(dy * O.layer_forward(cfg, layer, P, xx)))

    _assert_fd(s_of_x, x, dx)
    assert set(grads) == set(ALL7)
    for p in ALL7:
        A, B = P.lora[p]
        dA, dB = grads[p]

        def s_of_A(AA, p=p, B=B):
            P.lora[p] = (AA, B)
            try:
                return float(np.sum(dy * O.layer_forward(cfg, layer, P, x)))
            finally:
                P.lora[p] = (A, B)

        def s_of_B(BB, p=p, A=A):
            P.lora[p] = (A, BB)
            try:
                return float(np.sum(dy * O.layer_forward(cfg, layer, P, x)))
            finally:
                P.lora[p] = (A, B)

        _assert_fd(s_of_A, A, dA, n_dirs=2)
        _assert_fd(s_of_B, B, dB, n_dirs=2)


def test_block_backward_elementwise_fd_few_entries():
    cfg = TINY
    inp = make_inputs(cfg, seed=8)
    P = O.decompress_layer(cfg, inp, 0)
    rng = np.random.default_rng(12)
    x = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dy = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dx, _ = O.layer_backward(cfg, 0, P, x, dy)
    for (n, i) in [(0, 0), (3, 17), (6, 63), (7, 5), (13, 40)]:
        e = np.zeros_like(x)
        e[n, i] = 1.0
        fd = _fd_dir(lambda xx: float(np.sum(dy * O.layer_forward(cfg, 0, P, xx))), x, e)
        assert abs(fd - dx[n, i]) <= 1e-6 * max(1.0, abs(dx[n, i]))


def test_lm_head_rows_pins():
    # per-row form: FD of its own partial loss, consistency with the whole-batch head,
    # uniform logits give ln V per row, rows without a target contribute nothing
    cfg = TINY
    inp = make_inputs(cfg, seed=4, norm="random")
    E = O.decompress_embedding(cfg, inp)
    rng = np.random.default_rng(8)
    xL = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    n = cfg.batch * (cfg.seq - 1)
    tgt = np.full(cfg.n_tokens, -1)
    tgt.reshape(cfg.batch, cfg.seq)[:, :-1] = inp.ids[:, 1:]
    rows = np.array([0, 3, cfg.seq - 1, cfg.seq + 2])
    rl, dx = O.lm_head_ce_rows(cfg, E, inp.norm_final, xL[rows], tgt[rows], n)
    _assert_fd(lambda xx: float(np.sum(O.lm_head_ce_rows(cfg, E, inp.norm_final, xx, tgt[rows], n)[0])) / n,
               xL[rows], dx)
    assert rl[2] == 0 and np.all(dx[2] == 0)  # position T-1: no target
    loss, dx_all = O.lm_head_ce(cfg, E, inp.norm_final, xL, inp.ids)
    rl_all, dx_rows_all = O.lm_head_ce_rows(cfg, E, inp.norm_final, xL, tgt, n)
    assert abs(rl_all.sum() / n - loss) <= 1e-12 * abs(loss)
    np.testing.assert_allclose(dx_rows_all, dx_all, rtol=0, atol=1e-15)
    rl0, dx0 = O.lm_head_ce_rows(cfg, np.zeros_like(E), inp.norm_final, xL[rows], tgt[rows], n)
    np.testing.assert_allclose(rl0[[0, 1, 3]], math.log(cfg.vocab), rtol=1e-14)


def test_lm_head_block_finite_differences():
    cfg = TINY
    inp = make_inputs(cfg, seed=9, norm="random")
    E = O.decompress_embedding(cfg, inp)
    xL = np.random.default_rng(3).standard_normal((cfg.n_tokens, cfg.hidden))
    loss, dxL = O.lm_head_ce(cfg, E, inp.norm_final, xL, inp.ids)
    _assert_fd(lambda xx: O.lm_head_ce(cfg, E, inp.norm_final, xx, inp.ids)[0], xL, dxL)
    # the last position of every sequence has no target and no gradient through the head
    assert np.all(dxL.reshape(cfg.batch, cfg.seq, -1)[:, -1] == 0)


def test_full_step_lora_grads_fd_through_all_layers():
    cfg = TINY
    inp = make_inputs(cfg, seed=10, norm="random")
    res = O.train_step(cfg, inp)

    def loss_of(l, p, which, val):
        A, B = inp.lora[l][p]
        inp.lora[l][p] = (val, B) if which == 0 else (A, val)
        try:
            E = O.decompress_embedding(cfg, inp)
            x = O.embed(E, inp.ids)
            for j in range(cfg.n_layers):
                x = O.layer_forward(cfg, j, O.decompress_layer(cfg, inp, j), x)
            return O.lm_head_ce(cfg, E, inp.norm_final, x, inp.ids)[0]
        finally:
            inp.lora[l][p] = (A, B)

    for l, p in [(0, "q"), (0, "down"), (1, "v"), (1, "gate")]:
        A, B = (np.asarray(t, np.float64) for t in inp.lora[l][p])
        dA, dB = res.grads[l][p]
        _assert_fd(lambda a: loss_of(l, p, 0, a), A, dA, n_dirs=2, tol=1e-5)
        _assert_fd(lambda b: loss_of(l, p, 1, b), B, dB, n_dirs=2, tol=1e-5)


# ---------------------------------------------------------------------------------------
# P4: LoRA invariants
# ---------------------------------------------------------------------------------------
def test_lora_b_zero_is_identity_adapter_and_zero_dA():
    cfg = TINY
    inp0 = make_inputs(cfg, seed=13, lora_b_zero=True)
    P = O.decompress_layer(cfg, inp0, 0)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dy = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    y = O.layer_forward(cfg, 0, P, x)
    Pbase = O.LayerParams(P.W, P.norm_attn, P.norm_mlp, {})
    assert np.array_equal(y, O.layer_forward(cfg, 0, Pbase, x))
    _, grads = O.layer_backward(cfg, 0, P, x, dy)
    for p in ALL7:
        assert np.all(grads[p][0] == 0)
        assert np.any(grads[p][1] != 0)


def test_lora_merge_invariant():
    cfg = TINY
    inp = make_inputs(cfg, seed=14, norm="random")
    P = O.decompress_layer(cfg, inp, 1)
    s = cfg.lora_scale
    merged = O.LayerParams({p: P.W[p] + s * P.lora[p][1] @ P.lora[p][0] for p in PROJ},
                           P.norm_attn, P.norm_mlp, {})
    x = np.random.default_rng(4).standard_normal((cfg.n_tokens, cfg.hidden))
    np.testing.assert_allclose(O.layer_forward(cfg, 1, P, x), O.layer_forward(cfg, 1, merged, x),
                               rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------------------
# P8: checkpointing is exact (Algorithm 1; Sec. 5); P10: gradient accumulation (Sec. 3)
# ---------------------------------------------------------------------------------------
def test_checkpointed_equals_stored_activations():
    cfg = TINY
    inp = make_inputs(cfg, seed=15, norm="random")
    a = O.train_step(cfg, inp)
    b = O.train_step_stored(cfg, inp)
    assert a.loss == b.loss
    assert np.array_equal(a.dx0, b.dx0)
    for ga, gb in zip(a.grads, b.grads):
        for p in ga:
            assert np.array_equal(ga[p][0], gb[p][0]) and np.array_equal(ga[p][1], gb[p][1])


def test_batch_equals_accumulated_per_sequence_grads():
    cfg = TINY  # batch 2
    inp = make_inputs(cfg, seed=16, norm="random")
    full = O.train_step(cfg, inp)
    one = cfg.with_(batch=1)
    parts = []
    for b in range(2):
        sub = make_inputs(cfg, seed=16, norm="random")
        sub.cfg = one
        sub.ids = inp.ids[b:b + 1]
        parts.append(O.train_step(one, sub))
    # the batch loss is the mean over B*(T-1) targets; each sequence has T-1
    np.testing.assert_allclose(full.loss, 0.5 * (parts[0].loss + parts[1].loss), rtol=1e-13)
    for l in range(cfg.n_layers):
        for p in full.grads[l]:
            for i in range(2):
                acc = 0.5 * (parts[0].grads[l][p][i] + parts[1].grads[l][p][i])
                np.testing.assert_allclose(full.grads[l][p][i], acc, rtol=1e-10, atol=1e-14)


# ---------------------------------------------------------------------------------------
# P11: Table 1 trainable-parameter counts
# ---------------------------------------------------------------------------------------
def test_table1_trainable_param_counts():
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "lora_param_counts.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 5
    for name, L, d, H, Hkv, dh, F, printed in rows:
        cfg = Config(name=name, n_layers=int(L), hidden=int(d), n_heads=int(H),
                     n_kv_heads=int(Hkv), head_dim=int(dh), ffn=int(F), vocab=0,
                     lora_rank=8, lora_modules=ALL7)
        # printed to 0.01M; 4.399M is printed as 4.39 and 14.967M as 14.97, so the table
        # neither truncates nor rounds consistently: require agreement within 0.01M
        assert abs(cfg.lora_param_count() / 1e6 - float(printed)) < 0.01, name
        # the nearest alternative readings are far off (rank 16 on q,k,v,o; rank 16 on all)
        alt1 = cfg.with_(lora_rank=16, lora_modules=("q", "k", "v", "o")).lora_param_count()
        alt2 = cfg.with_(lora_rank=16).lora_param_count()
        assert abs(alt1 / 1e6 - float(printed)) > 0.5 and abs(alt2 / 1e6 - float(printed)) > 0.5


# ---------------------------------------------------------------------------------------
# P12: optimizer step on the LoRA parameters (AdamW, gradient accumulation)
# ---------------------------------------------------------------------------------------
HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


def test_adamw_constant_gradient_closed_form():
    # with a constant gradient from zero moments the bias-corrected moments are exactly g
    # and g^2, so every step moves p by lr * g / (|g| + eps) (no weight decay)
    rng = np.random.default_rng(40)
    p0 = rng.standard_normal(50)
    g = rng.standard_normal(50)
    p, m, v = p0, np.zeros(50), np.zeros(50)
    hp = dict(HP, weight_decay=0.0)
    for t in range(1, 8):
        p, m, v = O.adamw_step(p, g, m, v, t, **hp)
        np.testing.assert_allclose(p, p0 - t * hp["lr"] * g / (np.abs(g) + hp["eps"]), rtol=1e-12, atol=1e-15)


def test_adamw_zero_gradient_is_pure_decay():
    rng = np.random.default_rng(41)
    p0 = rng.standard_normal(30)
    p, m, v = p0, np.zeros(30), np.zeros(30)
    for t in range(1, 6):
        p, m, v = O.adamw_step(p, np.zeros(30), m, v, t, **HP)
    np.testing.assert_allclose(p, p0 * (1 - HP["lr"] * HP["weight_decay"]) ** 5, rtol=1e-14)
    assert not m.any() and not v.any()


def test_adamw_matches_torch_adamw_several_steps():
    # an independent implementation: torch.optim.AdamW in float64 on the CPU
    import torch
    rng = np.random.default_rng(42)
    shape = (16, 24)
    p0 = rng.standard_normal(shape)
    grads = [rng.standard_normal(shape) * (0.1 + t) for t in range(6)]
    tp = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([tp], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                            weight_decay=HP["weight_decay"])
    p, m, v = p0, np.zeros(shape), np.zeros(shape)
    for t, g in enumerate(grads, start=1):
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        p, m, v = O.adamw_step(p, g, m, v, t, **HP)
        st = opt.state[tp]
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-15)


def test_adamw_grad_scale_equals_scaled_gradient():
    rng = np.random.default_rng(43)
    p, g, m = rng.standard_normal((3, 40))
    v = np.abs(rng.standard_normal(40))
    a = O.adamw_step(p, g, m, v, 3, grad_scale=0.25, **HP)
    b = O.adamw_step(p, 0.25 * g, m, v, 3, **HP)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_grad_accumulation_of_micro_batches_equals_batch_gradient():
    # two single-sequence micro-batches accumulated with scale 1/2 give the gradient of
    # the batch of both (mean loss over B*(T-1) targets)
    cfg = TINY  # batch 2
    inp = make_inputs(cfg, seed=44, norm="random")
    full = O.train_step(cfg, inp)
    one = cfg.with_(batch=1)
    acc = {}
    for b in range(2):
        sub = make_inputs(cfg, seed=44, norm="random")
        sub.cfg = one
        sub.ids = inp.ids[b:b + 1]
        res = O.train_step(one, sub)
        for l in range(cfg.n_layers):
            for p, (dA, dB) in res.grads[l].items():
                acc[l, p, 0] = O.grad_accumulate(acc.get((l, p, 0)), dA, 0.5)
                acc[l, p, 1] = O.grad_accumulate(acc.get((l, p, 1)), dB, 0.5)
    for l in range(cfg.n_layers):
        for p in full.grads[l]:
            for i in range(2):
                np.testing.assert_allclose(acc[l, p, i], full.grads[l][p][i], rtol=1e-10, atol=1e-14)


# ---------------------------------------------------------------------------------------
# P13: architecture details (Qwen2.5 QKV bias; Gemma3 QK-norm, sandwich norms, embedding
# scale): finite differences through every new term, and invariants each one implies
# ---------------------------------------------------------------------------------------
ARCH = TINY.with_(qkv_bias=True, qk_norm=True, sandwich_norm=True, embed_scale=True)


@pytest.mark.parametrize("layer", [0, 1])
def test_arch_block_backward_finite_differences(layer):
    cfg = ARCH
    inp = make_inputs(cfg, seed=60, norm="random")
    P = O.decompress_layer(cfg, inp, layer)
    rng = np.random.default_rng(61)
    x = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dy = rng.standard_normal((cfg.n_tokens, cfg.hidden))
    dx, grads = O.layer_backward(cfg, layer, P, x, dy)
    _assert_fd(lambda xx: float(np.sum(dy * O.layer_forward(cfg, layer, P, xx))), x, dx)
    for p in ("q", "k", "o", "down"):
        A, B = P.lora[p]

        def s_of_A(AA, p=p, B=B, A=A):
            P.lora[p] = (AA, B)
            try:
                return float(np.sum(dy * O.layer_forward(cfg, layer, P, x)))
            finally:
                P.lora[p] = (A, B)

        _assert_fd(s_of_A, A, grads[p][0], n_dirs=2)


def test_arch_full_step_fd_with_embedding_scale():
    cfg = ARCH
    inp = make_inputs(cfg, seed=62, norm="random")
    res = O.train_step(cfg, inp)
    E = O.decompress_embedding(cfg, inp)
    np.testing.assert_array_equal(res.ckpts[0], np.sqrt(cfg.hidden) * E[inp.ids.reshape(-1)])

    def loss_of(val):
        A, B = inp.lora[1]["k"]
        inp.lora[1]["k"] = (val, B)
        try:
            x = O.embed(E, inp.ids, np.sqrt(cfg.hidden))
            for j in range(cfg.n_layers):
                x = O.layer_forward(cfg, j, O.decompress_layer(cfg, inp, j), x)
            return O.lm_head_ce(cfg, E, inp.norm_final, x, inp.ids)[0]
        finally:
            inp.lora[1]["k"] = (A, B)

    A = np.asarray(inp.lora[1]["k"][0], np.float64)
    _assert_fd(loss_of, A, res.grads[1]["k"][0], n_dirs=2, tol=1e-5)


def test_arch_norms_remove_the_scale_of_their_input():
    # QK-norm: scaling W_q, W_k, their biases and LoRA B by c > 0 leaves the block unchanged;
    # sandwich norms: the same for W_o (with B_o) and W_down (with B_down). Without the norm
    # the output would change by O(1). (eps is made negligible against the rows' mean
    # squares, which for the small o / down outputs of the tiny block are ~1e-5.)
    cfg = ARCH.with_(batch=1, rms_eps=1e-14)
    inp = make_inputs(cfg, seed=63, norm="random")
    x = np.random.default_rng(64).standard_normal((cfg.n_tokens, cfg.hidden))
    P = O.decompress_layer(cfg, inp, 0)
    y0 = O.layer_forward(cfg, 0, P, x)
    for group in (("q", "k"), ("o",), ("down",)):
        Q = O.decompress_layer(cfg, inp, 0)
        for p in group:
            Q.W[p] = 3.0 * Q.W[p]
            Q.lora[p] = (Q.lora[p][0], 3.0 * Q.lora[p][1])
            if Q.bias is not None and p in Q.bias:
                Q.bias[p] = 3.0 * Q.bias[p]
        y = O.layer_forward(cfg, 0, Q, x)
        assert np.max(np.abs(y - y0)) < 1e-9 * np.max(np.abs(y0)), group
    # and the normed heads have the weight's RMS: with unit weights every rotated head
    # vector has squared norm dh (RoPE preserves norms), up to eps
    one = ARCH.with_(batch=1)
    inp1 = make_inputs(one, seed=65, norm="ones")
    _, cache = O.layer_forward(one, 0, O.decompress_layer(one, inp1, 0), x, keep=True)
    sq = np.sum(cache["q4d"] ** 2, axis=-1)
    np.testing.assert_allclose(sq, one.head_dim, rtol=1e-4)


def test_arch_zero_bias_equals_no_bias():
    cfg = ARCH.with_(qkv_bias=True)
    inp = make_inputs(cfg, seed=66, norm="random")
    x = np.random.default_rng(67).standard_normal((cfg.n_tokens, cfg.hidden))
    P = O.decompress_layer(cfg, inp, 1)
    P.bias = {p: np.zeros_like(b) for p, b in P.bias.items()}
    Q = O.decompress_layer(cfg.with_(qkv_bias=False), inp, 1)
    np.testing.assert_array_equal(O.layer_forward(cfg, 1, P, x), O.layer_forward(cfg, 1, Q, x))
    # a nonzero bias changes the output
    R = O.decompress_layer(cfg, inp, 1)
    assert np.max(np.abs(O.layer_forward(cfg, 1, R, x) - O.layer_forward(cfg, 1, Q, x))) > 1e-3
