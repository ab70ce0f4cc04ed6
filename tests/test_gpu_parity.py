"""GPU parity of the HIP path against the CPU fp64 oracle, through the C ABI.

Bar: bit-exact for int4 unpacking / decompression; rel-L2 <= 2e-2 for every 16-bit-operand,
fp32-accumulate output and gradient; exact zeros where the mathematics gives zero
(LoRA B = 0); bit-identical reruns (no atomics anywhere).
"""
import numpy as np
import pytest
import torch

import oracle as O
from mebp_inputs import CONFIGS, MINI, PROJ, layer_input, make_inputs
from paper_2510_03425_amd import _lib as L
from paper_2510_03425_amd.device import DeviceModel, slot_index

from gpu_util import ROW_TOL, TOL, max_row_rel_l2, rel_l2, say, to_np

pytestmark = pytest.mark.gpu


def _dm(inp, gpu):
    return DeviceModel(inp, device=str(gpu))


# ------------------------------------------------------------------------ decompression
@pytest.mark.parametrize("name", ["block", "mini"])
def test_dequant_bit_exact(built_lib, gpu, name):
    cfg = CONFIGS.get(name, MINI)
    inp = make_inputs(cfg, seed=0)
    mats = [(p, inp.base[0][p], cfg.proj_shape(p)) for p in PROJ]
    if inp.emb is not None:
        mats.append(("emb", inp.emb, (cfg.vocab, cfg.hidden)))
    for p, (q4, sb), (rows, cols) in mats:
        say("dequant", name, p, rows, cols)
        tq = torch.from_numpy(q4).to(gpu)
        ts = torch.from_numpy(sb.view(np.int16)).to(gpu)
        f32 = torch.empty((rows, cols), dtype=torch.float32, device=gpu)
        b16 = torch.empty((rows, cols), dtype=torch.int16, device=gpu)
        w = L.MebpQ4(q4=tq.data_ptr(), scale=ts.data_ptr())
        L.mebp_dequant_q4(w, rows, cols, 32, f32.data_ptr(), b16.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ref = O.dequant(q4, sb, cols, 32)
        np.testing.assert_array_equal(f32.cpu().numpy().astype(np.float64), ref)
        np.testing.assert_array_equal(b16.cpu().numpy().view(np.uint16), O.dequant_bf16_bits(q4, sb, cols, 32))


def test_embed_exact(built_lib, gpu):
    inp = make_inputs(MINI, seed=1)
    dm = _dm(inp, gpu)
    x0 = torch.empty((dm.N, MINI.hidden), dtype=torch.float32, device=gpu)
    say("embed mini")
    dm.embed(x0)
    torch.cuda.synchronize()
    E = O.decompress_embedding(MINI, inp)
    np.testing.assert_array_equal(x0.cpu().numpy().astype(np.float64), O.embed(E, inp.ids))


# ------------------------------------------------------------------------ one layer
LAYER_CASES = [("block", 0, "ones"), ("block", 0, "random"), ("mini", 0, "random"), ("mini", 1, "random")]


def _layer_setup(name, layer, norm, gpu, seed=0, **kw):
    cfg = CONFIGS.get(name, MINI)
    inp = make_inputs(cfg, seed=seed, norm=norm, **kw)
    x, dy = (inp.x, inp.dy) if inp.x is not None else layer_input(cfg, seed + 100)
    return cfg, inp, x, dy, _dm(inp, gpu)


def _intermediates(dm, cfg):
    N, d, F = dm.N, cfg.hidden, cfg.ffn
    qd, kvd = cfg.n_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim
    bf = torch.float16  # forward activations are fp16
    return {
        "a": dm.ws_view(slot_index("a"), bf, (N, d)), "q": dm.ws_view(slot_index("q"), bf, (N, qd)),
        "k": dm.ws_view(slot_index("k"), bf, (N, kvd)), "v": dm.ws_view(slot_index("v"), bf, (N, kvd)),
        "o": dm.ws_view(slot_index("o"), bf, (N, qd)), "h": dm.ws_view(slot_index("h"), torch.float32, (N, d)),
        "c": dm.ws_view(slot_index("c"), bf, (N, d)), "z": dm.ws_view(slot_index("z"), bf, (N, F)),
        "lse": dm.ws_view(slot_index("lse"), torch.float32, (cfg.batch, cfg.n_heads, cfg.seq)),
    }


@pytest.mark.parametrize("name,layer,norm", LAYER_CASES)
def test_layer_forward_parity(built_lib, gpu, name, layer, norm):
    cfg, inp, x, dy, dm = _layer_setup(name, layer, norm, gpu)
    tx = torch.from_numpy(x).to(gpu)
    ty = torch.empty_like(tx)
    say("layer forward", name, layer, norm)
    dm.layer_forward(layer, tx, ty)
    torch.cuda.synchronize()
    P = O.decompress_layer(cfg, inp, layer)
    y_ref, cache = O.layer_forward(cfg, layer, P, x, keep=True)
    got = _intermediates(dm, cfg)
    N = dm.N
    ref = {"a": cache["a"], "q": cache["q4d"].reshape(N, -1), "k": cache["k4d"].reshape(N, -1),
           "v": cache["v4d"].reshape(N, -1), "o": cache["O"], "h": cache["h"], "c": cache["c"], "z": cache["z"]}
    errs = {k: rel_l2(to_np(got[k]), v) for k, v in ref.items()}
    errs["y"] = rel_l2(to_np(ty), y_ref)
    rows = {k: max_row_rel_l2(to_np(got[k]), v) for k, v in ref.items()}
    rows["y"] = max_row_rel_l2(to_np(ty), y_ref)
    say("rel-L2", {k: f"{v:.2e}" for k, v in errs.items()})
    say("max row rel-L2", {k: f"{v:.2e}" for k, v in rows.items()})
    for k, e in errs.items():
        assert e <= TOL, (k, e)
    for k, e in rows.items():
        assert e <= ROW_TOL, (k, "row", e)


@pytest.mark.parametrize("name,layer,norm", LAYER_CASES)
def test_layer_backward_parity(built_lib, gpu, name, layer, norm):
    cfg, inp, x, dy, dm = _layer_setup(name, layer, norm, gpu)
    tx = torch.from_numpy(x).to(gpu)
    tdy = torch.from_numpy(dy).to(gpu)
    tdx = torch.empty_like(tx)
    say("layer backward", name, layer, norm)
    dm.layer_backward(layer, tx, tdy, tdx)
    torch.cuda.synchronize()
    P = O.decompress_layer(cfg, inp, layer)
    dx_ref, grads = O.layer_backward(cfg, layer, P, x, dy)
    errs = {"dx": rel_l2(to_np(tdx), dx_ref)}
    for p, (dA, dB) in grads.items():
        errs["dA_" + p] = rel_l2(to_np(dm.dA[layer][p]), dA)
        errs["dB_" + p] = rel_l2(to_np(dm.dB[layer][p]), dB)
    row = max_row_rel_l2(to_np(tdx), dx_ref)
    say("rel-L2", {k: f"{v:.2e}" for k, v in errs.items()}, "dx max row", f"{row:.2e}")
    for k, e in errs.items():
        assert e <= TOL, (k, e)
    assert row <= ROW_TOL, ("dx row", row)


# Larger magnitudes than the random-init inputs: the layer input scaled by 30 (the residual
# stream of a deep model), and norm weights scaled by 8 (every normalised activation 8 times
# larger: attention scores 64 times, a sharply peaked softmax, gate/up products 64 times).
@pytest.mark.parametrize("case", ["x_times_30", "norm_times_8"])
def test_layer_parity_large_magnitudes(built_lib, gpu, case):
    cfg = MINI
    inp = make_inputs(cfg, seed=21, norm="random")
    x, dy = layer_input(cfg, 121)
    if case == "x_times_30":
        x = (x * 30.0).astype(np.float32)
    else:
        inp.norm_attn = [(w * 8.0).astype(np.float32) for w in inp.norm_attn]
        inp.norm_mlp = [(w * 8.0).astype(np.float32) for w in inp.norm_mlp]
    dm = _dm(inp, gpu)
    tx, tdy = torch.from_numpy(x).to(gpu), torch.from_numpy(dy).to(gpu)
    ty, tdx = torch.empty_like(tx), torch.empty_like(tx)
    say("large magnitudes", case)
    for layer in (0, 1):
        dm.layer_forward(layer, tx, ty)
        dm.layer_backward(layer, tx, tdy, tdx)
        torch.cuda.synchronize()
        P = O.decompress_layer(cfg, inp, layer)
        y_ref = O.layer_forward(cfg, layer, P, x)
        dx_ref, grads = O.layer_backward(cfg, layer, P, x, dy)
        errs = {"y": rel_l2(to_np(ty), y_ref), "dx": rel_l2(to_np(tdx), dx_ref)}
        for p, (dA, dB) in grads.items():
            errs["dA_" + p] = rel_l2(to_np(dm.dA[layer][p]), dA)
            errs["dB_" + p] = rel_l2(to_np(dm.dB[layer][p]), dB)
        rows = {"y": max_row_rel_l2(to_np(ty), y_ref), "dx": max_row_rel_l2(to_np(tdx), dx_ref)}
        say("layer", layer, "rel-L2", {k: f"{v:.2e}" for k, v in errs.items()},
            "max row", {k: f"{v:.2e}" for k, v in rows.items()})
        for k, e in errs.items():
            assert e <= TOL, (case, layer, k, e)
        for k, e in rows.items():
            assert e <= ROW_TOL, (case, layer, k, "row", e)


# Attention head dims 128 and 256, multi-head (one query head per KV head) and grouped-query,
# at a ragged length (T = 200: not a multiple of the 32/64/128-row attention tiles) and with
# a sliding-window layer (0) and a global layer (1). These short shapes run the attention
# loops split into chunks (few tiles per head); the last case has enough tiles to run them
# whole.
HEAD_DIM_CASES = {
    "dh128_mha": MINI.with_(name="dh128_mha", hidden=256, n_heads=2, n_kv_heads=2, head_dim=128, seq=200),
    "dh128_gqa": MINI.with_(name="dh128_gqa", hidden=256, n_heads=4, n_kv_heads=1, head_dim=128, seq=200),
    "dh256_mha": MINI.with_(name="dh256_mha", hidden=256, n_heads=2, n_kv_heads=2, head_dim=256, seq=200),
    "dh256_gqa": MINI.with_(name="dh256_gqa", hidden=256, n_heads=4, n_kv_heads=2, head_dim=256, seq=200),
    # enough 64-row tiles (9 x 8 heads x 4 sequences) that no attention loop is split
    "dh64_unsplit": MINI.with_(name="dh64_unsplit", n_heads=8, n_kv_heads=2, head_dim=64, batch=4, seq=520),
    # head dim 256 unsplit (17 x 4 heads x 4 sequences, 18 x 2 x 8 tiles of 64): the 32-key
    # wave-pair dK/dV kernel, grouped (partials) and ungrouped (direct store), ragged T
    "dh256_gqa_unsplit": MINI.with_(name="dh256_gqa_unsplit", hidden=256, n_heads=4, n_kv_heads=2, head_dim=256,
                                    batch=4, seq=1040),
    "dh256_mha_unsplit": MINI.with_(name="dh256_mha_unsplit", hidden=256, n_heads=2, n_kv_heads=2, head_dim=256,
                                    batch=8, seq=1100),
}


@pytest.mark.parametrize("layer", [0, 1])
@pytest.mark.parametrize("name", list(HEAD_DIM_CASES))
def test_layer_head_dims_parity(built_lib, gpu, name, layer):
    _layer_parity(HEAD_DIM_CASES[name], layer, gpu, name)


# The forward pass's gate/up product with z = act(g) * u formed in its epilogue (the
# large-tile kernel: 8192 tokens, 256 x 256 tiles) at an FFN width that is no multiple of its
# 128-feature column tile: 688 = 5 x 128 + 48, so in the last tile the first gate / up wave
# pair holds 48 of its 64 features and the second none.
RAGGED_FFN = MINI.with_(name="ragged_ffn", hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=688, batch=4,
                        seq=2048)


def test_layer_parity_fused_activation_ragged_ffn(built_lib, gpu):
    _layer_parity(RAGGED_FFN, 0, gpu, "ragged_ffn", rows=True)


def _layer_parity(cfg, layer, gpu, name, rows=False):
    inp = make_inputs(cfg, seed=7, norm="random")
    x, dy = layer_input(cfg, 107)
    dm = _dm(inp, gpu)
    tx, tdy = torch.from_numpy(x).to(gpu), torch.from_numpy(dy).to(gpu)
    ty, tdx = torch.empty_like(tx), torch.empty_like(tx)
    say("layer case", name, "layer", layer, "window", cfg.layer_window(layer))
    dm.layer_forward(layer, tx, ty)
    dm.layer_backward(layer, tx, tdy, tdx)
    torch.cuda.synchronize()
    P = O.decompress_layer(cfg, inp, layer)
    y_ref = O.layer_forward(cfg, layer, P, x)
    dx_ref, grads = O.layer_backward(cfg, layer, P, x, dy)
    errs = {"y": rel_l2(to_np(ty), y_ref), "dx": rel_l2(to_np(tdx), dx_ref)}
    for p, (dA, dB) in grads.items():
        errs["dA_" + p] = rel_l2(to_np(dm.dA[layer][p]), dA)
        errs["dB_" + p] = rel_l2(to_np(dm.dB[layer][p]), dB)
    say("rel-L2", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL, (k, e)
    if rows:
        row = {"y": max_row_rel_l2(to_np(ty), y_ref), "dx": max_row_rel_l2(to_np(tdx), dx_ref)}
        say("max row rel-L2", {k: f"{v:.2e}" for k, v in row.items()})
        for k, e in row.items():
            assert e <= ROW_TOL, (k, "row", e)


def test_dx_may_alias_dy(built_lib, gpu):
    cfg, inp, x, dy, dm = _layer_setup("mini", 0, "random", gpu)
    tx = torch.from_numpy(x).to(gpu)
    tdy = torch.from_numpy(dy).to(gpu)
    tdx = torch.empty_like(tx)
    say("alias dx=dy mini")
    dm.layer_backward(0, tx, tdy, tdx)
    g = tdy.clone()
    dm.layer_backward(0, tx, g, g)
    torch.cuda.synchronize()
    assert torch.equal(g, tdx)


def test_lora_b_zero_invariant(built_lib, gpu):
    cfg, inp, x, dy, dm = _layer_setup("mini", 1, "random", gpu, lora_b_zero=True)
    tx = torch.from_numpy(x).to(gpu)
    ty = torch.empty_like(tx)
    say("B=0 forward/backward mini")
    dm.layer_forward(1, tx, ty)
    base = DeviceModel(make_inputs(MINI.with_(lora_modules=()), seed=0, norm="random"), device=str(gpu))
    ty0 = torch.empty_like(tx)
    base.layer_forward(1, tx, ty0)
    dm.layer_backward(1, tx, torch.from_numpy(dy).to(gpu), None)
    torch.cuda.synchronize()
    assert torch.equal(ty, ty0)  # adapter output exactly zero
    for p in PROJ:
        assert torch.count_nonzero(dm.dA[1][p]).item() == 0, p
        assert torch.count_nonzero(dm.dB[1][p]).item() > 0, p


def test_deterministic_and_recompute_equals_forward(built_lib, gpu):
    cfg, inp, x, dy, dm = _layer_setup("mini", 0, "random", gpu)
    tx = torch.from_numpy(x).to(gpu)
    tdy = torch.from_numpy(dy).to(gpu)
    y1, y2 = torch.empty_like(tx), torch.empty_like(tx)
    say("determinism mini")
    dm.layer_forward(0, tx, y1)
    fwd = {k: v.clone() for k, v in _intermediates(dm, cfg).items()}
    dm.layer_forward(0, tx, y2)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    dx1, dx2 = torch.empty_like(tx), torch.empty_like(tx)
    dm.layer_backward(0, tx, tdy, dx1)
    rec = {k: v.clone() for k, v in _intermediates(dm, cfg).items()}
    g1 = {p: (dm.dA[0][p].clone(), dm.dB[0][p].clone()) for p in PROJ}
    dm.layer_backward(0, tx, tdy, dx2)
    torch.cuda.synchronize()
    assert torch.equal(dx1, dx2)
    for p in PROJ:
        assert torch.equal(g1[p][0], dm.dA[0][p]) and torch.equal(g1[p][1], dm.dB[0][p])
    # the recompute inside backward reproduces the stored forward's intermediates bit for bit
    for k in fwd:
        assert torch.equal(fwd[k], rec[k]), k


# ------------------------------------------------------------------------ LM head, full step
def test_lm_head_parity(built_lib, gpu):
    cfg = MINI
    inp = make_inputs(cfg, seed=3, norm="random")
    dm = _dm(inp, gpu)
    xL = np.random.default_rng(5).standard_normal((dm.N, cfg.hidden)).astype(np.float32)
    tx = torch.from_numpy(xL).to(gpu)
    tdx = torch.empty_like(tx)
    say("lm head mini")
    dm.lm_head(tx, tdx)
    torch.cuda.synchronize()
    E = O.decompress_embedding(cfg, inp)
    loss, dx = O.lm_head_ce(cfg, E, inp.norm_final, xL, inp.ids)
    row = max_row_rel_l2(to_np(tdx), dx)
    say("loss", dm.loss.item(), loss, "dx rel-L2", rel_l2(to_np(tdx), dx), "max row", row)
    assert abs(dm.loss.item() - loss) <= 1e-3 * abs(loss)
    assert rel_l2(to_np(tdx), dx) <= TOL
    assert row <= ROW_TOL
    # rows without a target (last position of each sequence) get exactly zero gradient
    assert torch.count_nonzero(tdx.view(cfg.batch, cfg.seq, -1)[:, -1]).item() == 0


# Logits far from the random-init regime. "wide": final-norm weight 45, so the logits have a
# standard deviation near 10 and row maxima near 35. "peaked": half of the rows are the
# decompressed embedding row of their own target (plus noise) and the final-norm weight is
# 4.75, which gives the target a probability near 0.99; the gradient of such a row is the
# small difference (P - onehot) E, where cancellation shows any rounding of the target term.
@pytest.mark.parametrize("case", ["wide", "peaked"])
def test_lm_head_parity_large_and_peaked_logits(built_lib, gpu, case):
    cfg = MINI
    inp = make_inputs(cfg, seed=33, norm="random")
    rng = np.random.default_rng(34)
    N, T = cfg.n_tokens, cfg.seq
    xL = rng.standard_normal((N, cfg.hidden)).astype(np.float32)
    E = O.decompress_embedding(cfg, inp)
    tgt = np.full(N, -1)
    tgt.reshape(cfg.batch, T)[:, :-1] = inp.ids[:, 1:]
    if case == "wide":
        inp.norm_final = np.full(cfg.hidden, 45.0, np.float32)
    else:
        inp.norm_final = np.full(cfg.hidden, 4.75, np.float32)
        rows = np.nonzero((tgt >= 0) & (np.arange(N) % 2 == 0))[0]
        xL[rows] = (E[tgt[rows]] * 50.0 + 0.05 * rng.standard_normal((rows.size, cfg.hidden))).astype(np.float32)
    dm = _dm(inp, gpu)
    tx = torch.from_numpy(xL).to(gpu)
    tdx = torch.empty_like(tx)
    say("lm head", case)
    dm.lm_head(tx, tdx)
    torch.cuda.synchronize()
    loss, dx = O.lm_head_ce(cfg, E, inp.norm_final, xL, inp.ids)
    if case == "peaked":
        z = O.lm_head_logits(cfg, E, inp.norm_final, xL[rows])
        p = np.exp(z - z.max(1, keepdims=True))
        pt = (p / p.sum(1, keepdims=True))[np.arange(rows.size), tgt[rows]]
        say("target probability of the peaked rows: median", float(np.median(pt)), "min", float(pt.min()))
        assert np.median(pt) > 0.95
    err, row = rel_l2(to_np(tdx), dx), max_row_rel_l2(to_np(tdx), dx)
    say("loss", dm.loss.item(), loss, "dx rel-L2", f"{err:.2e}", "max row", f"{row:.2e}")
    assert abs(dm.loss.item() - loss) <= 1e-3 * abs(loss)
    assert err <= TOL
    assert row <= ROW_TOL


def _step_parity(cfg, inp, gpu, ref=None):
    dm = _dm(inp, gpu)
    dx0 = torch.empty((dm.N, cfg.hidden), dtype=torch.float32, device=gpu)
    say("train step", cfg.name)
    dm.train_step(dx0)
    torch.cuda.synchronize()
    if ref is None:
        ref = O.train_step(cfg, inp)
    errs = {"dx0": rel_l2(to_np(dx0), ref.dx0)}
    for l in range(cfg.n_layers):
        for p, (dA, dB) in ref.grads[l].items():
            errs[f"dA{l}_{p}"] = rel_l2(to_np(dm.dA[l][p]), dA)
            errs[f"dB{l}_{p}"] = rel_l2(to_np(dm.dB[l][p]), dB)
    if ref.ckpts:
        for l in range(cfg.n_layers + 1):
            errs[f"ckpt{l}"] = rel_l2(to_np(dm.ckpt[l]), ref.ckpts[l])
    worst = max(errs, key=errs.get)
    say("loss", dm.loss.item(), ref.loss, "worst", worst, f"{errs[worst]:.2e}")
    assert abs(dm.loss.item() - ref.loss) <= 1e-3 * abs(ref.loss)
    for k, e in errs.items():
        assert e <= TOL, (k, e)
    return dm


def test_train_step_parity_mini(built_lib, gpu):
    _step_parity(MINI, make_inputs(MINI, seed=4, norm="random"), gpu)


def test_train_step_parity_qwen05b(built_lib, gpu):
    cfg = CONFIGS["qwen2.5-0.5b"]
    _step_parity(cfg, make_inputs(cfg, seed=0), gpu)


def test_train_step_parity_gemma1b(built_lib, gpu):
    # 26 layers with the 5 local : 1 global pattern, GeGLU, head_dim 256, one KV head,
    # LoRA r16, V = 262144: the whole step against the fp64 oracle
    cfg = CONFIGS["gemma3-1b"]
    _step_parity(cfg, make_inputs(cfg, seed=0), gpu)


def test_hip_graph_replay_matches_eager(built_lib, gpu):
    """The whole step captured as one HIP graph and replayed several times (with eager
    work and synchronisations between replays) reproduces the eager step bit for bit."""
    cfg = MINI
    inp = make_inputs(cfg, seed=6, norm="random")
    dm = _dm(inp, gpu)
    dx0 = torch.empty((dm.N, cfg.hidden), dtype=torch.float32, device=gpu)
    say("graph replay mini: eager reference")
    dm.train_step(dx0)
    torch.cuda.synchronize()
    ref_loss = dm.loss.clone()
    ref_dx = dx0.clone()
    ref = {(l, p): (dm.dA[l][p].clone(), dm.dB[l][p].clone()) for l in range(cfg.n_layers) for p in PROJ}
    s_cap = torch.cuda.Stream()
    s_cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s_cap):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s_cap):
            dm.train_step(dx0)
    torch.cuda.current_stream().wait_stream(s_cap)
    torch.cuda.synchronize()
    for rep in range(3):
        dx0.zero_()
        dm.loss.zero_()
        for (l, p) in ref:
            dm.dA[l][p].zero_()
        torch.cuda.synchronize()
        say("graph replay", rep)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dm.loss, ref_loss)
        assert torch.equal(dx0, ref_dx)
        for (l, p), (a, b) in ref.items():
            assert torch.equal(dm.dA[l][p], a) and torch.equal(dm.dB[l][p], b)
        dm.layer_forward(0, dm.ckpt[0].clone(), torch.empty_like(dm.ckpt[0]))  # eager work in between


# ------------------------------------------------------------------------ degenerate shapes
# One token per sequence (attention over a single key; 3 rows in every GEMM), a window of one
# (each query sees only itself), multi-head attention without grouping, a single-layer model,
# and the shortest sequence a training step allows (T = 2: one target per sequence).
DEGENERATE = {
    "T1": MINI.with_(name="T1", seq=1, batch=3),
    "window1": MINI.with_(name="window1", window=1, seq=70),
    "mha": MINI.with_(name="mha", n_kv_heads=4, seq=90),
}


@pytest.mark.parametrize("name", list(DEGENERATE))
def test_layer_degenerate_shapes(built_lib, gpu, name):
    cfg = DEGENERATE[name]
    inp = make_inputs(cfg, seed=80, norm="random")
    x, dy = layer_input(cfg, 180)
    dm = _dm(inp, gpu)
    tx, tdy = torch.from_numpy(x).to(gpu), torch.from_numpy(dy).to(gpu)
    ty, tdx = torch.empty_like(tx), torch.empty_like(tx)
    say("degenerate layer", name, "B", cfg.batch, "T", cfg.seq)
    dm.layer_forward(0, tx, ty)
    dm.layer_backward(0, tx, tdy, tdx)
    torch.cuda.synchronize()
    P = O.decompress_layer(cfg, inp, 0)
    y_ref = O.layer_forward(cfg, 0, P, x)
    dx_ref, grads = O.layer_backward(cfg, 0, P, x, dy)
    errs = {"y": rel_l2(to_np(ty), y_ref), "dx": rel_l2(to_np(tdx), dx_ref)}
    zero = ("q", "k") if cfg.window == 1 else ()
    for p, (dA, dB) in grads.items():
        if p in zero:
            continue
        errs["dA_" + p] = rel_l2(to_np(dm.dA[0][p]), dA)
        errs["dB_" + p] = rel_l2(to_np(dm.dB[0][p]), dB)
    say("rel-L2", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL, (k, e)
    # window 1: each query attends only to itself, the softmax is identically 1 and its
    # gradient vanishes, so q and k get exactly zero gradient. The HIP path computes
    # dS = P (dP - delta) from two separately rounded products; what remains must stay
    # within the parity bar measured against the scale of the v gradients.
    for p in zero:
        for i, t in enumerate((dm.dA[0][p], dm.dB[0][p])):
            ref_scale = np.linalg.norm(grads["v"][i])
            got = np.linalg.norm(to_np(t))
            say("window-1 zero gradient", p, i, f"{got / ref_scale:.2e} of the v gradient")
            assert np.linalg.norm(grads[p][i]) <= 1e-10 * ref_scale  # the oracle's is zero up to fp64 rounding
            assert got <= TOL * ref_scale


def test_train_step_shortest_sequence_one_layer(built_lib, gpu):
    cfg = MINI.with_(name="T2", seq=2, batch=2, n_layers=1)
    _step_parity(cfg, make_inputs(cfg, seed=81, norm="random"), gpu)
