"""GPU parity of the architecture options (Qwen2.5 QKV bias; Gemma3 per-head QK-norm,
sandwich norms, embedding scale) against the CPU fp64 oracle, through the C ABI: single
layers (forward output, dx, every LoRA gradient) at ragged sizes, sliding-window and
global layers, and whole training steps. Same bar as the plain block (rel-L2 <= 2e-2)."""
import numpy as np
import pytest
import torch

import oracle as O
from mebp_inputs import MINI, layer_input, make_inputs
from paper_2510_03425_amd.device import DeviceModel

from gpu_util import TOL, rel_l2, say, to_np

pytestmark = pytest.mark.gpu

ALL = dict(qkv_bias=True, qk_norm=True, sandwich_norm=True, embed_scale=True)
QWEN = dict(qkv_bias=True)
GEMMA = dict(qk_norm=True, sandwich_norm=True, embed_scale=True)
CASES = {
    "all_dh64": MINI.with_(name="arch_all", **ALL),
    "qwen_dh128": MINI.with_(name="arch_qwen", hidden=256, n_heads=4, n_kv_heads=2, head_dim=128, seq=200,
                             act="silu", **QWEN),
    "gemma_dh256": MINI.with_(name="arch_gemma", hidden=256, n_heads=4, n_kv_heads=1, head_dim=256, seq=200,
                              **GEMMA),
}


@pytest.mark.parametrize("layer", [0, 1])
@pytest.mark.parametrize("name", list(CASES))
def test_arch_layer_parity(built_lib, gpu, name, layer):
    cfg = CASES[name]
    inp = make_inputs(cfg, seed=70, norm="random")
    x, dy = layer_input(cfg, 170)
    dm = DeviceModel(inp, device=str(gpu))
    tx, tdy = torch.from_numpy(x).to(gpu), torch.from_numpy(dy).to(gpu)
    ty, tdx = torch.empty_like(tx), torch.empty_like(tx)
    say("arch layer", name, layer)
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


@pytest.mark.parametrize("name", ["all_dh64", "gemma_dh256"])
def test_arch_train_step_parity(built_lib, gpu, name):
    cfg = CASES[name].with_(n_layers=3)
    inp = make_inputs(cfg, seed=71, norm="random")
    dm = DeviceModel(inp, device=str(gpu))
    dx0 = torch.empty((dm.N, cfg.hidden), dtype=torch.float32, device=gpu)
    say("arch train step", name)
    dm.train_step(dx0)
    torch.cuda.synchronize()
    ref = O.train_step(cfg, inp)
    errs = {"dx0": rel_l2(to_np(dx0), ref.dx0)}
    for l in range(cfg.n_layers):
        for p, (dA, dB) in ref.grads[l].items():
            errs[f"dA{l}_{p}"] = rel_l2(to_np(dm.dA[l][p]), dA)
            errs[f"dB{l}_{p}"] = rel_l2(to_np(dm.dB[l][p]), dB)
        errs[f"ckpt{l + 1}"] = rel_l2(to_np(dm.ckpt[l + 1]), ref.ckpts[l + 1])
    # the embedding output is exact (scale sqrt(d) applied in fp32 to exact int4 values;
    # within one rounding of the fp64 value)
    np.testing.assert_allclose(to_np(dm.ckpt[0]), ref.ckpts[0], rtol=2 ** -23, atol=0)
    worst = max(errs, key=errs.get)
    say("loss", dm.loss.item(), ref.loss, "worst", worst, f"{errs[worst]:.2e}")
    assert abs(dm.loss.item() - ref.loss) <= 1e-3 * abs(ref.loss)
    for k, e in errs.items():
        assert e <= TOL, (k, e)
