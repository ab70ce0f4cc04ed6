"""The entry point for callers that cannot allocate (mebp_layer_recompute_backward_static):
its scratch is the library's own per-device buffer instead of a caller workspace. It must
give exactly what mebp_layer_recompute_backward gives with a workspace (same kernels, same
order), and the oracle's result within the parity bar, on consecutive calls of different
sizes (the buffer keeps the previous call's contents), and refuse a layer that does not fit.
"""
import numpy as np
import pytest
import torch

import oracle as O
from mebp_inputs import CONFIGS, MINI, layer_input, make_inputs
from paper_2510_03425_amd import _lib as L
from paper_2510_03425_amd.device import DeviceModel, ptr, stream_handle

from gpu_util import TOL, rel_l2, say, to_np

pytestmark = pytest.mark.gpu


def _case(cfg, seed):
    inp = make_inputs(cfg, seed=seed, norm="random")
    x, dy = layer_input(cfg, seed + 100)
    return inp, x, dy


def _grads_of(dm, layer):
    return {p: (dm.dA[layer][p].clone(), dm.dB[layer][p].clone()) for p in dm.dA[layer]}


def test_static_scratch_layer_backward_matches_workspace_call(built_lib, gpu):
    # first call: the mini model (2 sequences of 160 tokens), then a smaller one (1 x 96)
    cases = [(MINI, 1, 41), (MINI.with_(name="mini_small", batch=1, seq=96), 0, 42)]
    for cfg, layer, seed in cases:
        inp, x, dy = _case(cfg, seed)
        dm = DeviceModel(inp, device=str(gpu))
        tx, tdy = torch.from_numpy(x).to(gpu), torch.from_numpy(dy).to(gpu)
        dx_ws, dx_st = torch.empty_like(tx), torch.full_like(tx, float("nan"))
        say("workspace call", cfg.name, "B", cfg.batch, "T", cfg.seq, "layer", layer)
        dm.layer_backward(layer, tx, tdy, dx_ws)
        torch.cuda.synchronize()
        ref = _grads_of(dm, layer)
        for p in dm.dA[layer]:  # poison the outputs before the second call
            dm.dA[layer][p].fill_(float("nan"))
            dm.dB[layer][p].fill_(float("nan"))
        say("static-scratch call", cfg.name)
        L.mebp_layer_recompute_backward_static(dm.ccfg, layer, dm.base[layer], dm.lora[layer], ptr(tx), ptr(tdy),
                                               ptr(dx_st), dm.grads[layer], dm.B, dm.T, stream_handle())
        torch.cuda.synchronize()
        assert torch.equal(dx_st, dx_ws)
        for p, (a, b) in ref.items():
            assert torch.equal(dm.dA[layer][p], a) and torch.equal(dm.dB[layer][p], b), p
        # and the oracle, at the parity bar
        P = O.decompress_layer(cfg, inp, layer)
        dx_ref, grads = O.layer_backward(cfg, layer, P, x, dy)
        errs = {"dx": rel_l2(to_np(dx_st), dx_ref)}
        for p, (dA, dB) in grads.items():
            errs["dA_" + p] = rel_l2(to_np(dm.dA[layer][p]), dA)
            errs["dB_" + p] = rel_l2(to_np(dm.dB[layer][p]), dB)
        say("rel-L2", {k: f"{v:.2e}" for k, v in errs.items()})
        for k, e in errs.items():
            assert e <= TOL, (cfg.name, k, e)


def test_static_scratch_refuses_a_layer_that_does_not_fit(built_lib, gpu):
    cfg = CONFIGS["gemma3-1b"].with_(vocab=0)
    inp = make_inputs(cfg.with_(n_layers=1), seed=0, n_layers=1)
    dm = DeviceModel(inp, device=str(gpu))
    x = torch.zeros((dm.N, cfg.hidden), dtype=torch.float32, device=gpu)
    r = L.mebp_layer_recompute_backward_static(dm.ccfg, 0, dm.base[0], dm.lora[0], ptr(x), ptr(x), 0, dm.grads[0],
                                               dm.B, dm.T, stream_handle(), check=False)
    assert r == L.MEBP_EWORKSPACE, r
    assert "scratch" in L.mebp_last_error()
