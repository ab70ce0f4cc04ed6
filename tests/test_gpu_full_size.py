"""GPU parity at the full sizes of the model-shaped workloads (Gemma3-1B, Qwen2.5-1.5B and
Gemma3-4B shapes), in the launch configuration the benchmark uses: the same batch, sequence
length and widths, hence the same tile counts, split-K factors and attention grids.

The fp64 oracle cannot run a whole batch of these sizes in a test, so each check relies on a
property that makes a small oracle computation exact for the quantity compared:

* sequences are independent: the layer forward of the last sequence of the batch (all T
  rows, every column) is compared with the oracle run on that sequence alone;
* with an upstream gradient that is zero outside that sequence, the layer backward gives
  exactly zero dx on every other row, and its dx rows and every LoRA gradient equal the
  oracle's for the single sequence (the other rows contribute exact zeros to the sums);
* each row's LM-head loss term and input gradient depend on that row alone: sampled rows
  (first, middle and last positions of several sequences) are compared, and the loss is
  checked to be the mean of the per-row terms.

The Qwen2.5-0.5B shape is covered by the whole-step parity test.
"""
import numpy as np
import pytest
import torch

import oracle as O
from mebp_inputs import CONFIGS, make_inputs
from paper_2510_03425_amd.device import DeviceModel, slot_index

from gpu_util import ROW_TOL, TOL, max_row_rel_l2, rel_l2, say, to_np

pytestmark = pytest.mark.gpu

FULL = ["gemma3-1b", "qwen2.5-1.5b", "gemma3-4b"]


def _layers_to_test(cfg):
    # a local (sliding-window) and a global layer where the model has both
    if cfg.global_every:
        return [0, cfg.global_every - 1]
    return [0]


@pytest.mark.parametrize("name", FULL)
def test_layer_full_size(built_lib, gpu, name):
    cfg = CONFIGS[name].with_(vocab=0)
    layers = _layers_to_test(cfg)
    say("draw layers", name, "B", cfg.batch, "T", cfg.seq, "layers", layers)
    inp = make_inputs(cfg, seed=0, norm="random", n_layers=max(layers) + 1)
    dm = DeviceModel(inp, device=str(gpu))
    T, B, N = cfg.seq, cfg.batch, cfg.n_tokens
    b = B - 1
    rows = slice(b * T, (b + 1) * T)
    rows0 = slice(0, T)
    tx = torch.from_numpy(inp.x).to(gpu)
    dy = np.zeros_like(inp.dy)
    dy[rows] = inp.dy[rows]
    tdy = torch.from_numpy(dy).to(gpu)
    one = cfg.with_(batch=1)
    for l in layers:
        ty = torch.empty_like(tx)
        tdx = torch.empty_like(tx)
        say("layer", l, "forward + backward on GPU")
        dm.layer_forward(l, tx, ty)
        dm.layer_backward(l, tx, tdy, tdx)
        torch.cuda.synchronize()
        P = O.decompress_layer(cfg, inp, l)
        y_ref, cache = O.layer_forward(one, l, P, inp.x[rows], keep=True)
        dx_ref, grads = O.layer_backward(one, l, P, inp.x[rows], inp.dy[rows], cache=cache)
        dx = to_np(tdx)
        y = to_np(ty)
        # the first sequence's forward as well (other token tiles of the same launch)
        y0_ref = O.layer_forward(one, l, P, inp.x[rows0])
        errs = {"y": rel_l2(y[rows], y_ref), "y_first": rel_l2(y[rows0], y0_ref), "dx": rel_l2(dx[rows], dx_ref)}
        for p, (dA, dB) in grads.items():
            errs["dA_" + p] = rel_l2(to_np(dm.dA[l][p]), dA)
            errs["dB_" + p] = rel_l2(to_np(dm.dB[l][p]), dB)
        row = {"y": max_row_rel_l2(y[rows], y_ref), "y_first": max_row_rel_l2(y[rows0], y0_ref),
               "dx": max_row_rel_l2(dx[rows], dx_ref)}
        say("layer", l, "rel-L2", {k: f"{v:.2e}" for k, v in errs.items()},
            "max row", {k: f"{v:.2e}" for k, v in row.items()})
        for k, e in errs.items():
            assert e <= TOL, (name, l, k, e)
        for k, e in row.items():
            assert e <= ROW_TOL, (name, l, k, "row", e)
        other = np.ones(N, bool)
        other[rows] = False
        assert np.count_nonzero(dx[other]) == 0, "dx must be exactly zero outside the sequence"


@pytest.mark.parametrize("name", FULL)
def test_lm_head_full_size_sampled_rows(built_lib, gpu, name):
    cfg = CONFIGS[name]
    say("draw embedding", name, "V", cfg.vocab, "N", cfg.n_tokens)
    inp = make_inputs(cfg, seed=1, norm="random", n_layers=0)
    dm = DeviceModel(inp, device=str(gpu))
    N, T = cfg.n_tokens, cfg.seq
    xL = np.random.default_rng(2).standard_normal((N, cfg.hidden)).astype(np.float32)
    tx = torch.from_numpy(xL).to(gpu)
    tdx = torch.empty_like(tx)
    say("lm head on GPU")
    dm.lm_head(tx, tdx)
    torch.cuda.synchronize()
    row_loss = dm.ws_view(slot_index("ce_row_loss"), torch.float32, (N,)).cpu().numpy().astype(np.float64)
    n = cfg.batch * (T - 1)
    tgt = np.full(N, -1)
    tgt.reshape(cfg.batch, T)[:, :-1] = inp.ids[:, 1:]
    seqs = sorted({0, cfg.batch // 2, cfg.batch - 1})
    rows = np.array([b * T + t for b in seqs for t in (0, 1, T // 2, T - 2, T - 1)])
    E = O.decompress_embedding(cfg, inp)
    rl_ref, dx_ref = O.lm_head_ce_rows(cfg, E, inp.norm_final, xL[rows], tgt[rows], n)
    dx = to_np(tdx)
    err_dx = rel_l2(dx[rows], dx_ref)
    row_dx = max_row_rel_l2(dx[rows], dx_ref)
    err_rl = np.max(np.abs(row_loss[rows] - rl_ref) / np.maximum(np.abs(rl_ref), 1.0))
    loss = dm.loss.item()
    say("rows", rows.tolist(), "dx rel-L2", f"{err_dx:.2e}", "row-loss max rel err", f"{err_rl:.2e}", "loss", loss)
    assert err_dx <= TOL
    assert row_dx <= ROW_TOL, row_dx
    assert err_rl <= 1e-3
    # the loss is the mean of the per-row terms over the B*(T-1) target positions
    assert abs(loss - row_loss.sum() / n) <= 1e-4 * abs(loss)
    # rows without a target (last position) have exactly zero loss term and gradient
    last = np.arange(cfg.batch) * T + T - 1
    assert np.all(row_loss[last] == 0) and np.count_nonzero(dx[last]) == 0
    # random init: logits are ~N(0, s2) with s2 = 0.02^2 * d * mean(w^2), so the loss is
    # close to ln V + s2 / 2
    s2 = 0.02 ** 2 * cfg.hidden * float(np.mean(np.square(inp.norm_final, dtype=np.float64)))
    assert abs(loss - (np.log(cfg.vocab) + s2 / 2)) < 0.15
