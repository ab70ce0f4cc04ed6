"""Checkpoint offload (mebp_train_step_offload): the checkpoints go to pinned host memory
through a device ring and come back for the reverse loop. The kernels and their order
are those of mebp_train_step, so every result must be bit-identical to it (and through
it to the oracle, which the whole-step parity tests check): loss, every LoRA gradient,
the layer-0 input gradient, and the host checkpoints equal the device checkpoints."""
import pytest
import torch

from mebp_inputs import CONFIGS, MINI, PROJ, make_inputs
from paper_2510_03425_amd.device import DeviceModel

from gpu_util import say

pytestmark = pytest.mark.gpu


def _run_both(cfg, gpu, slots, seed=0):
    inp = make_inputs(cfg, seed=seed, norm="random")
    dm = DeviceModel(inp, device=str(gpu))
    N, d = dm.N, cfg.hidden
    dx_a = torch.empty((N, d), dtype=torch.float32, device=gpu)
    dx_b = torch.empty_like(dx_a)
    say("offload", cfg.name, "layers", cfg.n_layers, "slots", slots, ": reference step")
    dm.train_step(dx_a)
    torch.cuda.synchronize()
    ref = {"loss": dm.loss.clone(), "ckpt": dm.ckpt.clone()}
    ref_g = {(l, p): (dm.dA[l][p].clone(), dm.dB[l][p].clone()) for l in range(cfg.n_layers) for p in dm.dA[l]}
    host = torch.empty((cfg.n_layers + 1, N, d), dtype=torch.float32).pin_memory()
    ring = torch.empty((slots, N, d), dtype=torch.float32, device=gpu)
    for (l, p) in ref_g:
        dm.dA[l][p].zero_()
        dm.dB[l][p].zero_()
    dm.loss.zero_()
    torch.cuda.synchronize()
    say("offload step")
    dm.train_step_offload(host, ring, dx_b)
    torch.cuda.synchronize()
    return dm, ref, ref_g, host, ring, dx_a, dx_b


def _check_equal(dm, ref, ref_g, host, dx_a, dx_b):
    assert torch.equal(dm.loss, ref["loss"])
    assert torch.equal(dx_a, dx_b)
    for (l, p), (a, b) in ref_g.items():
        assert torch.equal(dm.dA[l][p], a) and torch.equal(dm.dB[l][p], b), (l, p)
    assert torch.equal(host, ref["ckpt"].cpu())


@pytest.mark.parametrize("layers,slots", [(7, 4), (2, 4), (9, 5)])
def test_offload_bit_identical_mini(built_lib, gpu, layers, slots):
    cfg = MINI.with_(n_layers=layers)
    dm, ref, ref_g, host, ring, dx_a, dx_b = _run_both(cfg, gpu, slots)
    _check_equal(dm, ref, ref_g, host, dx_a, dx_b)


def test_offload_bit_identical_qwen05b(built_lib, gpu):
    cfg = CONFIGS["qwen2.5-0.5b"]
    dm, ref, ref_g, host, ring, dx_a, dx_b = _run_both(cfg, gpu, 4)
    _check_equal(dm, ref, ref_g, host, dx_a, dx_b)


def test_offload_graph_replay(built_lib, gpu):
    """The offload step captured as a HIP graph (copy nodes included) and replayed three
    times, with eager work between replays, reproduces the eager step."""
    cfg = MINI.with_(n_layers=6)
    dm, ref, ref_g, host, ring, dx_a, dx_b = _run_both(cfg, gpu, 4, seed=3)
    _check_equal(dm, ref, ref_g, host, dx_a, dx_b)
    s_cap = torch.cuda.Stream()
    s_cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s_cap):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s_cap):
            dm.train_step_offload(host, ring, dx_b)
    torch.cuda.current_stream().wait_stream(s_cap)
    torch.cuda.synchronize()
    for rep in range(3):
        host.zero_()
        ring.zero_()
        dx_b.zero_()
        dm.loss.zero_()
        for (l, p) in ref_g:
            dm.dA[l][p].zero_()
        torch.cuda.synchronize()
        say("offload graph replay", rep)
        g.replay()
        torch.cuda.synchronize()
        _check_equal(dm, ref, ref_g, host, dx_a, dx_b)
        dm.train_step(dx_a)  # eager work in between
        torch.cuda.synchronize()
