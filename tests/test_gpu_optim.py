"""GPU parity of the optimizer step on the LoRA parameters (AdamW, gradient accumulation)
against the CPU fp64 oracle, through the C ABI.

Bar: both kernels are elementwise fp32 arithmetic (a dozen roundings per element for
AdamW, one or two for accumulation), so each result is within a few fp32 ulps of the
fp64 value: rel-L2 <= 1e-6 on parameters, moments and accumulated gradients. The
end-to-end step (model gradients from the HIP path) uses the model-gradient bar instead.
"""
import numpy as np
import pytest
import torch

import oracle as O
from mebp_inputs import CONFIGS, MINI, PROJ, make_inputs, make_optimizer_inputs
from paper_2510_03425_amd import _lib as L
from paper_2510_03425_amd.device import DeviceModel, make_config, stream_handle

from gpu_util import TOL, rel_l2, say

pytestmark = pytest.mark.gpu
OPT_TOL = 1e-6


def _upload(cfg, arrays, gpu):
    """arrays: per layer {proj: (A-shaped, B-shaped)} -> (torch tensors, ctypes struct array)."""
    n = len(arrays)
    st = (L.MebpLayerLoraState * n)()
    gr = (L.MebpLayerLoraGrad * n)()
    ts = []
    for l, mods in enumerate(arrays):
        td = {}
        for i, p in enumerate(PROJ):
            if p not in mods:
                continue
            a, b = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(gpu) for x in mods[p])
            td[p] = (a, b)
            st[l].A[i] = gr[l].dA[i] = a.data_ptr()
            st[l].B[i] = gr[l].dB[i] = b.data_ptr()
        ts.append(td)
    return ts, st, gr


@pytest.mark.parametrize("name", ["mini", "qwen2.5-0.5b"])
def test_adamw_parity_three_steps(built_lib, gpu, name):
    cfg = MINI if name == "mini" else CONFIGS[name]
    inp = make_inputs(cfg, seed=50, norm="random")
    opt = make_optimizer_inputs(cfg, seed=51)
    params = [{p: inp.lora[l][p] for p in inp.lora[l]} for l in range(cfg.n_layers)]
    grads = [{p: opt[l][p]["g"] for p in opt[l]} for l in range(cfg.n_layers)]
    ms = [{p: opt[l][p]["m"] for p in opt[l]} for l in range(cfg.n_layers)]
    vs = [{p: opt[l][p]["v"] for p in opt[l]} for l in range(cfg.n_layers)]
    tp, sp, _ = _upload(cfg, params, gpu)
    tg, _, sg = _upload(cfg, grads, gpu)  # the tensors must outlive the raw pointers
    tm, sm, _ = _upload(cfg, ms, gpu)
    tv, sv, _ = _upload(cfg, vs, gpu)
    ccfg = make_config(cfg)
    ref = {(l, p, k): (np.float64(params[l][p][k]), np.float64(ms[l][p][k]), np.float64(vs[l][p][k]))
           for l in range(cfg.n_layers) for p in params[l] for k in range(2)}
    steps = [dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_scale=1.0),
             dict(lr=2e-3, beta1=0.9, beta2=0.99, eps=1e-6, weight_decay=0.1, grad_scale=0.5),
             dict(lr=5e-4, beta1=0.8, beta2=0.999, eps=1e-8, weight_decay=0.0, grad_scale=2.0)]
    for t, hp in enumerate(steps, start=1):
        say("adamw", name, "step", t)
        L.mebp_lora_adamw_step(ccfg, sp, sg, sm, sv, L.MebpAdamwHparams(step=t, **hp), stream_handle())
        for (l, p, k), (rp, rm, rv) in ref.items():
            ref[l, p, k] = O.adamw_step(rp, grads[l][p][k], rm, rv, t, hp["lr"], hp["beta1"], hp["beta2"],
                                        hp["eps"], hp["weight_decay"], hp["grad_scale"])
        torch.cuda.synchronize()
        worst = 0.0
        for (l, p, k), (rp, rm, rv) in ref.items():
            for got, want in ((tp[l][p][k], rp), (tm[l][p][k], rm), (tv[l][p][k], rv)):
                e = rel_l2(got.cpu().numpy(), want)
                worst = max(worst, e)
                assert e <= OPT_TOL, (l, p, k, t, e)
        say("worst rel-L2", f"{worst:.2e}")


def test_grad_accumulate_parity(built_lib, gpu):
    cfg = MINI
    o1, o2 = make_optimizer_inputs(cfg, seed=52), make_optimizer_inputs(cfg, seed=53)
    g1 = [{p: o1[l][p]["g"] for p in o1[l]} for l in range(cfg.n_layers)]
    g2 = [{p: o2[l][p]["g"] for p in o2[l]} for l in range(cfg.n_layers)]
    acc0 = [{p: o1[l][p]["m"] for p in o1[l]} for l in range(cfg.n_layers)]  # overwritten by first=1
    t1, _, s1 = _upload(cfg, g1, gpu)  # the tensors must outlive the raw pointers
    t2, _, s2 = _upload(cfg, g2, gpu)
    ta, _, sa = _upload(cfg, acc0, gpu)
    ccfg = make_config(cfg)
    say("accumulate mini")
    L.mebp_lora_grad_accumulate(ccfg, s1, sa, 0.25, True, stream_handle())
    L.mebp_lora_grad_accumulate(ccfg, s2, sa, 0.75, False, stream_handle())
    # in place: acc aliases the gradients (a rescale of the micro-batch gradient itself)
    tg, _, sg = _upload(cfg, g2, gpu)
    L.mebp_lora_grad_accumulate(ccfg, sg, sg, 0.5, True, stream_handle())
    torch.cuda.synchronize()
    for l in range(cfg.n_layers):
        for p in g1[l]:
            for k in range(2):
                want = O.grad_accumulate(O.grad_accumulate(None, g1[l][p][k], 0.25), g2[l][p][k], 0.75)
                assert rel_l2(ta[l][p][k].cpu().numpy(), want) <= OPT_TOL
                assert rel_l2(tg[l][p][k].cpu().numpy(), O.grad_accumulate(None, g2[l][p][k], 0.5)) <= OPT_TOL


def test_optimizer_step_end_to_end_two_micro_batches(built_lib, gpu):
    """Two single-sequence micro-batches through mebp_train_step, their LoRA gradients
    accumulated with scale 1/2, one AdamW update; the same pipeline in the oracle.

    The accumulated gradient meets the model-gradient bar against the oracle's gradient of
    the whole batch. For the parameters: Adam moves each element by at most lr (for the
    first step, by lr * g / (|g| + eps)), so where the two gradients differ in sign the
    parameters differ by at most 2 lr; with lr = 1e-4 and parameters of std >= 0.02 the
    worst case is rel-L2 <= 1e-2, inside the bar."""
    cfg = MINI
    one = cfg.with_(batch=1)
    inp = make_inputs(cfg, seed=54, norm="random")
    dm = DeviceModel(inp, device=str(gpu))
    n = cfg.n_layers
    acc_t = [{p: (torch.empty_like(dm.dA[l][p]), torch.empty_like(dm.dB[l][p])) for p in dm.dA[l]} for l in range(n)]
    acc = (L.MebpLayerLoraGrad * n)()
    params = (L.MebpLayerLoraState * n)()
    m = (L.MebpLayerLoraState * n)()
    v = (L.MebpLayerLoraState * n)()
    keep = []
    for l in range(n):
        for i, p in enumerate(PROJ):
            if p not in acc_t[l]:
                continue
            acc[l].dA[i], acc[l].dB[i] = acc_t[l][p][0].data_ptr(), acc_t[l][p][1].data_ptr()
            params[l].A[i], params[l].B[i] = dm.lora[l].A[i], dm.lora[l].B[i]
            for s in (m, v):
                za, zb = torch.zeros_like(dm.dA[l][p]), torch.zeros_like(dm.dB[l][p])
                keep += [za, zb]
                s[l].A[i], s[l].B[i] = za.data_ptr(), zb.data_ptr()
    ck = dm.alloc_ckpt()
    T = cfg.seq
    ccfg = make_config(cfg)
    for b in range(2):
        say("micro-batch", b)
        L.mebp_train_step(ccfg, dm.emb, dm.base, dm.norm_final.data_ptr(), dm.lora, dm.ids.data_ptr() + 4 * b * T, 1,
                          T, ck.data_ptr(), dm.loss.data_ptr(), dm.grads, 0, dm.ws.data_ptr(), dm.ws_bytes,
                          stream_handle())
        L.mebp_lora_grad_accumulate(ccfg, dm.grads, acc, 0.5, b == 0, stream_handle())
    hp = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_scale=1.0)
    L.mebp_lora_adamw_step(ccfg, params, acc, m, v, L.MebpAdamwHparams(step=1, **hp), stream_handle())
    torch.cuda.synchronize()
    # oracle: the same pipeline in fp64
    full = O.train_step(cfg, inp, keep_ckpts=False)
    racc = {}
    for b in range(2):
        sub = make_inputs(cfg, seed=54, norm="random")
        sub.cfg = one
        sub.ids = inp.ids[b:b + 1]
        res = O.train_step(one, sub, keep_ckpts=False)
        for l in range(n):
            for p, g in res.grads[l].items():
                for k in range(2):
                    racc[l, p, k] = O.grad_accumulate(racc.get((l, p, k)), g[k], 0.5)
    errs = {}
    for (l, p, k), g in racc.items():
        np.testing.assert_allclose(g, full.grads[l][p][k], rtol=1e-9, atol=1e-13)  # oracle consistency
        errs[f"g{l}{p}{k}"] = rel_l2(acc_t[l][p][k].cpu().numpy(), g)
        p0 = np.float64(inp.lora[l][p][k])
        want, _, _ = O.adamw_step(p0, g, np.zeros_like(p0), np.zeros_like(p0), 1, **hp)
        got = params[l].A[PROJ.index(p)] if k == 0 else params[l].B[PROJ.index(p)]
        tens = [t for t in dm.keep if t.data_ptr() == got][0]
        errs[f"p{l}{p}{k}"] = rel_l2(tens.cpu().numpy(), want)
    worst = max(errs, key=errs.get)
    say("worst", worst, f"{errs[worst]:.2e}")
    for k_, e in errs.items():
        assert e <= TOL, (k_, e)
