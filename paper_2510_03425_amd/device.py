"""Device-memory plumbing for the C ABI: uploads a model's compressed weights, LoRA
adapters and token ids into torch tensors on the GPU, fills the ABI structs with their
addresses, owns the workspace, and calls the entry points on torch's current stream.

PyTorch is used only for device allocations and the stream handle; every step of the
training step runs inside ``libmebp.so``.
"""
from __future__ import annotations

import ctypes as C
from typing import List, Optional

import numpy as np
import torch

from mebp_inputs import PROJ, Config, Inputs

from . import _lib as L

ACT_CODE = {"silu": 0, "gelu_tanh": 1}


def make_config(cfg: Config) -> L.MebpConfig:
    return L.MebpConfig(
        n_layers=cfg.n_layers, hidden=cfg.hidden, n_heads=cfg.n_heads, n_kv_heads=cfg.n_kv_heads,
        head_dim=cfg.head_dim, ffn=cfg.ffn, vocab=cfg.vocab, act=ACT_CODE[cfg.act], rms_eps=cfg.rms_eps,
        rope_theta_global=cfg.rope_theta_global, rope_theta_local=cfg.rope_theta_local,
        window=cfg.window, global_every=cfg.global_every, group=cfg.group, lora_rank=cfg.lora_rank,
        lora_alpha=cfg.lora_alpha, lora_mask=cfg.lora_mask(), arch=cfg.arch_flags)


def stream_handle() -> int:
    return torch.cuda.current_stream().cuda_stream


def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


def ptr(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else t.data_ptr()


class DeviceModel:
    """A model's inputs resident in HBM plus the ABI structs that point at them."""

    def __init__(self, inp: Inputs, device: str = "cuda"):
        cfg = inp.cfg
        self.cfg = cfg
        self.inp = inp
        self.device = device
        self.ccfg = make_config(cfg)
        self.L = len(inp.base)
        if self.L != cfg.n_layers:
            # a truncated input set (per-layer or LM-head-only use); with no layer at all the
            # config still needs one for validation, and train_step is refused
            self.ccfg.n_layers = max(self.L, 1)
        self.keep: List[torch.Tensor] = []
        self.base = (L.MebpLayerBase * self.L)()
        self.lora = (L.MebpLayerLora * self.L)()
        self.grads = (L.MebpLayerLoraGrad * self.L)()
        self.dA: List[dict] = []
        self.dB: List[dict] = []
        for l in range(self.L):
            for i, p in enumerate(PROJ):
                q4, sb = inp.base[l][p]
                tq, ts = _dev(q4, device), _dev(sb, device)
                self.keep += [tq, ts]
                self.base[l].w[i].q4 = tq.data_ptr()
                self.base[l].w[i].scale = ts.data_ptr()
            na, nm = _dev(inp.norm_attn[l], device), _dev(inp.norm_mlp[l], device)
            self.keep += [na, nm]
            self.base[l].norm_attn = na.data_ptr()
            self.base[l].norm_mlp = nm.data_ptr()
            ex = inp.extra
            if ex.get("bias") and ex["bias"][l] is not None:
                for i, p in enumerate(("q", "k", "v")):
                    tb = _dev(ex["bias"][l][p], device)
                    self.keep.append(tb)
                    self.base[l].bias[i] = tb.data_ptr()
            if ex.get("qk_norm") and ex["qk_norm"][l] is not None:
                tq, tk = (_dev(w, device) for w in ex["qk_norm"][l])
                self.keep += [tq, tk]
                self.base[l].q_norm, self.base[l].k_norm = tq.data_ptr(), tk.data_ptr()
            if ex.get("post_norm") and ex["post_norm"][l] is not None:
                ta, tm = (_dev(w, device) for w in ex["post_norm"][l])
                self.keep += [ta, tm]
                self.base[l].post_attn_norm, self.base[l].post_mlp_norm = ta.data_ptr(), tm.data_ptr()
            dA, dB = {}, {}
            for i, p in enumerate(PROJ):
                if p not in inp.lora[l]:
                    continue
                A, B = inp.lora[l][p]
                tA, tB = _dev(A, device), _dev(B, device)
                self.keep += [tA, tB]
                self.lora[l].A[i] = tA.data_ptr()
                self.lora[l].B[i] = tB.data_ptr()
                gA = torch.empty(A.shape, dtype=torch.float32, device=device)
                gB = torch.empty(B.shape, dtype=torch.float32, device=device)
                dA[p], dB[p] = gA, gB
                self.grads[l].dA[i] = gA.data_ptr()
                self.grads[l].dB[i] = gB.data_ptr()
            self.dA.append(dA)
            self.dB.append(dB)
        self.emb = None
        if inp.emb is not None:
            eq, es = _dev(inp.emb[0], device), _dev(inp.emb[1], device)
            self.keep += [eq, es]
            self.emb = L.MebpQ4(q4=eq.data_ptr(), scale=es.data_ptr())
            self.norm_final = _dev(inp.norm_final, device)
        if inp.ids is not None:
            self.ids = _dev(inp.ids, device)
        self.B, self.T = cfg.batch, cfg.seq
        self.N = self.B * self.T
        self.ws_bytes = L.mebp_workspace_bytes(self.ccfg, self.B, self.T)
        if self.ws_bytes == 0:
            raise L.MebpError(L.MEBP_EINVAL, "invalid config for workspace sizing")
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.loss = torch.zeros(1, dtype=torch.float32, device=device)
        self.ckpt = None

    # ------------------------------------------------------------------ entry points
    def layer_forward(self, l: int, x_in: torch.Tensor, x_out: torch.Tensor):
        L.mebp_layer_forward_ckpt(self.ccfg, l, self.base[l], self.lora[l], ptr(x_in), ptr(x_out), self.B,
                                  self.T, ptr(self.ws), self.ws_bytes, stream_handle())

    def layer_backward(self, l: int, x_ckpt: torch.Tensor, dy: torch.Tensor, dx: Optional[torch.Tensor]):
        L.mebp_layer_recompute_backward(self.ccfg, l, self.base[l], self.lora[l], ptr(x_ckpt), ptr(dy), ptr(dx),
                                        self.grads[l], self.B, self.T, ptr(self.ws), self.ws_bytes,
                                        stream_handle())

    def lm_head(self, x_last: torch.Tensor, dx_last: torch.Tensor):
        L.mebp_lm_head_ce_backward(self.ccfg, self.emb, ptr(self.norm_final), ptr(x_last), ptr(self.ids), self.B,
                                   self.T, ptr(self.loss), ptr(dx_last), ptr(self.ws), self.ws_bytes,
                                   stream_handle())

    def embed(self, x0: torch.Tensor):
        L.mebp_embed(self.ccfg, self.emb, ptr(self.ids), self.B, self.T, ptr(x0), stream_handle())

    def alloc_ckpt(self):
        if self.ckpt is None:
            self.ckpt = torch.empty((self.L + 1, self.N, self.cfg.hidden), dtype=torch.float32,
                                    device=self.device)
        return self.ckpt

    def train_step(self, dx0: Optional[torch.Tensor] = None):
        if self.L == 0:
            raise ValueError("this input set has no layers")
        ck = self.alloc_ckpt()
        L.mebp_train_step(self.ccfg, self.emb, self.base, ptr(self.norm_final), self.lora, ptr(self.ids), self.B,
                          self.T, ptr(ck), ptr(self.loss), self.grads, ptr(dx0), ptr(self.ws), self.ws_bytes,
                          stream_handle())

    def train_step_offload(self, ckpt_host: torch.Tensor, ring: torch.Tensor, dx0: Optional[torch.Tensor] = None):
        """The step with checkpoints in pinned host memory ``ckpt_host`` [(L+1)][N][d] and a
        device ring ``ring`` [slots][N][d]."""
        if self.L == 0:
            raise ValueError("this input set has no layers")
        L.mebp_train_step_offload(self.ccfg, self.emb, self.base, ptr(self.norm_final), self.lora, ptr(self.ids),
                                  self.B, self.T, ptr(ckpt_host), ptr(ring), ring.shape[0], ptr(self.loss), self.grads,
                                  ptr(dx0), ptr(self.ws), self.ws_bytes, stream_handle())

    def grad_probe(self) -> torch.Tensor:
        """First and last layers' LoRA gradients, concatenated (a cheap result fingerprint)."""
        parts = [t.reshape(-1) for l in {0, self.L - 1} for d in (self.dA[l], self.dB[l]) for t in d.values()]
        return torch.cat(parts) if parts else torch.zeros(1, device=self.device)

    def ws_view(self, slot: int, dtype: torch.dtype, shape) -> torch.Tensor:
        """A view of a workspace intermediate (tests)."""
        off = L.mebp_workspace_offset(self.ccfg, self.B, self.T, slot)
        n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
        return self.ws[off:off + n].view(dtype).view(*shape)


def slot_index(name: str) -> int:
    i = 0
    while True:
        s = L.mebp_workspace_slot_name(i)
        if s is None:
            raise KeyError(name)
        if s == name:
            return i
        i += 1
