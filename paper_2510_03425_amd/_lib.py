"""ctypes binding of ``libmebp.so`` (declared in ``include/mebp.h``).

Argument marshalling only: every function here forwards to the C entry point of the
same name; all computation runs in the library's HIP kernels. Pointers are passed as
Python ints (device addresses), the stream as an int (``hipStream_t``, 0 = null stream).
Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# MEBP_LIB selects another build of the same library (the sanitizer build of the host-only
# tests); there is no fallback: a missing library raises.
LIB_PATH = os.environ.get("MEBP_LIB") or os.path.join(_HERE, "libmebp.so")

MEBP_OK, MEBP_EINVAL, MEBP_EUNSUPPORTED, MEBP_EWORKSPACE, MEBP_EHIP = 0, -1, -2, -3, -4
NPROJ = 7

EXPORTED = (
    "mebp_workspace_bytes", "mebp_layer_forward_ckpt", "mebp_layer_recompute_backward",
    "mebp_lm_head_ce_backward", "mebp_embed", "mebp_train_step", "mebp_last_error",
    "mebp_dequant_q4", "mebp_workspace_offset", "mebp_workspace_slot_name", "mebp_kernel_timing",
    "mebp_kernel_timing_report", "mebp_kernel_repeat", "mebp_lora_grad_accumulate", "mebp_lora_adamw_step",
    "mebp_train_step_offload", "mebp_test_gemm", "mebp_layer_recompute_backward_static",
    "mebp_set_workspace_guards", "mebp_workspace_guard_check",
)

STATIC_SCRATCH_BYTES = 64 << 20  # MEBP_STATIC_SCRATCH_BYTES

# mebp_test_gemm kinds
(TEST_GEMM_NT, TEST_GEMM_NT_BIG128, TEST_GEMM_NT_BIG256, TEST_GEMM_NT_LDS, TEST_GEMM_TN, TEST_GEMM_TN_BIG,
 TEST_GEMM_NT_LDS_W16, TEST_GEMM_TN_BIG_W16) = range(8)


class MebpConfig(C.Structure):
    _fields_ = [
        ("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
        ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
        ("vocab", C.c_int32), ("act", C.c_int32), ("rms_eps", C.c_float),
        ("rope_theta_global", C.c_float), ("rope_theta_local", C.c_float),
        ("window", C.c_int32), ("global_every", C.c_int32), ("group", C.c_int32),
        ("lora_rank", C.c_int32), ("lora_alpha", C.c_float), ("lora_mask", C.c_uint32), ("arch", C.c_uint32),
    ]


class MebpQ4(C.Structure):
    _fields_ = [("q4", C.c_void_p), ("scale", C.c_void_p)]


class MebpLayerBase(C.Structure):
    _fields_ = [("w", MebpQ4 * NPROJ), ("norm_attn", C.c_void_p), ("norm_mlp", C.c_void_p), ("bias", C.c_void_p * 3),
                ("q_norm", C.c_void_p), ("k_norm", C.c_void_p), ("post_attn_norm", C.c_void_p),
                ("post_mlp_norm", C.c_void_p)]


class MebpLayerLora(C.Structure):
    _fields_ = [("A", C.c_void_p * NPROJ), ("B", C.c_void_p * NPROJ)]


class MebpLayerLoraGrad(C.Structure):
    _fields_ = [("dA", C.c_void_p * NPROJ), ("dB", C.c_void_p * NPROJ)]


class MebpLayerLoraState(C.Structure):
    _fields_ = [("A", C.c_void_p * NPROJ), ("B", C.c_void_p * NPROJ)]


class MebpAdamwHparams(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float), ("grad_scale", C.c_float), ("step", C.c_int32)]


class MebpError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mebp status {code}: {msg}")
        self.code = code


_lib = None


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first (python -m paper_2510_03425_amd.build)")
        L = C.CDLL(LIB_PATH)
        P, I32, SZ = C.c_void_p, C.c_int32, C.c_size_t
        cfgp = C.POINTER(MebpConfig)
        sig = {
            "mebp_workspace_bytes": (SZ, [cfgp, I32, I32]),
            "mebp_layer_forward_ckpt": (C.c_int, [cfgp, I32, C.POINTER(MebpLayerBase), C.POINTER(MebpLayerLora),
                                                  P, P, I32, I32, P, SZ, P]),
            "mebp_layer_recompute_backward": (C.c_int, [cfgp, I32, C.POINTER(MebpLayerBase),
                                                        C.POINTER(MebpLayerLora), P, P, P,
                                                        C.POINTER(MebpLayerLoraGrad), I32, I32, P, SZ, P]),
            "mebp_layer_recompute_backward_static": (C.c_int, [cfgp, I32, C.POINTER(MebpLayerBase),
                                                               C.POINTER(MebpLayerLora), P, P, P,
                                                               C.POINTER(MebpLayerLoraGrad), I32, I32, P]),
            "mebp_lm_head_ce_backward": (C.c_int, [cfgp, C.POINTER(MebpQ4), P, P, P, I32, I32, P, P, P, SZ, P]),
            "mebp_embed": (C.c_int, [cfgp, C.POINTER(MebpQ4), P, I32, I32, P, P]),
            "mebp_train_step": (C.c_int, [cfgp, C.POINTER(MebpQ4), C.POINTER(MebpLayerBase), P,
                                          C.POINTER(MebpLayerLora), P, I32, I32, P, P,
                                          C.POINTER(MebpLayerLoraGrad), P, P, SZ, P]),
            "mebp_train_step_offload": (C.c_int, [cfgp, C.POINTER(MebpQ4), C.POINTER(MebpLayerBase), P,
                                                  C.POINTER(MebpLayerLora), P, I32, I32, P, P, I32, P,
                                                  C.POINTER(MebpLayerLoraGrad), P, P, SZ, P]),
            "mebp_last_error": (C.c_char_p, []),
            "mebp_dequant_q4": (C.c_int, [C.POINTER(MebpQ4), I32, I32, I32, P, P, P]),
            "mebp_test_gemm": (C.c_int, [I32, C.POINTER(MebpQ4), I32, I32, P, I32, P, P]),
            "mebp_workspace_offset": (SZ, [cfgp, I32, I32, I32]),
            "mebp_workspace_slot_name": (C.c_char_p, [I32]),
            "mebp_set_workspace_guards": (C.c_int, [I32]),
            "mebp_workspace_guard_check": (C.c_int, [cfgp, I32, I32, P, SZ, P]),
            "mebp_kernel_timing": (C.c_int, [I32, I32]),
            "mebp_kernel_timing_report": (C.c_int, [C.c_char_p, SZ]),
            "mebp_kernel_repeat": (C.c_int, [C.c_char_p, I32]),
            "mebp_lora_grad_accumulate": (C.c_int, [cfgp, C.POINTER(MebpLayerLoraGrad), C.POINTER(MebpLayerLoraGrad),
                                                    C.c_float, I32, P]),
            "mebp_lora_adamw_step": (C.c_int, [cfgp, C.POINTER(MebpLayerLoraState), C.POINTER(MebpLayerLoraGrad),
                                               C.POINTER(MebpLayerLoraState), C.POINTER(MebpLayerLoraState),
                                               C.POINTER(MebpAdamwHparams), P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(code: int) -> int:
    if code != MEBP_OK:
        raise MebpError(code, mebp_last_error())
    return code


def _ref(x):
    return None if x is None else C.byref(x)


def mebp_last_error() -> str:
    return lib().mebp_last_error().decode()


def mebp_workspace_bytes(cfg: MebpConfig, B: int, T: int) -> int:
    return lib().mebp_workspace_bytes(C.byref(cfg), B, T)


def mebp_workspace_offset(cfg: MebpConfig, B: int, T: int, slot: int) -> int:
    return lib().mebp_workspace_offset(C.byref(cfg), B, T, slot)


def mebp_set_workspace_guards(on: bool) -> bool:
    """Workspace guard debug mode on or off; returns the previous mode."""
    return bool(lib().mebp_set_workspace_guards(1 if on else 0))


def mebp_workspace_guard_check(cfg, B, T, ws, ws_bytes, stream=0, check=True):
    r = lib().mebp_workspace_guard_check(C.byref(cfg), B, T, ws, ws_bytes, stream)
    return _check(r) if check else r


def mebp_workspace_slot_name(slot: int):
    r = lib().mebp_workspace_slot_name(slot)
    return None if r is None else r.decode()


def mebp_layer_forward_ckpt(cfg, layer, base, lora, x_in, x_out, B, T, ws, ws_bytes, stream=0, check=True):
    r = lib().mebp_layer_forward_ckpt(C.byref(cfg), layer, _ref(base), _ref(lora), x_in, x_out, B, T, ws,
                                      ws_bytes, stream)
    return _check(r) if check else r


def mebp_layer_recompute_backward(cfg, layer, base, lora, x_ckpt, dy, dx, grads, B, T, ws, ws_bytes, stream=0,
                                  check=True):
    r = lib().mebp_layer_recompute_backward(C.byref(cfg), layer, _ref(base), _ref(lora), x_ckpt, dy, dx,
                                            _ref(grads), B, T, ws, ws_bytes, stream)
    return _check(r) if check else r


def mebp_layer_recompute_backward_static(cfg, layer, base, lora, x_ckpt, dy, dx, grads, B, T, stream=0,
                                         check=True):
    r = lib().mebp_layer_recompute_backward_static(C.byref(cfg), layer, _ref(base), _ref(lora), x_ckpt, dy, dx,
                                                   _ref(grads), B, T, stream)
    return _check(r) if check else r


def mebp_lm_head_ce_backward(cfg, emb, norm_final, x_last, ids, B, T, loss, dx_last, ws, ws_bytes, stream=0,
                             check=True):
    r = lib().mebp_lm_head_ce_backward(C.byref(cfg), _ref(emb), norm_final, x_last, ids, B, T, loss, dx_last, ws,
                                       ws_bytes, stream)
    return _check(r) if check else r


def mebp_embed(cfg, emb, ids, B, T, x0, stream=0, check=True):
    r = lib().mebp_embed(C.byref(cfg), _ref(emb), ids, B, T, x0, stream)
    return _check(r) if check else r


def mebp_train_step(cfg, emb, layers, norm_final, lora, ids, B, T, ckpt, loss, grads, dx0, ws, ws_bytes, stream=0,
                    check=True):
    r = lib().mebp_train_step(C.byref(cfg), _ref(emb), layers, norm_final, lora, ids, B, T, ckpt, loss, grads, dx0,
                              ws, ws_bytes, stream)
    return _check(r) if check else r


def mebp_train_step_offload(cfg, emb, layers, norm_final, lora, ids, B, T, ckpt_host, ring, ring_slots, loss, grads,
                            dx0, ws, ws_bytes, stream=0, check=True):
    r = lib().mebp_train_step_offload(C.byref(cfg), _ref(emb), layers, norm_final, lora, ids, B, T, ckpt_host, ring,
                                      ring_slots, loss, grads, dx0, ws, ws_bytes, stream)
    return _check(r) if check else r


def mebp_dequant_q4(w, rows, cols, group, out_f32, out_bf16, stream=0, check=True):
    r = lib().mebp_dequant_q4(_ref(w), rows, cols, group, out_f32, out_bf16, stream)
    return _check(r) if check else r


def mebp_test_gemm(kind, w, n_out, n_in, x, M, out, stream=0, check=True):
    r = lib().mebp_test_gemm(kind, _ref(w), n_out, n_in, x, M, out, stream)
    return _check(r) if check else r


def mebp_lora_grad_accumulate(cfg, grads, acc, scale: float, first: bool, stream=0, check=True):
    """grads, acc: ctypes arrays of MebpLayerLoraGrad (one entry per layer)."""
    r = lib().mebp_lora_grad_accumulate(C.byref(cfg), grads, acc, scale, int(first), stream)
    return _check(r) if check else r


def mebp_lora_adamw_step(cfg, params, grads, m, v, hp, stream=0, check=True):
    """params, m, v: ctypes arrays of MebpLayerLoraState; grads: of MebpLayerLoraGrad."""
    r = lib().mebp_lora_adamw_step(C.byref(cfg), params, grads, m, v, _ref(hp), stream)
    return _check(r) if check else r


def mebp_kernel_timing(enable: bool, capacity: int = 65536) -> int:
    return _check(lib().mebp_kernel_timing(int(enable), capacity))


def mebp_kernel_timing_report() -> list:
    import json
    n = lib().mebp_kernel_timing_report(None, 0)
    if n < 0:
        raise MebpError(n, mebp_last_error())
    buf = C.create_string_buffer(n)
    r = lib().mebp_kernel_timing_report(buf, n)
    if r < 0:
        raise MebpError(r, mebp_last_error())
    return json.loads(buf.value.decode())


def mebp_kernel_repeat(kernel, times: int) -> int:
    return _check(lib().mebp_kernel_repeat(None if kernel is None else kernel.encode(), times))
