"""Host-only checks of the C ABI: the library loads, exports every function that
include/mebp.h declares, and rejects invalid arguments before touching the GPU."""
import ctypes as C
import os
import re

import pytest

from mebp_inputs import CONFIGS, MINI
from paper_2510_03425_amd import _lib as L
from paper_2510_03425_amd.device import make_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "mebp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mebp_[a-z0-9_]+)\s*\(", src)))


def test_header_symbols_exported(built_lib):
    names = header_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(built_lib, n), n
    assert set(names) == set(L.EXPORTED)


def test_every_kernel_launch_stub_is_defined(built_lib):
    """Each launched kernel has its host-side launch stub in the library. The host pass can
    drop a kernel template's stub without an error (for instance when an argument of a target
    builtin in it needs an implicit conversion that only the device pass accepts); the library
    then fails to load with an undefined __device_stub__ symbol."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm is not available")
    out = subprocess.run([nm, "-u", L.LIB_PATH], capture_output=True, text=True, check=True).stdout
    missing = [ln.split()[-1] for ln in out.splitlines() if "__device_stub__" in ln]
    assert not missing, missing


def test_struct_sizes_match_header(built_lib):
    # mebp_config: 18 four-byte fields; the structs are arrays of pointers
    assert C.sizeof(L.MebpConfig) == 18 * 4
    assert C.sizeof(L.MebpQ4) == 16
    assert C.sizeof(L.MebpLayerBase) == 7 * 16 + 16 + 7 * 8
    assert C.sizeof(L.MebpLayerLora) == 14 * 8


def test_workspace_bytes(built_lib):
    for cfg in CONFIGS.values():
        assert L.mebp_workspace_bytes(make_config(cfg), cfg.batch, cfg.seq) > 0
    c = make_config(MINI)
    small = L.mebp_workspace_bytes(c, 1, 64)
    assert small < L.mebp_workspace_bytes(c, 2, 160)
    assert L.mebp_workspace_bytes(c, 0, 64) == 0


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, L.MEBP_EUNSUPPORTED), ("hidden", 100, L.MEBP_EUNSUPPORTED),
    ("n_kv_heads", 3, L.MEBP_EINVAL), ("group", 64, L.MEBP_EUNSUPPORTED),
    ("lora_rank", 4, L.MEBP_EUNSUPPORTED), ("act", 5, L.MEBP_EINVAL), ("ffn", 100, L.MEBP_EUNSUPPORTED),
    ("lora_mask", 1 << 9, L.MEBP_EINVAL), ("n_layers", 0, L.MEBP_EINVAL), ("vocab", 1000, L.MEBP_EUNSUPPORTED),
    ("arch", 1 << 4, L.MEBP_EINVAL),
])
def test_config_rejected(built_lib, field, value, code):
    c = make_config(MINI)
    setattr(c, field, value)
    r = L.mebp_layer_forward_ckpt(c, 0, None, None, 0, 0, 2, 160, 0, 0, 0, check=False)
    assert r == code
    assert L.mebp_last_error()


def _fake_layer():
    base = L.MebpLayerBase()
    lora = L.MebpLayerLora()
    for i in range(7):
        base.w[i].q4 = 0x1000 * (i + 1)
        base.w[i].scale = 0x1000 * (i + 1) + 0x800
        lora.A[i] = 0x100000 + 0x1000 * i
        lora.B[i] = 0x200000 + 0x1000 * i
    base.norm_attn = 0x300000
    base.norm_mlp = 0x300100
    return base, lora


def test_argument_errors_enqueue_nothing(built_lib):
    c = make_config(MINI)
    base, lora = _fake_layer()
    need = L.mebp_workspace_bytes(c, 2, 160)
    X, Y, WS = 0x400000, 0x800000, 0x1000000
    f = lambda **kw: L.mebp_layer_forward_ckpt(
        c, kw.get("layer", 0), kw.get("base", base), kw.get("lora", lora), kw.get("x", X), kw.get("y", Y),
        kw.get("B", 2), kw.get("T", 160), kw.get("ws", WS), kw.get("wsb", need), 0, check=False)
    assert f(layer=2) == L.MEBP_EINVAL
    assert f(layer=-1) == L.MEBP_EINVAL
    assert f(x=0) == L.MEBP_EINVAL
    assert f(x=X + 4) == L.MEBP_EINVAL  # misaligned activation
    assert f(y=X) == L.MEBP_EINVAL      # aliasing
    assert f(ws=0) == L.MEBP_EINVAL
    assert f(ws=WS + 16) == L.MEBP_EINVAL
    assert f(wsb=need - 1) == L.MEBP_EWORKSPACE
    assert f(B=0) == L.MEBP_EINVAL
    assert f(base=None) == L.MEBP_EINVAL
    bad = L.MebpLayerLora()
    C.memmove(C.byref(bad), C.byref(lora), C.sizeof(lora))
    bad.B[3] = None
    assert f(lora=bad) == L.MEBP_EINVAL
    assert "LoRA o" in L.mebp_last_error()
    badb = L.MebpLayerBase()
    C.memmove(C.byref(badb), C.byref(base), C.sizeof(base))
    badb.w[6].q4 = 0x1001
    assert f(base=badb) == L.MEBP_EINVAL
    # backward: missing gradient buffers
    g = L.MebpLayerLoraGrad()
    r = L.mebp_layer_recompute_backward(c, 0, base, lora, X, Y, 0, g, 2, 160, WS, need, 0, check=False)
    assert r == L.MEBP_EINVAL and "grad" in L.mebp_last_error()
    # LM head needs T >= 2 and a vocabulary
    emb = L.MebpQ4(q4=0x1000, scale=0x2000)
    r = L.mebp_lm_head_ce_backward(c, emb, 0x300000, X, 0x500000, 2, 1, 0x600000, Y, WS, need, 0, check=False)
    assert r == L.MEBP_EINVAL
    c0 = make_config(CONFIGS["block"])
    r = L.mebp_lm_head_ce_backward(c0, emb, 0x300000, X, 0x500000, 1, 128, 0x600000, Y, WS, 1 << 30, 0,
                                   check=False)
    assert r == L.MEBP_EINVAL and "vocab" in L.mebp_last_error()
    # dequant: unsupported column count
    assert L.mebp_dequant_q4(emb, 4, 12, 32, 0x10000, 0, 0, check=False) == L.MEBP_EUNSUPPORTED
    assert L.mebp_dequant_q4(emb, 4, 16, 32, 0, 0, 0, check=False) == L.MEBP_EINVAL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "nope.so"))
    monkeypatch.setattr(L, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        L.lib()


def _opt_arrays(cfg, fill=0x1000):
    """Per-layer optimizer structs whose adapted entries point at distinct fake, 16-byte
    aligned addresses (never dereferenced: every call below fails validation first)."""
    n = cfg.n_layers
    arrs = [(L.MebpLayerLoraState * n)(), (L.MebpLayerLoraGrad * n)(), (L.MebpLayerLoraState * n)(),
            (L.MebpLayerLoraState * n)()]
    addr = fill
    for l in range(n):
        for i in range(L.NPROJ):
            if not (cfg.lora_mask() >> i) & 1:
                continue
            for a in arrs:
                f0, f1 = ("dA", "dB") if isinstance(a[l], L.MebpLayerLoraGrad) else ("A", "B")
                getattr(a[l], f0)[i] = addr
                getattr(a[l], f1)[i] = addr + 0x100
                addr += 0x200
    return arrs


HP_OK = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_scale=1.0, step=1)


@pytest.mark.parametrize("bad", [dict(step=0), dict(beta1=1.0), dict(beta2=-0.1), dict(eps=-1.0),
                                 dict(lr=float("nan")), dict(grad_scale=float("inf"))])
def test_adamw_rejects_bad_hparams(built_lib, bad):
    p, g, m, v = _opt_arrays(MINI)
    hp = L.MebpAdamwHparams(**dict(HP_OK, **bad))
    r = L.mebp_lora_adamw_step(make_config(MINI), p, g, m, v, hp, 0, check=False)
    assert r == L.MEBP_EINVAL and L.mebp_last_error()


def test_adamw_rejects_null_misaligned_and_aliased(built_lib):
    c = make_config(MINI)
    hp = L.MebpAdamwHparams(**HP_OK)
    p, g, m, v = _opt_arrays(MINI)
    assert L.mebp_lora_adamw_step(c, p, g, None, v, hp, 0, check=False) == L.MEBP_EINVAL
    assert L.mebp_lora_adamw_step(c, p, g, m, v, None, 0, check=False) == L.MEBP_EINVAL
    p[1].B[6] = 0
    assert L.mebp_lora_adamw_step(c, p, g, m, v, hp, 0, check=False) == L.MEBP_EINVAL
    p, g, m, v = _opt_arrays(MINI)
    m[0].A[2] = m[0].A[2] + 4
    assert L.mebp_lora_adamw_step(c, p, g, m, v, hp, 0, check=False) == L.MEBP_EINVAL
    assert "aligned" in L.mebp_last_error()
    p, g, m, v = _opt_arrays(MINI)
    v[1].A[0] = m[1].A[0]
    assert L.mebp_lora_adamw_step(c, p, g, m, v, hp, 0, check=False) == L.MEBP_EINVAL
    assert "alias" in L.mebp_last_error()


def test_grad_accumulate_rejects(built_lib):
    c = make_config(MINI)
    _, g, _, _ = _opt_arrays(MINI)
    _, acc, _, _ = _opt_arrays(MINI, fill=0x900000)
    assert L.mebp_lora_grad_accumulate(c, g, None, 0.5, True, 0, check=False) == L.MEBP_EINVAL
    assert L.mebp_lora_grad_accumulate(c, g, acc, float("nan"), True, 0, check=False) == L.MEBP_EINVAL
    acc[0].dB[3] = 8
    assert L.mebp_lora_grad_accumulate(c, g, acc, 0.5, False, 0, check=False) == L.MEBP_EINVAL
    assert C.sizeof(L.MebpAdamwHparams) == 7 * 4
    assert C.sizeof(L.MebpLayerLoraState) == 14 * 8


def test_test_gemm_and_static_entry_validate_first(built_lib):
    w = L.MebpQ4(q4=0x1000, scale=0x2000)
    X, OUT = 0x400000, 0x800000
    g = lambda **kw: L.mebp_test_gemm(kw.get("kind", L.TEST_GEMM_NT), kw.get("w", w), kw.get("n_out", 64),
                                      kw.get("n_in", 64), kw.get("x", X), kw.get("M", 32), kw.get("out", OUT), 0,
                                      check=False)
    assert g(kind=8) == L.MEBP_EINVAL and g(kind=-1) == L.MEBP_EINVAL
    assert g(n_in=40) == L.MEBP_EUNSUPPORTED and g(n_out=8) == L.MEBP_EUNSUPPORTED
    assert g(M=0) == L.MEBP_EINVAL and g(M=70000) == L.MEBP_EUNSUPPORTED
    assert g(x=X + 8) == L.MEBP_EINVAL and g(out=0) == L.MEBP_EINVAL and g(w=None) == L.MEBP_EINVAL
    # the static-scratch layer backward refuses a layer larger than the library's buffer
    # (a Gemma3-1B-shaped layer at 512 tokens) before any device work
    cfg = CONFIGS["gemma3-1b"].with_(vocab=0)
    c = make_config(cfg)
    base, lora = _fake_layer()
    grads = L.MebpLayerLoraGrad()
    for i in range(7):
        grads.dA[i], grads.dB[i] = 0x1000000 + 0x1000 * i, 0x2000000 + 0x1000 * i
    need = L.mebp_workspace_bytes(c, 1, 512)
    assert need > L.STATIC_SCRATCH_BYTES
    r = L.mebp_layer_recompute_backward_static(c, 0, base, lora, X, OUT, 0, grads, 1, 512, 0, check=False)
    assert r == L.MEBP_EWORKSPACE and "scratch" in L.mebp_last_error()
    # ... and accepts the workspace sizes of the single block and a Qwen2.5-0.5B-shaped layer
    for name in ("block", "qwen2.5-0.5b"):
        cf = CONFIGS[name].with_(vocab=0)
        assert L.mebp_workspace_bytes(make_config(cf), cf.batch, cf.seq) <= L.STATIC_SCRATCH_BYTES, name


IN_PLACE = ["gemm_tn_act_bwd", "splitk_finalize_actbwd", "rope_fwd", "qkv_post", "headnorm_bwd", "ce_chunk_stats",
            "ce_probs", "ce_dh_accum", "ce_final", "lora_adamw", "lora_grad_accumulate"]


@pytest.mark.parametrize("name", IN_PLACE)
def test_kernel_repeat_refuses_in_place_kernels(built_lib, name):
    # repeating a kernel that updates its own input would change the result
    assert built_lib.mebp_kernel_repeat(name.encode(), 3) == L.MEBP_EINVAL
    assert "cannot be repeated" in L.mebp_last_error()


def test_kernel_repeat_accepts_pure_kernels_and_switches_off(built_lib):
    for name in ("gemm_nt_f16out", "gemm_tn_probs_dh", "attn_fwd", "lora_rows"):
        assert built_lib.mebp_kernel_repeat(name.encode(), 3) == L.MEBP_OK
    assert built_lib.mebp_kernel_repeat(None, 1) == L.MEBP_OK


def test_workspace_guard_mode_changes_the_layout_and_validates(built_lib):
    c = make_config(MINI)
    n = 0
    while L.mebp_workspace_slot_name(n) is not None:
        n += 1
    plain = L.mebp_workspace_bytes(c, 2, 160)
    offs = [L.mebp_workspace_offset(c, 2, 160, s) for s in range(n)]
    r = L.mebp_workspace_guard_check(c, 2, 160, 256, plain, 0, check=False)
    assert r == L.MEBP_EINVAL and "off" in L.mebp_last_error()
    assert L.mebp_set_workspace_guards(True) is False
    try:
        guarded = L.mebp_workspace_bytes(c, 2, 160)
        goffs = [L.mebp_workspace_offset(c, 2, 160, s) for s in range(n)]
        # every slot and every second copy gains a guard region of at least 256 bytes, plus
        # the status word's 256
        assert guarded >= plain + 256 * (n + 1)
        assert all(g >= o for g, o in zip(goffs, offs)) and all(g % 256 == 0 for g in goffs)
        assert all(b - a >= 256 for a, b in zip(goffs, goffs[1:]))
        # a workspace sized without the guards is refused, before anything is enqueued
        r = L.mebp_layer_forward_ckpt(c, 0, None, None, 0, 0, 2, 160, 256, plain, 0, check=False)
        assert r == L.MEBP_EINVAL  # base NULL is checked first
        r = L.mebp_workspace_guard_check(c, 2, 160, 256, plain, 0, check=False)
        assert r == L.MEBP_EWORKSPACE
        r = L.mebp_workspace_guard_check(c, 2, 160, 0, guarded, 0, check=False)
        assert r == L.MEBP_EINVAL
        r = L.mebp_workspace_guard_check(c, 0, 160, 256, guarded, 0, check=False)
        assert r == L.MEBP_EINVAL
    finally:
        assert L.mebp_set_workspace_guards(False) is True
    assert L.mebp_workspace_bytes(c, 2, 160) == plain
