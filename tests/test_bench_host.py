"""Host-side checks of the benchmark's bookkeeping (no GPU): the algorithmic work it prices
kernels and steps against, and the mapping from HIP kernel names (as rocprofv3 prints them) to
the timing-report names its traffic and counter summaries use."""
import importlib.util
import os
import re

import pytest

from mebp_inputs import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


# Per-step algorithmic work in TFLOP, computed independently from the model shapes (base GEMMs
# 6 N P L, LM head 4 N d V, attention 16 dh per visible pair per query head, LoRA 8 N r (in + out)
# per adapted module) when the workloads were specified.
@pytest.mark.parametrize("name,tflop", [("qwen2.5-0.5b", 0.703), ("gemma3-1b", 2.830),
                                        ("qwen2.5-1.5b", 38.07), ("gemma3-4b", 378.0)])
def test_algorithmic_flops_per_step(name, tflop):
    got = _bench().algorithmic_flops(CONFIGS[name]) / 1e12
    assert abs(got - tflop) <= 0.01 * tflop, (name, got, tflop)


# rocprofv3 kernel names of the library, normalised as the summaries do, and the report name
# each must land on (None: not one of the priced kernels)
KERNELS = [
    ("k_gemm_nt<0>", "gemm_nt_f16out"),
    ("k_gemm_nt_lds<0>", "gemm_nt_f16out"),
    ("k_gemm_nt_lds<0, false, 4>", "gemm_nt_f16out"),
    ("k_gemm_nt_lds<1, false, 4>", "gemm_nt_f32out"),
    ("k_gemm_nt_lds<2, false, 8>", "gemm_nt_logits"),
    ("k_gemm_nt_lds<0, false, 4, true>", "gemm_nt_f16out"),
    ("k_gemm_nt_lds<0, false, 4, false>", "gemm_nt_f16out"),
    ("k_gemm_nt_lds<1, false, 4, false>", "gemm_nt_f32out"),
    ("k_gemm_nt_lds<2, false, 8, false>", "gemm_nt_logits"),
    ("k_gemm_nt_big<256, 4, 0, true>", "gemm_nt_f16out"),
    ("k_gemm_nt_big<128, 2, 0, false>", "gemm_nt_f16out"),
    ("k_gemm_nt<1>", "gemm_nt_f32out"),
    ("k_gemm_nt_lds<1>", "gemm_nt_f32out"),
    ("k_gemm_nt_big<128, 2, 1, true>", "gemm_nt_f32out"),
    ("k_gemm_nt<2>", "gemm_nt_logits"),
    ("k_gemm_nt_lds<2>", "gemm_nt_logits"),
    ("k_gemm_nt_big<256, 4, 2, false>", "gemm_nt_logits"),
    ("k_gemm_tn<0>", "gemm_tn_f32out"),
    ("k_gemm_tn_big<128, 0>", "gemm_tn_f32out"),
    ("k_gemm_tn<1>", "gemm_tn_act_bwd"),
    ("k_gemm_tn_big<128, 1>", "gemm_tn_act_bwd"),
    ("k_gemm_tn<2>", "gemm_tn_probs_dh"),
    ("k_gemm_tn_big<128, 2>", "gemm_tn_probs_dh"),
    ("k_gemm_tn<3>", "gemm_tn_bf16out"),
    ("k_gemm_tn_big<128, 3>", "gemm_tn_bf16out"),
    ("k_gemm_tn_big<128, 0, true>", "gemm_tn_f32out"),
    ("k_gemm_tn_big<128, 1, true>", "gemm_tn_act_bwd"),
    ("k_gemm_tn_lds<1>", "gemm_tn_act_bwd"),
    ("k_gemm_tn_lds<3>", "gemm_tn_bf16out"),
    ("k_lora_rows<OpF16>", "lora_rows"),
    ("k_lora_outer<true>", "lora_outer"),
    ("k_attn_fwd32<256, 4>", "attn_fwd"),
    ("k_attn_bwd_kv32<128, 4>", "attn_bwd_dkdv"),
    ("k_attn_bwd_kv32p<2>", "attn_bwd_dkdv"),
    ("k_lora_rows<OpF16, 3>", "lora_rows"),
    ("k_lora_outer<true, 2>", "lora_outer"),
    ("k_attn_bwd_dkdv<64, 64>", "attn_bwd_dkdv"),
    ("k_attn_bwd_dq<256, 32, false>", "attn_bwd_dq"),
    ("k_nt_finalize<0>", None),
    ("k_tn_finalize_norm", None),
    ("k_ce_probs", None),
]


@pytest.mark.parametrize("kernel,report", KERNELS)
def test_kernel_name_patterns(kernel, report):
    pats = _bench().KERNEL_PATTERNS
    hits = [name for name, pat in pats.items() if re.search(pat, kernel)]
    assert hits == ([report] if report else []), (kernel, hits)
