"""Helpers shared by the GPU parity tests (no test functions here)."""
import sys

import numpy as np


def rel_l2(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def to_np(t):
    import torch
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.float().cpu().numpy()
    return t.cpu().numpy()


TOL = 2e-2  # rel-L2 bound for bf16-operand / fp32-accumulate outputs
