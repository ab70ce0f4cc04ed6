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


ROW_TOL = 5e-2  # per-row rel-L2 bound (each row of an activation-shaped output)


def max_row_rel_l2(got, ref, floor_frac=1e-3) -> float:
    """Largest rel-L2 over the rows of a 2-D output. A row whose reference norm is below
    ``floor_frac`` times the median row norm is measured against that floor instead of its
    own norm (rows that are exactly or nearly zero, such as positions without a target)."""
    got = np.asarray(got, np.float64).reshape(len(got), -1)
    ref = np.asarray(ref, np.float64).reshape(len(ref), -1)
    rn = np.linalg.norm(ref, axis=1)
    med = float(np.median(rn)) if rn.size else 0.0
    den = np.maximum(rn, floor_frac * med)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.linalg.norm(got - ref, axis=1) / den))
