"""Bit-exact check of the decompression that runs on the hot path: the int4 -> 16-bit
conversion fused into every dequant-GEMM kernel (Algorithm 1, LazyLoadAndDecompressWeights;
Sec. 3, base weight compression).

Each production GEMM kernel is run through ``mebp_test_gemm`` on a one-hot activation
(forward kernels) or a one-hot gradient (transposed kernels): every output is then a single
product 1 * W_op with fp32 accumulation, i.e. exactly the operand the kernel decompressed.
The forward kernels multiply fp16 operands, the transposed ones bf16, so the outputs must
equal the oracle's fp16 / bf16 round-to-nearest-even of ``q * s`` bit for bit.

Weights: the offline quantiser's output on seeded N(0, 0.02) weights, with some scales
replaced by hand: fp16 subnormals, the smallest normal, and large values, so that the
conversion's exponent handling is exercised. Shapes: a ragged reduction (688 = 10 K tiles
of 64 plus 48, groups of 32 with a 16-wide last one), ragged output tiles, several tiles in
every direction, and one aligned shape.
"""
import numpy as np
import pytest
import torch

import oracle as O
from mebp_inputs import quantize_q4
from paper_2510_03425_amd import _lib as L

from gpu_util import say

pytestmark = pytest.mark.gpu

FORWARD = {"nt": L.TEST_GEMM_NT, "nt_big128": L.TEST_GEMM_NT_BIG128, "nt_big256": L.TEST_GEMM_NT_BIG256,
           "nt_lds": L.TEST_GEMM_NT_LDS}
TRANSPOSED = {"tn": L.TEST_GEMM_TN, "tn_big": L.TEST_GEMM_TN_BIG}
# (n_out, n_in, M): ragged and aligned; M covers every input (forward) or output (transposed)
# index at least once and spans several token tiles with a ragged tail
SHAPES = [(592, 688, 808), (1024, 512, 1100)]


def _weights(n_out, n_in, seed):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((n_out, n_in)) * 0.02).astype(np.float32)
    q4, sb = quantize_q4(w, 32)
    sb = sb.copy()
    special = np.array([0x0001, 0x0003, 0x03FF, 0x0400, 0x0401, 0x1000, 0x3C00, 0x5800, 0x6400, 0x6ABC],
                       np.uint16)  # subnormals, smallest normals, 2^-11, 1, 128, 1024, 3448
    ng = sb.shape[1]
    for i in range(0, n_out, 7):
        sb[i, (i // 7) % ng] = special[(i // 7) % len(special)]
    return q4, sb


def _upload(q4, sb, gpu):
    tq = torch.from_numpy(np.ascontiguousarray(q4)).to(gpu)
    ts = torch.from_numpy(np.ascontiguousarray(sb).view(np.int16)).to(gpu)
    return tq, ts, L.MebpQ4(q4=tq.data_ptr(), scale=ts.data_ptr())


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("kind", list(FORWARD))
def test_forward_kernel_decompression_bit_exact(built_lib, gpu, kind, shape):
    n_out, n_in, M = shape
    q4, sb = _weights(n_out, n_in, seed=n_in + 1)
    tq, ts, w = _upload(q4, sb, gpu)
    x = torch.zeros((M, n_in), dtype=torch.float16, device=gpu)
    ks = torch.arange(M, device=gpu) % n_in
    x[torch.arange(M, device=gpu), ks] = 1.0
    out = torch.full((M, n_out), float("nan"), dtype=torch.float32, device=gpu)
    say("fused decompression", kind, "n_out", n_out, "n_in", n_in, "M", M)
    L.mebp_test_gemm(FORWARD[kind], w, n_out, n_in, x.data_ptr(), M, out.data_ptr(),
                     torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    ref = O.dequant_fp16_bits(q4, sb, n_in, 32).view(np.float16).astype(np.float32)  # [n_out][n_in]
    got = out.cpu().numpy()
    exp = ref[:, np.arange(M) % n_in].T
    bad = np.argwhere(got.view(np.uint32) != exp.view(np.uint32))
    assert bad.size == 0, f"{len(bad)} mismatches, first at (m, n) = {bad[0].tolist()}: " \
                          f"{got[tuple(bad[0])]!r} vs {exp[tuple(bad[0])]!r}"


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("kind", list(TRANSPOSED))
def test_transposed_kernel_decompression_bit_exact(built_lib, gpu, kind, shape):
    n_out, n_in, M = shape
    q4, sb = _weights(n_out, n_in, seed=n_out + 2)
    tq, ts, w = _upload(q4, sb, gpu)
    g = torch.zeros((M, n_out), dtype=torch.bfloat16, device=gpu)
    ns = torch.arange(M, device=gpu) % n_out
    g[torch.arange(M, device=gpu), ns] = 1.0
    out = torch.full((M, n_in), float("nan"), dtype=torch.float32, device=gpu)
    say("fused decompression", kind, "n_out", n_out, "n_in", n_in, "M", M)
    L.mebp_test_gemm(TRANSPOSED[kind], w, n_out, n_in, g.data_ptr(), M, out.data_ptr(),
                     torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    bits = O.dequant_bf16_bits(q4, sb, n_in, 32).astype(np.uint32) << 16  # [n_out][n_in]
    ref = bits.view(np.float32)
    got = out.cpu().numpy()
    exp = ref[np.arange(M) % n_out, :]
    bad = np.argwhere(got.view(np.uint32) != exp.view(np.uint32))
    assert bad.size == 0, f"{len(bad)} mismatches, first at (m, c) = {bad[0].tolist()}: " \
                          f"{got[tuple(bad[0])]!r} vs {exp[tuple(bad[0])]!r}"


@pytest.mark.parametrize("fwd", [True, False], ids=["forward", "transposed"])
def test_16bit_weight_mode_is_the_same_kernel(built_lib, gpu, fwd):
    # the 16-bit-weight modes (used to measure what the decompression costs) fed the
    # decompressed weights multiply exactly the operands of the int4 kernels in the same
    # order: outputs identical bit for bit on random inputs
    n_out, n_in, M = 592, 688, 808
    q4, sb = _weights(n_out, n_in, seed=5)
    tq, ts, w = _upload(q4, sb, gpu)
    wf = torch.from_numpy(O.dequant(q4, sb, n_in, 32).astype(np.float32)).to(gpu)
    w16 = (wf.half() if fwd else wf.bfloat16()).contiguous()
    ww = L.MebpQ4(q4=w16.data_ptr(), scale=0)
    if fwd:
        x = (torch.randn(M, n_in, device=gpu)).half()
        kinds, cols = (L.TEST_GEMM_NT_LDS, L.TEST_GEMM_NT_LDS_W16), n_out
    else:
        x = (torch.randn(M, n_out, device=gpu) * 0.01).bfloat16()
        kinds, cols = (L.TEST_GEMM_TN_BIG, L.TEST_GEMM_TN_BIG_W16), n_in
    outs = []
    for kind, wt in zip(kinds, (w, ww)):
        out = torch.full((M, cols), float("nan"), dtype=torch.float32, device=gpu)
        say("16-bit weight mode", "forward" if fwd else "transposed", kind)
        L.mebp_test_gemm(kind, wt, n_out, n_in, x.data_ptr(), M, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
        outs.append(out)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
