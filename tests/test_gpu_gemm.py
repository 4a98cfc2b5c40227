"""The update step's bf16 GEMM kernels alone (trace_debug_gemm), in every
operand orientation and mode they are used with, on both tile kernels, against
an fp64 product of the same operand values: fp32 rounded to bf16 as read, fp32
split into bf16 hi + lo, and operands stored as bf16.  Shapes leave partial
tiles in m, n and k.  (The 256-tile kernel's bf16-operand loads otherwise run
only on products of the large workload, which the oracle does not reach.)"""
import numpy as np
import pytest
import torch

import paper_2203_16114_amd as P

pytestmark = pytest.mark.gpu

M, N, K = 200, 136, 264  # partial 128 / 256 tiles; K a multiple of 8, not of 32


def bf16_bits(x):
    return torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16)


def bf16_vals(x):
    return torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def operand(rng, rows, kc, mode):
    """Returns (device tensor as the kernel reads it, fp64 [rows][K] values of the product)."""
    v = rng.standard_normal((rows, K)) * np.exp(rng.uniform(-3, 3, (rows, 1)))
    mem = v if kc else v.T.copy()                     # [rows][K] or [K][rows]
    if mode == 0:
        eff = bf16_vals(v)
        dev = torch.from_numpy(mem.astype(np.float32)).cuda()
    elif mode == 1:
        hi = bf16_vals(v)
        eff = hi + bf16_vals(v.astype(np.float32).astype(np.float64) - hi)
        dev = torch.from_numpy(mem.astype(np.float32)).cuda()
    else:
        eff = bf16_vals(v)
        dev = bf16_bits(mem).cuda()
    return dev, eff


MODES = [(0, 0), (1, 0), (0, 1), (2, 0), (0, 2), (2, 2), (2, 1), (1, 2)]


@pytest.mark.parametrize("kernel", [1, 2])
@pytest.mark.parametrize("a_kc,b_kc", [(True, True), (True, False), (False, True), (False, False)])
@pytest.mark.parametrize("modes", MODES)
def test_bf16_gemm_modes_orientations_and_tiles(kernel, a_kc, b_kc, modes):
    ma, mb = modes
    rng = np.random.default_rng(1000 * kernel + 10 * ma + mb + 2 * a_kc + b_kc)
    A, a = operand(rng, M, a_kc, ma)
    B, b = operand(rng, N, b_kc, mb)
    ref = a @ b.T
    bound = np.abs(a) @ np.abs(b).T
    C = P.debug_gemm(A, B, M, N, K, a_kc, ma, b_kc, mb, kernel=kernel).cpu().numpy().astype(np.float64)
    # fp32 accumulation in a different order than the fp64 sum
    assert np.all(np.abs(C - ref) <= 1e-5 * bound + 1e-30), np.max(np.abs(C - ref) / (bound + 1e-30))


@pytest.mark.parametrize("kernel", [1, 2])
def test_bf16_gemm_writes_a_rounded_result(kernel):
    rng = np.random.default_rng(7 + kernel)
    A, a = operand(rng, M, True, 0)
    B, b = operand(rng, N, True, 2)
    C = P.debug_gemm(A, B, M, N, K, True, 0, True, 2, half_c=True, kernel=kernel)
    full = P.debug_gemm(A, B, M, N, K, True, 0, True, 2, kernel=kernel)
    # the bf16 result is the fp32 result rounded to nearest even
    assert torch.equal(C.cpu(), full.cpu().to(torch.bfloat16).view(torch.int16))


def test_bf16_gemm_rejects_what_it_cannot_read():
    rng = np.random.default_rng(3)
    A = torch.from_numpy(rng.standard_normal((M, 260)).astype(np.float32)).to(torch.bfloat16).view(torch.int16).cuda()
    B = torch.from_numpy(rng.standard_normal((N, 260)).astype(np.float32)).cuda()
    with pytest.raises(P.TraceError) as ei:  # bf16 with k contiguous needs K a multiple of 8
        P.debug_gemm(A, B, M, N, 260, True, 2, True, 0)
    assert ei.value.code == P.TRACE_EUNSUPPORTED
