"""GPU parity of the transposed-weight GEMV (nmm_gemv_nt: W given row-major as Wt[N, K]) against
the oracle's plain product, through the C ABI.

The oracle takes W as [K, N]; the tests draw W that way and hand the GPU its transpose, so the
expected values are the same plain product as for nmm_gemv.  Floating-point cases meet the fp32
bar, integer-valued cases match bit for bit.  Shapes cover the decode chain's matrices as torch
stores them, split and unsplit K, ragged K (row padding filled with NaN, which must not reach the
sums) and ragged N, M above the 4-row block, fp16, and K = 0.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import assert_parity, dev16

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")


def transposed(W: np.ndarray, K: int, N: int, ldwt: int, fill: int = 0x7FC0) -> np.ndarray:
    """Wt[n, k] = W[k, n], rows padded to ldwt with `fill` (a NaN pattern by default)."""
    Wt = np.full((N, ldwt), fill, dtype=np.uint16)
    Wt[:, :K] = W[:K, :N].T
    return Wt


def run_nt(c: syn.GemvCase, ldwt: int, ldy=None):
    Wt = transposed(c.W, c.K, c.N, ldwt)
    ldy = c.N if ldy is None else ldy
    y = torch.full((c.M, ldy), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv_nt(dev16(c.x, c.dt), dev16(Wt, c.dt), y, K=c.K)
    torch.cuda.synchronize()
    return y


def check_nt(c: syn.GemvCase, ldwt: int, ldy=None):
    y = run_nt(c, ldwt, ldy)
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt, K=c.K, N=c.N)
    assert_parity(y[:, :c.N], y_ref, a_ref, integer=c.integer, what=c.name)
    if ldy is not None and ldy > c.N:
        assert torch.isnan(y[:, c.N:]).all(), "columns past N were written"


@pytest.mark.parametrize("K,N,name", [(16384, 7168, "W_O^T"), (7168, 2112, "down^T"), (1536, 24576, "W_UQ^T"),
                                      (7168, 576, "MatMul 2^T")])
@pytest.mark.parametrize("integer", [False, True])
def test_nt_decode_shapes(K, N, name, integer):
    c = syn.gemv_case(500 + K % 97, 1, K, N, syn.BF16, integer=integer, name=name)
    check_nt(c, K)


@pytest.mark.parametrize("M,K,N,dt,ldx,ldwt", [
    (1, 1021, 1031, syn.BF16, 1024, 1024),   # ragged K inside a 16-byte chunk, ragged N
    (1, 13, 8, syn.F16, 16, 16),
    (2, 20000, 40, syn.BF16, 20000, 20000),  # split K, few rows
    (3, 4099, 520, syn.F16, 4104, 4104),
    (4, 9000, 4200, syn.BF16, 9000, 9008),
    (5, 777, 300, syn.BF16, 784, 800),       # two 4-row blocks
    (16, 1536, 3000, syn.BF16, 1536, 1536),
    (1, 1, 1, syn.BF16, 8, 8),
    (1, 100000, 64, syn.BF16, 100000, 100000),
    (1, 16385, 300, syn.BF16, 16392, 16392),  # one k past the unsplit limit
])
def test_nt_ragged_shapes(M, K, N, dt, ldx, ldwt):
    c = syn.gemv_case(600 + M + K % 89, M, K, N, dt, ldx=ldx, name=f"nt_{M}x{K}x{N}")
    check_nt(c, ldwt, ldy=N + 3)
    ci = syn.gemv_case(700 + M + K % 89, M, K, N, dt, integer=True, ldx=ldx, name=f"nt_int_{M}x{K}x{N}")
    check_nt(ci, ldwt)


@pytest.mark.parametrize("case", syn.random_nt_shapes(), ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}")
def test_nt_random_shapes_integer_exact(case):
    # a seeded sweep (the launch-bounds model checks the same cases): small integers, so every
    # output is exact, with the output rows padded past N to catch stray writes
    M, K, N, dt, ldx, ldwt = case
    c = syn.gemv_case(800 + M + K % 83, M, K, N, dt, integer=True, ldx=ldx, name=f"nt_random_{M}x{K}x{N}")
    check_nt(c, ldwt, ldy=N + 5)


def test_nt_agrees_with_the_row_major_path_within_the_bar():
    # the same product from the two layouts: both within the bar of the oracle, and close to each
    # other (the summation orders differ)
    c = syn.gemv_case(801, 1, 7168, 2112, syn.BF16, name="down")
    y_nt = run_nt(c, 7168)
    y_rm = torch.empty((1, 2112), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv(dev16(c.x, syn.BF16), dev16(c.W, syn.BF16), y_rm)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x, c.W, syn.BF16)
    assert_parity(y_nt, y_ref, a_ref, what="nt")
    assert_parity(y_rm, y_ref, a_ref, what="row-major")


def test_nt_is_deterministic_and_reuses_its_workspace():
    c = syn.gemv_case(802, 1, 16384, 7168, syn.BF16, name="wo")
    Wt = dev16(transposed(c.W, c.K, c.N, c.K), syn.BF16)
    x = dev16(c.x, syn.BF16)
    ws = nmm.Workspace()
    outs = []
    for _ in range(3):
        y = torch.empty((1, c.N), dtype=torch.float32, device="cuda")
        nmm.nmm_gemv_nt(x, Wt, y, workspace=ws)
        outs.append(y)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])


def test_nt_zero_k_writes_zeros():
    y = torch.full((2, 16), float("nan"), dtype=torch.float32, device="cuda")
    x = torch.zeros((2, 8), dtype=torch.bfloat16, device="cuda")
    Wt = torch.zeros((16, 8), dtype=torch.bfloat16, device="cuda")
    nmm.nmm_gemv_nt(x, Wt, y, K=0)
    torch.cuda.synchronize()
    assert torch.equal(y, torch.zeros_like(y))
