"""GPU parity of nmm_gemv_noalloc (the GEMV on the library's own scratch) through the C ABI.

Each call is compared with nmm_gemv on its own workspace bit for bit (same plan, same kernels) and
with the oracle at the GEMV's tolerance.  Calls come in a row on the one scratch array, the later
ones smaller, so a counter left non-zero or a partial sum read from an earlier call would show.
"""
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import assert_parity, dev16

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _noalloc(c: syn.GemvCase, path: int) -> tuple[int, torch.Tensor]:
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    y = torch.full((c.M, c.N), float("nan"), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    st = nmm.lib().nmm_gemv_noalloc(c.M, c.K, c.N, c.dt, x.data_ptr(), x.stride(0), W.data_ptr(),
                                    W.stride(0), y.data_ptr(), c.N, path, _stream())
    torch.cuda.synchronize()
    return st, y


def _with_workspace(c: syn.GemvCase, path: int) -> torch.Tensor:
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    y = torch.full((c.M, c.N), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv(x, W, y, N=c.N, path=path, workspace=nmm.Workspace())
    torch.cuda.synchronize()
    return y


def _check(c: syn.GemvCase, path: int):
    st, y = _noalloc(c, path)
    assert st == nmm.NMM_OK, (c.name, st)
    ref = _with_workspace(c, path)
    assert torch.equal(y, ref), f"{c.name}: differs from nmm_gemv"
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt)
    assert_parity(y, y_ref, a_ref, what=c.name)
    return y


def test_calls_in_a_row_each_smaller():
    # the streaming path at 8 rows of W_O [16384, 7168] (7.4 MB of scratch, split K), then the
    # MFMA path at 3 rows of [7168, 2112], then one row of [7168, 2112] on the streaming path
    wo8 = syn.gemv_case(41, 8, 16384, 7168, syn.BF16, name="wo_M8")
    down3 = syn.gemv_case(42, 3, 7168, 2112, syn.BF16, name="down_M3")
    assert nmm.nmm_gemv_workspace_size(8, 16384, 7168, syn.BF16, nmm.NMM_PATH_GEMV) <= nmm.NMM_NOALLOC_SCRATCH_BYTES
    first = _check(wo8, nmm.NMM_PATH_GEMV)
    _check(down3, nmm.NMM_PATH_MFMA)
    _check(syn.down_projection(), nmm.NMM_PATH_GEMV)
    st, again = _noalloc(wo8, nmm.NMM_PATH_GEMV)
    assert st == nmm.NMM_OK and torch.equal(again, first)


def test_integer_exact_two_calls():
    big = syn.gemv_case(43, 4, 16384, 7168, syn.BF16, integer=True, name="wo_M4_int")
    small = syn.down_projection(integer=True)
    for c in (big, small):
        st, y = _noalloc(c, nmm.NMM_PATH_AUTO)
        assert st == nmm.NMM_OK
        y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt)
        assert_parity(y, y_ref, a_ref, integer=True, what=c.name)


def test_scratch_too_small_is_rejected_before_any_launch():
    # 16 rows of W_O on the streaming path would need 29 MB of partial sums
    M, K, N = 16, 16384, 7168
    assert nmm.nmm_gemv_workspace_size(M, K, N, syn.BF16, nmm.NMM_PATH_GEMV) > nmm.NMM_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((M, K), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((K, N), dtype=torch.bfloat16, device="cuda")
    y = torch.full((M, N), 3.0, device="cuda")
    st = nmm.lib().nmm_gemv_noalloc(M, K, N, syn.BF16, x.data_ptr(), K, W.data_ptr(), N, y.data_ptr(), N,
                                    nmm.NMM_PATH_GEMV, _stream())
    torch.cuda.synchronize()
    assert st == nmm.NMM_ERR_WORKSPACE and torch.all(y == 3.0)
    # the same call on the MFMA path fits, and still agrees with the oracle afterwards
    _check(syn.gemv_case(44, 16, K, N, syn.BF16, name="wo_M16"), nmm.NMM_PATH_MFMA)


def test_empty_and_k_zero():
    x = torch.zeros((2, 8), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((1, 16), dtype=torch.bfloat16, device="cuda")
    y = torch.full((2, 16), 5.0, device="cuda")
    st = nmm.lib().nmm_gemv_noalloc(0, 8, 16, syn.BF16, x.data_ptr(), 8, W.data_ptr(), 16, y.data_ptr(), 16,
                                    0, _stream())
    torch.cuda.synchronize()
    assert st == nmm.NMM_OK and torch.all(y == 5.0)
    st = nmm.lib().nmm_gemv_noalloc(2, 0, 16, syn.BF16, x.data_ptr(), 8, W.data_ptr(), 16, y.data_ptr(), 16,
                                    0, _stream())
    torch.cuda.synchronize()
    assert st == nmm.NMM_OK and torch.all(y == 0)
