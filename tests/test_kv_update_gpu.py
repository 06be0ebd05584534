"""GPU parity of the bf16 output cast (nmm_gemv_bf16) and of MatMul 2 with its cache entry
(nmm_mla_kv_update) against the oracle, through the C ABI.

* bf16 outputs: the GPU rounds its own fp32 sum, so its bf16 must be exactly the oracle's
  rounding (same mode) of the GPU's fp32 y, and that y must pass the fp32 acceptance.  Integer
  inputs whose sums land on bf16 ties fix the tie rule bit for bit.
* MatMul 2: mm passes the fp32 acceptance; the cache entry is checked step-wise (the oracle's
  RMSNorm / RoPE in fp64 applied to the GPU's own mm: the GPU's bf16 must round a value within
  1e-4 relative of it, and at least 99 % of entries must match the oracle's rounding bit for bit)
  and end to end (against the oracle's own mm, within the acceptance propagated through RMSNorm
  plus one bf16 step).  A constructed case with exact ties checks the epilogue's rounding mode
  bit for bit, and rows other than `position` must be untouched.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import ABS_TOL, REL_TOL, assert_parity, dev16, host_bits

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")

SENTINEL = 0x7FC1   # a NaN pattern the kernels never write


def bf16_step(v: np.ndarray) -> np.ndarray:
    """Spacing of the bf16 grid at |v| (normal range; the subnormal step below 2^-126)."""
    a = np.abs(np.asarray(v, dtype=np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 2.0 ** -126)))
    return 2.0 ** (np.maximum(e, -126) - 7)


# ---------------------------------------------------------------- nmm_gemv_bf16

BF16_CASES = [  # M, K, N, dt, ldx, ldw, path
    (1, 7168, 576, syn.BF16, 7168, 576, nmm.NMM_PATH_GEMV),
    (1, 1021, 1031, syn.F16, 1024, 1032, nmm.NMM_PATH_GEMV),
    (2, 1536, 3000, syn.BF16, 1536, 3000, nmm.NMM_PATH_GEMV),
    (16, 4099, 520, syn.BF16, 4104, 520, nmm.NMM_PATH_GEMV),
    (4, 1536, 24576, syn.BF16, 1536, 24576, nmm.NMM_PATH_MFMA),
    (33, 4099, 520, syn.F16, 4104, 520, nmm.NMM_PATH_MFMA),
    (17, 16384, 7168, syn.BF16, 16384, 7168, nmm.NMM_PATH_AUTO),
]


@pytest.mark.parametrize("mode", [nmm.NMM_ROUND_EVEN, nmm.NMM_ROUND_AWAY])
@pytest.mark.parametrize("M,K,N,dt,ldx,ldw,path", BF16_CASES)
def test_gemv_bf16_rounds_the_fp32_sum(M, K, N, dt, ldx, ldw, path, mode):
    c = syn.gemv_case(300 + M + K % 11, M, K, N, dt, ldx=ldx, ldw=ldw, name=f"bf16_{M}x{K}x{N}")
    x, W = dev16(c.x, dt), dev16(c.W, dt)
    ldyb = N + 5
    yb = torch.full((M, ldyb), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv_bf16(x, W, yb, round=mode, y=y, N=N, path=path)
    yb_only = torch.full((M, ldyb), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    nmm.nmm_gemv_bf16(x, W, yb_only, round=mode, N=N, path=path)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x, c.W, dt, K=K, N=N)
    assert_parity(y, y_ref, a_ref, what=c.name)
    got = host_bits(yb)
    assert np.all(got[:, N:] == SENTINEL), "padding columns of y_bf16 were written"
    want = oracle.round_bf16(y.cpu().numpy(), mode)
    assert np.array_equal(got[:, :N], want), "bf16 is not the rounding of the GPU's own fp32 sum"
    assert np.array_equal(host_bits(yb_only), got), "the bf16-only call must give the same bits"


@pytest.mark.parametrize("path", [nmm.NMM_PATH_GEMV, nmm.NMM_PATH_MFMA])
@pytest.mark.parametrize("mode", [nmm.NMM_ROUND_EVEN, nmm.NMM_ROUND_AWAY])
def test_gemv_bf16_integer_ties(path, mode):
    # x = [1, 1, 0, ...]; column n sums W[0, n] + W[1, n]: 256 + {1, 3, -1 ...} lands on the
    # ties 257, 259, 255.5 ... of the bf16 grid; every sum is exact in fp32
    M, K, N = 3, 64, 136
    rng = np.random.default_rng(17)
    hi = rng.choice([256.0, -256.0, 512.0, 128.0], size=N)
    lo = rng.choice([1.0, 3.0, -1.0, 0.5, 2.0, 0.25], size=N)
    Wf = np.zeros((K, N), np.float32)
    Wf[0], Wf[1] = hi, lo
    W = syn.bits_from_f32(Wf, syn.BF16)
    xf = np.zeros((M, K), np.float32)
    xf[:, 0], xf[:, 1] = 1.0, 1.0
    xf[1, 1] = -1.0
    xf[2] = 0.0
    x = syn.bits_from_f32(xf, syn.BF16)
    yb = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv_bf16(dev16(x, syn.BF16), dev16(W, syn.BF16), yb, round=mode, y=y, path=path)
    torch.cuda.synchronize()
    y_ref, _ = oracle.gemv(x, W, syn.BF16)
    assert np.array_equal(y.cpu().numpy().astype(np.float64), y_ref)
    ties = np.count_nonzero(oracle.round_bf16(y_ref, 0) != oracle.round_bf16(y_ref, 1))
    assert ties > N // 4, "the case must contain ties"
    assert np.array_equal(host_bits(yb), oracle.round_bf16(y_ref, mode))


def test_gemv_bf16_zero_k_writes_zero():
    yb = torch.full((2, 16), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    x = torch.zeros((2, 8), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((0, 16), dtype=torch.bfloat16, device="cuda")
    nmm.nmm_gemv_bf16(x, W, yb, N=16, round=nmm.NMM_ROUND_AWAY)
    torch.cuda.synchronize()
    assert np.all(host_bits(yb) == 0)


# ---------------------------------------------------------------- nmm_mla_kv_update

def run_kv(c: syn.KvUpdateCase, mode, cache_rows=None, ld_cache=None, workspace=None):
    n = c.kv_lora + c.rope
    cache_rows = c.position + 3 if cache_rows is None else cache_rows
    ld_cache = n + 8 if ld_cache is None else ld_cache
    hidden = c.w.shape[0]
    hpad = np.zeros((1, (hidden + 7) // 8 * 8), np.uint16)
    hpad[0, :hidden] = c.h.reshape(-1)
    h = dev16(hpad, syn.BF16)
    cache = torch.full((cache_rows, ld_cache), SENTINEL, dtype=torch.int16, device="cuda")
    mm = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_mla_kv_update(h, dev16(c.w, syn.BF16), dev16(c.gamma, syn.BF16), mm, cache.view(torch.bfloat16),
                          kv_lora=c.kv_lora, rope=c.rope, eps=c.eps, theta=c.theta, position=c.position,
                          round=mode, workspace=workspace)
    torch.cuda.synchronize()
    return mm.cpu().numpy().astype(np.float64), cache


def check_kv(c: syn.KvUpdateCase, mode, **kw):
    n, kv = c.kv_lora + c.rope, c.kv_lora
    mm, cache = run_kv(c, mode, **kw)
    mm_ref, mm_abs, row_ref, bits_ref = oracle.mla_kv_update(c.h, c.w, c.gamma, kv, c.rope, c.eps, c.theta,
                                                             c.position, mode)
    assert_parity(mm, mm_ref, mm_abs, what="MatMul 2 product")

    # the written row, and nothing else
    row = cache[c.position].view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.all(row[n:] == SENTINEL), "columns past kv_lora + rope were written"
    for r in {0, c.position - 1, c.position + 1, cache.shape[0] - 1} - {c.position}:
        if 0 <= r < cache.shape[0]:
            other = cache[r].view(torch.int16).cpu().numpy().view(np.uint16)
            assert np.all(other == SENTINEL), f"cache row {r} was written"
    got = oracle.decode(row[:n], syn.BF16)

    # step-wise: the oracle's epilogue on the GPU's own product
    row2, bits2 = oracle.kv_entry(mm, c.gamma, kv, c.eps, c.theta, c.position, mode)
    slack = 1e-4 * np.abs(row2) + np.concatenate([np.zeros(kv), 1e-6 * np.repeat(
        np.abs(mm[kv::2]) + np.abs(mm[kv + 1::2]), 2)])
    bad = np.abs(got - row2) > 0.5 * bf16_step(row2) + slack
    assert not bad.any(), f"{np.count_nonzero(bad)} entries are not a rounding of the fp64 epilogue " \
                          f"(first {np.argmax(bad)}: {got[np.argmax(bad)]} vs {row2[np.argmax(bad)]})"
    same = np.count_nonzero(row[:n] == bits2) / n
    assert same >= 0.99, f"only {same:.3%} of entries round like the oracle"

    # end to end: the oracle's own product, with the acceptance propagated through the epilogue
    tol = REL_TOL * mm_abs + ABS_TOL
    c_ref = mm_ref[:kv]
    ms = np.mean(c_ref ** 2) + c.eps
    inv = 1.0 / math.sqrt(ms)
    g = np.abs(oracle.decode(c.gamma, syn.BF16))
    d_inv = inv * float(np.sum(np.abs(c_ref) * tol[:kv])) / (kv * ms)
    bound_c = g * (inv * tol[:kv] + np.abs(c_ref) * d_inv)
    bound_k = np.repeat(tol[kv::2] + tol[kv + 1::2], 2)
    bound = np.concatenate([bound_c, bound_k]) + bf16_step(row_ref) + 1e-4 * np.abs(row_ref)
    bad = np.abs(got - row_ref) > bound
    assert not bad.any(), f"{np.count_nonzero(bad)} entries outside the propagated tolerance"
    return row, bits_ref


@pytest.mark.parametrize("mode", [nmm.NMM_ROUND_EVEN, nmm.NMM_ROUND_AWAY])
def test_kv_update_deepseek_shape(mode):
    check_kv(syn.kv_update_case(), mode)


@pytest.mark.parametrize("hidden,kv,rope,ldw,position", [
    (200, 48, 16, 64, 0), (77, 5, 2, 8, 9), (4100, 1000, 88, 1088, 123), (33, 4096, 0, 4096, 2),
    (1536, 128, 64, 200, 70000), (9, 1, 0, 8, 0), (7168, 512, 64, 576, 1_000_003), (64, 8, 512, 520, 3),
])
def test_kv_update_ragged_shapes(hidden, kv, rope, ldw, position):
    c = syn.kv_update_case(seed=hidden + kv, hidden=hidden, kv_lora=kv, rope=rope, position=position, ldw=ldw)
    check_kv(c, nmm.NMM_ROUND_EVEN, cache_rows=position + 1 if position > 1000 else None,
             ld_cache=kv + rope if position > 1000 else None)


@pytest.mark.parametrize("mode", [nmm.NMM_ROUND_EVEN, nmm.NMM_ROUND_AWAY])
def test_kv_update_rounding_mode_on_exact_ties(mode):
    # h = (1, 1): mm = W[0] + W[1] = (257, 0, 0, -257 | 259, -257) exactly; eps = 32511.5 makes
    # the RMS root 256, gamma = 256 keeps the latent values at the ties +-257; position 0 leaves
    # the RoPE values as they are
    hidden, kv, rope = 2, 4, 2
    W0 = [256.0, 0.0, 0.0, -256.0, 258.0, -256.0]
    W1 = [1.0, 0.0, 0.0, -1.0, 1.0, -1.0]
    w = syn.bits_from_f32(np.array([W0, W1], np.float32), syn.BF16)
    w = syn.padded(w, 8)
    h = syn.bits_from_f32(np.array([[1.0, 1.0]], np.float32), syn.BF16)
    gamma = syn.bits_from_f32(np.array([256.0, 1.0, 1.0, 256.0], np.float32), syn.BF16)
    c = syn.KvUpdateCase(h, w, gamma, kv, rope, 0, eps=32511.5)
    mm, cache = run_kv(c, mode, cache_rows=2, ld_cache=8)
    assert mm.tolist() == [257.0, 0.0, 0.0, -257.0, 259.0, -257.0]
    row = cache[0].view(torch.int16).cpu().numpy().view(np.uint16)[:6]
    if mode == nmm.NMM_ROUND_EVEN:
        assert row.tolist() == [0x4380, 0x0000, 0x0000, 0xC380, 0x4382, 0xC380]
    else:
        assert row.tolist() == [0x4381, 0x0000, 0x0000, 0xC381, 0x4382, 0xC381]
    _, bits = oracle.kv_entry(mm, gamma, kv, 32511.5, c.theta, 0, mode)
    assert np.array_equal(row, bits)


def test_kv_update_back_to_back_calls_share_a_workspace():
    # the panel counter must return to zero: a second call (another shape and position) on the
    # same workspace must still build its entry exactly once and correctly
    ws = nmm.Workspace()
    a = syn.kv_update_case(seed=21, position=5)
    b = syn.kv_update_case(seed=22, hidden=1536, kv_lora=128, rope=64, position=7, ldw=200)
    for c in (a, b, a):
        check_kv(c, nmm.NMM_ROUND_EVEN, workspace=ws)
