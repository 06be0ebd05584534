"""GPU parity of nmm_gemv / nmm_batched_gemv against the oracle, through the C ABI.

Floating-point cases must satisfy |y - y_ref| <= 4e-3 * sum_k |x_k W_kn| + 1e-6 elementwise;
integer-valued cases (every partial sum exact in fp32) must match bit for bit.  Sizes span
several panels, K-slices and ragged tails; the workload shapes are the full decode shapes.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import assert_parity, dev16, host_bits

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")


def run_gemv(c: syn.GemvCase, path=None, ldy=None, fill=np.nan):
    path = nmm.NMM_PATH_AUTO if path is None else path
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    ldy = c.N if ldy is None else ldy
    y = torch.full((c.M, ldy), fill, dtype=torch.float32, device="cuda")
    nmm.nmm_gemv(x, W, y, N=c.N, path=path)
    torch.cuda.synchronize()
    return y


def check_case(c: syn.GemvCase, path=None):
    y = run_gemv(c, path)
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt, K=c.K, N=c.N)
    return assert_parity(y, y_ref, a_ref, integer=c.integer, what=c.name)


@pytest.mark.parametrize("integer", [False, True])
def test_single_gemv_512_fp16(integer):
    check_case(syn.single_gemv_512(integer))


@pytest.mark.parametrize("integer", [False, True])
def test_down_projection_7168x2112(integer):
    check_case(syn.down_projection(integer))


def test_paper_matmul2_7168x576():
    check_case(syn.down_projection(n=576))


@pytest.mark.parametrize("M", [1, 2, 4, 8, 16, 32])
def test_uq_sweep_gemv_path(M):
    check_case(syn.uq_sweep(M), path=nmm.NMM_PATH_GEMV)


@pytest.mark.parametrize("M", [1, 16])
def test_uq_sweep_integer_exact(M):
    check_case(syn.uq_sweep(M, integer=True), path=nmm.NMM_PATH_GEMV)


def test_output_projection_16384x7168():
    check_case(syn.gemv_case(40, 1, 16384, 7168, syn.BF16, name="wo_16384x7168"))


RAGGED = [  # (M, K, N, dt, ldx, ldw)
    (3, 1021, 1031, syn.BF16, 1024, 1032),
    (1, 1, 1, syn.BF16, 8, 8),
    (5, 77, 3, syn.F16, 80, 8),
    (16, 4099, 520, syn.BF16, 4104, 520),
    (7, 9000, 4200, syn.F16, 9000, 4200),
    (1, 13, 8, syn.BF16, 16, 8),
    (2, 300, 64, syn.F16, 304, 64),
    (1, 33000, 24, syn.BF16, 33000, 24),
    (9, 1536, 3000, syn.BF16, 1536, 3000),
    (1, 2048, 8200, syn.BF16, 2048, 8200),
]


@pytest.mark.parametrize("M,K,N,dt,ldx,ldw", RAGGED)
def test_ragged_shapes_and_padding(M, K, N, dt, ldx, ldw):
    c = syn.gemv_case(1000 + M * K % 97, M, K, N, dt, ldx=ldx, ldw=ldw, name=f"ragged_{M}x{K}x{N}")
    check_case(c, path=nmm.NMM_PATH_GEMV)


@pytest.mark.parametrize("M,K,N,dt", [(3, 1021, 1031, syn.BF16), (16, 4099, 520, syn.F16),
                                      (1, 7168, 2112, syn.F16)])
def test_ragged_integer_exact(M, K, N, dt):
    c = syn.gemv_case(7, M, K, N, dt, integer=True, ldx=(K + 7) // 8 * 8, ldw=(N + 7) // 8 * 8,
                      name="ragged_int")
    check_case(c, path=nmm.NMM_PATH_GEMV)


@pytest.mark.parametrize("case", syn.random_gemv_shapes(), ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}_{c[6]}")
def test_random_shapes_integer_exact(case):
    # a seeded sweep over M, K, N, both 16-bit types, padded pitches and the three path choices
    # (the launch-bounds model checks the same cases): small integers, so every output is exact
    M, K, N, dt, ldx, ldw, path = case
    c = syn.gemv_case(500 + M + K % 97, M, K, N, dt, integer=True, ldx=ldx, ldw=ldw, name=f"random_{M}x{K}x{N}_{path}")
    check_case(c, path={"gemv": nmm.NMM_PATH_GEMV, "mfma": nmm.NMM_PATH_MFMA, "auto": nmm.NMM_PATH_AUTO}[path])


def test_largest_weight_extent_on_every_path():
    # one weight [65521, 16384] bf16 whose extent, 65521 * 16384 * 2 = 2^31 - 491,520 bytes, is just
    # under the 2^31-byte limit, so the 32-bit buffer offsets take their largest values.  As W
    # [65521, 16383] (padding column NaN) it feeds the GEMV (one row, every output) and the matrix
    # cores (16 rows, sampled columns); the same bytes as Wt [65521 rows, 16383 + 1] feed the
    # transposed path (sampled rows).  Values are small integers, so every sum is exact in fp32.
    K, N, ldw = 65521, 16383, 16384
    c = syn.large_int_case(61, 16, K, N, ldw)
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    rng = np.random.default_rng(5)
    y1 = torch.full((1, N), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv(x[:1], W, y1, N=N, path=nmm.NMM_PATH_GEMV)
    y16 = torch.full((16, N), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv(x, W, y16, N=N, path=nmm.NMM_PATH_MFMA)
    Kt, Nt = ldw - 1, K
    yt = torch.full((1, Nt), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv_nt(x[:1, :Kt], W, yt, K=Kt)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x[:1], c.W, c.dt, K=K, N=N)
    assert_parity(y1, y_ref, a_ref, integer=True, what="GEMV at the largest extent")
    cols = np.unique(np.r_[0, 1, 127, 128, 8191, 8192, N - 129, N - 2, N - 1, rng.choice(N, 119, replace=False)])
    y_ref, a_ref = oracle.gemv(c.x, np.ascontiguousarray(c.W[:, cols]), c.dt, K=K, N=len(cols))
    assert_parity(y16[:, cols], y_ref, a_ref, integer=True, what="MFMA at the largest extent")
    rows = np.unique(np.r_[0, 1, 31, 32, Nt // 2, Nt - 33, Nt - 2, Nt - 1, rng.choice(Nt, 120, replace=False)])
    Ws = np.ascontiguousarray(c.W[rows, :Kt].T)           # [Kt, len(rows)]: the sampled rows of Wt as W
    y_ref, a_ref = oracle.gemv(c.x[:1], Ws, c.dt, K=Kt, N=len(rows))
    assert_parity(yt[:, rows], y_ref, a_ref, integer=True, what="transposed path at the largest extent")


def test_output_padding_untouched():
    c = syn.gemv_case(3, 2, 500, 70, syn.BF16, ldx=504, ldw=72)
    y = run_gemv(c, ldy=80, fill=-7.0)
    assert torch.all(y[:, 70:] == -7.0)
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt, N=70)
    assert_parity(y[:, :70], y_ref, a_ref)


def test_deterministic_and_workspace_reuse():
    big = syn.down_projection()
    small = syn.gemv_case(9, 1, 4000, 1000, syn.BF16)
    ws = nmm.Workspace()
    outs = []
    for c in (big, small, big, small):
        x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
        y = torch.empty((1, c.N), dtype=torch.float32, device="cuda")
        nmm.nmm_gemv(x, W, y, workspace=ws)
        torch.cuda.synchronize()
        outs.append(y.cpu())
    assert torch.equal(outs[0], outs[2]) and torch.equal(outs[1], outs[3])
    y_ref, a_ref = oracle.gemv(small.x, small.W, small.dt)
    assert_parity(outs[3], y_ref, a_ref)
    # every arrival counter (the workspace's first 64 KiB) is back at zero after the calls
    tickets = ws.buf[:65536].view(torch.int32)
    assert int(tickets.abs().sum()) == 0


@pytest.mark.parametrize("K,N", [(7168, 2112), (16384, 7168), (7168, 576)], ids=["down", "w_o", "matmul2"])
def test_split_k_soak_bit_identical(K, N):
    # 1000 launches of a split-K shape on one workspace: every result equals the first bit for
    # bit (the gather sums the slices in a fixed order, whichever XCD finishes first), and the
    # arrival counters are back at zero after the last
    c = syn.gemv_case(50, 1, K, N, syn.BF16, name=f"soak_{K}x{N}")
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    ws = nmm.Workspace()
    assert nmm.nmm_gemv_plan(1, K, N, syn.BF16, nmm.NMM_PATH_AUTO)["split_k_full"] > 1
    ref = torch.empty((1, N), dtype=torch.float32, device="cuda")
    nmm.nmm_gemv(x, W, ref, workspace=ws)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt)
    assert_parity(ref, y_ref, a_ref, what=c.name)
    ys = torch.empty((20, 1, N), dtype=torch.float32, device="cuda")
    for batch in range(50):
        ys.fill_(float("nan"))
        for i in range(20):
            nmm.nmm_gemv(x, W, ys[i], workspace=ws)
        same = (ys == ref).all(dim=2).view(-1)
        if not bool(same.all()):
            first = batch * 20 + int((~same).nonzero()[0])
            raise AssertionError(f"{c.name}: launch {first} differs from the first result")
    assert int(ws.buf[:65536].view(torch.int32).abs().sum()) == 0


def test_k_zero_writes_zeros_and_empty_is_noop():
    x = torch.zeros((2, 8), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((1, 16), dtype=torch.bfloat16, device="cuda")
    y = torch.full((2, 16), 5.0, device="cuda")
    st = nmm.lib().nmm_gemv(2, 0, 16, nmm.NMM_BF16, x.data_ptr(), 8, W.data_ptr(), 16, y.data_ptr(), 16,
                            0, None, 0, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == nmm.NMM_OK and torch.all(y == 0)
    y.fill_(5.0)
    st = nmm.lib().nmm_gemv(0, 8, 16, nmm.NMM_BF16, x.data_ptr(), 8, W.data_ptr(), 16, y.data_ptr(), 16,
                            0, None, 0, None)
    torch.cuda.synchronize()
    assert st == nmm.NMM_OK and torch.all(y == 5.0)


def test_invalid_call_enqueues_nothing():
    c = syn.gemv_case(5, 1, 256, 256, syn.BF16)
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    y = torch.full((1, 256), 3.0, device="cuda")
    st = nmm.lib().nmm_gemv(1, 256, 256, nmm.NMM_BF16, x.data_ptr(), 256, W.data_ptr() + 2, 256,
                            y.data_ptr(), 256, 0, None, 0, None)
    torch.cuda.synchronize()
    assert st == nmm.NMM_ERR_ALIGN and torch.all(y == 3.0)


def _loaded_hip_runtime():
    """The HIP runtime library this process has loaded (the one libnmm's calls go to)."""
    import ctypes
    with open("/proc/self/maps") as f:
        paths = {line.split()[-1] for line in f if "libamdhip64.so" in line}
    assert paths, "no HIP runtime loaded"
    return ctypes.CDLL(sorted(paths)[0])


def test_hip_error_reaches_the_caller_as_nmm_err_hip():
    # NMM_ERR_HIP reports what the HIP runtime says after the launch: here an error left unread
    # by an earlier runtime call on this thread (an invalid device ordinal, refused on the host;
    # nothing reaches the GPU), which the call reports once and so clears
    c = syn.gemv_case(5, 1, 256, 256, syn.BF16)
    x, W = dev16(c.x, c.dt), dev16(c.W, c.dt)
    y = torch.empty((1, 256), device="cuda")
    torch.cuda.synchronize()
    hip = _loaded_hip_runtime()
    assert hip.hipSetDevice(1 << 20) != 0
    args = (1, 256, 256, nmm.NMM_BF16, x.data_ptr(), 256, W.data_ptr(), 256, y.data_ptr(), 256, 0, None, 0, None)
    assert nmm.lib().nmm_gemv(*args) == nmm.NMM_ERR_HIP
    torch.cuda.synchronize()
    assert nmm.lib().nmm_gemv(*args) == nmm.NMM_OK
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt)
    assert_parity(y, y_ref, a_ref)


def test_infinity_propagates_to_its_column_only():
    c = syn.gemv_case(6, 1, 3000, 700, syn.BF16, ldw=704)
    W = c.W.copy()
    W[1234, 321] = 0x7F80          # +inf
    x = c.x.copy()
    x[0, 1234] = 0x3F80            # 1.0
    y = run_gemv(syn.GemvCase(1, 3000, 700, syn.BF16, x, W, name="inf"))
    y = y.cpu().numpy()[0]
    assert np.isposinf(y[321])
    mask = np.ones(700, bool)
    mask[321] = False
    assert np.isfinite(y[mask]).all()


# ------------------------------------------------------------------ batched (per-head)

def test_absorbed_heads_two_steps():
    h = syn.absorbed_heads()
    q = dev16(h.q_nope, h.dt)
    uk, uv = dev16(h.w_uk, h.dt), dev16(h.w_uv, h.dt)
    lat = torch.empty((128, 1, 512), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(q, uk, lat)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.batched_gemv(h.q_nope, h.w_uk, h.dt)
    assert_parity(lat, y_ref, a_ref, what="q_nope . W_UK")
    # step 2 consumes the GPU's step-1 result rounded to bf16 (ties to even)
    lat_bits = oracle.round_bf16(lat.cpu().numpy())
    o = torch.empty((128, 1, 128), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(dev16(lat_bits, h.dt), uv, o)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.batched_gemv(lat_bits, h.w_uv, h.dt)
    assert_parity(o, y_ref, a_ref, what="latent . W_UV")


def test_absorbed_heads_integer_exact():
    h = syn.absorbed_heads(integer=True)
    lat = torch.empty((128, 1, 512), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(dev16(h.q_nope, h.dt), dev16(h.w_uk, h.dt), lat)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.batched_gemv(h.q_nope, h.w_uk, h.dt)
    assert_parity(lat, y_ref, a_ref, integer=True, what="int q_nope . W_UK")


def test_batched_strided_query_slice():
    # q_nope is the first 128 of each head's 192 columns: a strided view, stride 192
    rng = np.random.default_rng(8)
    q_full = syn.normal_bits(rng, (128, 1, 192), 1.0, syn.BF16)
    h = syn.absorbed_heads()
    qd = dev16(q_full, syn.BF16)[:, :, :128]
    lat = torch.empty((128, 1, 512), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(qd, dev16(h.w_uk, h.dt), lat)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.batched_gemv(np.ascontiguousarray(q_full[:, :, :128]), h.w_uk, h.dt)
    assert_parity(lat, y_ref, a_ref, what="strided q_nope")


@pytest.mark.parametrize("B,M,K,N", [(3, 2, 1000, 72), (128, 1, 512, 128), (5, 16, 96, 1000), (2, 1, 20000, 40)])
def test_batched_ragged(B, M, K, N):
    rng = np.random.default_rng(B * 1000 + K)
    x = syn.normal_bits(rng, (B, M, K), 1.0, syn.BF16)
    W = syn.normal_bits(rng, (B, K, N), 1.0 / np.sqrt(K), syn.BF16)
    y = torch.empty((B, M, N), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(dev16(x, syn.BF16), dev16(W, syn.BF16), y, path=nmm.NMM_PATH_GEMV)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.batched_gemv(x, W, syn.BF16)
    assert_parity(y, y_ref, a_ref, what=f"batched {B}x{M}x{K}x{N}")


@pytest.mark.parametrize("case", syn.random_batched_shapes(), ids=lambda c: "x".join(map(str, c)))
def test_batched_random_shapes_integer_exact(case):
    # a seeded sweep (the launch-bounds model checks the same cases): small integers, so every
    # output of every batch entry is exact
    B, M, K, N = case
    rng = np.random.default_rng(B * 7919 + K + N)
    x = syn.int_bits(rng, (B, M, K), syn.BF16)
    W = syn.int_bits(rng, (B, K, N), syn.BF16)
    y = torch.full((B, M, N), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(dev16(x, syn.BF16), dev16(W, syn.BF16), y, path=nmm.NMM_PATH_GEMV)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.batched_gemv(x, W, syn.BF16)
    assert_parity(y, y_ref, a_ref, integer=True, what=f"batched {B}x{M}x{K}x{N}")


# ------------------------------------------------------------------ matrix-core path

@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 8, 16, 17, 32])
def test_uq_sweep_mfma_path(M):
    check_case(syn.uq_sweep(min(M, 32)) if M <= 32 else None, path=nmm.NMM_PATH_MFMA)


@pytest.mark.parametrize("M", [4, 32])
def test_uq_sweep_mfma_integer_exact(M):
    check_case(syn.uq_sweep(M, integer=True), path=nmm.NMM_PATH_MFMA)


@pytest.mark.parametrize("M,K,N,dt,ldx,ldw", [(5, 1021, 1031, syn.BF16, 1024, 1032), (33, 4099, 520, syn.F16, 4104, 520),
                                              (8, 100, 8, syn.BF16, 104, 8), (32, 20000, 300, syn.F16, 20000, 304),
                                              (17, 16384, 7168, syn.BF16, 16384, 7168)])
def test_mfma_ragged(M, K, N, dt, ldx, ldw):
    c = syn.gemv_case(77 + M, M, K, N, dt, ldx=ldx, ldw=ldw, name=f"mfma_{M}x{K}x{N}")
    check_case(c, path=nmm.NMM_PATH_MFMA)
    ci = syn.gemv_case(78 + M, M, K, N, dt, integer=True, ldx=ldx, ldw=ldw, name=f"mfma_int_{M}x{K}x{N}")
    check_case(ci, path=nmm.NMM_PATH_MFMA)


def test_auto_path_switches_at_crossover():
    # one row streams; W_UQ's matrix-core plan has a single K-slice, so two rows take the matrix
    # cores there, while W_O's (split K) keeps the streaming GEMV at two rows
    assert nmm.nmm_gemv_plan(1, 1536, 24576)["path"] == nmm.NMM_PATH_GEMV
    assert nmm.nmm_gemv_plan(2, 16384, 7168)["path"] == nmm.NMM_PATH_GEMV
    for M in (2, 3, 4, 16, 32):
        assert nmm.nmm_gemv_plan(M, 1536, 24576)["path"] == nmm.NMM_PATH_MFMA
    assert nmm.nmm_gemv_plan(16, 128, 512, batch=8)["path"] == nmm.NMM_PATH_GEMV


@pytest.mark.parametrize("M", [17, 20])
def test_remnant_split_on_two_streams(M):
    # the paper's Condition 4 split: rows [0, 16q) on the matrix cores and the remnant rows on
    # the streaming GEMV, concurrently on two streams into one y; both parts meet the fp32 bar
    c = syn.uq_sweep(32)
    q16 = M // 16 * 16
    x, W = dev16(c.x[:M], syn.BF16), dev16(c.W, syn.BF16)
    y = torch.full((M, c.N), float("nan"), dtype=torch.float32, device="cuda")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    start = torch.cuda.Event()
    start.record()
    sa.wait_event(start)
    sb.wait_event(start)
    nmm.nmm_gemv(x[:q16], W, y[:q16], path=nmm.NMM_PATH_MFMA, workspace=nmm.Workspace(), stream=sa)
    nmm.nmm_gemv(x[q16:], W, y[q16:], path=nmm.NMM_PATH_GEMV, workspace=nmm.Workspace(), stream=sb)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x[:M], c.W, syn.BF16)
    assert_parity(y, y_ref, a_ref, what=f"remnant split M={M}")
