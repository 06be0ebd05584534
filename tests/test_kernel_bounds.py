"""CPU model of the GEMV kernel's address arithmetic (gemv.hip), run over the planned grid for
every shape the GPU tests use: every W load must stay inside the W extent, every x read inside
x, every LDS access inside the launch's dynamic LDS, and every y / partial-sum / ticket access
inside its buffer.  This is the check that a launch cannot fault before it runs on a GPU.
"""
import numpy as np
import pytest

nmm = pytest.importorskip("paper_2609_16009_amd")
import synthetic as syn  # noqa: E402

WAVES, THREADS = 4, 256


def check_launch(batch, M, K, N, ldx, ldw, ldy, sx=None, sw=None, sy=None):
    p = nmm.nmm_gemv_plan(M, K, N, nmm.NMM_BF16, nmm.NMM_PATH_GEMV, batch=batch)
    if K == 0 or M == 0 or N == 0:
        return
    mt, items, mblocks = p["m_tile"], p["items"], p["m_blocks"]
    sx = M * ldx if sx is None else sx
    sw = K * ldw if sw is None else sw
    sy = M * ldy if sy is None else sy
    extent = ((K - 1) * ldw + (N + 7) // 8 * 8) * 2
    assert extent < 2 ** 31
    n_panels = p["n_full_panels"] + (1 if p["tail_chunks"] else 0)
    ks_max = max(p["split_k_full"], p["split_k_tail"])
    part_floats = batch * mblocks * n_panels * ks_max * mt * 512
    lg_tail = (p["tail_width"] - 1).bit_length() if p["tail_chunks"] else 0
    rows_max = max(p["rows_full"], p["rows_tail"])
    mg = min(mt, 4)
    lds_floats = max(rows_max * mt, mg * THREADS * 8)
    unroll = p["unroll"]
    tid = np.arange(THREADS)
    lane, wave = tid & 63, tid >> 6
    x_total = (batch - 1) * sx + (M - 1) * ldx + K       # elements a dense x needs
    y_total = (batch - 1) * sy + (M - 1) * ldy + N
    for item in range(items):
        full_lg = (p["panel_width"] - 1).bit_length()
        if item < p["n_full_panels"] * p["split_k_full"]:
            panel, sl = divmod(item, p["split_k_full"])
            lg, ks, rows, valid = full_lg, p["split_k_full"], p["rows_full"], p["panel_width"]
        else:
            panel, sl = p["n_full_panels"], item - p["n_full_panels"] * p["split_k_full"]
            lg, ks, rows, valid = lg_tail, p["split_k_tail"], p["rows_tail"], p["tail_chunks"]
        cw = 1 << lg
        c = lane & (cw - 1)
        rstep = WAVES << (6 - lg)
        rin = wave * (64 >> lg) + (lane >> lg)
        k0 = sl * rows
        assert rows % (rstep * unroll) == 0 and rows * mt <= lds_floats
        cc = np.minimum(c, valid - 1)
        nsteps = rows // rstep
        guard = k0 + rows > K
        for s in range(nsteps):
            row = k0 + rin + s * rstep
            off = row * ldw * 2 + ((panel << full_lg) + cc) * 16
            issued = row < K if guard else np.ones_like(row, bool)
            if not guard:
                assert np.all(row < K)
            assert np.all(off[issued] >= 0) and np.all(off[issued] + 16 <= extent)
            assert np.all((s * rstep + rin) * mt + mt - 1 < lds_floats)
        # reduction buffer and outputs
        assert np.max(((wave * mg + mg - 1) * cw + c) * 8 + 7) < lds_floats
        pcols = cw * 8
        for mb in range(mblocks):
            m0 = mb * mt
            for b in (0, batch - 1):
                ms = np.arange(mt)[:, None]
                cols = np.arange(pcols)[None, :]
                n = (panel << full_lg) * 8 + cols
                keep = (m0 + ms < M) & (n < N)
                yi = b * sy + (m0 + ms) * ldy + n
                assert np.all(yi[keep] < y_total) and np.all(yi[keep] >= 0)
                if ks > 1:
                    pbase = ((b * mblocks + mb) * n_panels + panel) * ks_max * mt * 512
                    pi = pbase + (ks - 1) * mt * 512 + ms * 512 + cols
                    assert np.all(pi < part_floats)
                    assert (b * mblocks + mb) * n_panels + panel < min(batch * mblocks * n_panels, 16384)
                xk = k0 + min(rows, K - k0) - 1
                xi = b * sx + (m0 + ms[keep.any(axis=1)]) * ldx + xk
                assert np.all(xi < x_total)


SHAPES = [  # batch, M, K, N, ldx, ldw
    (1, 1, 512, 512, 512, 512), (1, 1, 7168, 2112, 7168, 2112), (1, 1, 7168, 576, 7168, 576),
    (1, 1, 1536, 24576, 1536, 24576), (1, 16, 1536, 24576, 1536, 24576), (1, 32, 1536, 24576, 1536, 24576),
    (1, 2, 1536, 24576, 1536, 24576), (1, 1, 16384, 7168, 16384, 7168),
    (1, 3, 1021, 1031, 1024, 1032), (1, 1, 1, 1, 8, 8), (1, 5, 77, 3, 80, 8), (1, 16, 4099, 520, 4104, 520),
    (1, 7, 9000, 4200, 9000, 4200), (1, 1, 13, 8, 16, 8), (1, 2, 300, 64, 304, 64),
    (1, 1, 33000, 24, 33000, 24), (1, 9, 1536, 3000, 1536, 3000), (1, 1, 2048, 8200, 2048, 8200),
    (1, 2, 500, 70, 504, 72), (1, 1, 4000, 1000, 4000, 1000), (1, 1, 3000, 700, 3000, 704),
    (128, 1, 128, 512, 128, 512), (128, 1, 512, 128, 512, 128), (3, 2, 1000, 72, 1000, 72),
    (5, 16, 96, 1000, 96, 1000), (2, 1, 20000, 40, 20000, 40),
    (1, 1, 65521, 16383, 65528, 16384),   # W's extent 2^31 - 491,520 bytes: the largest offsets
]


@pytest.mark.parametrize("batch,M,K,N,ldx,ldw", SHAPES)
def test_gemv_launch_stays_in_bounds(batch, M, K, N, ldx, ldw):
    check_launch(batch, M, K, N, ldx, ldw, ldy=N)


def test_strided_query_slice_in_bounds():
    # x rows of 128 taken every 192 elements (q_nope inside [128, 192])
    check_launch(128, 1, 128, 512, ldx=128, ldw=512, ldy=512, sx=192)


@pytest.mark.parametrize("M,K,N,ldx,ldw", [(1, 1536, 24576, 1536, 24576), (16, 1536, 24576, 1536, 24576),
                                           (32, 1536, 24576, 1536, 24576), (5, 1021, 1031, 1024, 1032),
                                           (33, 4099, 520, 4104, 520), (17, 16384, 7168, 16384, 7168),
                                           (8, 100, 8, 104, 8), (32, 20000, 300, 20000, 304),
                                           (16, 65521, 16383, 65528, 16384)])
def test_mfma_launch_stays_in_bounds(M, K, N, ldx, ldw):
    check_mfma_launch(M, K, N, ldx, ldw)


def check_mfma_launch(M, K, N, ldx, ldw, dt=None):
    p = nmm.nmm_gemv_plan(M, K, N, nmm.NMM_BF16 if dt is None else dt, nmm.NMM_PATH_MFMA)
    mt, rows, ks, panels = p["m_tile"], p["rows_full"], p["split_k_full"], p["n_full_panels"]
    assert mt in (16, 32) and rows % 64 == 0 and ks * rows >= K and (ks - 1) * rows < K
    assert panels * 128 >= N and (panels - 1) * 128 < N
    # LDS: two stage buffers, each a W tile [64][136] and an x tile [mt][72], 16-bit elements
    assert 2 * (64 * 136 + mt * 72) * 2 <= 65536
    extent = ((K - 1) * ldw + (N + 7) // 8 * 8) * 2
    tid = np.arange(256)
    wc, wr0 = tid & 15, tid >> 4
    xm, xc = tid >> 3, tid & 7
    for mb in {0, p["m_blocks"] - 1}:
        m0 = mb * mt
        mrows = min(mt, M - m0)
        x_extent = ((mrows - 1) * ldx + (K + 7) // 8 * 8) * 2
        for sl in {0, ks - 1}:
            k0 = sl * rows
            stages = (min(rows, K - k0) + 63) // 64
            for st in range(stages):
                k = k0 + st * 64 + 8 * xc
                ok = (xm < mrows) & (k < K)
                off = (xm * ldx + k) * 2
                assert np.all(off[ok] + 16 <= x_extent)
                # the LDS x tile row of every loading thread exists
                assert np.all(xm[tid < mt * 8] < mt)
    for panel in {0, panels - 1}:
        n0 = panel * 128
        valid = min(16, (N - n0 + 7) // 8)
        for sl in {0, ks - 1}:
            k0 = sl * rows
            for st in range(rows // 64):
                for q in range(4):
                    row = k0 + st * 64 + wr0 + 16 * q
                    ok = (row < K) & (wc < valid)
                    off = row * ldw * 2 + (n0 // 8 + wc) * 16
                    assert np.all(off[ok] + 16 <= extent)
        # outputs of the tile stay inside y / the partial buffer
        assert n0 + 127 >= min(N - 1, n0)
    assert p["grid"] == p["m_blocks"] * panels * ks


@pytest.mark.parametrize("case", syn.random_gemv_shapes(), ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}_{c[6]}")
def test_random_gemv_shapes_stay_in_bounds(case):
    """The seeded sweep the GPU tests run (synthetic.random_gemv_shapes), through the model of the
    path each call takes."""
    M, K, N, dt, ldx, ldw, path = case
    code = {"gemv": nmm.NMM_PATH_GEMV, "mfma": nmm.NMM_PATH_MFMA, "auto": nmm.NMM_PATH_AUTO}[path]
    taken = nmm.nmm_gemv_plan(M, K, N, dt, code)["path"]
    if taken == nmm.NMM_PATH_MFMA:
        check_mfma_launch(M, K, N, ldx, ldw, dt)
    else:
        assert taken == nmm.NMM_PATH_GEMV
        check_launch(1, M, K, N, ldx, ldw, ldy=N)


@pytest.mark.parametrize("nope", [64, 128, 192, 512])
def test_head_pair_loads_stay_in_bounds(nope):
    # head_pair_kernel: W_UK[h] is nope rows of 1 KB, W_UV[h] 512 rows of 256 B; 16 row-steps
    # in flight, W_UK's last 16 steps reload with W_UV's first 16, W_UV's last reload past the end
    U, lat, v = 16, 512, 128
    assert nope % (4 * U) == 0
    tid = np.arange(256)
    lane, wave = tid & 63, tid >> 6
    ta, tb = nope // 4, lat // 16
    uk_bytes, uv_bytes = nope * lat * 2, lat * v * 2
    off_a = lambda t: (4 * t + wave) * lat * 2 + lane * 16
    off_b = lambda t: (16 * t + 4 * wave + (lane >> 4)) * v * 2 + (lane & 15) * 16 if t < tb else None
    issued_a = list(range(U)) + [t0 + u + U for t0 in range(0, ta - U, U) for u in range(U)]
    assert sorted(issued_a) == list(range(ta))                 # every W_UK step exactly once
    for t in issued_a:
        assert np.all(off_a(t) + 16 <= uk_bytes) and np.all(off_a(t) >= 0)
    issued_b = list(range(U)) + [t + u + U for t in range(0, tb, U) for u in range(U)]
    assert sorted(x for x in issued_b if x < tb) == list(range(tb))   # every W_UV step once
    for t in issued_b:
        o = off_b(t)
        if o is not None:
            assert np.all(o + 16 <= uv_bytes)
    # rows used by the multiply-adds: x of W_UK and the latent of W_UV
    assert max(4 * t + 3 for t in range(ta)) < nope
    assert max(16 * t + 15 for t in range(tb)) < lat
    # q_nope: 8 values per lane, lanes with tid * 8 < nope
    assert np.all((tid * 16 + 16)[tid * 8 < nope] <= nope * 2)


KV_SHAPES = [  # hidden, kv_lora, rope, ldw
    (7168, 512, 64, 576), (200, 48, 16, 64), (77, 5, 2, 8), (4100, 1000, 88, 1088), (33, 4096, 0, 4096),
    (1536, 128, 64, 200), (9, 1, 0, 8), (64, 8, 512, 520),
]


@pytest.mark.parametrize("hidden,kv,rope,ldw", KV_SHAPES)
def test_kv_update_launch_stays_in_bounds(hidden, kv, rope, ldw):
    """MatMul 2 with its cache-entry epilogue (gemv_kv_kernel): the GEMV part is the plain
    launch; the epilogue counts every panel of [0, kv + rope) exactly once, keeps its counter in
    the counter block, and stages kv + rope values, kv gamma values and one word per wave in the
    launch's LDS."""
    n = kv + rope
    ldx = (hidden + 7) // 8 * 8
    check_launch(1, 1, hidden, n, ldx, ldw, ldy=n)
    p = nmm.nmm_gemv_plan(1, hidden, n, nmm.NMM_BF16, nmm.NMM_PATH_GEMV)
    pcols = p["panel_width"] * 8
    panels_total = p["n_full_panels"] + (1 if p["tail_chunks"] else 0)
    first, last = 0, (n - 1) // pcols
    assert first == 0 and last == panels_total - 1     # every panel of the launch counts in once
    n_tickets = panels_total if max(p["split_k_full"], p["split_k_tail"]) > 1 else 0
    assert panels_total + 1 <= 16384 and n_tickets < 16384   # the panel counter sits after the tickets
    rows_max = max(p["rows_full"], p["rows_tail"])
    lds_floats = max(rows_max * p["m_tile"], min(p["m_tile"], 4) * THREADS * 8, n + kv + WAVES)
    assert n + kv + WAVES <= lds_floats and lds_floats * 4 <= 64 * 1024   # y values, gamma, per-wave sums
    assert rope // 2 <= THREADS                         # one RoPE pair per thread



NT_SHAPES = [  # M, K, N, ldx, ldwt
    (1, 16384, 7168, 16384, 16384), (1, 7168, 2112, 7168, 7168), (1, 1536, 24576, 1536, 1536),
    (1, 1021, 1031, 1024, 1024), (1, 13, 8, 16, 16), (2, 20000, 40, 20000, 20000), (3, 4099, 520, 4104, 4104),
    (4, 9000, 4200, 9000, 9000), (5, 777, 300, 784, 784), (16, 1536, 3000, 1536, 1536), (1, 1, 1, 8, 8),
    (1, 100000, 64, 100000, 100000),
    (1, 16383, 65521, 65528, 16384),      # Wt's extent 2^31 - 491,520 bytes: the largest offsets
]


@pytest.mark.parametrize("M,K,N,ldx,ldwt", NT_SHAPES)
def test_gemv_nt_launch_stays_in_bounds(M, K, N, ldx, ldwt):
    """The transposed-weight GEMV (gemv_nt_kernel): every Wt load inside Wt's extent, x's staged
    slice (16-bit) inside the 32 KB staging limit and the launch's LDS, every LDS read of x inside it,
    partial sums and tickets inside the workspace, y writes inside y."""
    import ctypes
    L = nmm.lib()
    mt = 1 if M <= 1 else 2 if M <= 2 else 4
    mblocks = -(-M // mt)
    slice_max = 16384 // mt
    ks = -(-K // slice_max)
    slice_k = -(-(-(-K // ks)) // 512) * 512
    ks = -(-K // slice_k)
    target_rb = max(1, 256 // (ks * mblocks))
    r = min(8, max(1, N // (4 * target_rb)))
    rg = 1 if r < 2 else 2 if mt == 1 else 4
    r = -(-r // rg) * rg
    R = 4 * r
    row_blocks = -(-N // R)
    grid = mblocks * row_blocks * ks
    ws = L.nmm_gemv_nt_workspace_size(M, K, N, nmm.NMM_BF16)
    if ks > 1:
        assert ws == 64 * 1024 + grid * mt * R * 4 and mblocks * row_blocks <= 16384
    else:
        assert ws == 0
    extent = ((N - 1) * ldwt + (K + 7) // 8 * 8) * 2
    lds_halves = slice_k * mt
    lane = np.arange(64)
    part_floats = grid * mt * R
    for sl in sorted({0, ks - 1}):
        k0 = sl * slice_k
        klen = min(slice_k, K - k0)
        J = -(-klen // 512)
        assert J * 512 * mt <= 16384 and J * 512 * mt <= lds_halves         # staged x fits
        for rb in sorted({0, row_blocks - 1}):
            for wave in range(4):
                row0 = rb * R + wave * r
                for i in range(r):
                    n = row0 + i
                    for j in range(J):
                        k = k0 + j * 512 + 8 * lane
                        issued = (n < N) & (k < K)
                        off = n * ldwt * 2 + k * 2
                        assert np.all(off[issued] + 16 <= extent)
                        kb = j * 512 + 8 * lane
                        assert np.all((kb + 7) * mt + mt - 1 < lds_halves)   # LDS reads of x
                    if ks > 1:
                        for mb in range(mblocks):
                            pbase = ((mb * row_blocks + rb) * ks + sl) * mt * R
                            assert pbase + (mt - 1) * R + wave * r + i < part_floats


@pytest.mark.parametrize("case", syn.random_batched_shapes(), ids=lambda c: "x".join(map(str, c)))
def test_random_batched_shapes_stay_in_bounds(case):
    """The seeded sweep of the batched GEMV the GPU tests run (synthetic.random_batched_shapes)."""
    B, M, K, N = case
    check_launch(B, M, K, N, ldx=K, ldw=N, ldy=N)


@pytest.mark.parametrize("case", syn.random_nt_shapes(), ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}")
def test_random_nt_shapes_stay_in_bounds(case):
    """The seeded sweep of the transposed-weight GEMV the GPU tests run (synthetic.random_nt_shapes)."""
    M, K, N, dt, ldx, ldwt = case
    test_gemv_nt_launch_stays_in_bounds(M, K, N, ldx, ldwt)


@pytest.mark.parametrize("heads,nope,rope,kv,ldq", [(128, 128, 64, 512, 576), (6, 40, 24, 136, 160), (4, 16, 8, 24, 40),
                                                    (3, 8, 512, 8, 520), (1, 8, 2, 8, 10), (7, 16, 0, 8, 8)])
def test_qrope_workgroup_covers_each_pair_once(heads, nope, rope, kv, ldq):
    """The extra workgroup of the query launch (gemv_qrope_kernel): thread t takes pair
    t % (rope/2) of heads t / (rope/2), t / (rope/2) + 256 / (rope/2), ...; every (head, pair) is
    written exactly once, reads stay inside q [heads, nope + rope] and writes inside
    q_out[h * ldq + kv .. kv + rope)."""
    pairs = rope // 2
    if pairs == 0:
        return
    qk = nope + rope
    seen = np.zeros((heads, pairs), int)
    hstep = THREADS // pairs
    for t in range(THREADS):
        j, h0 = t % pairs, t // pairs
        if h0 >= hstep:
            continue
        for h in range(h0, heads, hstep):
            seen[h, j] += 1
            assert h * qk + nope + 2 * j + 1 < heads * qk
            assert kv + 2 * j + 1 < ldq and h * ldq + kv + 2 * j + 1 < heads * ldq
    assert np.all(seen == 1)


def default_spans(heads, seq):
    """The default partition before the span is rounded to whole chunks: about 64 (32-head block,
    span) pairs, or spans of at most 8 chunks, or of about 4 (chunks // 4 spans) while a grid of 16-head blocks
    still holds them at 256 workgroups (a multiple of 8 from 8 on), but spans of at least 2 chunks."""
    fit = 256 // -(-heads // 16) if heads else 256
    fit = fit // 8 * 8 if fit >= 8 else fit
    want = max(64 // max(1, -(-heads // 32)), -(-seq // 512), min(max(1, -(-seq // 64) // 4), fit))
    return max(1, min(-(-seq // 128), want))


@pytest.mark.parametrize("K,N", [(16384, 7168), (144, 1032), (2048, 512)])
def test_gemv_attention_launch_shares_lds_and_grid(K, N):
    """gemv_attention_kernel: workgroups [0, gemv_grid) run the GEMV exactly as its own launch
    (same ids, so the same items), the rest are attention workgroups 0 .. attention grid - 1; the
    GEMV's x slice (rows_max * 4 bytes, or the 4 x 256 x 8 floats of its reduction) must fit the
    first attention chunk buffer of 64 x 592 bf16.  Its attention workgroups take blocks of 32 heads."""
    p = nmm.nmm_gemv_plan(1, K, N, nmm.NMM_BF16, nmm.NMM_PATH_GEMV)
    assert p["m_tile"] == 1 and p["unroll"] in (8, 16)
    rows_max = max(p["rows_full"], p["rows_tail"])
    gemv_lds = max(rows_max * 1 * 4, 1 * 256 * 8 * 4)
    assert gemv_lds <= 64 * 592 * 2
    for heads, seq, splits in ((128, 4096, 16), (128, 4096, 0), (70, 300, 3), (1, 64, 1)):
        ws = nmm.nmm_latent_attention_workspace_size(heads, seq, 576, 512)
        n_hb = (heads + 31) // 32
        span = -(-seq // max(1, min(splits or default_spans(heads, seq),
                                     -(-seq // 64))))
        span = -(-span // 64) * 64
        nsp = -(-seq // span)
        agrid = n_hb * ((nsp + 7) // 8 * 8 if (nsp % 8 == 0 or nsp > 8) else nsp)
        total = p["grid"] + agrid
        ids = np.arange(total)
        gemv_ids, attn_ids = ids[ids < p["grid"]], ids[ids >= p["grid"]] - p["grid"]
        assert np.array_equal(gemv_ids, np.arange(p["grid"]))
        assert np.array_equal(attn_ids, np.arange(agrid)) and total < 2 ** 31
        assert ws >= 0


@pytest.mark.parametrize("heads", [1, 15, 16, 17, 20, 32, 33, 70, 128, 129])
@pytest.mark.parametrize("seq,splits", [(4096, 0), (4096, 16), (4096, 32), (300, 3), (65535, 64), (64, 0),
                                         (8192, 0), (16384, 0), (32768, 0), (1000, 0), (4097, 0), (8300, 0)])
def test_attention_spans_and_workspace_serve_both_head_blocks(heads, seq, splits):
    """The attention launch takes blocks of 16 heads (32 where 16 would take over 256 workgroups),
    workgroups beside a GEMV blocks of 32, over the same spans (default_spans).  Each form's span partials,
    [n_hb][nsp][block heads][d_v] floats then [n_hb][nsp][block heads][2], must fit past the counter
    block of the one workspace size the library reports for the call."""
    dv, ticket = 512, 64 * 1024
    L = nmm.lib()
    ws = L.nmm_latent_attention_workspace_size(heads, seq, 576, dv) if splits == 0 else \
        L.nmm_latent_attention_ex_workspace_size(heads, seq, 576, dv, splits)
    nsp = splits or default_spans(heads, seq)
    nsp = min(nsp, -(-seq // 64), 64)
    span = -(-(-(-seq // nsp)) // 64) * 64
    nsp = -(-seq // span)
    if nsp == 1:
        assert ws == 0
        return
    for hbh in (16, 32):
        n_hb = -(-heads // hbh)
        need = ticket + n_hb * nsp * hbh * (dv + 2) * 4
        assert need <= ws, (hbh, need, ws)
    assert ws == ticket + -(-heads // 32) * 32 * nsp * (dv + 2) * 4


@pytest.mark.parametrize("heads,dv,nsp,hbh", [(128, 512, 16, 16), (128, 512, 16, 32), (70, 512, 3, 16),
                                             (20, 64, 5, 32), (5, 272, 64, 16), (33, 16, 2, 32)])
def test_merge_blocks_cover_every_output_once(heads, dv, nsp, hbh):
    """The two merge forms over heads x ceil(d_v / 256) blocks: merge_block (256 threads, one column
    each) and merge_block_wide (64 threads, four columns each) must each write every (head,
    column < d_v) exactly once, and read the span partials [n_hb][nsp][hbh][d_v] and
    [n_hb][nsp][hbh][2] only inside those arrays."""
    n_cb = -(-dv // 256)
    blocks = heads * n_cb
    n_hb = -(-heads // hbh)
    o_size, ml_size = n_hb * nsp * hbh * dv, n_hb * nsp * hbh * 2
    for threads, width in ((256, 1), (64, 4)):
        seen = np.zeros((heads, dv), dtype=np.int64)
        for blk in range(blocks):
            h, cb = divmod(blk, n_cb)
            hb, hl = divmod(h, hbh)
            base = hb * nsp * hbh + hl
            for t in range(threads):
                c = cb * 256 + width * t
                if c >= dv:
                    continue
                for s_ in range(nsp):
                    first = (base + s_ * hbh) * dv + c
                    assert 0 <= first and first + width <= o_size
                    assert (base + s_ * hbh) * 2 + 2 <= ml_size
                seen[h, c:c + width] += 1
        assert np.all(seen == 1), (threads, width)


@pytest.mark.parametrize("n_hb,nsp,vsplit", [(2, 16, 1), (2, 11, 1), (2, 32, 1), (1, 9, 1), (3, 22, 1), (2, 3, 1),
                                            (1, 1, 1), (2, 64, 1), (8, 16, 2), (8, 8, 2), (5, 21, 2), (1, 3, 2),
                                            (1, 32, 4), (2, 32, 4), (1, 64, 4), (2, 3, 4)])
def test_attention_workgroups_cover_every_head_block_and_span_once(n_hb, nsp, vsplit):
    """attention_block's workgroup -> (head block, column part, span) map, with nb = n_hb x vsplit
    (head block hb, column part v at hb vsplit + v): from 8 spans on (xcd_map) the grid holds nsp
    padded to a multiple of 8 per nb, workgroup b takes span (b % 8) + 8 (b / 8 nb) of index
    (b / 8) % nb, and the padding spans exit; otherwise the plain order.  Every (head block,
    column part, span) runs once, and with xcd_map the workgroups of one span sit 8 ids apart, on
    one XCD (ids are dealt to the 8 XCDs round robin; the decode step's shared launches put the
    attention's workgroups first)."""
    nb = n_hb * vsplit
    xcd_map = nsp % 8 == 0 or nsp > 8
    grid_sp = (nsp + 7) // 8 * 8 if xcd_map else nsp
    seen = {}
    for b in range(nb * grid_sp):
        if xcd_map:
            sp, hbv = (b & 7) + 8 * (b // (8 * nb)), (b >> 3) % nb
            if sp >= nsp:
                continue
        else:
            hbv, sp = b % nb, b // nb
        key = (hbv // vsplit, hbv % vsplit, sp)
        assert key not in seen
        seen[key] = b
    assert set(seen) == {(h, v, s_) for h in range(n_hb) for v in range(vsplit) for s_ in range(nsp)}
    if xcd_map:
        for s_ in range(nsp):
            assert len({seen[(h, v, s_)] % 8 for h in range(n_hb) for v in range(vsplit)}) == 1
