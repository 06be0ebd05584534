"""GPU parity of the MLA decode chain (nmm_mla_decode_chain), checked step by step.

Each step is compared with the oracle fed exactly the bf16 operand the GPU consumed; every bf16
hand-off must equal the oracle's ties-to-even rounding of the GPU's own fp32 result bit for bit
(the rounding decision is taken in the same precision on both sides).  The chain also runs
concurrently with latent attention on a second stream and inside a captured HIP graph; both
must reproduce the eager, serial results exactly.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import assert_parity, dev16, host_bits

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")


def alloc_chain(step, device="cuda"):
    d = step.dims
    n_down = d["q_lora"] + d["kv_lora"] + d["rope"]
    qk = d["nope"] + d["rope"]
    f32 = lambda n: torch.full((n,), np.nan, dtype=torch.float32, device=device)
    b16 = lambda n: torch.zeros((n,), dtype=torch.bfloat16, device=device)
    bufs = dict(x=dev16(step.x, syn.BF16), w_down=dev16(step.w_down, syn.BF16), w_uq=dev16(step.w_uq, syn.BF16),
                w_uk=dev16(step.w_uk, syn.BF16), w_uv=dev16(step.w_uv, syn.BF16), w_o=dev16(step.w_o, syn.BF16),
                down_f32=f32(n_down), q_f32=f32(d["heads"] * qk), lat_f32=f32(d["heads"] * d["kv_lora"]),
                o_f32=f32(d["heads"] * d["v_head"]), y=f32(d["hidden"]), cq_bf16=b16(d["q_lora"]),
                qnope_bf16=b16(d["heads"] * d["nope"]), lat_bf16=b16(d["heads"] * d["kv_lora"]),
                o_bf16=b16(d["heads"] * d["v_head"]))
    return bufs


def small_step(seed=11):
    # the decode step's structure at reduced sizes (several panels, ragged tails, split K)
    rng = np.random.default_rng(seed)
    d = dict(hidden=1032, q_lora=264, kv_lora=136, rope=24, heads=6, nope=40, v_head=24)
    nb = lambda shape, k: syn.normal_bits(rng, shape, 1 / math.sqrt(k), syn.BF16)
    n_down = d["q_lora"] + d["kv_lora"] + d["rope"]
    qk = d["nope"] + d["rope"]
    s = syn.DecodeStep(x=syn.normal_bits(rng, (1, d["hidden"]), 1.0, syn.BF16),
                       w_down=nb((d["hidden"], n_down), d["hidden"]),
                       w_uq=nb((d["q_lora"], d["heads"] * qk), d["q_lora"]),
                       w_uk=nb((d["heads"], d["nope"], d["kv_lora"]), d["nope"]),
                       w_uv=nb((d["heads"], d["kv_lora"], d["v_head"]), d["kv_lora"]),
                       w_o=nb((d["heads"] * d["v_head"], d["hidden"]), d["heads"] * d["v_head"]),
                       q=None, kv=None)
    s.dims = d
    return s


def check_chain_stepwise(step, bufs):
    d = step.dims
    qk = d["nope"] + d["rope"]
    H = d["heads"]
    get = lambda k: bufs[k].cpu().numpy()
    # 1) down-projection (the paper's MatMul 2, widened)
    y_ref, a_ref = oracle.gemv(step.x, step.w_down, syn.BF16)
    assert_parity(get("down_f32")[None], y_ref, a_ref, what="down-projection")
    cq = host_bits(bufs["cq_bf16"])
    assert np.array_equal(cq, oracle.round_bf16(get("down_f32")[:d["q_lora"]])), "c_q bf16 hand-off"
    # 2) W_UQ
    y_ref, a_ref = oracle.gemv(cq[None], step.w_uq, syn.BF16)
    assert_parity(get("q_f32")[None], y_ref, a_ref, what="W_UQ")
    qn = host_bits(bufs["qnope_bf16"]).reshape(H, d["nope"])
    assert np.array_equal(qn, oracle.round_bf16(get("q_f32").reshape(H, qk)[:, :d["nope"]])), "q_nope hand-off"
    # 3) per-head W_UK
    y_ref, a_ref = oracle.batched_gemv(qn[:, None, :], step.w_uk, syn.BF16)
    assert_parity(get("lat_f32").reshape(H, 1, -1), y_ref, a_ref, what="W_UK")
    lat = host_bits(bufs["lat_bf16"]).reshape(H, 1, d["kv_lora"])
    assert np.array_equal(lat.reshape(-1), oracle.round_bf16(get("lat_f32"))), "latent hand-off"
    # 4) per-head W_UV
    y_ref, a_ref = oracle.batched_gemv(lat, step.w_uv, syn.BF16)
    assert_parity(get("o_f32").reshape(H, 1, -1), y_ref, a_ref, what="W_UV")
    o = host_bits(bufs["o_bf16"])
    assert np.array_equal(o, oracle.round_bf16(get("o_f32"))), "o hand-off"
    # 5) W_O
    y_ref, a_ref = oracle.gemv(o[None], step.w_o, syn.BF16)
    assert_parity(get("y")[None], y_ref, a_ref, what="W_O")
    return get("y")


def run_chain(step, bufs, stream=None, events=None, workspace=None):
    nmm.nmm_mla_decode_chain(step.dims, bufs, stream=stream, events=events, workspace=workspace)


def test_chain_small_stepwise():
    step = small_step()
    bufs = alloc_chain(step)
    run_chain(step, bufs)
    torch.cuda.synchronize()
    check_chain_stepwise(step, bufs)


def test_chain_decode_step_full_size():
    step = syn.decode_step()
    bufs = alloc_chain(step)
    events = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    run_chain(step, bufs, events=events)
    torch.cuda.synchronize()
    y = check_chain_stepwise(step, bufs)
    # W_UK and W_UV run as one launch here: events 2 and 3 are recorded together before it
    gaps = [events[i].elapsed_time(events[i + 1]) for i in range(5)]
    assert all(g >= 0 for g in gaps) and all(gaps[i] > 0 for i in (0, 1, 3, 4)), gaps
    # end to end against the oracle's own chain: the bf16 hand-offs may round differently near
    # ties, so only the overall agreement is checked here
    y_chain = oracle.mla_chain(step)[0]
    rel = np.linalg.norm(y - y_chain) / np.linalg.norm(y_chain)
    assert rel < 1e-2, rel


def test_chain_concurrent_with_attention_matches_serial():
    step = small_step(5)
    q, kv, scale = syn.attention_case(6, 128, 4096)
    qd, kvd = dev16(q, syn.BF16), dev16(kv, syn.BF16)
    ref_bufs = alloc_chain(step)
    run_chain(step, ref_bufs)
    att_ref = torch.empty((128, 512), device="cuda")
    nmm.nmm_latent_attention(qd, kvd, att_ref, scale)
    torch.cuda.synchronize()

    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    ws_a, ws_b = nmm.Workspace(), nmm.Workspace()
    bufs = alloc_chain(step)
    att = torch.empty((128, 512), device="cuda")
    start = torch.cuda.Event()
    start.record()
    a.wait_event(start)
    b.wait_event(start)
    for _ in range(3):
        run_chain(step, bufs, stream=a, workspace=ws_a)
        nmm.nmm_latent_attention(qd, kvd, att, scale, stream=b, workspace=ws_b)
    torch.cuda.synchronize()
    for k in nmm.CHAIN_BUFFERS[6:]:
        assert torch.equal(bufs[k], ref_bufs[k]), k
    assert torch.equal(att, att_ref)
    ref, ref_abs = oracle.latent_attention(q, kv, scale)
    assert_parity(att, ref, ref_abs, what="attention on stream B")


def test_default_workspaces_on_two_streams_unsized_and_unsynchronised():
    # no workspace given and nothing sized beforehand: each stream gets its own default
    # workspace, zeroed on that stream before the call's kernels, so the chain on one stream and
    # the attention on the other share no partial sums or counters
    step = small_step(13)
    q, kv, scale = syn.attention_case(14, 128, 4096)
    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(a):
        bufs = alloc_chain(step)
    with torch.cuda.stream(b):
        qd, kvd = dev16(q, syn.BF16), dev16(kv, syn.BF16)
        att = torch.full((128, 512), float("nan"), device="cuda")
    for _ in range(2):
        run_chain(step, bufs, stream=a)
        nmm.nmm_latent_attention(qd, kvd, att, scale, stream=b)
    torch.cuda.synchronize()
    check_chain_stepwise(step, bufs)
    ref, ref_abs = oracle.latent_attention(q, kv, scale)
    assert_parity(att, ref, ref_abs, what="attention on the second stream")


def test_chain_graph_replays_match_eager():
    step = small_step(7)
    eager = alloc_chain(step)
    run_chain(step, eager)
    torch.cuda.synchronize()
    bufs = alloc_chain(step)
    ws = nmm.Workspace()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        run_chain(step, bufs, workspace=ws)      # sizes the workspace before capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            run_chain(step, bufs, workspace=ws)
    torch.cuda.synchronize()
    for rep in range(3):
        for k in ("y", "down_f32", "q_f32", "lat_f32", "o_f32"):
            bufs[k].fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in nmm.CHAIN_BUFFERS[6:]:
            assert torch.equal(bufs[k], eager[k]), (rep, k)
        junk = torch.randn(1 << 20, device="cuda").sum()   # eager work between replays
        torch.cuda.synchronize()
        del junk


def test_workspace_garbage_past_counter_block_is_harmless():
    # Only the first 64 KiB of a workspace hold arrival counters; whatever earlier calls left in
    # the rest (partial sums of other shapes) must not matter.
    step = small_step(3)
    ref = alloc_chain(step)
    run_chain(step, ref)
    torch.cuda.synchronize()
    ws = nmm.Workspace()
    ws.get(32 << 20)
    ws.buf[65536:].fill_(0x7F)
    bufs = alloc_chain(step)
    run_chain(step, bufs, workspace=ws)
    torch.cuda.synchronize()
    for k in nmm.CHAIN_BUFFERS[6:]:
        assert torch.equal(bufs[k], ref[k]), k
    assert int(ws.buf[:65536].view(torch.int32).abs().sum()) == 0
    # a single split-K GEMV and the attention merge on the same dirty workspace
    c = syn.down_projection()
    y = torch.empty((1, c.N), device="cuda")
    nmm.nmm_gemv(dev16(c.x, c.dt), dev16(c.W, c.dt), y, workspace=ws)
    q, kv, scale = syn.attention_case(2, 128, 4096)
    att = torch.empty((128, 512), device="cuda")
    nmm.nmm_latent_attention(dev16(q, syn.BF16), dev16(kv, syn.BF16), att, scale, workspace=ws)
    torch.cuda.synchronize()
    y_ref, a_ref = oracle.gemv(c.x, c.W, c.dt)
    assert_parity(y, y_ref, a_ref, what="gemv on a dirty workspace")
    ref_att, ref_abs = oracle.latent_attention(q, kv, scale)
    assert_parity(att, ref_att, ref_abs, what="attention on a dirty workspace")


def pair_step(seed, heads, nope):
    # dimensions for which W_UK and W_UV run as one launch (kv_lora 512, v_head 128)
    rng = np.random.default_rng(seed)
    d = dict(hidden=520, q_lora=200, kv_lora=512, rope=16, heads=heads, nope=nope, v_head=128)
    nb = lambda shape, k: syn.normal_bits(rng, shape, 1 / math.sqrt(k), syn.BF16)
    n_down = d["q_lora"] + d["kv_lora"] + d["rope"]
    qk = d["nope"] + d["rope"]
    s = syn.DecodeStep(x=syn.normal_bits(rng, (1, d["hidden"]), 1.0, syn.BF16),
                       w_down=nb((d["hidden"], n_down), d["hidden"]),
                       w_uq=nb((d["q_lora"], d["heads"] * qk), d["q_lora"]),
                       w_uk=nb((d["heads"], d["nope"], d["kv_lora"]), d["nope"]),
                       w_uv=nb((d["heads"], d["kv_lora"], d["v_head"]), d["kv_lora"]),
                       w_o=nb((d["heads"] * d["v_head"], d["hidden"]), d["heads"] * d["v_head"]),
                       q=None, kv=None)
    s.dims = d
    return s


@pytest.mark.parametrize("heads,nope", [(3, 64), (5, 128), (2, 512)])
def test_chain_paired_heads_stepwise(heads, nope):
    # the single-launch W_UK -> W_UV at its smallest, the model's and its largest nope
    step = pair_step(heads * 100 + nope, heads, nope)
    bufs = alloc_chain(step)
    run_chain(step, bufs)
    torch.cuda.synchronize()
    check_chain_stepwise(step, bufs)


def test_chain_pair_agrees_with_two_batched_launches():
    # the pair sums the same per-head products as two nmm_batched_gemv launches, in another order:
    # the latents agree to rounding, and the pair's hand-offs pass the oracle step by step
    step = syn.decode_step()
    one = alloc_chain(step)
    run_chain(step, one)
    torch.cuda.synchronize()
    d = step.dims
    uk = dev16(step.w_uk, syn.BF16)
    lat = torch.empty((d["heads"], 1, d["kv_lora"]), dtype=torch.float32, device="cuda")
    nmm.nmm_batched_gemv(one["qnope_bf16"].view(d["heads"], 1, d["nope"]), uk, lat)
    torch.cuda.synchronize()
    a, b = one["lat_f32"].cpu().numpy().reshape(-1), lat.cpu().numpy().reshape(-1)
    assert np.abs(a - b).max() <= 1e-5 * np.abs(b).max()
    check_chain_stepwise(step, one)


def kv_for(step, seed, position, cache_rows, mode=0):
    d = step.dims
    rng = np.random.default_rng(seed)
    gamma = syn.bits_from_f32((1.0 + 0.1 * rng.standard_normal(d["kv_lora"], dtype=np.float32)), syn.BF16)
    n = d["kv_lora"] + d["rope"]
    cache = torch.full((cache_rows, n + 8), 0x7FC1, dtype=torch.int16, device="cuda")
    return dict(gamma=dev16(gamma, syn.BF16), cache=cache.view(torch.bfloat16), eps=syn.KV_EPS,
                theta=syn.ROPE_THETA, position=position, round=mode), gamma


def check_kv_row(step, bufs, kv, gamma):
    d = step.dims
    q, kvl, n = d["q_lora"], d["kv_lora"], d["kv_lora"] + d["rope"]
    mm = bufs["down_f32"].cpu().numpy().astype(np.float64)[q:q + n]
    row_ref, bits_ref = oracle.kv_entry(mm, gamma, kvl, kv["eps"], kv["theta"], kv["position"], kv["round"])
    cache = kv["cache"].view(torch.int16).cpu().numpy().view(np.uint16)
    row = cache[kv["position"]]
    got = oracle.decode(row[:n], syn.BF16)
    step_ = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(row_ref), 2.0 ** -126))) - 7)
    slack = 1e-4 * np.abs(row_ref) + np.concatenate([np.zeros(kvl), 1e-6 * np.repeat(
        np.abs(mm[kvl::2]) + np.abs(mm[kvl + 1::2]), 2)])
    assert np.all(np.abs(got - row_ref) <= 0.5 * step_ + slack), "cache entry is not a rounding of the oracle's"
    assert np.count_nonzero(row[:n] == bits_ref) >= 0.99 * n
    assert np.all(row[n:] == 0x7FC1)
    others = np.delete(cache, kv["position"], axis=0)
    assert np.all(others == 0x7FC1), "another cache row was written"


@pytest.mark.parametrize("full", [False, True])
def test_chain_with_cache_entry(full):
    step = syn.decode_step() if full else small_step(7)
    pos = 4096 if full else 37
    kv, gamma = kv_for(step, 3, pos, pos + 2, mode=nmm.NMM_ROUND_AWAY if not full else nmm.NMM_ROUND_EVEN)
    bufs = alloc_chain(step)
    run_chain_kv = lambda b, k: nmm.nmm_mla_decode_chain(step.dims, b, kv=k)
    run_chain_kv(bufs, kv)
    ref = alloc_chain(step)
    run_chain(step, ref)
    torch.cuda.synchronize()
    check_chain_stepwise(step, bufs)
    check_kv_row(step, bufs, kv, gamma)
    # the entry changes nothing else the chain writes
    for k in nmm.CHAIN_BUFFERS[6:]:
        assert torch.equal(bufs[k].view(torch.int32) if bufs[k].dtype == torch.float32 else bufs[k].view(torch.int16),
                           ref[k].view(torch.int32) if ref[k].dtype == torch.float32 else ref[k].view(torch.int16)), k


def test_chain_with_cache_entry_in_graph_replays():
    # captured once, replayed several times with eager work between replays: the entry's panel
    # counter must return to zero every time and each replay must write the same row
    step = small_step(8)
    kv, gamma = kv_for(step, 4, 5, 9)
    bufs = alloc_chain(step)
    s = torch.cuda.Stream()
    ws = nmm.Workspace()
    nmm.nmm_mla_decode_chain(step.dims, bufs, kv=kv, workspace=ws)
    torch.cuda.synchronize()
    first = kv["cache"].view(torch.int16).clone()
    with torch.cuda.stream(s):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            nmm.nmm_mla_decode_chain(step.dims, bufs, kv=kv, workspace=ws, stream=s)
    for _ in range(4):
        kv["cache"].view(torch.int16).fill_(0x7FC1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(kv["cache"].view(torch.int16), first)
    check_chain_stepwise(step, bufs)
    check_kv_row(step, bufs, kv, gamma)
