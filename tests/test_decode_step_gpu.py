"""GPU parity of the decode step (nmm_mla_decode_step: the MLA chain and an independent latent
attention, the attention's workgroups sharing W_UQ's launch and its merge the W_UK -> W_UV pair's
(W_O's for chains without the pair), or with a cache entry the attention in W_O's launch),
through the C ABI.

The step must reproduce, bit for bit, what the chain (nmm_mla_decode_chain) and the attention
(nmm_latent_attention_ex with the same partition) write when run on their own: the shared launch
runs the same per-workgroup code.  Both are also checked against the oracle (the chain step by
step, the attention against the fp64 softmax attention).  Shapes the shared launch does not take
(a non-576/512 attention) must give the same results through the two launches in order.  An
attention that reads what the chain writes is refused before anything runs.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import assert_parity, dev16, host_bits
from test_chain_gpu import alloc_chain, check_chain_stepwise, check_kv_row, kv_for, pair_step, small_step

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")

OUTPUTS = ("down_f32", "q_f32", "lat_f32", "o_f32", "y", "cq_bf16", "qnope_bf16", "lat_bf16", "o_bf16")


def attn_bufs(q_bits, kv_bits, dv, bf16_copy=True):
    heads = q_bits.shape[0]
    out = torch.full((heads, dv), float("nan"), dtype=torch.float32, device="cuda")
    outb = torch.zeros((heads, dv + 8), dtype=torch.bfloat16, device="cuda") if bf16_copy else None
    return dev16(q_bits, syn.BF16), dev16(kv_bits, syn.BF16), out, outb


def run_separately(step, q, kv, scale, splits, dqk, dv, kv_entry=None):
    bufs = alloc_chain(step)
    nmm.nmm_mla_decode_chain(step.dims, bufs, kv=kv_entry)
    heads = q.shape[0]
    out = torch.full((heads, dv), float("nan"), dtype=torch.float32, device="cuda")
    outb = torch.zeros((heads, dv + 8), dtype=torch.bfloat16, device="cuda")
    nmm.nmm_latent_attention_ex(q, kv, out, scale, splits=splits, out_bf16=outb, d_qk=dqk, d_v=dv)
    torch.cuda.synchronize()
    return bufs, out, outb


def assert_same(bufs_a, bufs_b, out_a, out_b, outb_a, outb_b):
    for k in OUTPUTS:
        assert torch.equal(bufs_a[k].view(torch.int16) if bufs_a[k].dtype == torch.bfloat16 else bufs_a[k],
                           bufs_b[k].view(torch.int16) if bufs_b[k].dtype == torch.bfloat16 else bufs_b[k]), k
    assert torch.equal(out_a, out_b), "attention output"
    if outb_a is not None:
        assert torch.equal(outb_a.view(torch.int16), outb_b.view(torch.int16)), "attention bf16 copy"


@pytest.mark.parametrize("splits", [16, 0, 1, 12])   # 12: 11 spans, the grid padded to 16 spans
def test_full_size_step_matches_chain_and_attention(splits):
    step = syn.decode_step()
    q, kv, out, outb = attn_bufs(step.q, step.kv, syn.ATTN_DV)
    bufs = alloc_chain(step)
    events = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=q, kv=kv, out=out, out_bf16=outb, scale=step.scale,
                                                  splits=splits), events=events)
    torch.cuda.synchronize()
    gaps = [events[i].elapsed_time(events[i + 1]) for i in range(5)]
    assert all(g >= 0 for g in gaps), gaps
    sep, out2, outb2 = run_separately(step, q, kv, step.scale, splits, syn.ATTN_DQK, syn.ATTN_DV)
    assert_same(bufs, sep, out, out2, outb, outb2)
    if splits in (16, 12):
        check_chain_stepwise(step, bufs)
        ref, ref_abs = oracle.latent_attention(step.q, step.kv, step.scale)
        assert_parity(out, ref, ref_abs, what="decode-step attention")
        bits = host_bits(outb)
        assert np.array_equal(bits[:, :syn.ATTN_DV], oracle.round_bf16(out.cpu().numpy()))
        assert np.all(bits[:, syn.ATTN_DV:] == 0)


@pytest.mark.parametrize("heads,seq,dqk,dv,splits", [
    (6, 4096, 576, 512, 16),   # the shared launch beside a small chain
    (70, 300, 576, 512, 3),    # ragged heads (two head blocks) and a ragged last span
    (5, 1000, 128, 64, 4),     # a shape the shared launch does not take: two launches in order
])
def test_small_step_matches_chain_and_attention(heads, seq, dqk, dv, splits):
    step = small_step(17)
    qb, kvb, scale = syn.attention_case(40 + heads, heads, seq, dqk=dqk, dv=dv)
    q, kv, out, outb = attn_bufs(qb, kvb, dv)
    bufs = alloc_chain(step)
    nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=q, kv=kv, out=out, out_bf16=outb, scale=scale, splits=splits,
                                                  d_qk=dqk, d_v=dv))
    torch.cuda.synchronize()
    sep, out2, outb2 = run_separately(step, q, kv, scale, splits, dqk, dv)
    assert_same(bufs, sep, out, out2, outb, outb2)
    check_chain_stepwise(step, bufs)
    ref, ref_abs = oracle.latent_attention(qb, kvb, scale, dqk=dqk, dv=dv)
    assert_parity(out, ref, ref_abs, what=f"attention {heads}x{seq} {dqk}/{dv}")


@pytest.mark.parametrize("heads,nope,a_heads,seq,dqk,dv,splits", [
    (3, 64, 20, 1000, 576, 512, 5),   # the pair's 4-wave form: one merge block per extra workgroup
    (5, 128, 5, 700, 128, 64, 4),     # 8-wave form, two blocks per workgroup, an odd number of blocks
])
def test_paired_step_carries_the_merge(heads, nope, a_heads, seq, dqk, dv, splits):
    step = pair_step(heads * 100 + nope, heads, nope)
    qb, kvb, scale = syn.attention_case(60 + a_heads, a_heads, seq, dqk=dqk, dv=dv)
    q, kv, out, outb = attn_bufs(qb, kvb, dv)
    bufs = alloc_chain(step)
    nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=q, kv=kv, out=out, out_bf16=outb, scale=scale, splits=splits,
                                                  d_qk=dqk, d_v=dv))
    torch.cuda.synchronize()
    sep, out2, outb2 = run_separately(step, q, kv, scale, splits, dqk, dv)
    assert_same(bufs, sep, out, out2, outb, outb2)
    check_chain_stepwise(step, bufs)
    ref, ref_abs = oracle.latent_attention(qb, kvb, scale, dqk=dqk, dv=dv)
    assert_parity(out, ref, ref_abs, what=f"attention {a_heads}x{seq} {dqk}/{dv} merged beside the pair")


def test_step_with_cache_entry_and_no_bf16_copy():
    step = small_step(19)
    kv_entry, gamma = kv_for(step, 3, position=5, cache_rows=9)
    qb, kvb, scale = syn.attention_case(77, 6, 4096)
    q, kv, out, _ = attn_bufs(qb, kvb, syn.ATTN_DV, bf16_copy=False)
    bufs = alloc_chain(step)
    nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=q, kv=kv, out=out, scale=scale, splits=16), kv=kv_entry)
    torch.cuda.synchronize()
    check_chain_stepwise(step, bufs)
    check_kv_row(step, bufs, kv_entry, gamma)
    ref, ref_abs = oracle.latent_attention(qb, kvb, scale)
    assert_parity(out, ref, ref_abs, what="attention beside the chain with a cache entry")


def test_attention_reading_the_chains_writes_is_refused_before_any_launch():
    step = small_step(23)
    kv_entry, _ = kv_for(step, 5, position=2, cache_rows=64)
    cache = kv_entry["cache"]                       # [64, kv_lora + rope + 8]
    qb, _, scale = syn.attention_case(78, 6, 64, dqk=128, dv=64)
    bufs = alloc_chain(step)
    out = torch.full((6, 64), float("nan"), dtype=torch.float32, device="cuda")
    # the attention reads the cache the chain writes its new row into
    with pytest.raises(nmm.NmmError) as e:
        nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=dev16(qb, syn.BF16), kv=cache, out=out, scale=scale,
                                                      d_qk=128, d_v=64), kv=kv_entry)
    assert e.value.status == nmm.NMM_ERR_ARG
    # the attention's output on top of the chain's input x
    with pytest.raises(nmm.NmmError) as e:
        x_as_out = bufs["x"].view(-1).view(torch.float32)[:96].view(6, 16)
        nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=dev16(qb, syn.BF16), kv=cache[8:], out=x_as_out,
                                                      scale=scale, d_qk=128, d_v=16))
    assert e.value.status == nmm.NMM_ERR_ARG
    # a misaligned q (2-byte offset) is an argument error of the attention, also before any launch
    qd = dev16(np.concatenate([np.zeros((6, 1), np.uint16), qb], axis=1), syn.BF16)[:, 1:]
    other = torch.zeros((64, 136), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(nmm.NmmError) as e:
        nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=qd, kv=other, out=out, scale=scale, d_qk=128, d_v=64))
    assert e.value.status == nmm.NMM_ERR_ALIGN
    torch.cuda.synchronize()
    for k in ("down_f32", "y"):
        assert torch.isnan(bufs[k]).all(), f"{k} was written by a refused call"
    assert torch.isnan(out).all()


def test_step_graph_replays_match_eager():
    step = syn.decode_step()
    q, kv, out, outb = attn_bufs(step.q, step.kv, syn.ATTN_DV)
    bufs = alloc_chain(step)
    ws = nmm.Workspace()
    prep = nmm.PreparedStep(step.dims, bufs, dict(q=q, kv=kv, out=out, out_bf16=outb, scale=step.scale, splits=16),
                            workspace=ws)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        prep.launch(stream=s)
    torch.cuda.synchronize()
    ref = {k: bufs[k].clone() for k in OUTPUTS}
    ref_out, ref_outb = out.clone(), outb.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        prep.launch(stream=s)
    for r in range(3):
        for k in OUTPUTS:
            bufs[k].zero_()
        out.fill_(float("nan"))
        outb.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in OUTPUTS:
            assert torch.equal(bufs[k], ref[k]), (r, k)
        assert torch.equal(out, ref_out) and torch.equal(outb, ref_outb), r


def test_step_with_no_attention_heads_is_the_chain():
    step = small_step(29)
    q = torch.zeros((0, 576), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((64, 576), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((0, 512), dtype=torch.float32, device="cuda")
    bufs = alloc_chain(step)
    nmm.nmm_mla_decode_step(step.dims, bufs, dict(q=q, kv=kv, out=out, scale=0.1, splits=16))
    torch.cuda.synchronize()
    sep = alloc_chain(step)
    nmm.nmm_mla_decode_chain(step.dims, sep)
    torch.cuda.synchronize()
    for k in OUTPUTS:
        assert torch.equal(bufs[k].view(torch.int16) if bufs[k].dtype == torch.bfloat16 else bufs[k],
                           sep[k].view(torch.int16) if sep[k].dtype == torch.bfloat16 else sep[k]), k


def test_full_size_step_soak_bit_identical():
    # 200 full-size steps on one workspace: the chain's split-K gathers, the attention beside
    # W_UQ and its merge beside the pair give every output the same bits each time, and the
    # chain's arrival counters are back at zero after the last
    step = syn.decode_step()
    q, kv, out, outb = attn_bufs(step.q, step.kv, syn.ATTN_DV)
    bufs = alloc_chain(step)
    ws = nmm.Workspace()
    prepared = nmm.PreparedStep(step.dims, bufs, dict(q=q, kv=kv, out=out, out_bf16=outb, scale=step.scale,
                                                      splits=16), workspace=ws)
    prepared.launch()
    torch.cuda.synchronize()
    first = {k: bufs[k].clone() for k in OUTPUTS}
    out0, outb0 = out.clone(), outb.clone()
    saved = {k: torch.empty((20,) + tuple(v.shape), dtype=v.dtype, device="cuda") for k, v in first.items()}
    outs = torch.empty((20,) + tuple(out.shape), dtype=out.dtype, device="cuda")
    outbs = torch.empty((20,) + tuple(outb.shape), dtype=outb.dtype, device="cuda")
    for batch in range(10):
        for i in range(20):
            prepared.launch()
            for k in OUTPUTS:
                saved[k][i].copy_(bufs[k])
            outs[i].copy_(out)
            outbs[i].copy_(outb)
        torch.cuda.synchronize()
        for k in OUTPUTS:
            a, b = saved[k], first[k].unsqueeze(0).expand_as(saved[k])
            if a.dtype == torch.bfloat16:
                a, b = a.view(torch.int16), b.view(torch.int16)
            assert torch.equal(a, b), f"step {batch * 20}..{batch * 20 + 19}: {k} differs from the first step"
        assert torch.equal(outs, out0.unsqueeze(0).expand_as(outs)), f"steps {batch * 20}..: attention output"
        assert torch.equal(outbs.view(torch.int16), outb0.view(torch.int16).unsqueeze(0).expand_as(outbs)), \
            f"steps {batch * 20}..: attention bf16 copy"
    assert int(ws.buf[:65536].view(torch.int32).abs().sum()) == 0
