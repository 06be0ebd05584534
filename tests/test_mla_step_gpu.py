"""GPU parity of one MLA single-token decode step in its real dependency order, composed from the
library's calls on two streams (the paper's overlap: MatMul 2 and the vector work behind it run
beside the matrix-unit work of the query path, Section IV-A):

  stream A   c_q = x . W_DQ  ->  q = c_q . W_UQ  ->  query = [q_nope . W_UK | RoPE(q_pe)]
  stream B   [c_kv | k_pe] = x . (W_DKV | W_KR)  ->  cache[t] = bf16([RMSNorm(c_kv) | RoPE(k_pe)])
  then       attention(query, cache[0 .. t])  ->  o = attention . W_UV (per head)  ->  y = o . W_O

Each stage is checked against the oracle fed exactly the bf16 operands the GPU consumed; every
bf16 hand-off must equal the oracle's rounding of the GPU's own fp32 result; the RoPE'd parts
must round a value within the stated slack of the oracle's fp64 rotation.  The two-stream step
must reproduce the one-stream step bit for bit.
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


def make_step(seq):
    s = syn.decode_step(seq=seq)
    d = s.dims
    rng = np.random.default_rng(12)
    gamma = syn.bits_from_f32((1.0 + 0.1 * rng.standard_normal(d["kv_lora"], dtype=np.float32)), syn.BF16)
    n_kv = d["kv_lora"] + d["rope"]
    H, qk = d["heads"], d["nope"] + d["rope"]
    dev = dict(x=dev16(s.x, syn.BF16), w_down=dev16(s.w_down, syn.BF16), w_uq=dev16(s.w_uq, syn.BF16),
               w_uk=dev16(s.w_uk, syn.BF16), w_uv=dev16(s.w_uv, syn.BF16), w_o=dev16(s.w_o, syn.BF16),
               gamma=dev16(gamma, syn.BF16))
    cache = torch.zeros((seq + 1, n_kv), dtype=torch.bfloat16, device="cuda")
    cache[:seq] = dev16(s.kv, syn.BF16)
    f32 = lambda *shape: torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    b16 = lambda *shape: torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    bufs = dict(cq=f32(1, d["q_lora"]), cq_b=b16(1, d["q_lora"]), q=f32(1, H * qk), q_b=b16(1, H * qk),
                qlat=f32(H, d["kv_lora"]), query=b16(H, n_kv), kv=f32(n_kv), att=f32(H, d["kv_lora"]),
                att_b=b16(H, d["kv_lora"]), o=f32(H, d["v_head"]), o_b=b16(H, d["v_head"]), y=f32(1, d["hidden"]),
                cache=cache)
    return s, gamma, dev, bufs


def run_step(s, dev, bufs, seq, sa=None, sb=None, ws_a=None, ws_b=None):
    """The step; with sb given, MatMul 2 and its cache entry run on sb beside the query path."""
    d = s.dims
    H, ql, kvl, rp = d["heads"], d["q_lora"], d["kv_lora"], d["rope"]
    w_dq = dev["w_down"][:, :ql]                       # [hidden, q_lora] view, row pitch 2112
    w_dkv = dev["w_down"][:, ql:]                      # [hidden, kv_lora + rope] view (MatMul 2)
    cur = sa if sa is not None else torch.cuda.current_stream()
    kvs = sb if sb is not None else cur
    if sb is not None:
        fork = torch.cuda.Event()
        fork.record(cur)
        sb.wait_event(fork)
    nmm.nmm_mla_kv_update(dev["x"], w_dkv, dev["gamma"], bufs["kv"], bufs["cache"], kv_lora=kvl, rope=rp,
                          eps=syn.KV_EPS, theta=syn.ROPE_THETA, position=seq, workspace=ws_b, stream=kvs)
    nmm.nmm_gemv_bf16(dev["x"], w_dq, bufs["cq_b"], y=bufs["cq"], workspace=ws_a, stream=cur)
    nmm.nmm_gemv_bf16(bufs["cq_b"], dev["w_uq"], bufs["q_b"], y=bufs["q"], workspace=ws_a, stream=cur)
    nmm.nmm_mla_query(bufs["q"], bufs["q_b"], dev["w_uk"], bufs["qlat"], bufs["query"], nope=d["nope"], rope=rp,
                      position=seq, theta=syn.ROPE_THETA, workspace=ws_a, stream=cur)
    if sb is not None:
        join = torch.cuda.Event()
        join.record(sb)
        cur.wait_event(join)
    nmm.nmm_latent_attention_bf16(bufs["query"], bufs["cache"][:seq + 1], bufs["att"], bufs["att_b"], s.scale,
                                  d_v=kvl, workspace=ws_a, stream=cur)
    nmm.nmm_batched_gemv_bf16(bufs["att_b"].view(H, 1, kvl), dev["w_uv"], bufs["o_b"].view(H, 1, -1),
                              y=bufs["o"].view(H, 1, -1), workspace=ws_a, stream=cur)
    nmm.nmm_gemv(bufs["o_b"].view(1, -1), dev["w_o"], bufs["y"], workspace=ws_a, stream=cur)


def rounds_within(bits, ref, slack):
    got = oracle.decode(bits, syn.BF16)
    step = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7)
    return np.all(np.abs(got - ref) <= 0.5 * step + slack)


def check_step(s, gamma, bufs, seq):
    d = s.dims
    H, ql, kvl, rp, nope = d["heads"], d["q_lora"], d["kv_lora"], d["rope"], d["nope"]
    qk = nope + rp
    g = lambda k: bufs[k].cpu().numpy()
    # q path
    y_ref, a_ref = oracle.gemv(s.x, s.w_down[:, :ql], syn.BF16, N=ql)
    assert_parity(g("cq"), y_ref, a_ref, what="c_q")
    cq_b = host_bits(bufs["cq_b"])
    assert np.array_equal(cq_b, oracle.round_bf16(g("cq"))), "c_q hand-off"
    y_ref, a_ref = oracle.gemv(cq_b, s.w_uq, syn.BF16)
    assert_parity(g("q"), y_ref, a_ref, what="W_UQ")
    q_b = host_bits(bufs["q_b"])
    assert np.array_equal(q_b, oracle.round_bf16(g("q"))), "q hand-off"
    qn = q_b.reshape(H, qk)[:, :nope]
    y_ref, a_ref = oracle.batched_gemv(np.ascontiguousarray(qn)[:, None, :], s.w_uk, syn.BF16)
    assert_parity(g("qlat").reshape(H, 1, kvl), y_ref, a_ref, what="W_UK")
    query = host_bits(bufs["query"])
    assert np.array_equal(query[:, :kvl], oracle.round_bf16(g("qlat"))), "query: latent part"
    qpe = g("q").reshape(H, qk)[:, nope:].astype(np.float64)
    rot = np.stack([oracle.rope(qpe[h], seq, syn.ROPE_THETA) for h in range(H)])
    slack = 1e-4 * np.abs(rot) + 1e-6 * np.repeat(np.abs(qpe[:, 0::2]) + np.abs(qpe[:, 1::2]), 2, axis=1)
    assert rounds_within(query[:, kvl:], rot, slack), "query: RoPE part"
    same = np.count_nonzero(query[:, kvl:] == oracle.round_bf16_exact(rot)) / rot.size
    assert same >= 0.99, same
    # kv path: MatMul 2 and the cache entry (row seq), other rows untouched
    y_ref, a_ref = oracle.gemv(s.x, s.w_down[:, ql:], syn.BF16, N=kvl + rp)
    assert_parity(g("kv")[None], y_ref, a_ref, what="MatMul 2")
    cache = host_bits(bufs["cache"])
    assert np.array_equal(cache[:seq], s.kv), "earlier cache rows changed"
    row_ref, bits_ref = oracle.kv_entry(g("kv").astype(np.float64), gamma, kvl, syn.KV_EPS, syn.ROPE_THETA, seq)
    assert np.count_nonzero(cache[seq] == bits_ref) >= 0.99 * (kvl + rp)
    # attention over the seq + 1 rows, its bf16 output, then W_UV and W_O
    att_ref, att_abs = oracle.latent_attention(query, cache, s.scale, dv=kvl)
    assert_parity(g("att"), att_ref, att_abs, what="attention")
    att_b = host_bits(bufs["att_b"])
    assert np.array_equal(att_b, oracle.round_bf16(g("att"))), "attention hand-off"
    y_ref, a_ref = oracle.batched_gemv(att_b[:, None, :], s.w_uv, syn.BF16)
    assert_parity(g("o").reshape(H, 1, -1), y_ref, a_ref, what="W_UV")
    o_b = host_bits(bufs["o_b"])
    assert np.array_equal(o_b, oracle.round_bf16(g("o"))), "o hand-off"
    y_ref, a_ref = oracle.gemv(o_b.reshape(1, -1), s.w_o, syn.BF16)
    assert_parity(g("y"), y_ref, a_ref, what="W_O")


@pytest.mark.parametrize("seq", [300, 4096])
def test_mla_step_stepwise_and_two_streams_match_one(seq):
    s, gamma, dev, bufs = make_step(seq)
    run_step(s, dev, bufs, seq)
    torch.cuda.synchronize()
    check_step(s, gamma, bufs, seq)
    ref = {k: v.clone() for k, v in bufs.items()}
    for v in bufs.values():
        if v.dtype == torch.float32:
            v.fill_(float("nan"))
    bufs["cache"][seq].zero_()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(sa):
        run_step(s, dev, bufs, seq, sa=sa, sb=sb, ws_a=nmm.Workspace(), ws_b=nmm.Workspace())
    torch.cuda.synchronize()
    for k in bufs:
        a, b = bufs[k], ref[k]
        view = torch.int32 if a.dtype == torch.float32 else torch.int16
        assert torch.equal(a.view(view), b.view(view)), k


def test_mla_query_rope_only_heads():
    # nope part empty of meaning: W_UK = 0 gives a zero latent query, so the query is exactly
    # [0 | bf16(RoPE(q_pe))]; position 0 leaves q_pe unrotated
    H, nope, rope, kvl = 4, 16, 8, 24
    rng = np.random.default_rng(3)
    q = rng.standard_normal((H, nope + rope)).astype(np.float32)
    qt = torch.from_numpy(q).cuda()
    qb = qt.to(torch.bfloat16)
    w_uk = torch.zeros((H, nope, kvl), dtype=torch.bfloat16, device="cuda")
    qlat = torch.empty((H, kvl), dtype=torch.float32, device="cuda")
    out = torch.full((H, kvl + rope + 8), 1.0, dtype=torch.bfloat16, device="cuda")
    nmm.nmm_mla_query(qt, qb, w_uk, qlat, out, nope=nope, rope=rope, position=0, theta=10000.0)
    torch.cuda.synchronize()
    o = host_bits(out)
    assert np.all(o[:, :kvl] == 0) and torch.equal(qlat, torch.zeros_like(qlat))
    assert np.array_equal(o[:, kvl:kvl + rope], oracle.round_bf16(q[:, nope:]))
    assert np.all(o[:, kvl + rope:] == 0x3F80), "padding past the query was written"


def run_step_fused(s, dev, bufs, seq):
    """The same step with everything before attention in one call (down as one GEMV over
    [W_DQ | W_DKV | W_KR], the cache entry on a spare workgroup of W_UQ, then the query)."""
    d = s.dims
    H, ql, kvl = d["heads"], d["q_lora"], d["kv_lora"]
    down = torch.full((1, ql + kvl + d["rope"]), float("nan"), dtype=torch.float32, device="cuda")
    qp = nmm.PreparedQueryPath(d, dict(x=dev["x"], w_down=dev["w_down"], w_uq=dev["w_uq"], w_uk=dev["w_uk"],
                                       kv_gamma=dev["gamma"], kv_cache=bufs["cache"], down_f32=down,
                                       cq_bf16=bufs["cq_b"], q_f32=bufs["q"], q_bf16=bufs["q_b"],
                                       qlat_f32=bufs["qlat"], query=bufs["query"]),
                               eps=syn.KV_EPS, theta=syn.ROPE_THETA, position=seq)
    qp.launch()
    nmm.nmm_latent_attention_bf16(bufs["query"], bufs["cache"][:seq + 1], bufs["att"], bufs["att_b"], s.scale,
                                  d_v=kvl)
    nmm.nmm_batched_gemv_bf16(bufs["att_b"].view(H, 1, kvl), dev["w_uv"], bufs["o_b"].view(H, 1, -1),
                              y=bufs["o"].view(H, 1, -1))
    nmm.nmm_gemv(bufs["o_b"].view(1, -1), dev["w_o"], bufs["y"])
    bufs["cq"] = down[:, :ql]
    bufs["kv"] = down[0, ql:]


@pytest.mark.parametrize("seq", [300, 4096])
def test_mla_step_fused_query_path_stepwise(seq):
    s, gamma, dev, bufs = make_step(seq)
    run_step_fused(s, dev, bufs, seq)
    torch.cuda.synchronize()
    check_step(s, gamma, bufs, seq)
