"""GPU parity of nmm_latent_attention against the oracle's fp64 softmax attention.

Acceptance per output: |o - o_ref| <= 4e-3 * sum_j p_ref,j |V_jn| + 1e-6 (the oracle returns the
weighted absolute sum).  P is rounded to bf16 for the matrix-core product, a relative error of at
most 2^-9 per weight, inside that bound.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as syn
from gpu_util import assert_parity, dev16, host_bits

pytestmark = pytest.mark.gpu

nmm = pytest.importorskip("paper_2609_16009_amd")


def run_attention(q_bits, kv_bits, scale, dqk, dv, ldo=None):
    q, kv = dev16(q_bits, syn.BF16), dev16(kv_bits, syn.BF16)
    heads = q_bits.shape[0]
    out = torch.full((heads, ldo or dv), np.nan, dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention(q, kv, out, scale, d_qk=dqk, d_v=dv)
    torch.cuda.synchronize()
    return out


def check(q_bits, kv_bits, scale, dqk, dv, what):
    out = run_attention(q_bits, kv_bits, scale, dqk, dv)
    ref, ref_abs = oracle.latent_attention(q_bits, kv_bits, scale, dqk=dqk, dv=dv)
    return assert_parity(out, ref, ref_abs, what=what), out


def test_decode_step_attention_full_size():
    q, kv, scale = syn.attention_case(4, 128, 4096)
    check(q, kv, scale, 576, 512, "attention 128x4096x576/512")


@pytest.mark.parametrize("splits", [1, 8, 16, 21, 64])
def test_decode_step_attention_every_partition(splits):
    # the span count changes the summation order, never the result beyond tolerance
    q, kv, scale = syn.attention_case(14, 128, 4096)
    out = torch.full((128, 512), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, scale, splits=splits)
    torch.cuda.synchronize()
    ref, ref_abs = oracle.latent_attention(q, kv, scale)
    assert_parity(out, ref, ref_abs, what=f"attention 128x4096, {splits} spans")


@pytest.mark.parametrize("splits", [1, 4])
def test_attention_rising_scores_rescale_every_chunk(splits):
    # scores that grow along the cache: each 64-position chunk's maximum exceeds the running one by
    # far more than the lazy-rescale threshold, so the running output is rescaled at every chunk
    rng = np.random.default_rng(77)
    heads, seq, dqk, dv = 40, 700, 576, 512
    qf = rng.standard_normal((heads, dqk), dtype=np.float32)
    u = np.sign(rng.standard_normal(dqk)).astype(np.float32)
    qf[:, :] = np.abs(qf) * u                       # every head leans towards u
    t = np.linspace(0.0, 3.0, seq, dtype=np.float32)
    kvf = rng.standard_normal((seq, dqk), dtype=np.float32) * 0.5 + t[:, None] * u[None, :]
    q, kv = syn.bits_from_f32(qf, syn.BF16), syn.bits_from_f32(kvf, syn.BF16)
    scale = 0.05
    out = torch.full((heads, dv), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, scale, splits=splits, d_v=dv)
    torch.cuda.synchronize()
    ref, ref_abs = oracle.latent_attention(q, kv, scale, dqk=dqk, dv=dv)
    assert_parity(out, ref, ref_abs, what=f"rising scores, {splits} spans")


@pytest.mark.parametrize("heads,seq,dqk,dv,ldkv", [
    (20, 1000, 96, 48, 104),      # ragged heads and positions, padded cache rows
    (16, 50, 64, 64, 64),         # one span: no cross-workgroup merge
    (3, 1, 32, 16, 40),           # a single position
    (128, 4097, 576, 512, 576),   # one position past a chunk boundary
    (33, 777, 576, 512, 584),
])
def test_attention_ragged(heads, seq, dqk, dv, ldkv):
    q, kv, scale = syn.attention_case(heads * 7 + seq, heads, seq, dqk=dqk, dv=dv, ldkv=ldkv)
    check(q, kv, scale, dqk, dv, f"attention {heads}x{seq}x{dqk}/{dv}")


@pytest.mark.parametrize("splits", [1, 3, 16])
def test_attention_identical_keys_give_the_value_row(splits):
    # a closed form, independent of the oracle: when every cache row is the same, every score of
    # a head is the same, P = 2^0 = 1 at every position and the output is that row's first d_v
    # values.  The sums are exact (integer multiples of bf16 values below 2^24), so a merge of
    # spans returns the row bit for bit; one span multiplies by the rounded 1 / l, within one ulp.
    rng = np.random.default_rng(91)
    heads, seq, dqk, dv = 40, 1000, 576, 512
    q = syn.bits_from_f32(rng.standard_normal((heads, dqk), dtype=np.float32), syn.BF16)
    row = syn.bits_from_f32(rng.standard_normal(dqk, dtype=np.float32), syn.BF16)
    kv = np.ascontiguousarray(np.broadcast_to(row, (seq, dqk)))
    out = torch.full((heads, dv), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, 0.07, splits=splits)
    torch.cuda.synchronize()
    v = np.broadcast_to(oracle.decode(row[:dv], syn.BF16).astype(np.float32), (heads, dv))
    got = out.cpu().numpy()
    if splits == 1:
        assert np.all(np.abs(got - v) <= np.abs(v) * 2.0 ** -23), "one span: within one ulp of the row"
    else:
        assert np.array_equal(got, v), f"{splits} spans: the row bit for bit"


def test_attention_largest_cache():
    # a cache at the largest extent the ABI accepts: 65,535 rows of 16,384 elements (576 of them
    # data, the rest a NaN pattern that must never be read), ((seq - 1) * ldkv + 576) * 2 =
    # 2^31 - 64,384 bytes, so the chunks' 32-bit row offsets take their largest values; one ragged
    # block of 20 heads over the default partition (64 spans of 1,024 positions)
    seq, ldkv = 65535, 16384
    q, kv, scale = syn.attention_case_large(67, 20, seq, ldkv)
    assert ((seq - 1) * ldkv + 576) * 2 < 2 ** 31
    out = torch.full((20, 512), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, scale)
    torch.cuda.synchronize()
    ref, ref_abs = oracle.latent_attention(q, kv, scale, dqk=576, dv=512)
    assert_parity(out, ref, ref_abs, what=f"attention 20 heads x {seq} positions, rows of {ldkv}")


def test_attention_sharp_softmax_and_determinism():
    # a large scale makes the softmax nearly one-hot: stresses the running max and rescaling
    q, kv, _ = syn.attention_case(9, 32, 2000, dqk=128, dv=64)
    _, out1 = check(q, kv, 2.0, 128, 64, "sharp softmax")
    out2 = run_attention(q, kv, 2.0, 128, 64)
    assert torch.equal(out1, out2)


def test_attention_rejects_bad_arguments():
    q = torch.zeros((16, 576), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((64, 576), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((16, 512), device="cuda")
    L = nmm.lib()
    s = torch.cuda.current_stream().cuda_stream
    args = lambda **k: dict(dict(h=16, seq=64, dqk=576, dv=512, q=q.data_ptr(), ldq=576, kv=kv.data_ptr(),
                                 ldkv=576, scale=0.1, out=out.data_ptr(), ldo=512), **k)
    call = lambda a: L.nmm_latent_attention(a["h"], a["seq"], a["dqk"], a["dv"], a["q"], a["ldq"], a["kv"],
                                            a["ldkv"], a["scale"], a["out"], a["ldo"], None, 0, s)
    assert call(args(seq=0)) == nmm.NMM_ERR_SHAPE
    assert call(args(dqk=100)) == nmm.NMM_ERR_SHAPE
    assert call(args(dqk=608, ldq=608, ldkv=608)) == nmm.NMM_ERR_SHAPE   # d_qk above 576
    assert call(args(dv=520)) == nmm.NMM_ERR_SHAPE
    assert call(args(scale=float("inf"))) == nmm.NMM_ERR_ARG
    assert call(args(q=None)) == nmm.NMM_ERR_NULL
    assert call(args(ldkv=500)) == nmm.NMM_ERR_SHAPE
    assert call(args(kv=kv.data_ptr() + 2)) == nmm.NMM_ERR_ALIGN
    assert call(args(h=128, seq=4096)) == nmm.NMM_ERR_WORKSPACE


@pytest.mark.parametrize("splits", [16, 3, 0])
def test_attention_ex_partition_and_bf16_copy(splits):
    # the caller-chosen partition meets the same bar, and the bf16 copy is the ties-to-even
    # rounding of the fp32 output bit for bit
    q, kv, scale = syn.attention_case(31, 128, 4096)
    out = torch.full((128, 512), float("nan"), dtype=torch.float32, device="cuda")
    outb = torch.zeros((128, 520), dtype=torch.bfloat16, device="cuda")
    nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, scale, splits=splits, out_bf16=outb)
    torch.cuda.synchronize()
    ref, ref_abs = oracle.latent_attention(q, kv, scale)
    assert_parity(out, ref, ref_abs, what=f"attention splits={splits}")
    bits = host_bits(outb)
    assert np.array_equal(bits[:, :512], oracle.round_bf16(out.cpu().numpy()))
    assert np.all(bits[:, 512:] == 0)


def test_attention_random_shapes_and_partitions():
    # a seeded sweep over head counts (ragged 16- and 32-head blocks), lengths (one chunk, ragged
    # last chunks and spans) and partitions (the default, one span, fewer or more spans than 8,
    # so both workgroup maps and the padded grid, with and without the two-workgroup column
    # split): every head of every case against the oracle
    rng = np.random.default_rng(2024)
    for case in range(16):
        heads = int(rng.integers(1, 150))
        seq = int(rng.integers(1, 2600))
        splits = int(rng.choice([0, 0, 1, 2, 3, 5, 8, 11, 16, 23, 32, 64]))
        q, kv, scale = syn.attention_case(300 + case, heads, seq)
        out = torch.full((heads, 512), float("nan"), dtype=torch.float32, device="cuda")
        nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, scale, splits=splits)
        torch.cuda.synchronize()
        ref, ref_abs = oracle.latent_attention(q, kv, scale, dqk=576, dv=512)
        assert_parity(out, ref, ref_abs, what=f"case {case}: {heads} heads x {seq} positions, splits {splits}")


def test_attention_wide_head_blocks_match_narrow_bit_for_bit():
    # 128 heads over 64 spans would take 512 workgroups in blocks of 16 heads, so the launch takes
    # blocks of 32; the same heads in two calls of 64 stay in blocks of 16 (256 workgroups).  A
    # head's arithmetic does not depend on its block: the two agree bit for bit, and both meet the
    # oracle; then the default partition at 32,768 positions, which widens the blocks by itself
    q, kv, scale = syn.attention_case(41, 128, 8192)
    qd, kvd = dev16(q, syn.BF16), dev16(kv, syn.BF16)
    wide = torch.full((128, 512), float("nan"), dtype=torch.float32, device="cuda")
    narrow = torch.full((128, 512), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(qd, kvd, wide, scale, splits=64)
    for h0 in (0, 64):
        nmm.nmm_latent_attention_ex(qd[h0:h0 + 64], kvd, narrow[h0:h0 + 64], scale, splits=64)
    torch.cuda.synchronize()
    assert torch.equal(wide, narrow)
    ref, ref_abs = oracle.latent_attention(q, kv, scale, dqk=576, dv=512)
    assert_parity(wide, ref, ref_abs, what="attention 128 heads x 8192 positions, 64 spans")
    q, kv, scale = syn.attention_case(43, 128, 32768)
    out = torch.full((128, 512), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(dev16(q, syn.BF16), dev16(kv, syn.BF16), out, scale)
    torch.cuda.synchronize()
    ref, ref_abs = oracle.latent_attention(q, kv, scale, dqk=576, dv=512)
    assert_parity(out, ref, ref_abs, what="attention 128 heads x 32768 positions, default partition")


def test_attention_wide_head_blocks_general_shape():
    # the general (not 576 / 512) kernel in blocks of 32 heads: 160 heads over 32 spans would take
    # 320 workgroups in blocks of 16; the same heads in two calls of 80 stay in blocks of 16 (160
    # workgroups).  Bit for bit alike, and against the oracle (ragged dims, padded cache rows)
    heads, seq, dqk, dv, ldkv = 160, 2000, 96, 48, 104
    q, kv, scale = syn.attention_case(47, heads, seq, dqk=dqk, dv=dv, ldkv=ldkv)
    qd, kvd = dev16(q, syn.BF16), dev16(kv, syn.BF16)
    wide = torch.full((heads, dv), float("nan"), dtype=torch.float32, device="cuda")
    narrow = torch.full((heads, dv), float("nan"), dtype=torch.float32, device="cuda")
    nmm.nmm_latent_attention_ex(qd, kvd, wide, scale, splits=40, d_v=dv)
    for h0 in (0, 80):
        nmm.nmm_latent_attention_ex(qd[h0:h0 + 80], kvd, narrow[h0:h0 + 80], scale, splits=40, d_v=dv)
    torch.cuda.synchronize()
    assert torch.equal(wide, narrow)
    ref, ref_abs = oracle.latent_attention(q, kv, scale, dqk=dqk, dv=dv)
    assert_parity(wide, ref, ref_abs, what=f"attention {heads}x{seq}x{dqk}/{dv}, 32 spans in 32-head blocks")
