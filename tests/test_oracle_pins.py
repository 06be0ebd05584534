"""Pins for the CPU oracle: it is checked against what the paper and the mathematics fix, never
against itself or the HIP path.  CPU only.

What pins what:
  * 16-bit decoders: every one of the 65,536 patterns against numpy's float16 and torch's bfloat16.
  * fp32 -> bf16 rounding: constructed ties, neighbours of ties, and 2^21 random patterns against
    torch's round-to-nearest-even conversion.
  * Narrow MatMul (problem statement, Section II-E; Condition 2, Section III-A; eq. 4): identity,
    one-hot W, one-hot x on a non-square W (catches a transposed operand), rank-1 closed forms,
    exact rational brute force on tiny shapes, and integer-valued workloads against int64 sums.
  * Latent attention: seq = 1, uniform scores, a two-key case whose softmax is (3/4, 1/4) by
    construction, a dominant key, permutation invariance.
  * Decode chain: permutation-matrix weights make the chain a closed-form gather of x.
  * Ties away from zero and the single rounding of fp64 values: constructed ties and a
    neighbour search over the decoded bf16 grid.
  * RMSNorm: a 3-4-5 closed form, eps on a one-element vector, unit RMS and scale invariance.
  * RoPE: identity at t = 0, a quarter turn, the relative-position property of RoFormer
    (<R_m q, R_n k> depends on m - n only), composition, the pair frequency ladder, and the
    rotation's direction.
  * MatMul 2 and the cache entry: a one-hot token selects a row of W, and the entry splits
    into RMSNorm of the first kv_lora values and RoPE of the rest.
"""
from __future__ import annotations

import math
import random
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synthetic as syn

ONE = {syn.F16: 0x3C00, syn.BF16: 0x3F80}


def exact_bits(vals, dt):
    """Bit patterns of values that are exact in dt (checked)."""
    v = np.asarray(vals, dtype=np.float32)
    b = syn.bits_from_f32(v, dt)
    back = oracle.decode(b, dt)
    assert np.array_equal(back, v.astype(np.float64)), "value not exact in the 16-bit type"
    return b


# ---------------------------------------------------------------- decoders

def test_decode_f16_all_patterns():
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(b, syn.F16)
    ref = b.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_decode_bf16_all_patterns():
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(b, syn.BF16)
    ref = torch.from_numpy(b.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))
    # subnormal and extreme anchors
    assert got[0x0001] == 2.0 ** -133
    assert got[0x0080] == 2.0 ** -126
    assert got[0x7F7F] == (2 - 2 ** -7) * 2.0 ** 127
    assert got[0xBF80] == -1.0


# ---------------------------------------------------------------- fp32 -> bf16

def _torch_rne(f32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(f32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_round_bf16_ties_to_even():
    # every finite positive bf16 b and the float exactly halfway to the next bf16
    b = np.arange(0x0000, 0x7F7F, dtype=np.uint32)
    mid = ((b << 16) | 0x8000).view(np.float32)
    got = oracle.round_bf16(mid)
    even = np.where(b & 1, b + 1, b).astype(np.uint16)
    assert np.array_equal(got, even)
    # one float ulp either side of the tie
    below = ((b << 16) | 0x7FFF).view(np.float32)
    above = ((b << 16) | 0x8001).view(np.float32)
    assert np.array_equal(oracle.round_bf16(below), b.astype(np.uint16))
    assert np.array_equal(oracle.round_bf16(above), (b + 1).astype(np.uint16))
    # negative side mirrors
    assert np.array_equal(oracle.round_bf16(-mid), even | 0x8000)


def test_round_bf16_against_torch_random_patterns():
    rng = np.random.default_rng(123)
    u = rng.integers(0, 2 ** 32, size=1 << 21, dtype=np.uint64).astype(np.uint32)
    f = u.view(np.float32)
    f = f[np.isfinite(f)]
    assert np.array_equal(oracle.round_bf16(f), _torch_rne(f))


def test_round_bf16_overflow_and_specials():
    assert oracle.round_bf16(np.array([np.inf, -np.inf], np.float32)).tolist() == [0x7F80, 0xFF80]
    big = np.float32(3.4e38)   # above the largest finite bf16's rounding boundary
    assert int(oracle.round_bf16(np.array([big]))[0]) == int(_torch_rne(np.array([big]))[0])
    assert np.isnan(oracle.decode(oracle.round_bf16(np.array([np.nan], np.float32)), syn.BF16)[0])
    assert oracle.round_bf16(np.array([0.0, -0.0], np.float32)).tolist() == [0x0000, 0x8000]


# ---------------------------------------------------------------- narrow MatMul

@pytest.mark.parametrize("dt", [syn.F16, syn.BF16])
def test_gemv_identity(dt):
    c = syn.gemv_case(11, 3, 40, 40, dt)
    W = np.zeros((40, 40), np.uint16)
    W[np.arange(40), np.arange(40)] = ONE[dt]
    y, a = oracle.gemv(c.x, W, dt)
    xd = oracle.decode(c.x, dt)
    assert np.array_equal(y, xd)
    assert np.array_equal(a, np.abs(xd))


@pytest.mark.parametrize("dt", [syn.F16, syn.BF16])
def test_gemv_one_hot_w(dt):
    c = syn.gemv_case(12, 2, 37, 29, dt)
    for k0, n0 in [(0, 0), (36, 28), (17, 5)]:
        W = np.zeros((37, 29), np.uint16)
        W[k0, n0] = ONE[dt]
        y, _ = oracle.gemv(c.x, W, dt)
        exp = np.zeros((2, 29))
        exp[:, n0] = oracle.decode(c.x[:, k0], dt)
        assert np.array_equal(y, exp)


def test_gemv_one_hot_x_reads_rows_of_w():
    # non-square W with all-distinct entries: x = e_k must return row k of W, not column k
    K, N = 23, 41
    i = np.arange(K * N)
    # all-distinct bf16-exact values: 8-bit significands over 8 binades, alternating sign
    vals = ((128 + i % 128) * 2.0 ** (i // 128 - 7) * (-1.0) ** i).astype(np.float32).reshape(K, N)
    W = exact_bits(vals, syn.BF16)
    for k in [0, 7, 22]:
        x = np.zeros((1, K), np.uint16)
        x[0, k] = ONE[syn.BF16]
        y, _ = oracle.gemv(x, W, syn.BF16)
        assert np.array_equal(y[0], vals[k].astype(np.float64))


def test_gemv_rank1_closed_form():
    rng = np.random.default_rng(5)
    pool = np.array([-2, -1, -0.5, 0.5, 1, 2], np.float32)
    K, N, M = 64, 48, 4
    u = rng.choice(pool, K)
    v = rng.choice(pool, N)
    xs = rng.integers(-3, 4, (M, K)).astype(np.float32)
    W = exact_bits(np.outer(u, v), syn.BF16)
    x = exact_bits(xs, syn.BF16)
    y, a = oracle.gemv(x, W, syn.BF16)
    exp = np.outer(xs.astype(np.float64) @ u.astype(np.float64), v.astype(np.float64))
    assert np.array_equal(y, exp)
    assert np.array_equal(a, np.outer(np.abs(xs.astype(np.float64)) @ np.abs(u.astype(np.float64)),
                                      np.abs(v.astype(np.float64))))


@pytest.mark.parametrize("seed", range(6))
def test_gemv_bruteforce_fractions(seed):
    rnd = random.Random(seed)
    for dt in (syn.F16, syn.BF16):
        M, K, N = rnd.randint(1, 3), rnd.randint(1, 4), rnd.randint(1, 4)
        # random 16-bit values with a modest exponent range: every partial sum is exact in fp64
        vals = lambda r, c: np.array([[rnd.choice([-1, 1]) * rnd.uniform(0.0625, 16) for _ in range(c)]
                                      for _ in range(r)], np.float32)
        x = syn.bits_from_f32(vals(M, K), dt)
        W = syn.bits_from_f32(vals(K, N), dt)
        xf = [[Fraction(float(v)) for v in row] for row in
              (x.view(np.float16).astype(np.float64) if dt == syn.F16 else
               torch.from_numpy(x.astype(np.int16)).view(torch.bfloat16).double().numpy())]
        Wf = [[Fraction(float(v)) for v in row] for row in
              (W.view(np.float16).astype(np.float64) if dt == syn.F16 else
               torch.from_numpy(W.astype(np.int16)).view(torch.bfloat16).double().numpy())]
        y, a = oracle.gemv(x, W, dt)
        for m in range(M):
            for n in range(N):
                s = sum(xf[m][k] * Wf[k][n] for k in range(K))
                sa = sum(abs(xf[m][k] * Wf[k][n]) for k in range(K))
                assert Fraction(y[m, n]) == s
                assert Fraction(a[m, n]) == sa


def _int_values(bits, dt):
    f = bits.view(np.float16).astype(np.float32) if dt == syn.F16 else \
        (bits.astype(np.uint32) << 16).view(np.float32)
    i = f.astype(np.int64)
    assert np.array_equal(i.astype(np.float32), f)
    return i


@pytest.mark.parametrize("make", [lambda: syn.single_gemv_512(True), lambda: syn.down_projection(True),
                                  lambda: syn.uq_sweep(4, True)])
def test_gemv_integer_workloads_exact(make):
    c = make()
    y, a = oracle.gemv(c.x, c.W, c.dt)
    ref = _int_values(c.x, c.dt) @ _int_values(c.W, c.dt)
    assert np.array_equal(y, ref.astype(np.float64))
    assert np.all(np.abs(ref) < 2 ** 24)      # exact in fp32 in any summation order
    assert np.all(a >= np.abs(y))


def test_gemv_padding_is_ignored():
    c = syn.gemv_case(21, 3, 50, 70, syn.BF16)
    cp = syn.gemv_case(21, 3, 50, 70, syn.BF16, ldx=64, ldw=80)   # NaN in the padding
    y0, a0 = oracle.gemv(c.x, c.W, syn.BF16)
    y1, a1 = oracle.gemv(cp.x, cp.W, syn.BF16, K=50, N=70)
    assert np.isfinite(y1).all()
    assert np.array_equal(y0, y1) and np.array_equal(a0, a1)


def test_gemv_abs_sum_properties():
    c = syn.gemv_case(22, 2, 300, 33, syn.F16)
    y, a = oracle.gemv(c.x, c.W, syn.F16)
    assert np.all(a >= np.abs(y))
    pos = np.abs(oracle.decode(c.W, syn.F16)).astype(np.float32)
    Wp = syn.bits_from_f32(pos, syn.F16)
    xp = syn.bits_from_f32(np.abs(oracle.decode(c.x, syn.F16)).astype(np.float32), syn.F16)
    y2, a2 = oracle.gemv(xp, Wp, syn.F16)
    assert np.array_equal(y2, a2)


def test_gemv_zero_k_is_empty_sum():
    y, a = oracle.gemv(np.zeros((2, 0), np.uint16), np.zeros((0, 5), np.uint16), syn.BF16, K=0, N=5)
    assert np.array_equal(y, np.zeros((2, 5))) and np.array_equal(a, np.zeros((2, 5)))


def test_batched_strides_select_each_batch():
    B, K, N = 5, 12, 9
    W = np.zeros((B, K, N), np.uint16)
    for b in range(B):
        W[b, b, (2 * b) % N] = ONE[syn.BF16]        # batch b: one-hot at (b, 2b mod N)
    x = syn.normal_bits(np.random.default_rng(3), (B, 1, K), 1.0, syn.BF16)
    y, _ = oracle.batched_gemv(x, W, syn.BF16)
    for b in range(B):
        exp = np.zeros(N)
        exp[(2 * b) % N] = oracle.decode(x[b, 0, b:b + 1], syn.BF16)[0]
        assert np.array_equal(y[b, 0], exp)


# ---------------------------------------------------------------- latent attention

def _bf16_mat(vals):
    return exact_bits(np.asarray(vals, np.float32), syn.BF16)


def test_attention_single_position_returns_v():
    q, kv, scale = syn.attention_case(1, 4, 1, dqk=40, dv=24)
    out, oabs = oracle.latent_attention(q, kv, scale, dv=24)
    v = oracle.decode(kv[0, :24], syn.BF16)
    assert np.array_equal(out, np.tile(v, (4, 1)))
    assert np.array_equal(oabs, np.tile(np.abs(v), (4, 1)))


def test_attention_uniform_scores_average_v():
    _, kv, scale = syn.attention_case(2, 3, 64, dqk=32, dv=16)
    q = np.zeros((3, 32), np.uint16)
    out, _ = oracle.latent_attention(q, kv, scale, dv=16)
    mean = oracle.decode(kv[:, :16], syn.BF16).mean(axis=0)
    assert np.allclose(out, np.tile(mean, (3, 1)), rtol=0, atol=1e-14)


def test_attention_two_keys_three_to_one():
    # q.k0 - q.k1 = 1 exactly; scale = ln 3 makes the softmax weights (3/4, 1/4)
    q = _bf16_mat([[1.0, 0.0, 0.0, 0.0]])
    kv = _bf16_mat([[1.0, 0.0, 2.0, -8.0], [0.0, 0.0, 6.0, 4.0]])
    out, _ = oracle.latent_attention(q, kv, math.log(3.0), dv=4)
    assert np.allclose(out[0], 0.75 * np.array([1, 0, 2, -8]) + 0.25 * np.array([0, 0, 6, 4]),
                       rtol=0, atol=1e-14)


def test_attention_dominant_key_and_permutation():
    q, kv, scale = syn.attention_case(3, 2, 50, dqk=32, dv=16)
    out, _ = oracle.latent_attention(q, kv, scale, dv=16)
    perm = np.random.default_rng(0).permutation(50)
    out_p, _ = oracle.latent_attention(q, kv[perm], scale, dv=16)
    assert np.allclose(out, out_p, rtol=0, atol=1e-13)
    # a key far ahead of all others takes all the weight (the rest underflow to zero)
    qd = _bf16_mat([[1.0] + [0.0] * 31])
    kvd = kv.copy()
    kvd[:, 0] = exact_bits(np.zeros(50, np.float32), syn.BF16)
    kvd[7, 0] = exact_bits(np.array([8.0], np.float32), syn.BF16)[0]
    out_d, _ = oracle.latent_attention(qd, kvd, 1000.0, dv=16)
    assert np.array_equal(out_d[0], oracle.decode(kvd[7, :16], syn.BF16))


# ---------------------------------------------------------------- decode chain

def test_chain_with_permutation_weights_is_a_gather():
    # tiny dims; every weight is a 0/1 selection so each step only moves bf16 values around
    d = dict(hidden=8, q_lora=4, kv_lora=4, rope=2, heads=2, nope=2, v_head=3)
    ndown = d["q_lora"] + d["kv_lora"] + d["rope"]
    nq = d["heads"] * (d["nope"] + d["rope"])
    one = ONE[syn.BF16]
    x = _bf16_mat([[1.5, -2.0, 3.25, 0.5, -0.75, 6.0, 7.0, -1.0]])
    w_down = np.zeros((8, ndown), np.uint16)
    for j in range(ndown):
        w_down[(3 * j + 1) % 8, j] = one           # down[j] = x[(3j+1) % 8]
    w_uq = np.zeros((4, nq), np.uint16)
    for j in range(nq):
        w_uq[j % 4, j] = one                       # q[j] = c_q[j % 4]
    w_uk = np.zeros((2, 2, 4), np.uint16)
    for h in range(2):
        for j in range(4):
            w_uk[h, (j + h) % 2, j] = one          # lat[h, j] = qn[h, (j+h) % 2]
    w_uv = np.zeros((2, 4, 3), np.uint16)
    for h in range(2):
        for j in range(3):
            w_uv[h, (2 * j + h) % 4, j] = one      # o[h, j] = lat[h, (2j+h) % 4]
    w_o = np.zeros((6, 8), np.uint16)
    for j in range(8):
        w_o[(5 * j) % 6, j] = one                  # y[j] = o[(5j) % 6]

    class Step:
        pass
    s = Step()
    s.x, s.w_down, s.w_uq, s.w_uk, s.w_uv, s.w_o, s.dims = x, w_down, w_uq, w_uk, w_uv, w_o, d
    y = oracle.mla_chain(s)

    xv = oracle.decode(x[0], syn.BF16)
    down = [xv[(3 * j + 1) % 8] for j in range(ndown)]
    cq = down[:4]
    q = [cq[j % 4] for j in range(nq)]
    qn = [[q[h * 4 + t] for t in range(2)] for h in range(2)]     # nope slice of each head
    lat = [[qn[h][(j + h) % 2] for j in range(4)] for h in range(2)]
    o = [[lat[h][(2 * j + h) % 4] for j in range(3)] for h in range(2)]
    of = [v for row in o for v in row]
    exp = [of[(5 * j) % 6] for j in range(8)]
    assert np.array_equal(y[0], np.array(exp))


def test_chain_rounds_intermediates_to_bf16():
    # 3 * (1 + 2^-7) = 3 + 1.5 * 2^-6 sits exactly between the bf16 neighbours 3 + 2^-6 (odd)
    # and 3 + 2^-5 (even); every later step is a 1.0 multiply, so y shows the rounded value
    d = dict(hidden=2, q_lora=1, kv_lora=1, rope=1, heads=1, nope=1, v_head=1)
    three = exact_bits(np.array([3.0], np.float32), syn.BF16)[0]
    x = _bf16_mat([[1.0 + 2 ** -7, 0.0]])
    one = ONE[syn.BF16]
    w_down = np.zeros((2, 3), np.uint16); w_down[0, 0] = three          # 3 + 3*2^-7 (not bf16)
    w_uq = np.zeros((1, 2), np.uint16); w_uq[0, 0] = one
    w_uk = np.full((1, 1, 1), one, np.uint16)
    w_uv = np.full((1, 1, 1), one, np.uint16)
    w_o = np.zeros((1, 2), np.uint16); w_o[0, 1] = one

    class Step:
        pass
    s = Step()
    s.x, s.w_down, s.w_uq, s.w_uk, s.w_uv, s.w_o, s.dims = x, w_down, w_uq, w_uk, w_uv, w_o, d
    y = oracle.mla_chain(s)
    exact = 3 * (1 + 2 ** -7)
    expect = oracle.decode(oracle.round_bf16(np.array([exact], np.float32)), syn.BF16)[0]
    assert expect != exact and expect == 3 + 2 ** -5
    assert y[0, 1] == expect and y[0, 0] == 0.0


# ---------------------------------------------------------------- rounding modes

def _neighbour_search(v: float, away: bool) -> int:
    """Nearest bf16 to v by searching the decoded grid (independent of the oracle's arithmetic)."""
    sign = 0x8000 if math.copysign(1.0, v) < 0 else 0
    a = abs(v)
    grid = oracle.decode(np.arange(0, 0x7F81, dtype=np.uint16), syn.BF16)   # 0 .. inf, ascending
    hi = int(np.searchsorted(grid, a, side="left"))
    if grid[hi] == a:
        return sign | hi
    lo = hi - 1
    dlo, dhi = a - grid[lo], grid[hi] - a
    if dlo < dhi:
        return sign | lo
    if dhi < dlo:
        return sign | hi
    return sign | (hi if away or (hi & 1) == 0 else lo)


def test_round_bf16_ties_away_from_zero():
    b = np.arange(0x0000, 0x7F7F, dtype=np.uint32)
    mid = ((b << 16) | 0x8000).view(np.float32)
    assert np.array_equal(oracle.round_bf16(mid, oracle.ROUND_AWAY), (b + 1).astype(np.uint16))
    assert np.array_equal(oracle.round_bf16(-mid, oracle.ROUND_AWAY), (b + 1).astype(np.uint16) | 0x8000)
    below = ((b << 16) | 0x7FFF).view(np.float32)
    assert np.array_equal(oracle.round_bf16(below, oracle.ROUND_AWAY), b.astype(np.uint16))
    # integers: 257 and 259 are ties on the bf16 grid of step 2 above 256
    ints = np.array([257.0, 259.0, -257.0, 258.0], np.float32)
    assert oracle.round_bf16(ints, oracle.ROUND_EVEN).tolist() == [0x4380, 0x4382, 0xC380, 0x4381]
    assert oracle.round_bf16(ints, oracle.ROUND_AWAY).tolist() == [0x4381, 0x4382, 0xC381, 0x4381]
    # the largest finite bf16 plus half a step rounds away to infinity
    top = np.array([(2 - 2 ** -8) * 2.0 ** 127], np.float64)
    assert oracle.round_bf16_exact(top, oracle.ROUND_AWAY).tolist() == [0x7F80]
    assert oracle.round_bf16_exact(top, oracle.ROUND_EVEN).tolist() == [0x7F80]


@pytest.mark.parametrize("away", [False, True])
def test_round_bf16_exact_matches_neighbour_search(away):
    rng = random.Random(7 + away)
    vals = []
    for _ in range(400):
        e = rng.randint(-140, 127)
        vals.append(rng.choice([-1, 1]) * rng.random() * 2.0 ** e)
    # exact ties and values a hair off them, in the normal and subnormal ranges
    for b in (0x0001, 0x0042, 0x3F80, 0x4380, 0x7F00):
        lo = float(oracle.decode(np.array([b], np.uint16), syn.BF16)[0])
        hi = float(oracle.decode(np.array([b + 1], np.uint16), syn.BF16)[0])
        m = (lo + hi) / 2
        vals += [m, -m, math.nextafter(m, 0), math.nextafter(m, math.inf)]
    mode = oracle.ROUND_AWAY if away else oracle.ROUND_EVEN
    got = oracle.round_bf16_exact(np.array(vals), mode).tolist()
    assert got == [_neighbour_search(v, away) for v in vals]


def test_round_bf16_exact_rounds_once():
    # 257 + 2^-20 lies above the tie 257 (so rounds to 258), but narrowing it to float32 first
    # lands on the tie, which then rounds to even (256)
    v = np.array([257.0 + 2.0 ** -20])
    assert oracle.round_bf16_exact(v).tolist() == [0x4381]
    assert oracle.round_bf16(v).tolist() == [0x4380]


# ---------------------------------------------------------------- RMSNorm and RoPE

def _gamma(vals):
    return exact_bits(np.asarray(vals, np.float32), syn.BF16)


def test_rmsnorm_closed_forms():
    # mean of squares of (3, 4) is 12.5; each value divides by sqrt(12.5) = 5 / sqrt(2)
    out = oracle.rmsnorm([3.0, 4.0], _gamma([1.0, 1.0]), 0.0)
    assert np.allclose(out, [3 * math.sqrt(2) / 5, 4 * math.sqrt(2) / 5], rtol=1e-15, atol=0)
    # eps enters under the root: 2 / sqrt(4 + 5) = 2/3
    assert np.allclose(oracle.rmsnorm([2.0], _gamma([1.0]), 5.0), [2.0 / 3.0], rtol=1e-15)
    # gamma scales each output on its own
    g = oracle.rmsnorm([3.0, 4.0], _gamma([2.0, -0.5]), 0.0)
    assert np.allclose(g, out * np.array([2.0, -0.5]), rtol=1e-15)


def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(11)
    c = rng.standard_normal(512) * 7.0
    ones = _gamma(np.ones(512))
    out = oracle.rmsnorm(c, ones, 0.0)
    assert abs(math.sqrt(np.mean(out ** 2)) - 1.0) < 1e-13
    assert np.allclose(oracle.rmsnorm(c * 1000.0, ones, 0.0), out, rtol=1e-13)
    # with eps > 0 the output's RMS falls below 1 by exactly sqrt(ms / (ms + eps))
    ms = np.mean(c ** 2)
    out_e = oracle.rmsnorm(c, ones, ms)
    assert abs(math.sqrt(np.mean(out_e ** 2)) - math.sqrt(0.5)) < 1e-13


def test_rope_identity_at_position_zero():
    k = np.random.default_rng(3).standard_normal(64)
    assert np.array_equal(oracle.rope(k, 0, 10000.0), k)


def test_rope_quarter_turn_and_direction():
    # d = 4: pair 1 turns at theta^(-1/2); theta = (2/pi)^2 makes that pi/2 per position
    th = (2 / math.pi) ** 2
    out = oracle.rope([0.0, 0.0, 1.0, 0.0], 1, th)
    assert np.allclose(out, [0.0, 0.0, 0.0, 1.0], atol=1e-15)
    out = oracle.rope([0.0, 0.0, 0.0, 1.0], 1, th)
    assert np.allclose(out, [0.0, 0.0, -1.0, 0.0], atol=1e-15)
    # pair 0 always turns by t radians: a small t moves (1, 0) towards +second component
    small = oracle.rope([1.0, 0.0], 1, 10000.0)
    assert small[1] > 0.8 and 0.5 < small[0] < 0.6


def test_rope_relative_position_property():
    rng = np.random.default_rng(5)
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    for m, n in [(7, 3), (4100, 4096), (12, 0), (300, 450)]:
        lhs = float(np.dot(oracle.rope(q, m, 10000.0), oracle.rope(k, n, 10000.0)))
        rhs = float(np.dot(oracle.rope(q, m - n, 10000.0), k))
        assert abs(lhs - rhs) < 1e-10 * (1 + abs(rhs))


def test_rope_composes_and_preserves_pair_norms():
    rng = np.random.default_rng(6)
    k = rng.standard_normal(64)
    two = oracle.rope(oracle.rope(k, 100, 10000.0), 23, 10000.0)
    assert np.allclose(two, oracle.rope(k, 123, 10000.0), rtol=0, atol=1e-12)
    r = oracle.rope(k, 4096, 10000.0)
    assert np.allclose(np.hypot(r[0::2], r[1::2]), np.hypot(k[0::2], k[1::2]), rtol=1e-14)


def test_rope_frequency_ladder():
    # pair i turns theta^(2/d) times slower than pair i-1: with d = 8 and theta = 16, pair 2 at
    # t = 16 turns as far as pair 0 at t = 4 (16 * 16^(-4/8) = 4)
    e = np.zeros(8); e[4] = 1.0
    r = oracle.rope(e, 16, 16.0)
    r0 = oracle.rope([1.0, 0.0] + [0.0] * 6, 4, 16.0)
    assert np.allclose(r[4:6], r0[0:2], atol=1e-14)
    assert np.array_equal(r[:4], np.zeros(4)) and np.array_equal(r[6:], np.zeros(2))


# ---------------------------------------------------------------- MatMul 2 and the cache entry

def test_kv_entry_splits_into_rmsnorm_and_rope():
    rng = np.random.default_rng(9)
    mm = rng.standard_normal(12)
    gamma = syn.normal_bits(rng, (8,), 1.0, syn.BF16)
    row, bits = oracle.kv_entry(mm, gamma, 8, 1e-6, 10000.0, 37)
    assert np.array_equal(row[:8], oracle.rmsnorm(mm[:8], gamma, 1e-6))
    assert np.array_equal(row[8:], oracle.rope(mm[8:], 37, 10000.0))
    assert np.array_equal(bits, oracle.round_bf16_exact(row))


def test_kv_entry_rounding_mode_reaches_the_cache():
    # c = (257, 0, 0, -257): mean square 33024.5, and eps = 32511.5 makes the root 256, so with
    # gamma = 256 the normalised values are the bf16 ties +-257; the RoPE part at t = 0 passes
    # the ties 259 (even and away agree: 260) and -257 through unchanged
    mm = np.array([257.0, 0.0, 0.0, -257.0, 259.0, -257.0])
    g = exact_bits(np.array([256.0, 1.0, 1.0, 256.0], np.float32), syn.BF16)
    row, even = oracle.kv_entry(mm, g, 4, 32511.5, 10000.0, 0, oracle.ROUND_EVEN)
    _, away = oracle.kv_entry(mm, g, 4, 32511.5, 10000.0, 0, oracle.ROUND_AWAY)
    assert row.tolist() == [257.0, 0.0, 0.0, -257.0, 259.0, -257.0]
    assert even.tolist() == [0x4380, 0x0000, 0x0000, 0xC380, 0x4382, 0xC380]
    assert away.tolist() == [0x4381, 0x0000, 0x0000, 0xC381, 0x4382, 0xC381]


def test_mla_kv_update_one_hot_token_selects_a_row():
    rng = np.random.default_rng(10)
    hidden, kv, rp = 24, 8, 4
    W = syn.padded(syn.normal_bits(rng, (hidden, kv + rp), 0.2, syn.BF16), kv + rp + 4)
    gamma = syn.normal_bits(rng, (kv,), 1.0, syn.BF16)
    h = np.zeros(hidden, np.uint16); h[13] = ONE[syn.BF16]
    mm, mm_abs, row, bits = oracle.mla_kv_update(h, W, gamma, kv, rp, 1e-6, 10000.0, 5)
    w13 = oracle.decode(W[13, :kv + rp], syn.BF16)
    assert np.array_equal(mm, w13) and np.array_equal(mm_abs, np.abs(w13))
    row2, bits2 = oracle.kv_entry(w13, gamma, kv, 1e-6, 10000.0, 5)
    assert np.array_equal(row, row2) and np.array_equal(bits, bits2)
