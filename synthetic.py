"""Seeded synthetic inputs for narrow MatMul at DeepSeek-V3 MLA single-token decode shapes.

This module only draws numbers. It holds none of the method's arithmetic: it samples Gaussian or
small-integer values with numpy and stores them as 16-bit float bit patterns (numpy ``uint16``
arrays). The CPU oracle and the HIP path both consume exactly these bytes, so neither side has to
trust the other's input handling.

Recipe (the same for every workload):

* ``rng = numpy.random.default_rng(seed)``; tensors are drawn in the order the workload lists them.
* Gaussian tensors: ``rng.standard_normal(shape, dtype=float32) * sigma``, then rounded to the
  16-bit type with round-to-nearest-even.
* Integer-valued variants: ``rng.integers(-3, 4, shape)`` from a fresh generator with the same
  seed; every such value is exact in fp16 and bf16.

The trained DeepSeek-V3 weights are not available; these draws stand in for them at the same shapes
(hidden 7168, q_lora 1536, kv_lora 512, rope 64, 128 heads, nope 128, v 128).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

F16 = 1   # numeric codes of the two 16-bit input types (the same values as the C ABI's enum)
BF16 = 2

# DeepSeek-V3 MLA dimensions.
HIDDEN, Q_LORA, KV_LORA, ROPE, HEADS, NOPE, V_HEAD = 7168, 1536, 512, 64, 128, 128, 128
DOWN_N = Q_LORA + KV_LORA + ROPE          # 2112: q_lora | kv_lora | rope columns of the fused down-projection
QK_HEAD = NOPE + ROPE                     # 192 per-head query width
ATTN_SEQ, ATTN_DQK, ATTN_DV = 4096, KV_LORA + ROPE, KV_LORA   # latent cache [4096, 576], V = kv[:, :512]


def bits_from_f32(a: np.ndarray, dt: int) -> np.ndarray:
    """Round float32 values to fp16 or bf16 (ties to even) and return the raw 16-bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dt == F16:
        return a.astype(np.float16).view(np.uint16)
    if dt == BF16:
        u = a.view(np.uint32).astype(np.uint64)
        u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
        return u.astype(np.uint16)
    raise ValueError(f"unknown dtype code {dt}")


def normal_bits(rng: np.random.Generator, shape, sigma: float, dt: int) -> np.ndarray:
    g = rng.standard_normal(shape, dtype=np.float32)
    if sigma != 1.0:
        g *= np.float32(sigma)
    return bits_from_f32(g, dt)


def int_bits(rng: np.random.Generator, shape, dt: int) -> np.ndarray:
    return bits_from_f32(rng.integers(-3, 4, size=shape).astype(np.float32), dt)


def padded(a: np.ndarray, ld: int, fill: int = 0x7FC0) -> np.ndarray:
    """Copy a [rows, cols] bit array into a [rows, ld] array; the padding holds ``fill`` (a NaN)."""
    rows, cols = a.shape
    out = np.full((rows, ld), fill, dtype=np.uint16)
    out[:, :cols] = a
    return out


def large_int_case(seed: int, M: int, K: int, N: int, ldw: int, dt: int = BF16) -> "GemvCase":
    """Integer-valued x[M, K] and W[K, N] (values -3..3, as 16-bit float bits) for weights of up to
    2 GiB: drawn as int8 row blocks and mapped through a table, so no wider temporary of W's size
    exists.  x rows are padded to a multiple of 8; W's padding columns [N, ldw) hold a NaN
    pattern."""
    rng = np.random.default_rng(seed)
    table = bits_from_f32(np.arange(-3, 4, dtype=np.float32), dt)
    x = padded(table[rng.integers(0, 7, size=(M, K), dtype=np.int8)], (K + 7) // 8 * 8)
    W = np.empty((K, ldw), dtype=np.uint16)
    for r0 in range(0, K, 4096):
        r1 = min(K, r0 + 4096)
        W[r0:r1, :N] = table[rng.integers(0, 7, size=(r1 - r0, N), dtype=np.int8)]
    W[:, N:] = 0x7FC0
    return GemvCase(M, K, N, dt, x, W, True, f"int_{M}x{K}x{N}")


@dataclass
class GemvCase:
    """One narrow MatMul y[M,N] = x[M,K] . W[K,N] (row-major, 16-bit inputs, fp32 output)."""
    M: int
    K: int
    N: int
    dt: int
    x: np.ndarray          # uint16 [M, ldx]
    W: np.ndarray          # uint16 [K, ldw]
    integer: bool = False
    name: str = ""

    @property
    def ldx(self) -> int:
        return self.x.shape[1]

    @property
    def ldw(self) -> int:
        return self.W.shape[1]


def gemv_case(seed: int, M: int, K: int, N: int, dt: int = BF16, *, integer: bool = False,
              sigma_x: float = 1.0, sigma_w: float | None = None, ldx: int | None = None,
              ldw: int | None = None, w_first: bool = False, name: str = "") -> GemvCase:
    """Generic narrow MatMul case. W ~ N(0, 1/K) by default; ``w_first`` draws W before x."""
    rng = np.random.default_rng(seed)
    if sigma_w is None:
        sigma_w = 1.0 / math.sqrt(max(K, 1))
    draw = (lambda shape, s: int_bits(rng, shape, dt)) if integer else \
           (lambda shape, s: normal_bits(rng, shape, s, dt))
    if w_first:
        W = draw((K, N), sigma_w)
        x = draw((M, K), sigma_x)
    else:
        x = draw((M, K), sigma_x)
        W = draw((K, N), sigma_w)
    if ldx is not None and ldx != K:
        x = padded(x, ldx)
    if ldw is not None and ldw != N:
        W = padded(W, ldw)
    return GemvCase(M, K, N, dt, x, W, integer, name)


# ---------------------------------------------------------------- the five workloads

def single_gemv_512(integer: bool = False) -> GemvCase:
    """x[1,512] fp16 . W[512,512] fp16 (W ~ N(0,1)/sqrt(512)), seed 0; integer variant {-3..3}."""
    return gemv_case(0, 1, 512, 512, F16, integer=integer, name="gemv512_fp16")


def down_projection(integer: bool = False, n: int = DOWN_N) -> GemvCase:
    """x[1,7168] bf16 . W[7168,2112] bf16 (q_lora 1536 | kv_lora 512 | rope 64), seed 1.

    ``n=576`` gives the kv_lora | rope down-projection of the paper's MatMul 2 (eq. 4)."""
    return gemv_case(1, 1, HIDDEN, n, BF16, integer=integer, name=f"down_7168x{n}")


def uq_sweep(M: int, integer: bool = False) -> GemvCase:
    """x[M,1536] . W_UQ[1536,24576] bf16, seed 3; W is drawn first, then x[32,1536], then x[:M]."""
    full = gemv_case(3, 32, Q_LORA, HEADS * QK_HEAD, BF16, integer=integer, w_first=True,
                     name="uq_1536x24576")
    return GemvCase(M, full.K, full.N, BF16, np.ascontiguousarray(full.x[:M]), full.W, integer,
                    f"uq_M{M}")


@dataclass
class HeadsCase:
    """Per-head absorbed MLA matmuls: q_nope[128,1,128] . W_UK[128,128,512], then . W_UV[128,512,128]."""
    q_nope: np.ndarray     # uint16 [128, 1, 128]
    w_uk: np.ndarray       # uint16 [128, 128, 512]
    w_uv: np.ndarray       # uint16 [128, 512, 128]
    dt: int = BF16


def absorbed_heads(integer: bool = False) -> HeadsCase:
    """Seed 2. Every tensor ~ N(0, 1/K) with K the contraction length it feeds (128, 128, 512)."""
    rng = np.random.default_rng(2)
    if integer:
        q = int_bits(rng, (HEADS, 1, NOPE), BF16)
        uk = int_bits(rng, (HEADS, NOPE, KV_LORA), BF16)
        uv = int_bits(rng, (HEADS, KV_LORA, V_HEAD), BF16)
    else:
        q = normal_bits(rng, (HEADS, 1, NOPE), 1 / math.sqrt(NOPE), BF16)
        uk = normal_bits(rng, (HEADS, NOPE, KV_LORA), 1 / math.sqrt(NOPE), BF16)
        uv = normal_bits(rng, (HEADS, KV_LORA, V_HEAD), 1 / math.sqrt(KV_LORA), BF16)
    return HeadsCase(q, uk, uv)


@dataclass
class DecodeStep:
    """One MLA single-token decode step: the narrow chain (stream A) and latent attention (stream B)."""
    x: np.ndarray          # [1, 7168]
    w_down: np.ndarray     # [7168, 2112]
    w_uq: np.ndarray       # [1536, 24576]
    w_uk: np.ndarray       # [128, 128, 512]
    w_uv: np.ndarray       # [128, 512, 128]
    w_o: np.ndarray        # [16384, 7168]
    q: np.ndarray          # [128, 576]   latent-space query (attention, stream B)
    kv: np.ndarray         # [4096, 576]  latent KV cache; V = kv[:, :512]
    scale: float = 1.0 / math.sqrt(QK_HEAD)
    dims: dict = field(default_factory=lambda: dict(hidden=HIDDEN, q_lora=Q_LORA, kv_lora=KV_LORA,
                                                    rope=ROPE, heads=HEADS, nope=NOPE, v_head=V_HEAD))


def decode_step(seed: int = 4, seq: int = ATTN_SEQ) -> DecodeStep:
    """Seed 4. Weights ~ N(0, 1/K); x, q and the latent cache ~ N(0, 1); bf16 throughout."""
    rng = np.random.default_rng(seed)
    x = normal_bits(rng, (1, HIDDEN), 1.0, BF16)
    w_down = normal_bits(rng, (HIDDEN, DOWN_N), 1 / math.sqrt(HIDDEN), BF16)
    w_uq = normal_bits(rng, (Q_LORA, HEADS * QK_HEAD), 1 / math.sqrt(Q_LORA), BF16)
    w_uk = normal_bits(rng, (HEADS, NOPE, KV_LORA), 1 / math.sqrt(NOPE), BF16)
    w_uv = normal_bits(rng, (HEADS, KV_LORA, V_HEAD), 1 / math.sqrt(KV_LORA), BF16)
    w_o = normal_bits(rng, (HEADS * V_HEAD, HIDDEN), 1 / math.sqrt(HEADS * V_HEAD), BF16)
    q = normal_bits(rng, (HEADS, ATTN_DQK), 1.0, BF16)
    kv = normal_bits(rng, (seq, ATTN_DQK), 1.0, BF16)
    return DecodeStep(x, w_down, w_uq, w_uk, w_uv, w_o, q, kv)


def attention_case(seed: int, heads: int, seq: int, dqk: int = ATTN_DQK, dv: int = ATTN_DV,
                   ldkv: int | None = None) -> tuple[np.ndarray, np.ndarray, float]:
    """Smaller latent-attention cases with the decode step's distributions: q, kv ~ N(0,1) bf16."""
    rng = np.random.default_rng(seed)
    q = normal_bits(rng, (heads, dqk), 1.0, BF16)
    kv = normal_bits(rng, (seq, dqk), 1.0, BF16)
    if ldkv is not None and ldkv != dqk:
        kv = padded(kv, ldkv)
    return q, kv, 1.0 / math.sqrt(QK_HEAD)


def attention_case_large(seed: int, heads: int, seq: int, ldkv: int, dqk: int = ATTN_DQK) -> tuple[np.ndarray, np.ndarray, float]:
    """attention_case's distributions in a cache of rows padded to ``ldkv`` (the padding holds a
    NaN pattern), for caches of up to 2 GiB: the rows are drawn in blocks, so no float32 temporary
    of the cache's size exists."""
    rng = np.random.default_rng(seed)
    q = normal_bits(rng, (heads, dqk), 1.0, BF16)
    kv = np.full((seq, ldkv), 0x7FC0, dtype=np.uint16)
    for r0 in range(0, seq, 1 << 16):
        r1 = min(seq, r0 + (1 << 16))
        kv[r0:r1, :dqk] = normal_bits(rng, (r1 - r0, dqk), 1.0, BF16)
    return q, kv, 1.0 / math.sqrt(QK_HEAD)


# MatMul 2 of the paper (one token times (W^DKV | W^KR)^T) and the cache entry behind it.
KV_EPS, ROPE_THETA = 1e-6, 10000.0      # DeepSeek-V3's RMSNorm epsilon; RoFormer's RoPE base


@dataclass
class KvUpdateCase:
    """MatMul 2 [1, hidden] . [hidden, kv_lora + rope] and the RMSNorm / RoPE / cache-append behind it."""
    h: np.ndarray          # [1, hidden] token
    w: np.ndarray          # [hidden, ldw]: columns 0..kv_lora-1 are W^DKV^T, then rope columns of W^KR^T
    gamma: np.ndarray      # [kv_lora] RMSNorm weight
    kv_lora: int
    rope: int
    position: int          # the token's position: its RoPE angle and its cache row
    eps: float = KV_EPS
    theta: float = ROPE_THETA


def kv_update_case(seed: int = 5, hidden: int = HIDDEN, kv_lora: int = KV_LORA, rope: int = ROPE,
                   position: int = ATTN_SEQ, ldw: int | None = None) -> KvUpdateCase:
    """Seed 5. h ~ N(0,1), W ~ N(0, 1/hidden), gamma ~ 1 + 0.1 N(0,1) (a trained norm weight sits
    near 1); bf16 throughout.  The default position appends after a 4096-row cache."""
    rng = np.random.default_rng(seed)
    h = normal_bits(rng, (1, hidden), 1.0, BF16)
    w = normal_bits(rng, (hidden, kv_lora + rope), 1 / math.sqrt(hidden), BF16)
    gamma = bits_from_f32((1.0 + 0.1 * rng.standard_normal(kv_lora, dtype=np.float32)).astype(np.float32), BF16)
    if ldw is not None and ldw != kv_lora + rope:
        w = padded(w, ldw)
    return KvUpdateCase(h, w, gamma, kv_lora, rope, position)


def random_gemv_shapes(seed: int = 31, n: int = 20) -> list[tuple[int, int, int, int, int, int, str]]:
    """Seeded (M, K, N, dt, ldx, ldw, path) cases for a sweep of the GEMV entry points: M 1-40,
    K 1-9000, N 1-3000, either 16-bit type, row pitches rounded up to 8 elements plus 0, 8 or 64
    more, and the path asked for ("gemv", "mfma" or "auto").  Shapes only: the GPU tests draw
    their inputs with gemv_case, and the launch-bounds model checks the same cases."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        M = int(rng.integers(1, 41))
        K = int(rng.integers(1, 9001))
        N = int(rng.integers(1, 3001))
        dt = int(rng.choice([F16, BF16]))
        ldx = (K + 7) // 8 * 8 + int(rng.choice([0, 8]))
        ldw = (N + 7) // 8 * 8 + int(rng.choice([0, 8, 64]))
        out.append((M, K, N, dt, ldx, ldw, str(rng.choice(["gemv", "mfma", "auto"]))))
    return out


def random_nt_shapes(seed: int = 37, n: int = 16) -> list[tuple[int, int, int, int, int, int]]:
    """Seeded (M, K, N, dt, ldx, ldwt) cases for a sweep of the transposed-weight GEMV: M 1-20,
    K 1-20000 (past the unsplit limit of 16384 now and then), N 1-3000, either 16-bit type, row
    pitches rounded up to 8 elements plus 0 or 8 more."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        M = int(rng.integers(1, 21))
        K = int(rng.integers(1, 20001))
        N = int(rng.integers(1, 3001))
        dt = int(rng.choice([F16, BF16]))
        ldx = (K + 7) // 8 * 8 + int(rng.choice([0, 8]))
        ldwt = (K + 7) // 8 * 8 + int(rng.choice([0, 8]))
        out.append((M, K, N, dt, ldx, ldwt))
    return out


def random_batched_shapes(seed: int = 41, n: int = 12) -> list[tuple[int, int, int, int]]:
    """Seeded (batch, M, K, N) cases for a sweep of the batched GEMV over contiguous [batch, M, K] x
    [batch, K, N] operands: batch 1-130, M 1-4, K and N multiples of 8 (the row pitch rule) up to
    1536 and 520."""
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(1, 131)), int(rng.integers(1, 5)), 8 * int(rng.integers(1, 193)),
             8 * int(rng.integers(1, 66))) for _ in range(n)]
