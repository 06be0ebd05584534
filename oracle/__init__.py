"""CPU oracle for narrow MatMul -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package. The HIP product path (``paper_2609_16009_amd``) never imports it, and the two share
no code: this side is plain C (``nmm_oracle.c``, fp64, built with gcc) plus numpy marshalling.

Functions (each cites the passage it follows in ``nmm_oracle.c``):

* ``gemv``            -- y = x . W and sum |x_k W_kn| in fp64 (problem statement, Section II-E;
                         Condition 2, Section III-A; eq. 4, Section IV-B).
* ``batched_gemv``    -- the same per batch index (per-head absorbed MLA matmuls).
* ``round_bf16``      -- fp32 -> bf16, ties to even or away (Algorithm 2's final cast, Section IV-E).
* ``round_bf16_exact``-- the same for fp64 values, rounded once.
* ``rmsnorm``, ``rope``, ``kv_entry``, ``mla_kv_update`` -- MatMul 2 of Section IV-A and the
                         vector work behind it (RMSNorm, RoPE, the cache entry).
* ``latent_attention``-- textbook softmax attention in fp64 (the decode step's independent work).
* ``mla_chain``       -- the decode step's narrow chain composed from the above.

``alg2_schedule`` (a separate module) models the MatMul 2 work split of Section IV-E.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "nmm_oracle.c")
_DEFAULT_LIB = os.path.join(_HERE, "libnmm_oracle.so")
# The mutation tests point this at a copy of the oracle with a planted mistake.
_LIB_PATH = os.environ.get("NMM_ORACLE_LIB") or _DEFAULT_LIB
_lib = None

F16, BF16 = 1, 2

_i64 = ctypes.c_int64
_p = ctypes.c_void_p


def build(force: bool = False, src: str = _SRC, out: str = _DEFAULT_LIB) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction); returns the .so path."""
    if force or not os.path.exists(out):
        tmp = out + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                        "-shared", "-Wall", "-o", tmp, src, "-lm"], check=True)
        os.replace(tmp, out)
    return out


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            if _LIB_PATH != _DEFAULT_LIB:
                raise FileNotFoundError(_LIB_PATH)
            build()
        L = ctypes.CDLL(_LIB_PATH)
        L.nmmo_dec_f16.restype = ctypes.c_double
        L.nmmo_dec_f16.argtypes = [ctypes.c_uint16]
        L.nmmo_dec_bf16.restype = ctypes.c_double
        L.nmmo_dec_bf16.argtypes = [ctypes.c_uint16]
        L.nmmo_round_bf16_rne.restype = ctypes.c_uint16
        L.nmmo_round_bf16_rne.argtypes = [ctypes.c_float]
        L.nmmo_round_bf16_rne_array.argtypes = [_p, _p, _i64]
        L.nmmo_round_bf16_array.argtypes = [_p, _p, _i64, ctypes.c_int]
        L.nmmo_rmsnorm.argtypes = [_i64, _p, _p, ctypes.c_double, _p]
        L.nmmo_rope.argtypes = [_i64, _p, _i64, ctypes.c_double, _p]
        L.nmmo_kv_entry.restype = ctypes.c_int
        L.nmmo_kv_entry.argtypes = [_i64, _i64, _p, _p, ctypes.c_double, ctypes.c_double, _i64,
                                    ctypes.c_int, _p, _p]
        L.nmmo_mla_kv_update.restype = ctypes.c_int
        L.nmmo_mla_kv_update.argtypes = [_i64, _i64, _i64, _p, _p, _i64, _p, ctypes.c_double,
                                         ctypes.c_double, _i64, ctypes.c_int, _p, _p, _p, _p,
                                         ctypes.c_int]
        L.nmmo_decode_array.argtypes = [ctypes.c_int, _p, _p, _i64]
        L.nmmo_max_threads.restype = ctypes.c_int
        L.nmmo_gemv.restype = ctypes.c_int
        L.nmmo_gemv.argtypes = [_i64, _i64, _i64, ctypes.c_int, _p, _i64, _p, _i64, _p, _p, _i64,
                                ctypes.c_int]
        L.nmmo_batched_gemv.restype = ctypes.c_int
        L.nmmo_batched_gemv.argtypes = [_i64, _i64, _i64, _i64, ctypes.c_int, _p, _i64, _i64, _p,
                                        _i64, _i64, _p, _p, _i64, _i64, ctypes.c_int]
        L.nmmo_latent_attention.restype = ctypes.c_int
        L.nmmo_latent_attention.argtypes = [_i64, _i64, _i64, _i64, _p, _i64, _p, _i64,
                                            ctypes.c_double, _p, _p, _i64, ctypes.c_int]
        L.nmmo_mla_chain.restype = ctypes.c_int
        L.nmmo_mla_chain.argtypes = [_i64] * 7 + [_p] * 7 + [ctypes.c_int]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _u16(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype != np.uint16:
        raise TypeError("oracle inputs are 16-bit float bit patterns (numpy uint16)")
    return np.ascontiguousarray(a)


def max_threads() -> int:
    return int(lib().nmmo_max_threads())


def decode(bits, dt: int) -> np.ndarray:
    """Decode fp16 (dt=1) or bf16 (dt=2) bit patterns to float64 with the oracle's own decoder."""
    b = _u16(bits)
    out = np.empty(b.shape, dtype=np.float64)
    lib().nmmo_decode_array(dt, _ptr(b), _ptr(out), b.size)
    return out


ROUND_EVEN, ROUND_AWAY = 0, 1


def round_bf16(values, mode: int = ROUND_EVEN) -> np.ndarray:
    """Round values, first narrowed to float32, to bf16 bit patterns (the paper's output cast);
    ties to even (mode 0) or away from zero (mode 1)."""
    v = np.ascontiguousarray(np.asarray(values, dtype=np.float32), dtype=np.float64)
    out = np.empty(v.shape, dtype=np.uint16)
    lib().nmmo_round_bf16_array(_ptr(v), _ptr(out), v.size, int(mode))
    return out


def round_bf16_exact(values, mode: int = ROUND_EVEN) -> np.ndarray:
    """Round float64 values to bf16 bit patterns with one rounding (no float32 step)."""
    v = np.ascontiguousarray(values, dtype=np.float64)
    out = np.empty(v.shape, dtype=np.uint16)
    lib().nmmo_round_bf16_array(_ptr(v), _ptr(out), v.size, int(mode))
    return out


def rmsnorm(c, gamma, eps: float) -> np.ndarray:
    """c / sqrt(mean(c^2) + eps) * gamma in float64 (gamma: bf16 bits)."""
    c = np.ascontiguousarray(c, dtype=np.float64)
    g = _u16(gamma)
    if g.size != c.size:
        raise ValueError("gamma must match c")
    out = np.empty(c.shape, dtype=np.float64)
    lib().nmmo_rmsnorm(c.size, _ptr(c), _ptr(g), float(eps), _ptr(out))
    return out


def rope(k, t: int, theta: float) -> np.ndarray:
    """RoFormer rotation of adjacent pairs of k at position t, base theta, in float64."""
    k = np.ascontiguousarray(k, dtype=np.float64)
    if k.size % 2:
        raise ValueError("RoPE needs an even width")
    out = np.empty(k.shape, dtype=np.float64)
    lib().nmmo_rope(k.size, _ptr(k), int(t), float(theta), _ptr(out))
    return out


def kv_entry(mm, gamma, kv_lora: int, eps: float, theta: float, t: int,
             mode: int = ROUND_EVEN) -> tuple[np.ndarray, np.ndarray]:
    """The cache entry [RMSNorm(mm[:kv_lora]) | RoPE(mm[kv_lora:], t)]: (float64 row, bf16 bits)."""
    mm = np.ascontiguousarray(mm, dtype=np.float64).reshape(-1)
    g = _u16(gamma)
    rope_w = mm.size - kv_lora
    row = np.empty(mm.size, dtype=np.float64)
    bits = np.empty(mm.size, dtype=np.uint16)
    rc = lib().nmmo_kv_entry(kv_lora, rope_w, _ptr(mm), _ptr(g), float(eps), float(theta), int(t),
                             int(mode), _ptr(row), _ptr(bits))
    if rc:
        raise ValueError(f"oracle kv_entry rejected its arguments ({rc})")
    return row, bits


def mla_kv_update(h, W, gamma, kv_lora: int, rope_w: int, eps: float, theta: float, t: int,
                  mode: int = ROUND_EVEN, threads: int = 0):
    """MatMul 2 (h[1, hidden] . W[hidden, >= kv_lora + rope_w]) and the cache entry behind it.

    Returns (mm, mm_abs, row, row_bits): the product and sum |h_k W_kn| in float64, the float64
    entry before rounding, and its bf16 bits."""
    h = _u16(h).reshape(-1)
    W = _u16(W)
    g = _u16(gamma)
    hidden, ldw = W.shape
    n = kv_lora + rope_w
    if h.size != hidden or g.size != kv_lora or ldw < n:
        raise ValueError("MatMul 2 operand shapes do not match")
    mm = np.empty(n, dtype=np.float64)
    mm_abs = np.empty(n, dtype=np.float64)
    row = np.empty(n, dtype=np.float64)
    bits = np.empty(n, dtype=np.uint16)
    rc = lib().nmmo_mla_kv_update(hidden, kv_lora, rope_w, _ptr(h), _ptr(W), ldw, _ptr(g), float(eps),
                                  float(theta), int(t), int(mode), _ptr(mm), _ptr(mm_abs), _ptr(row),
                                  _ptr(bits), threads)
    if rc:
        raise ValueError(f"oracle mla_kv_update rejected its arguments ({rc})")
    return mm, mm_abs, row, bits


def gemv(x, W, dt: int, M: int | None = None, K: int | None = None, N: int | None = None,
         threads: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """y[M,N] and abs[M,N] (float64) for x[M, ldx] and W[K, ldw] bit arrays."""
    x = _u16(x)
    W = _u16(W)
    M = x.shape[0] if M is None else M
    K = W.shape[0] if K is None else K
    N = W.shape[1] if N is None else N
    y = np.empty((M, N), dtype=np.float64)
    a = np.empty((M, N), dtype=np.float64)
    rc = lib().nmmo_gemv(M, K, N, dt, _ptr(x), x.shape[1], _ptr(W), W.shape[1], _ptr(y), _ptr(a),
                         N, threads)
    if rc:
        raise ValueError(f"oracle gemv rejected its arguments ({rc})")
    return y, a


def batched_gemv(x, W, dt: int, N: int | None = None, threads: int = 0):
    """x[B, M, ldx] . W[B, K, ldw] -> y[B, M, N], abs[B, M, N] in float64."""
    x = _u16(x)
    W = _u16(W)
    B, M, ldx = x.shape
    _, K, ldw = W.shape
    N = ldw if N is None else N
    y = np.empty((B, M, N), dtype=np.float64)
    a = np.empty((B, M, N), dtype=np.float64)
    rc = lib().nmmo_batched_gemv(B, M, K, N, dt, _ptr(x), ldx, M * ldx, _ptr(W), ldw, K * ldw,
                                 _ptr(y), _ptr(a), N, M * N, threads)
    if rc:
        raise ValueError(f"oracle batched_gemv rejected its arguments ({rc})")
    return y, a


def latent_attention(q, kv, scale: float, dqk: int | None = None, dv: int = 512,
                     threads: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """out[h, :dv] and sum_j p_hj |V_jn| (float64) for q[heads, ldq], kv[seq, ldkv] (bf16 bits)."""
    q = _u16(q)
    kv = _u16(kv)
    heads, ldq = q.shape
    seq, ldkv = kv.shape
    dqk = ldq if dqk is None else dqk
    out = np.empty((heads, dv), dtype=np.float64)
    oabs = np.empty((heads, dv), dtype=np.float64)
    rc = lib().nmmo_latent_attention(heads, seq, dqk, dv, _ptr(q), ldq, _ptr(kv), ldkv,
                                     float(scale), _ptr(out), _ptr(oabs), dv, threads)
    if rc:
        raise ValueError(f"oracle latent_attention rejected its arguments ({rc})")
    return out, oabs


def mla_chain(step, threads: int = 0) -> np.ndarray:
    """The decode step's narrow chain end to end (bf16 between steps); returns y[1, hidden] fp64."""
    d = step.dims
    args = [_u16(a) for a in (step.x, step.w_down, step.w_uq, step.w_uk, step.w_uv, step.w_o)]
    y = np.empty((1, d["hidden"]), dtype=np.float64)
    rc = lib().nmmo_mla_chain(d["hidden"], d["q_lora"], d["kv_lora"], d["rope"], d["heads"],
                              d["nope"], d["v_head"], *[_ptr(a) for a in args], _ptr(y), threads)
    if rc:
        raise ValueError(f"oracle mla_chain failed ({rc})")
    return y


def within_tolerance(y, y_ref, abs_ref, rel: float = 4e-3, atol: float = 1e-6) -> np.ndarray:
    """Elementwise acceptance |y - y_ref| <= rel * sum_k |x_k W_kn| + atol."""
    return np.abs(np.asarray(y, dtype=np.float64) - y_ref) <= rel * abs_ref + atol
