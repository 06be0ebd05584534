"""CPU oracle for narrow MatMul -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package. The HIP product path (``paper_2609_16009_amd``) never imports it, and the two share
no code: this side is plain C (``nmm_oracle.c``, fp64, built with gcc) plus numpy marshalling.

Functions (each cites the passage it follows in ``nmm_oracle.c``):

* ``gemv``            -- y = x . W and sum |x_k W_kn| in fp64 (problem statement, Section II-E;
                         Condition 2, Section III-A; eq. 4, Section IV-B).
* ``batched_gemv``    -- the same per batch index (per-head absorbed MLA matmuls).
* ``round_bf16``      -- fp32 -> bf16 ties-to-even (Algorithm 2's final cast, Section IV-E).
* ``latent_attention``-- textbook softmax attention in fp64 (the decode step's independent work).
* ``mla_chain``       -- the decode step's narrow chain composed from the above.

``alg2_schedule`` (a separate module) models the partition of Algorithm 2 in the paper's notation.
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


def round_bf16(values) -> np.ndarray:
    """Round float32 values to bf16 bit patterns, ties to even (the paper's output cast)."""
    v = np.ascontiguousarray(values, dtype=np.float32)
    out = np.empty(v.shape, dtype=np.uint16)
    lib().nmmo_round_bf16_rne_array(_ptr(v), _ptr(out), v.size)
    return out


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
