"""Narrow MatMul on AMD MI355X (gfx950): the Python binding of libnmm.so.

Argument marshalling only.  Every step of the computation runs in the HIP kernels of libnmm.so
behind the C ABI declared in include/nmm.h; torch supplies device memory, streams and events.
The functions carry the C names (nmm_gemv, nmm_batched_gemv, nmm_mla_decode_chain,
nmm_latent_attention, ...) and take torch tensors, from which they read pointers, sizes and
strides.  There is no fallback: if libnmm.so is missing, importing the binding's functions
raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnmm.so")

NMM_OK, NMM_ERR_NULL, NMM_ERR_SHAPE, NMM_ERR_DTYPE, NMM_ERR_ALIGN, NMM_ERR_WORKSPACE, \
    NMM_ERR_HIP, NMM_ERR_PATH, NMM_ERR_ARG = range(9)
NMM_F16, NMM_BF16 = 1, 2
NMM_PATH_AUTO, NMM_PATH_GEMV, NMM_PATH_MFMA = 0, 1, 2
NMM_ROUND_EVEN, NMM_ROUND_AWAY = 0, 1
NMM_NOALLOC_SCRATCH_BYTES = 8 << 20   # nmm_gemv_noalloc's scratch per GPU

_i64 = ctypes.c_int64
_p = ctypes.c_void_p
_sz = ctypes.c_size_t
_lib = None


class NmmError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {nmm_status_string(status)}")


class nmm_plan_info(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("m_tile", ctypes.c_int32), ("m_blocks", ctypes.c_int32),
                ("panel_width", ctypes.c_int32), ("n_full_panels", ctypes.c_int32),
                ("tail_chunks", ctypes.c_int32),
                ("tail_width", ctypes.c_int32), ("split_k_full", ctypes.c_int32),
                ("rows_full", ctypes.c_int32), ("split_k_tail", ctypes.c_int32),
                ("rows_tail", ctypes.c_int32), ("items", ctypes.c_int32),
                ("threads", ctypes.c_int32), ("unroll", ctypes.c_int32), ("grid", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


class nmm_mla_chain(ctypes.Structure):
    _fields_ = [(n, _i64) for n in ("hidden", "q_lora", "kv_lora", "rope", "heads", "nope", "v_head")] + \
               [(n, _p) for n in ("x", "w_down", "w_uq", "w_uk", "w_uv", "w_o", "down_f32", "q_f32",
                                  "lat_f32", "o_f32", "y", "cq_bf16", "qnope_bf16", "lat_bf16",
                                  "o_bf16", "events")] + [("n_events", ctypes.c_int)] + \
               [("kv_gamma", _p), ("kv_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("position", _i64), ("kv_cache", _p), ("ld_cache", _i64), ("cache_rows", _i64),
                ("round", ctypes.c_int)]


class nmm_mla_kv(ctypes.Structure):
    _fields_ = [("hidden", _i64), ("kv_lora", _i64), ("rope", _i64), ("h", _p), ("w", _p), ("ldw", _i64),
                ("gamma", _p), ("eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("position", _i64),
                ("mm", _p), ("cache", _p), ("ld_cache", _i64), ("cache_rows", _i64), ("round", ctypes.c_int)]


class nmm_latent_attn(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("heads", "seq", "d_qk", "d_v")] + [
        ("q", ctypes.c_void_p), ("ldq", ctypes.c_int64), ("kv", ctypes.c_void_p), ("ld_kv", ctypes.c_int64),
        ("scale", ctypes.c_float), ("out", ctypes.c_void_p), ("ldo", ctypes.c_int64), ("out_bf16", ctypes.c_void_p),
        ("ldob", ctypes.c_int64), ("splits", ctypes.c_int64)]


class nmm_mla_query_path(ctypes.Structure):
    _fields_ = [(n, _i64) for n in ("hidden", "q_lora", "kv_lora", "rope", "heads", "nope")] + \
               [(n, _p) for n in ("x", "w_down", "w_uq", "w_uk", "kv_gamma")] + \
               [("kv_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("position", _i64), ("kv_cache", _p),
                ("ld_cache", _i64), ("cache_rows", _i64), ("round", ctypes.c_int)] + \
               [(n, _p) for n in ("down_f32", "cq_bf16", "q_f32", "q_bf16", "qlat_f32", "query")] + [("ldq", _i64)]


EXPORTS = {
    "nmm_gemv": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_int, _p, _i64, _p, _i64, _p, _i64,
                                ctypes.c_int, _p, _sz, _p]),
    "nmm_gemv_noalloc": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_int, _p, _i64, _p, _i64, _p, _i64, ctypes.c_int, _p]),
    "nmm_batched_gemv": (ctypes.c_int, [_i64, _i64, _i64, _i64, ctypes.c_int, _p, _i64, _i64, _p,
                                        _i64, _i64, _p, _i64, _i64, ctypes.c_int, _p, _sz, _p]),
    "nmm_gemv_bf16": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_int, _p, _i64, _p, _i64, _p, _i64,
                                     ctypes.c_int, _p, _i64, ctypes.c_int, _p, _sz, _p]),
    "nmm_mla_kv_update": (ctypes.c_int, [ctypes.POINTER(nmm_mla_kv), _p, _sz, _p]),
    "nmm_batched_gemv_bf16": (ctypes.c_int, [_i64, _i64, _i64, _i64, ctypes.c_int, _p, _i64, _i64, _p, _i64, _i64,
                                             _p, _i64, _i64, ctypes.c_int, _p, _i64, _i64, ctypes.c_int, _p, _sz, _p]),
    "nmm_mla_query": (ctypes.c_int, [_i64, _i64, _i64, _i64, _p, _p, _p, _i64, ctypes.c_float, _p, _p, _i64, _p,
                                     _sz, _p]),
    "nmm_mla_query_workspace_size": (_sz, [_i64, _i64, _i64]),
    "nmm_mla_query_path_run": (ctypes.c_int, [ctypes.POINTER(nmm_mla_query_path), _p, _sz, _p]),
    "nmm_mla_query_path_workspace_size": (_sz, [ctypes.POINTER(nmm_mla_query_path)]),
    "nmm_latent_attention_bf16": (ctypes.c_int, [_i64, _i64, _i64, _i64, _p, _i64, _p, _i64, ctypes.c_float, _p, _i64,
                                                 _p, _i64, _p, _sz, _p]),
    "nmm_latent_attention_ex": (ctypes.c_int, [_i64, _i64, _i64, _i64, _p, _i64, _p, _i64, ctypes.c_float, _p, _i64,
                                               _p, _i64, _i64, _p, _sz, _p]),
    "nmm_latent_attention_ex_workspace_size": (_sz, [_i64, _i64, _i64, _i64, _i64]),
    "nmm_gemv_nt": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_int, _p, _i64, _p, _i64, _p, _i64, _p, _sz, _p]),
    "nmm_gemv_nt_workspace_size": (_sz, [_i64, _i64, _i64, ctypes.c_int]),
    "nmm_mla_kv_update_workspace_size": (_sz, [ctypes.POINTER(nmm_mla_kv)]),
    "nmm_mla_decode_chain": (ctypes.c_int, [ctypes.POINTER(nmm_mla_chain), _p, _sz, _p]),
    "nmm_mla_decode_step": (ctypes.c_int, [ctypes.POINTER(nmm_mla_chain), ctypes.POINTER(nmm_latent_attn), _p, _sz,
                                           _p]),
    "nmm_mla_decode_step_workspace_size": (_sz, [ctypes.POINTER(nmm_mla_chain), ctypes.POINTER(nmm_latent_attn)]),
    "nmm_latent_attention": (ctypes.c_int, [_i64, _i64, _i64, _i64, _p, _i64, _p, _i64,
                                            ctypes.c_float, _p, _i64, _p, _sz, _p]),
    "nmm_gemv_workspace_size": (_sz, [_i64, _i64, _i64, ctypes.c_int, ctypes.c_int]),
    "nmm_batched_gemv_workspace_size": (_sz, [_i64, _i64, _i64, _i64, ctypes.c_int, ctypes.c_int]),
    "nmm_mla_decode_chain_workspace_size": (_sz, [ctypes.POINTER(nmm_mla_chain)]),
    "nmm_latent_attention_workspace_size": (_sz, [_i64, _i64, _i64, _i64]),
    "nmm_workspace_init": (ctypes.c_int, [_p, _sz, _p]),
    "nmm_gemv_plan": (ctypes.c_int, [_i64, _i64, _i64, _i64, ctypes.c_int, ctypes.c_int,
                                     ctypes.POINTER(nmm_plan_info)]),
    "nmm_read_probe": (ctypes.c_int, [_p, _sz, _p, _i64, ctypes.c_int, _p]),
    "nmm_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "nmm_version": (ctypes.c_char_p, []),
}


def lib() -> ctypes.CDLL:
    """Load libnmm.so (raises if it has not been built: there is no other implementation)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_16009_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def nmm_status_string(status: int) -> str:
    return lib().nmm_status_string(status).decode()


def nmm_version() -> str:
    return lib().nmm_version().decode()


def _check(status: int, where: str) -> None:
    if status != NMM_OK:
        raise NmmError(status, where)


def _dtype_code(t: torch.Tensor, dt: int | None) -> int:
    if t.dtype == torch.bfloat16:
        return NMM_BF16
    if t.dtype == torch.float16:
        return NMM_F16
    if t.dtype in (torch.int16, torch.uint16) and dt in (NMM_F16, NMM_BF16):
        return dt
    raise TypeError("x and W must be bfloat16/float16 tensors, or int16 bit patterns with dt given")


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ld(t: torch.Tensor) -> int:
    if t.stride(-1) != 1:
        raise ValueError("the last dimension must be contiguous")
    return t.stride(-2) if t.dim() >= 2 else t.shape[-1]


class Workspace:
    """Device memory for split-K partial sums and arrival counters, grown on demand.

    A workspace serves one stream at a time: calls that may overlap need different workspaces.
    A new buffer is zeroed on the stream of the call that needs it (allocated there too, so that
    torch's allocator orders its reuse with that stream); the buffers it replaces are kept until
    the Workspace is dropped, because kernels enqueued earlier may still be using them."""

    def __init__(self, device=None):
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
        self.buf = None
        self._retired = []

    def get(self, nbytes: int, stream=None) -> tuple[int, int]:
        if nbytes == 0:
            return 0, 0
        if self.buf is None or self.buf.numel() < nbytes:
            ts = _torch_stream(stream, self.device)
            size = max(nbytes, 1 << 20, 2 * self.buf.numel() if self.buf is not None else 0)
            with torch.cuda.stream(ts):
                buf = torch.empty(size, dtype=torch.uint8, device=self.device)
            _check(lib().nmm_workspace_init(buf.data_ptr(), size, ts.cuda_stream), "nmm_workspace_init")
            if self.buf is not None:
                self._retired.append(self.buf)
            self.buf = buf
        return self.buf.data_ptr(), self.buf.numel()


def _torch_stream(stream, device) -> torch.cuda.Stream:
    if stream is None:
        return torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=device)


_default_ws: dict = {}


def _workspace(ws, nbytes: int, device, stream=None) -> tuple[int, int]:
    """The workspace of one call.  Without one given, each (device, stream) pair has its own, so
    calls on different streams never share partial sums or counters."""
    if ws is None:
        dev = torch.device(device)
        key = (dev.index, _stream(stream))
        ws = _default_ws.get(key)
        if ws is None:
            ws = _default_ws[key] = Workspace(dev)
    if isinstance(ws, Workspace):
        return ws.get(nbytes, stream)
    return ws.data_ptr(), ws.numel() * ws.element_size()


def _prepared_workspace(ws, nbytes: int, device):
    """The workspace of a prepared call, which is launched later on any stream: without one
    given, a private one.  Either way it is sized and zeroed before this returns.  Returns the
    (pointer, bytes) pair and the private Workspace (None for a given one) to keep alive."""
    own = Workspace(device) if ws is None else None
    out = _workspace(own if ws is None else ws, nbytes, device)
    torch.cuda.current_stream(torch.device(device)).synchronize()
    return out, own


def nmm_gemv(x: torch.Tensor, W: torch.Tensor, y: torch.Tensor, *, N: int | None = None,
             path: int = NMM_PATH_AUTO, dt: int | None = None, workspace=None, stream=None) -> torch.Tensor:
    """y[M,N] = x[M,K] . W[K,N].  x [M, ldx], W [K, ldw], y [M, ldy] (fp32), row-major."""
    code = _dtype_code(x, dt)
    M, K = x.shape[0], W.shape[0]
    N = W.shape[1] if N is None else N
    need = lib().nmm_gemv_workspace_size(M, K, N, code, path)
    wp, wb = _workspace(workspace, need, x.device, stream)
    _check(lib().nmm_gemv(M, K, N, code, x.data_ptr(), _ld(x), W.data_ptr(), _ld(W), y.data_ptr(),
                          _ld(y), path, wp, wb, _stream(stream)), "nmm_gemv")
    return y


def nmm_gemv_noalloc(x: torch.Tensor, W: torch.Tensor, y: torch.Tensor, *, N: int | None = None,
                     path: int = NMM_PATH_AUTO, dt: int | None = None, stream=None) -> torch.Tensor:
    """nmm_gemv with the library's own scratch instead of a workspace (allocates nothing)."""
    code = _dtype_code(x, dt)
    M, K = x.shape[0], W.shape[0]
    N = W.shape[1] if N is None else N
    _check(lib().nmm_gemv_noalloc(M, K, N, code, x.data_ptr(), _ld(x), W.data_ptr(), _ld(W), y.data_ptr(), _ld(y),
                                  path, _stream(stream)), "nmm_gemv_noalloc")
    return y


def nmm_gemv_bf16(x: torch.Tensor, W: torch.Tensor, y_bf16: torch.Tensor, *, round: int = NMM_ROUND_EVEN,
                  y: torch.Tensor | None = None, N: int | None = None, path: int = NMM_PATH_AUTO,
                  dt: int | None = None, workspace=None, stream=None) -> torch.Tensor:
    """y_bf16[M,N] = bf16(x[M,K] . W[K,N]) rounded once per ``round``; ``y`` (fp32) optional."""
    code = _dtype_code(x, dt)
    M, K = x.shape[0], W.shape[0]
    N = W.shape[1] if N is None else N
    need = lib().nmm_gemv_workspace_size(M, K, N, code, path)
    wp, wb = _workspace(workspace, need, x.device, stream)
    _check(lib().nmm_gemv_bf16(M, K, N, code, x.data_ptr(), _ld(x), W.data_ptr(), _ld(W), y_bf16.data_ptr(),
                               _ld(y_bf16), round, y.data_ptr() if y is not None else None,
                               _ld(y) if y is not None else 0, path, wp, wb, _stream(stream)), "nmm_gemv_bf16")
    return y_bf16


def nmm_batched_gemv_bf16(x: torch.Tensor, W: torch.Tensor, y_bf16: torch.Tensor, *, y: torch.Tensor | None = None,
                          N: int | None = None, round: int = NMM_ROUND_EVEN, path: int = NMM_PATH_AUTO,
                          dt: int | None = None, workspace=None, stream=None) -> torch.Tensor:
    """y_bf16[b] = bf16(x[b] . W[b]) for 3-D x, W, y_bf16 (strided views allowed); ``y`` fp32 optional."""
    code = _dtype_code(x, dt)
    B, M, K = x.shape[0], x.shape[1], W.shape[1]
    N = W.shape[2] if N is None else N
    need = lib().nmm_batched_gemv_workspace_size(B, M, K, N, code, path)
    wp, wb = _workspace(workspace, need, x.device, stream)
    _check(lib().nmm_batched_gemv_bf16(B, M, K, N, code, x.data_ptr(), _ld(x), x.stride(0), W.data_ptr(), _ld(W),
                                       W.stride(0), y_bf16.data_ptr(), _ld(y_bf16), y_bf16.stride(0), round,
                                       y.data_ptr() if y is not None else None, _ld(y) if y is not None else 0,
                                       y.stride(0) if y is not None else 0, path, wp, wb, _stream(stream)),
           "nmm_batched_gemv_bf16")
    return y_bf16


def nmm_mla_query(q: torch.Tensor, q_bf16: torch.Tensor, w_uk: torch.Tensor, qlat: torch.Tensor, q_out: torch.Tensor,
                  *, nope: int, rope: int, position: int, theta: float, workspace=None, stream=None) -> torch.Tensor:
    """q_out[h] = bf16([q_nope[h] . W_UK[h] | RoPE(q[h, nope:], position)]) for q [heads, nope + rope] fp32,
    q_bf16 its bf16 rounding, w_uk [heads, nope, kv_lora]; qlat [heads, kv_lora] fp32 receives the products."""
    heads, kv_lora = w_uk.shape[0], w_uk.shape[2]
    need = lib().nmm_mla_query_workspace_size(heads, nope, kv_lora)
    wp, wb = _workspace(workspace, need, q.device, stream)
    _check(lib().nmm_mla_query(heads, nope, rope, kv_lora, q.data_ptr(), q_bf16.data_ptr(), w_uk.data_ptr(),
                               int(position), float(theta), qlat.data_ptr(), q_out.data_ptr(), _ld(q_out), wp, wb,
                               _stream(stream)), "nmm_mla_query")
    return q_out


class PreparedQueryPath:
    """nmm_mla_query_path_run with its argument struct built once.  ``dims``: hidden, q_lora,
    kv_lora, rope, heads, nope; ``bufs``: x, w_down, w_uq, w_uk, kv_gamma, kv_cache, down_f32,
    cq_bf16, q_f32, q_bf16, qlat_f32, query (tensors); ``eps``, ``theta``, ``position``."""

    def __init__(self, dims: dict, bufs: dict, *, eps: float, theta: float, position: int,
                 round: int = NMM_ROUND_EVEN, workspace=None):
        self._bufs = bufs
        c = nmm_mla_query_path()
        for k in ("hidden", "q_lora", "kv_lora", "rope", "heads", "nope"):
            setattr(c, k, int(dims[k]))
        for k in ("x", "w_down", "w_uq", "w_uk", "kv_gamma", "kv_cache", "down_f32", "cq_bf16", "q_f32", "q_bf16",
                  "qlat_f32", "query"):
            setattr(c, k, bufs[k].data_ptr())
        c.kv_eps, c.rope_theta, c.position, c.round = float(eps), float(theta), int(position), int(round)
        c.ld_cache, c.cache_rows = _ld(bufs["kv_cache"]), bufs["kv_cache"].shape[0]
        c.ldq = _ld(bufs["query"])
        self._c = c
        need = lib().nmm_mla_query_path_workspace_size(ctypes.byref(c))
        (self._wp, self._wb), self._ws = _prepared_workspace(workspace, need, bufs["x"].device)

    def launch(self, stream=None) -> None:
        _check(lib().nmm_mla_query_path_run(ctypes.byref(self._c), self._wp, self._wb, _stream(stream)),
               "nmm_mla_query_path_run")


def nmm_gemv_nt(x: torch.Tensor, Wt: torch.Tensor, y: torch.Tensor, *, K: int | None = None,
                dt: int | None = None, workspace=None, stream=None) -> torch.Tensor:
    """y[M,N] = x[M,K] . Wt[N,K]^T for Wt row-major [N, ldwt] (a torch Linear weight's layout)."""
    code = _dtype_code(x, dt)
    M, N = x.shape[0], Wt.shape[0]
    K = Wt.shape[1] if K is None else K
    need = lib().nmm_gemv_nt_workspace_size(M, K, N, code)
    wp, wb = _workspace(workspace, need, x.device, stream)
    _check(lib().nmm_gemv_nt(M, K, N, code, x.data_ptr(), _ld(x), Wt.data_ptr(), _ld(Wt), y.data_ptr(), _ld(y),
                             wp, wb, _stream(stream)), "nmm_gemv_nt")
    return y


def _kv_struct(h, w, gamma, mm, cache, *, kv_lora: int, rope: int, eps: float, theta: float,
               position: int, round: int):
    k = nmm_mla_kv()
    k.hidden = w.shape[0] if w is not None else 0      # h may be padded to a multiple of 8
    k.kv_lora, k.rope = int(kv_lora), int(rope)
    for name, t in (("h", h), ("w", w), ("gamma", gamma), ("mm", mm), ("cache", cache)):
        setattr(k, name, t.data_ptr() if t is not None else None)
    k.ldw = _ld(w) if w is not None else 0
    k.eps, k.rope_theta, k.position = float(eps), float(theta), int(position)
    k.ld_cache = _ld(cache) if cache is not None else 0
    k.cache_rows = cache.shape[0] if cache is not None else 0
    k.round = int(round)
    return k


def nmm_mla_kv_update(h: torch.Tensor, w: torch.Tensor, gamma: torch.Tensor, mm: torch.Tensor,
                      cache: torch.Tensor, *, kv_lora: int, rope: int, eps: float, theta: float,
                      position: int, round: int = NMM_ROUND_EVEN, workspace=None, stream=None) -> None:
    """MatMul 2 (h . w -> mm fp32) and the cache entry cache[position] = bf16([RMSNorm | RoPE])."""
    k = _kv_struct(h, w, gamma, mm, cache, kv_lora=kv_lora, rope=rope, eps=eps, theta=theta,
                   position=position, round=round)
    need = lib().nmm_mla_kv_update_workspace_size(ctypes.byref(k))
    wp, wb = _workspace(workspace, need, h.device, stream)
    _check(lib().nmm_mla_kv_update(ctypes.byref(k), wp, wb, _stream(stream)), "nmm_mla_kv_update")


def nmm_batched_gemv(x: torch.Tensor, W: torch.Tensor, y: torch.Tensor, *, N: int | None = None,
                     path: int = NMM_PATH_AUTO, dt: int | None = None, workspace=None,
                     stream=None) -> torch.Tensor:
    """y[b] = x[b] . W[b] for 3-D x [B, M, ldx], W [B, K, ldw], y [B, M, ldy] (strided views allowed)."""
    code = _dtype_code(x, dt)
    B, M, K = x.shape[0], x.shape[1], W.shape[1]
    N = W.shape[2] if N is None else N
    need = lib().nmm_batched_gemv_workspace_size(B, M, K, N, code, path)
    wp, wb = _workspace(workspace, need, x.device, stream)
    _check(lib().nmm_batched_gemv(B, M, K, N, code, x.data_ptr(), _ld(x), x.stride(0), W.data_ptr(),
                                  _ld(W), W.stride(0), y.data_ptr(), _ld(y), y.stride(0), path, wp,
                                  wb, _stream(stream)), "nmm_batched_gemv")
    return y


def nmm_gemv_plan(M: int, K: int, N: int, dt: int = NMM_BF16, path: int = NMM_PATH_AUTO,
                  batch: int = 1) -> dict:
    info = nmm_plan_info()
    _check(lib().nmm_gemv_plan(batch, M, K, N, dt, path, ctypes.byref(info)), "nmm_gemv_plan")
    return info.as_dict()


def nmm_gemv_workspace_size(M, K, N, dt=NMM_BF16, path=NMM_PATH_AUTO) -> int:
    return int(lib().nmm_gemv_workspace_size(M, K, N, dt, path))


def nmm_batched_gemv_workspace_size(batch, M, K, N, dt=NMM_BF16, path=NMM_PATH_AUTO) -> int:
    return int(lib().nmm_batched_gemv_workspace_size(batch, M, K, N, dt, path))


def nmm_workspace_init(ws: torch.Tensor, stream=None) -> None:
    _check(lib().nmm_workspace_init(ws.data_ptr(), ws.numel() * ws.element_size(), _stream(stream)),
           "nmm_workspace_init")


CHAIN_DIMS = ("hidden", "q_lora", "kv_lora", "rope", "heads", "nope", "v_head")
CHAIN_BUFFERS = ("x", "w_down", "w_uq", "w_uk", "w_uv", "w_o", "down_f32", "q_f32", "lat_f32",
                 "o_f32", "y", "cq_bf16", "qnope_bf16", "lat_bf16", "o_bf16")


def _chain_struct(dims: dict, bufs: dict, events=None, kv: dict | None = None):
    """``kv`` (optional): the cache entry behind the down-projection, a dict with the tensors
    ``gamma`` and ``cache`` and the numbers ``eps``, ``theta``, ``position`` and ``round``."""
    c = nmm_mla_chain()
    for k in CHAIN_DIMS:
        setattr(c, k, int(dims[k]))
    for k in CHAIN_BUFFERS:
        t = bufs.get(k)
        setattr(c, k, t.data_ptr() if t is not None else None)
    if kv is not None:
        cache = kv["cache"]
        c.kv_gamma = kv["gamma"].data_ptr()
        c.kv_eps, c.rope_theta = float(kv["eps"]), float(kv["theta"])
        c.position = int(kv["position"])
        c.kv_cache = cache.data_ptr()
        c.ld_cache, c.cache_rows = _ld(cache), cache.shape[0]
        c.round = int(kv.get("round", NMM_ROUND_EVEN))
    keep = None
    if events is not None:
        for e in events:
            if not e.cuda_event:      # torch creates the HIP event at its first record
                e.record()
        handles = [e.cuda_event for e in events]
        keep = (_p * len(handles))(*handles)
        c.events = ctypes.cast(keep, _p)
        c.n_events = len(handles)
    return c, keep


class PreparedChain:
    """A decode chain whose argument struct is built once, so that a launch is a single C call
    (for tight loops where Python overhead would otherwise show).  ``events`` is an optional
    list of event lists, one per slot; ``launch(slot)`` uses slot ``slot``'s events."""

    def __init__(self, dims: dict, bufs: dict, workspace=None, events=None, kv: dict | None = None):
        self._bufs = bufs                       # keep the tensors alive
        self._kv = kv
        self._slots = []
        for evs in (events or [None]):
            c, keep = _chain_struct(dims, bufs, evs, kv)
            self._slots.append((c, keep))
        need = lib().nmm_mla_decode_chain_workspace_size(ctypes.byref(self._slots[0][0]))
        (self._wp, self._wb), self._ws = _prepared_workspace(workspace, need, bufs["x"].device)

    def launch(self, slot: int = 0, stream=None) -> None:
        c = self._slots[slot][0]
        _check(lib().nmm_mla_decode_chain(ctypes.byref(c), self._wp, self._wb, _stream(stream)),
               "nmm_mla_decode_chain")


def _attn_struct(attn: dict) -> nmm_latent_attn:
    """nmm_latent_attn from {q, kv, out, scale[, out_bf16, splits, d_qk, d_v]} (q [heads, >= d_qk] and
    kv [seq, >= max(d_qk, d_v)] bf16, out [heads, >= d_v] fp32)."""
    q, kv, out = attn["q"], attn["kv"], attn["out"]
    ob = attn.get("out_bf16")
    a = nmm_latent_attn()
    a.heads, a.seq = q.shape[0], kv.shape[0]
    a.d_qk = attn.get("d_qk", q.shape[1])
    a.d_v = attn.get("d_v", 512)
    a.q, a.ldq, a.kv, a.ld_kv = q.data_ptr(), _ld(q), kv.data_ptr(), _ld(kv)
    a.scale = float(attn["scale"])
    a.out, a.ldo = out.data_ptr(), _ld(out)
    a.out_bf16, a.ldob = (ob.data_ptr(), _ld(ob)) if ob is not None else (None, 0)
    a.splits = int(attn.get("splits", 0))
    return a


class PreparedStep:
    """A decode step (nmm_mla_decode_step: the chain and an independent latent attention, the
    attention sharing W_O's launch) with its argument structs built once, so that a launch is a
    single C call.  ``attn`` is {q, kv, out, scale[, out_bf16, splits, d_qk, d_v]}."""

    def __init__(self, dims: dict, bufs: dict, attn: dict, workspace=None, events=None, kv: dict | None = None):
        self._bufs, self._attn_bufs, self._kv = bufs, attn, kv   # keep the tensors alive
        self._a = _attn_struct(attn)
        self._slots = []
        for evs in (events or [None]):
            c, keep = _chain_struct(dims, bufs, evs, kv)
            self._slots.append((c, keep))
        need = lib().nmm_mla_decode_step_workspace_size(ctypes.byref(self._slots[0][0]), ctypes.byref(self._a))
        if need == 0:
            raise ValueError("nmm_mla_decode_step: invalid chain or attention sizes")
        (self._wp, self._wb), self._ws = _prepared_workspace(workspace, need, bufs["x"].device)

    def launch(self, slot: int = 0, stream=None) -> None:
        c = self._slots[slot][0]
        _check(lib().nmm_mla_decode_step(ctypes.byref(c), ctypes.byref(self._a), self._wp, self._wb, _stream(stream)),
               "nmm_mla_decode_step")


def nmm_mla_decode_step(dims: dict, bufs: dict, attn: dict, *, workspace=None, stream=None, events=None,
                        kv: dict | None = None) -> None:
    """One decode step (see nmm.h): the chain of nmm_mla_decode_chain and the attention ``attn``
    ({q, kv, out, scale[, out_bf16, splits, d_qk, d_v]}) beside it (its workgroups in W_UQ's
    launch, its merge in the W_UK -> W_UV pair's)."""
    PreparedStep(dims, bufs, attn, workspace=workspace, events=None if events is None else [events],
                 kv=kv).launch(stream=stream)


def nmm_mla_decode_step_workspace_size(dims: dict, attn: dict) -> int:
    c, _ = _chain_struct(dims, {})
    a = _attn_struct(attn)
    return int(lib().nmm_mla_decode_step_workspace_size(ctypes.byref(c), ctypes.byref(a)))


def nmm_mla_decode_chain_workspace_size(dims: dict) -> int:
    c, _ = _chain_struct(dims, {})
    return int(lib().nmm_mla_decode_chain_workspace_size(ctypes.byref(c)))


def nmm_mla_decode_chain(dims: dict, bufs: dict, *, workspace=None, stream=None, events=None,
                         kv: dict | None = None) -> None:
    """One decode chain (see nmm.h).  ``bufs`` maps the nmm_mla_chain field names to tensors;
    ``events`` is an optional list of >= 6 torch.cuda.Event(enable_timing=True); ``kv`` the
    optional cache entry (see _chain_struct)."""
    c, keep = _chain_struct(dims, bufs, events, kv)
    need = lib().nmm_mla_decode_chain_workspace_size(ctypes.byref(c))
    wp, wb = _workspace(workspace, need, bufs["x"].device, stream)
    _check(lib().nmm_mla_decode_chain(ctypes.byref(c), wp, wb, _stream(stream)), "nmm_mla_decode_chain")
    del keep


def nmm_latent_attention_workspace_size(heads, seq, d_qk, d_v) -> int:
    return int(lib().nmm_latent_attention_workspace_size(heads, seq, d_qk, d_v))


def nmm_latent_attention(q: torch.Tensor, kv: torch.Tensor, out: torch.Tensor, scale: float, *,
                         d_qk: int | None = None, d_v: int = 512, workspace=None, stream=None) -> torch.Tensor:
    """out[h, :d_v] = softmax(scale * q[h] . kv[:, :d_qk]^T) . kv[:, :d_v]  (bf16 in, fp32 out)."""
    heads, seq = q.shape[0], kv.shape[0]
    d_qk = q.shape[1] if d_qk is None else d_qk
    need = lib().nmm_latent_attention_workspace_size(heads, seq, d_qk, d_v)
    wp, wb = _workspace(workspace, need, q.device, stream)
    _check(lib().nmm_latent_attention(heads, seq, d_qk, d_v, q.data_ptr(), _ld(q), kv.data_ptr(),
                                      _ld(kv), float(scale), out.data_ptr(), _ld(out), wp, wb,
                                      _stream(stream)), "nmm_latent_attention")
    return out


def nmm_latent_attention_bf16(q: torch.Tensor, kv: torch.Tensor, out: torch.Tensor, out_bf16: torch.Tensor,
                              scale: float, *, d_qk: int | None = None, d_v: int = 512, workspace=None,
                              stream=None) -> torch.Tensor:
    """nmm_latent_attention, also writing out_bf16 = bf16(out)."""
    heads, seq = q.shape[0], kv.shape[0]
    d_qk = q.shape[1] if d_qk is None else d_qk
    need = lib().nmm_latent_attention_workspace_size(heads, seq, d_qk, d_v)
    wp, wb = _workspace(workspace, need, q.device, stream)
    _check(lib().nmm_latent_attention_bf16(heads, seq, d_qk, d_v, q.data_ptr(), _ld(q), kv.data_ptr(), _ld(kv),
                                           float(scale), out.data_ptr(), _ld(out), out_bf16.data_ptr(), _ld(out_bf16),
                                           wp, wb, _stream(stream)), "nmm_latent_attention_bf16")
    return out


def nmm_latent_attention_ex(q: torch.Tensor, kv: torch.Tensor, out: torch.Tensor, scale: float, *, splits: int = 0,
                            out_bf16: torch.Tensor | None = None, d_qk: int | None = None, d_v: int = 512,
                            workspace=None, stream=None) -> torch.Tensor:
    """nmm_latent_attention with `splits` position spans (0: default) and an optional bf16 copy
    of the output."""
    heads, seq = q.shape[0], kv.shape[0]
    d_qk = q.shape[1] if d_qk is None else d_qk
    need = lib().nmm_latent_attention_ex_workspace_size(heads, seq, d_qk, d_v, splits)
    wp, wb = _workspace(workspace, need, q.device, stream)
    _check(lib().nmm_latent_attention_ex(heads, seq, d_qk, d_v, q.data_ptr(), _ld(q), kv.data_ptr(), _ld(kv),
                                         float(scale), out.data_ptr(), _ld(out),
                                         out_bf16.data_ptr() if out_bf16 is not None else None,
                                         _ld(out_bf16) if out_bf16 is not None else 0, int(splits), wp, wb,
                                         _stream(stream)), "nmm_latent_attention_ex")
    return out


def nmm_read_probe(buf: torch.Tensor, out: torch.Tensor, grid: int, unroll: int = 4, stream=None) -> None:
    """Read all of ``buf`` once on the GPU (bandwidth calibration); ``out`` holds >= grid uint32."""
    if out.numel() * out.element_size() < 4 * grid:
        raise ValueError("out must hold one uint32 per workgroup")
    _check(lib().nmm_read_probe(buf.data_ptr(), buf.numel() * buf.element_size(), out.data_ptr(), grid,
                                unroll, _stream(stream)), "nmm_read_probe")
