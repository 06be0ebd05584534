"""The C ABI without a GPU: the library loads, exports every function include/nmm.h declares,
rejects every invalid argument before touching the device, and plans partitions that cover W
exactly once.  No compute call is made here.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nmm.h")

nmm = pytest.importorskip("paper_2609_16009_amd")
if not os.path.exists(nmm.LIB_PATH):
    pytest.skip("libnmm.so not built", allow_module_level=True)

L = nmm.lib()
ALIGNED = 1 << 20          # a fake, 256-byte aligned "device address"; never dereferenced here


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return sorted(set(re.findall(r"\b(nmm_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_function_is_exported():
    names = declared_functions()
    assert "nmm_gemv" in names and "nmm_mla_decode_chain" in names and "nmm_latent_attention" in names
    raw = ctypes.CDLL(nmm.LIB_PATH)
    missing = [n for n in names if not hasattr(raw, n)]
    assert not missing, f"declared but not exported: {missing}"
    assert set(names) <= set(nmm.EXPORTS), "the binding must cover every declared function"


def test_status_strings_and_version():
    for s in range(9):
        assert L.nmm_status_string(s).decode().startswith("NMM_")
    assert nmm.nmm_version().count(".") == 2


def gemv(**kw):
    a = dict(M=1, K=64, N=64, dt=nmm.NMM_BF16, x=ALIGNED, ldx=64, W=ALIGNED, ldw=64, y=ALIGNED, ldy=64,
             path=nmm.NMM_PATH_AUTO, ws=ALIGNED, wsb=1 << 30, stream=None)
    a.update(kw)
    return L.nmm_gemv(a["M"], a["K"], a["N"], a["dt"], a["x"], a["ldx"], a["W"], a["ldw"], a["y"],
                      a["ldy"], a["path"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), nmm.NMM_ERR_NULL),
    (dict(W=None), nmm.NMM_ERR_NULL),
    (dict(y=None), nmm.NMM_ERR_NULL),
    (dict(dt=3), nmm.NMM_ERR_DTYPE),
    (dict(dt=0), nmm.NMM_ERR_DTYPE),
    (dict(path=9), nmm.NMM_ERR_PATH),
    (dict(M=-1), nmm.NMM_ERR_SHAPE),
    (dict(K=-5), nmm.NMM_ERR_SHAPE),
    (dict(ldx=32), nmm.NMM_ERR_SHAPE),
    (dict(ldw=32), nmm.NMM_ERR_SHAPE),
    (dict(ldy=32), nmm.NMM_ERR_SHAPE),
    (dict(N=61, ldw=61, ldy=61), nmm.NMM_ERR_ALIGN),
    (dict(x=ALIGNED + 2), nmm.NMM_ERR_ALIGN),
    (dict(W=ALIGNED + 8), nmm.NMM_ERR_ALIGN),
    (dict(ldx=66), nmm.NMM_ERR_ALIGN),
    (dict(y=ALIGNED + 2), nmm.NMM_ERR_ALIGN),
    (dict(M=1, K=1 << 31), nmm.NMM_ERR_SHAPE),
    (dict(K=40000, N=40000, ldw=40000, ldy=40000, ldx=40000), nmm.NMM_ERR_SHAPE),  # W > 2 GiB
    (dict(M=2, ldx=1 << 30), nmm.NMM_ERR_SHAPE),    # two x rows 2 GiB apart: one block > 2 GiB
    (dict(M=40, ldx=1 << 26), nmm.NMM_ERR_SHAPE),   # a 32-row block of x spans > 2 GiB
    (dict(K=4096, N=4096, ldw=4096, ldy=4096, ldx=4096, ws=None), nmm.NMM_ERR_WORKSPACE),
    (dict(K=4096, N=4096, ldw=4096, ldy=4096, ldx=4096, wsb=16), nmm.NMM_ERR_WORKSPACE),
    (dict(K=4096, N=4096, ldw=4096, ldy=4096, ldx=4096, ws=ALIGNED + 64), nmm.NMM_ERR_WORKSPACE),
])
def test_gemv_rejects_invalid_arguments(kw, status):
    assert gemv(**kw) == status


@pytest.mark.parametrize("kw", [dict(M=0), dict(N=0), dict(M=0, x=None, W=None, y=None)])
def test_empty_problems_are_noops_without_device_access(kw):
    assert gemv(**kw) == nmm.NMM_OK


def test_batched_rejects_misaligned_strides():
    st = L.nmm_batched_gemv(4, 1, 64, 64, nmm.NMM_BF16, ALIGNED, 64, 68, ALIGNED, 64, 64 * 64,
                            ALIGNED, 64, 64, 0, ALIGNED, 1 << 30, None)
    assert st == nmm.NMM_ERR_ALIGN
    st = L.nmm_batched_gemv(4, 1, 64, 64, nmm.NMM_BF16, ALIGNED, 64, -64, ALIGNED, 64, 64 * 64,
                            ALIGNED, 64, 64, 0, ALIGNED, 1 << 30, None)
    assert st == nmm.NMM_ERR_SHAPE
    assert L.nmm_batched_gemv(0, 1, 64, 64, nmm.NMM_BF16, None, 64, 64, None, 64, 64, None, 64, 64,
                              0, None, 0, None) == nmm.NMM_OK


def test_chain_rejects_null_and_bad_dims():
    assert L.nmm_mla_decode_chain(None, None, 0, None) == nmm.NMM_ERR_NULL
    dims = dict(hidden=7168, q_lora=1536, kv_lora=512, rope=64, heads=128, nope=128, v_head=128)
    bufs = {k: None for k in nmm.CHAIN_BUFFERS}
    c, _ = nmm._chain_struct(dims, {})
    assert L.nmm_mla_decode_chain(ctypes.byref(c), ALIGNED, 1 << 30, None) == nmm.NMM_ERR_NULL
    for k in nmm.CHAIN_BUFFERS:
        setattr(c, k, ALIGNED)
    c.hidden = 0
    assert L.nmm_mla_decode_chain(ctypes.byref(c), ALIGNED, 1 << 30, None) == nmm.NMM_ERR_SHAPE
    c.hidden = 7168
    assert L.nmm_mla_decode_chain(ctypes.byref(c), None, 0, None) == nmm.NMM_ERR_WORKSPACE
    c.x = ALIGNED + 2
    assert L.nmm_mla_decode_chain(ctypes.byref(c), ALIGNED, 1 << 30, None) == nmm.NMM_ERR_ALIGN
    assert nmm.nmm_mla_decode_chain_workspace_size(dims) > 0
    del bufs


def test_workspace_init_validates():
    assert L.nmm_workspace_init(None, 16, None) == nmm.NMM_ERR_NULL
    assert L.nmm_workspace_init(ALIGNED + 4, 16, None) == nmm.NMM_ERR_WORKSPACE
    assert L.nmm_workspace_init(None, 0, None) == nmm.NMM_OK


SHAPES = [(1, 512, 512), (1, 7168, 2112), (1, 7168, 576), (1, 1536, 24576), (1, 16384, 7168),
          (2, 1536, 24576), (4, 1536, 24576), (8, 1536, 24576), (16, 1536, 24576), (32, 1536, 24576),
          (3, 1021, 1031), (1, 1, 1), (1, 13, 8), (5, 77, 3), (16, 4099, 520), (1, 128, 512),
          (1, 512, 128), (7, 9000, 4200)]


@pytest.mark.parametrize("M,K,N", SHAPES)
@pytest.mark.parametrize("batch", [1, 128])
def test_plan_covers_w_exactly_once(M, K, N, batch):
    p = nmm.nmm_gemv_plan(M, K, N, nmm.NMM_BF16, nmm.NMM_PATH_GEMV, batch=batch)
    chunks = -(-N // 8)
    pw = p["panel_width"]
    assert pw in (8, 16, 32, 64)
    assert p["n_full_panels"] == chunks // pw and p["tail_chunks"] == chunks % pw
    assert p["m_blocks"] * p["m_tile"] >= M and (p["m_blocks"] - 1) * p["m_tile"] < M
    waves = p["threads"] // 64
    for ks, rows, width, present in [(p["split_k_full"], p["rows_full"], pw, p["n_full_panels"] > 0),
                                     (p["split_k_tail"], p["rows_tail"], p["tail_width"], p["tail_chunks"] > 0)]:
        if not present:
            continue
        assert width >= 1 and (width & (width - 1)) == 0
        rstep = waves * 64 // width
        assert rows % (rstep * p["unroll"]) == 0          # whole unrolled row-steps per K-slice
        assert ks * rows >= K and (ks - 1) * rows < K     # slices tile K, none empty
        assert rows * p["m_tile"] * 4 <= 32 * 1024         # staged x slice fits its LDS budget
    if p["tail_chunks"]:
        assert p["tail_width"] >= p["tail_chunks"]
    items = p["n_full_panels"] * p["split_k_full"] + (p["split_k_tail"] if p["tail_chunks"] else 0)
    assert p["items"] == items and p["grid"] == batch * p["m_blocks"] * items
    split = max(p["split_k_full"], p["split_k_tail"]) > 1
    assert (p["workspace_bytes"] > 0) == split
    assert nmm.nmm_batched_gemv_workspace_size(batch, M, K, N, nmm.NMM_BF16, nmm.NMM_PATH_GEMV) == p["workspace_bytes"]


def test_plan_rejects_unavailable_path_and_bad_dtype():
    info = nmm.nmm_plan_info()
    assert L.nmm_gemv_plan(1, 1, 64, 64, 7, 0, ctypes.byref(info)) == nmm.NMM_ERR_DTYPE
    assert L.nmm_gemv_plan(1, 1, 64, 64, nmm.NMM_BF16, 5, ctypes.byref(info)) == nmm.NMM_ERR_PATH
    assert L.nmm_gemv_plan(1, 1, 64, 64, nmm.NMM_BF16, 0, None) == nmm.NMM_ERR_NULL


def gemv_bf16(**kw):
    a = dict(M=1, K=64, N=64, dt=nmm.NMM_BF16, x=ALIGNED, ldx=64, W=ALIGNED, ldw=64, yb=ALIGNED, ldyb=64,
             round=nmm.NMM_ROUND_EVEN, y=None, ldy=0, path=nmm.NMM_PATH_AUTO, ws=ALIGNED, wsb=1 << 30,
             stream=None)
    a.update(kw)
    return L.nmm_gemv_bf16(a["M"], a["K"], a["N"], a["dt"], a["x"], a["ldx"], a["W"], a["ldw"], a["yb"],
                           a["ldyb"], a["round"], a["y"], a["ldy"], a["path"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(yb=None), nmm.NMM_ERR_NULL),
    (dict(round=2), nmm.NMM_ERR_ARG),
    (dict(round=-1), nmm.NMM_ERR_ARG),
    (dict(ldyb=63), nmm.NMM_ERR_SHAPE),
    (dict(yb=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
    (dict(y=ALIGNED, ldy=32), nmm.NMM_ERR_SHAPE),
    (dict(y=ALIGNED + 2, ldy=64), nmm.NMM_ERR_ALIGN),
    (dict(x=None), nmm.NMM_ERR_NULL),
    (dict(M=-1), nmm.NMM_ERR_SHAPE),
    (dict(K=4096, N=4096, ldw=4096, ldyb=4096, ldx=4096, ws=None), nmm.NMM_ERR_WORKSPACE),
])
def test_gemv_bf16_rejects_invalid_arguments(kw, status):
    assert gemv_bf16(**kw) == status


@pytest.mark.parametrize("kw", [dict(M=0), dict(N=0, ldyb=0), dict(M=0, yb=None, x=None)])
def test_gemv_bf16_empty_problems_are_noops(kw):
    assert gemv_bf16(**kw) == nmm.NMM_OK


def kv_struct(**kw):
    k = nmm.nmm_mla_kv()
    vals = dict(hidden=7168, kv_lora=512, rope=64, h=ALIGNED, w=ALIGNED, ldw=576, gamma=ALIGNED, eps=1e-6,
                rope_theta=10000.0, position=4096, mm=ALIGNED, cache=ALIGNED, ld_cache=576, cache_rows=4097,
                round=nmm.NMM_ROUND_EVEN)
    vals.update(kw)
    for name, v in vals.items():
        setattr(k, name, v)
    return k


def test_kv_update_workspace_covers_the_counter_block():
    k = kv_struct()
    need = L.nmm_mla_kv_update_workspace_size(ctypes.byref(k))
    plan = nmm.nmm_gemv_plan(1, 7168, 576, path=nmm.NMM_PATH_GEMV)
    assert need >= 64 * 1024 and need >= plan["workspace_bytes"]
    assert L.nmm_mla_kv_update_workspace_size(ctypes.byref(kv_struct(rope=63))) == 0
    assert L.nmm_mla_kv_update_workspace_size(None) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(h=None), nmm.NMM_ERR_NULL),
    (dict(w=None), nmm.NMM_ERR_NULL),
    (dict(gamma=None), nmm.NMM_ERR_NULL),
    (dict(mm=None), nmm.NMM_ERR_NULL),
    (dict(cache=None), nmm.NMM_ERR_NULL),
    (dict(hidden=0), nmm.NMM_ERR_SHAPE),
    (dict(kv_lora=0), nmm.NMM_ERR_SHAPE),
    (dict(rope=63, ldw=576), nmm.NMM_ERR_SHAPE),
    (dict(rope=-2), nmm.NMM_ERR_SHAPE),
    (dict(rope=514, ldw=1032, ld_cache=1032), nmm.NMM_ERR_SHAPE),
    (dict(kv_lora=4096, rope=64, ldw=4160, ld_cache=4160), nmm.NMM_ERR_SHAPE),
    (dict(ldw=568), nmm.NMM_ERR_SHAPE),
    (dict(ld_cache=575), nmm.NMM_ERR_SHAPE),
    (dict(position=4097), nmm.NMM_ERR_SHAPE),
    (dict(position=-1), nmm.NMM_ERR_SHAPE),
    (dict(cache_rows=0, position=0), nmm.NMM_ERR_SHAPE),
    (dict(eps=-1.0), nmm.NMM_ERR_ARG),
    (dict(eps=float("nan")), nmm.NMM_ERR_ARG),
    (dict(rope_theta=0.0), nmm.NMM_ERR_ARG),
    (dict(rope_theta=float("inf")), nmm.NMM_ERR_ARG),
    (dict(round=5), nmm.NMM_ERR_ARG),
    (dict(ldw=580), nmm.NMM_ERR_ALIGN),
    (dict(h=ALIGNED + 8), nmm.NMM_ERR_ALIGN),
    (dict(gamma=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
    (dict(cache=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
    (dict(mm=ALIGNED + 2), nmm.NMM_ERR_ALIGN),
])
def test_kv_update_rejects_invalid_arguments(kw, status):
    k = kv_struct(**kw)
    assert L.nmm_mla_kv_update(ctypes.byref(k), ALIGNED, 1 << 30, None) == status


def test_kv_update_rejects_small_or_missing_workspace():
    k = kv_struct()
    need = L.nmm_mla_kv_update_workspace_size(ctypes.byref(k))
    assert L.nmm_mla_kv_update(ctypes.byref(k), None, 0, None) == nmm.NMM_ERR_WORKSPACE
    assert L.nmm_mla_kv_update(ctypes.byref(k), ALIGNED, need - 1, None) == nmm.NMM_ERR_WORKSPACE
    assert L.nmm_mla_kv_update(None, ALIGNED, need, None) == nmm.NMM_ERR_NULL


@pytest.mark.parametrize("kw,status", [
    (dict(kv_gamma=None), nmm.NMM_ERR_NULL),
    (dict(position=4097), nmm.NMM_ERR_SHAPE),
    (dict(ld_cache=575), nmm.NMM_ERR_SHAPE),
    (dict(kv_eps=float("nan")), nmm.NMM_ERR_ARG),
    (dict(rope_theta=-1.0), nmm.NMM_ERR_ARG),
    (dict(round=3), nmm.NMM_ERR_ARG),
    (dict(kv_cache=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
    (dict(kv_gamma=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
])
def test_chain_rejects_bad_cache_entry(kw, status):
    dims = dict(hidden=7168, q_lora=1536, kv_lora=512, rope=64, heads=128, nope=128, v_head=128)
    c, _ = nmm._chain_struct(dims, {})
    for k in nmm.CHAIN_BUFFERS:
        setattr(c, k, ALIGNED)
    vals = dict(kv_gamma=ALIGNED, kv_eps=1e-6, rope_theta=10000.0, position=4096, kv_cache=ALIGNED,
                ld_cache=576, cache_rows=4097, round=0)
    vals.update(kw)
    for k, v in vals.items():
        setattr(c, k, v)
    assert L.nmm_mla_decode_chain(ctypes.byref(c), ALIGNED, 1 << 30, None) == status


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structures have the C layout of include/nmm.h (compiled with gcc)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    probes = {"nmm_mla_chain": ["x", "events", "n_events", "kv_gamma", "kv_eps", "position", "kv_cache", "round"],
              "nmm_mla_kv": ["h", "ldw", "gamma", "eps", "rope_theta", "position", "mm", "cache_rows", "round"],
              "nmm_plan_info": ["path", "grid", "workspace_bytes"],
              "nmm_mla_query_path": ["x", "kv_gamma", "kv_eps", "position", "round", "down_f32", "query", "ldq"],
              "nmm_latent_attn": ["heads", "q", "ldq", "kv", "scale", "out", "ldo", "out_bf16", "ldob", "splits"]}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "nmm.h"', "int main(void) {"]
    for st, fields in probes.items():
        lines.append(f'  printf("{st} sizeof %zu\\n", sizeof({st}));')
        for f in fields:
            lines.append(f'  printf("{st} {f} %zu\\n", offsetof({st}, {f}));')
    lines.append("  return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for st, fields in probes.items():
        cls = getattr(nmm, st)
        assert got[(st, "sizeof")] == ctypes.sizeof(cls), st
        for f in fields:
            assert got[(st, f)] == getattr(cls, f).offset, (st, f)


def gemv_nt(**kw):
    a = dict(M=1, K=64, N=64, dt=nmm.NMM_BF16, x=ALIGNED, ldx=64, W=ALIGNED, ldw=64, y=ALIGNED, ldy=64,
             ws=ALIGNED, wsb=1 << 30, stream=None)
    a.update(kw)
    return L.nmm_gemv_nt(a["M"], a["K"], a["N"], a["dt"], a["x"], a["ldx"], a["W"], a["ldw"], a["y"], a["ldy"],
                         a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), nmm.NMM_ERR_NULL),
    (dict(W=None), nmm.NMM_ERR_NULL),
    (dict(y=None), nmm.NMM_ERR_NULL),
    (dict(dt=0), nmm.NMM_ERR_DTYPE),
    (dict(M=-1), nmm.NMM_ERR_SHAPE),
    (dict(ldx=56), nmm.NMM_ERR_SHAPE),
    (dict(ldw=56), nmm.NMM_ERR_SHAPE),              # ldwt < K
    (dict(ldy=60), nmm.NMM_ERR_SHAPE),
    (dict(K=60, ldw=60, ldx=64), nmm.NMM_ERR_ALIGN),  # ldwt not a multiple of 8
    (dict(W=ALIGNED + 8), nmm.NMM_ERR_ALIGN),
    (dict(y=ALIGNED + 2), nmm.NMM_ERR_ALIGN),
    (dict(N=40000, K=40000, ldw=40000, ldx=40000, ldy=40000), nmm.NMM_ERR_SHAPE),   # Wt > 2 GiB
    (dict(K=20000, ldw=20000, ldx=20000, ws=None), nmm.NMM_ERR_WORKSPACE),          # split K needs one
])
def test_gemv_nt_rejects_invalid_arguments(kw, status):
    assert gemv_nt(**kw) == status


def test_gemv_nt_workspace_only_when_k_splits():
    assert L.nmm_gemv_nt_workspace_size(1, 16384, 7168, nmm.NMM_BF16) == 0
    assert L.nmm_gemv_nt_workspace_size(1, 16385, 7168, nmm.NMM_BF16) > 64 * 1024
    assert L.nmm_gemv_nt_workspace_size(4, 4096, 100, nmm.NMM_BF16) == 0
    assert L.nmm_gemv_nt_workspace_size(4, 4097, 100, nmm.NMM_BF16) > 0       # 4096 k per slice at mt = 4
    assert gemv_nt(M=0, x=None, W=None, y=None) == nmm.NMM_OK


def mla_query(**kw):
    a = dict(heads=128, nope=128, rope=64, kv=512, q=ALIGNED, qb=ALIGNED, w=ALIGNED, pos=4096, theta=10000.0,
             qlat=ALIGNED, out=ALIGNED, ldq=576, ws=ALIGNED, wsb=1 << 30)
    a.update(kw)
    return L.nmm_mla_query(a["heads"], a["nope"], a["rope"], a["kv"], a["q"], a["qb"], a["w"], a["pos"], a["theta"],
                           a["qlat"], a["out"], a["ldq"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), nmm.NMM_ERR_NULL),
    (dict(qb=None), nmm.NMM_ERR_NULL),
    (dict(w=None), nmm.NMM_ERR_NULL),
    (dict(qlat=None), nmm.NMM_ERR_NULL),
    (dict(out=None), nmm.NMM_ERR_NULL),
    (dict(rope=63), nmm.NMM_ERR_SHAPE),
    (dict(rope=514), nmm.NMM_ERR_SHAPE),
    (dict(nope=0), nmm.NMM_ERR_SHAPE),
    (dict(ldq=575), nmm.NMM_ERR_SHAPE),
    (dict(pos=-1), nmm.NMM_ERR_SHAPE),
    (dict(theta=0.0), nmm.NMM_ERR_ARG),
    (dict(theta=float("nan")), nmm.NMM_ERR_ARG),
    (dict(q=ALIGNED + 2), nmm.NMM_ERR_ALIGN),
    (dict(out=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
    (dict(nope=120, rope=6), nmm.NMM_ERR_ALIGN),      # head stride nope + rope = 126: not a multiple of 8
    (dict(qb=ALIGNED + 8), nmm.NMM_ERR_ALIGN),
])
def test_mla_query_rejects_invalid_arguments(kw, status):
    assert mla_query(**kw) == status


def test_mla_query_empty_and_workspace():
    assert mla_query(heads=0, q=None, qb=None, w=None, qlat=None, out=None) == nmm.NMM_OK
    need = L.nmm_mla_query_workspace_size(128, 128, 512)
    assert need == nmm.nmm_batched_gemv_workspace_size(128, 1, 128, 512)


@pytest.mark.parametrize("kw,status", [
    (dict(yb=None), nmm.NMM_ERR_NULL),
    (dict(round=7), nmm.NMM_ERR_ARG),
    (dict(ldyb=60), nmm.NMM_ERR_SHAPE),
    (dict(syb=-1), nmm.NMM_ERR_SHAPE),
    (dict(yb=ALIGNED + 1), nmm.NMM_ERR_ALIGN),
    (dict(sx=68), nmm.NMM_ERR_ALIGN),
])
def test_batched_gemv_bf16_rejects_invalid_arguments(kw, status):
    a = dict(B=4, M=1, K=64, N=64, x=ALIGNED, ldx=64, sx=64, W=ALIGNED, ldw=64, sw=64 * 64, yb=ALIGNED, ldyb=64,
             syb=64, round=0, y=None, ldy=0, sy=0)
    a.update(kw)
    assert L.nmm_batched_gemv_bf16(a["B"], a["M"], a["K"], a["N"], nmm.NMM_BF16, a["x"], a["ldx"], a["sx"], a["W"],
                                   a["ldw"], a["sw"], a["yb"], a["ldyb"], a["syb"], a["round"], a["y"], a["ldy"],
                                   a["sy"], nmm.NMM_PATH_AUTO, ALIGNED, 1 << 30, None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(splits=-1), nmm.NMM_ERR_ARG),
    (dict(ob=ALIGNED + 1, ldob=512), nmm.NMM_ERR_ALIGN),
    (dict(ob=ALIGNED, ldob=500), nmm.NMM_ERR_SHAPE),
    (dict(out=None), nmm.NMM_ERR_NULL),
    (dict(scale=float("inf")), nmm.NMM_ERR_ARG),
])
def test_attention_ex_rejects_invalid_arguments(kw, status):
    a = dict(q=ALIGNED, kv=ALIGNED, out=ALIGNED, ob=None, ldob=0, splits=16, scale=0.07)
    a.update(kw)
    assert L.nmm_latent_attention_ex(128, 4096, 576, 512, a["q"], 576, a["kv"], 576, a["scale"], a["out"], 512, a["ob"],
                                     a["ldob"], a["splits"], ALIGNED, 1 << 30, None) == status


def test_attention_ex_workspace_follows_the_partition():
    w16 = L.nmm_latent_attention_ex_workspace_size(128, 4096, 576, 512, 16)
    w32 = L.nmm_latent_attention_ex_workspace_size(128, 4096, 576, 512, 32)
    # the default partition: 16 spans for 128 heads (one workspace size for either head block)
    assert 0 < w16 < w32 and w16 == nmm.nmm_latent_attention_workspace_size(128, 4096, 576, 512)
    assert L.nmm_latent_attention_ex_workspace_size(128, 4096, 576, 512, 1) == 0     # one span: no merge
    assert L.nmm_latent_attention_ex_workspace_size(128, 4096, 576, 512, -1) == 0


def test_query_path_rejects_invalid_arguments():
    c = nmm.nmm_mla_query_path()
    for k, v in dict(hidden=7168, q_lora=1536, kv_lora=512, rope=64, heads=128, nope=128).items():
        setattr(c, k, v)
    assert L.nmm_mla_query_path_run(None, ALIGNED, 1 << 30, None) == nmm.NMM_ERR_NULL
    assert L.nmm_mla_query_path_run(ctypes.byref(c), ALIGNED, 1 << 30, None) == nmm.NMM_ERR_NULL
    for k in ("x", "w_down", "w_uq", "w_uk", "kv_gamma", "kv_cache", "down_f32", "cq_bf16", "q_f32", "q_bf16",
              "qlat_f32", "query"):
        setattr(c, k, ALIGNED)
    c.kv_eps, c.rope_theta, c.position, c.ld_cache, c.cache_rows, c.ldq = 1e-6, 10000.0, 4096, 576, 4097, 576
    need = L.nmm_mla_query_path_workspace_size(ctypes.byref(c))
    assert need > 0
    assert L.nmm_mla_query_path_run(ctypes.byref(c), ALIGNED, need - 1, None) == nmm.NMM_ERR_WORKSPACE
    c.position = 4097
    assert L.nmm_mla_query_path_run(ctypes.byref(c), ALIGNED, need, None) == nmm.NMM_ERR_SHAPE
    c.position, c.ldq = 4096, 570
    assert L.nmm_mla_query_path_run(ctypes.byref(c), ALIGNED, need, None) == nmm.NMM_ERR_SHAPE
    c.ldq, c.rope = 576, 65
    assert L.nmm_mla_query_path_run(ctypes.byref(c), ALIGNED, need, None) == nmm.NMM_ERR_SHAPE
    c.rope, c.query = 64, ALIGNED + 1
    assert L.nmm_mla_query_path_run(ctypes.byref(c), ALIGNED, need, None) == nmm.NMM_ERR_ALIGN


def fake_step(chain_kv=False):
    """A decode step's argument structs over fake, disjoint 1 GiB "device" regions (validation only)."""
    c = nmm.nmm_mla_chain()
    for k, v in dict(hidden=7168, q_lora=1536, kv_lora=512, rope=64, heads=128, nope=128, v_head=128).items():
        setattr(c, k, v)
    region = iter(range(1 << 34, 1 << 40, 1 << 30))
    for k in nmm.CHAIN_BUFFERS:
        setattr(c, k, next(region))
    if chain_kv:
        c.kv_gamma, c.kv_cache = next(region), next(region)
        c.kv_eps, c.rope_theta, c.position, c.ld_cache, c.cache_rows = 1e-6, 10000.0, 4096, 576, 4097
    a = nmm.nmm_latent_attn()
    a.heads, a.seq, a.d_qk, a.d_v, a.ldq, a.ld_kv, a.ldo, a.scale, a.splits = 128, 4096, 576, 512, 576, 576, 512, 0.07, 16
    a.q, a.kv, a.out = next(region), next(region), next(region)
    return c, a


def test_decode_step_workspace_and_validation():
    c, a = fake_step()
    chain_ws = L.nmm_mla_decode_chain_workspace_size(ctypes.byref(c))
    need = L.nmm_mla_decode_step_workspace_size(ctypes.byref(c), ctypes.byref(a))
    att_ws = L.nmm_latent_attention_ex_workspace_size(128, 4096, 576, 512, 16)
    assert need == (chain_ws + 255) // 256 * 256 + att_ws and att_ws > 0
    step = lambda wsb=need: L.nmm_mla_decode_step(ctypes.byref(c), ctypes.byref(a), ALIGNED, wsb, None)
    assert L.nmm_mla_decode_step(None, ctypes.byref(a), ALIGNED, need, None) == nmm.NMM_ERR_NULL
    assert L.nmm_mla_decode_step(ctypes.byref(c), None, ALIGNED, need, None) == nmm.NMM_ERR_NULL
    assert L.nmm_mla_decode_step_workspace_size(ctypes.byref(c), None) == 0
    assert step(need - 1) == nmm.NMM_ERR_WORKSPACE
    # the attention reads what the chain writes (its q on the chain's q_f32)
    q = a.q
    a.q = c.q_f32
    assert step() == nmm.NMM_ERR_ARG
    # ... or writes what the chain reads (its output on W_O; its bf16 copy on x)
    a.q, out = q, a.out
    a.out = c.w_o + 4096
    assert step() == nmm.NMM_ERR_ARG
    a.out, a.out_bf16, a.ldob = out, c.x, 512
    assert step() == nmm.NMM_ERR_ARG
    a.out_bf16, a.ldob = None, 0
    # the attention's own limits, all before any launch
    a.out = out + 4
    assert step() == nmm.NMM_ERR_ALIGN
    a.out, a.ldq = out, 1 << 40
    assert step() == nmm.NMM_ERR_SHAPE
    a.ldq, a.d_qk = 576, 577
    assert L.nmm_mla_decode_step_workspace_size(ctypes.byref(c), ctypes.byref(a)) == 0
    assert step() == nmm.NMM_ERR_SHAPE
    a.d_qk, a.splits = 576, -1
    assert step() == nmm.NMM_ERR_ARG


def test_decode_step_refuses_attention_over_the_new_cache_row():
    c, a = fake_step(chain_kv=True)
    need = L.nmm_mla_decode_step_workspace_size(ctypes.byref(c), ctypes.byref(a))
    step = lambda: L.nmm_mla_decode_step(ctypes.byref(c), ctypes.byref(a), ALIGNED, need, None)
    a.kv = c.kv_cache                       # rows 0 .. 4095; the chain writes row 4096
    a.seq = 4097
    assert step() == nmm.NMM_ERR_ARG
    a.seq = 4096                            # stops short of the new row: independent, but this would
    assert L.nmm_mla_decode_step_workspace_size(ctypes.byref(c), ctypes.byref(a)) > 0   # launch; not run here


def test_prepared_step_refuses_invalid_sizes_before_any_launch():
    """The binding's PreparedStep queries the workspace size first: an invalid attention shape
    (d_qk not a multiple of 32) gives 0 and a ValueError, with nothing allocated or launched."""
    import torch
    dims = dict(hidden=7168, q_lora=1536, kv_lora=512, rope=64, heads=128, nope=128, v_head=128)
    t = torch.zeros(8, dtype=torch.bfloat16)
    bufs = {k: t for k in nmm.CHAIN_BUFFERS}
    attn = dict(q=torch.zeros((4, 577), dtype=torch.bfloat16), kv=torch.zeros((16, 577), dtype=torch.bfloat16),
                out=torch.zeros((4, 512)), scale=0.1, d_qk=577)
    with pytest.raises(ValueError):
        nmm.PreparedStep(dims, bufs, attn)
    a = nmm._attn_struct(dict(attn, d_qk=576, splits=12))
    assert (a.heads, a.seq, a.d_qk, a.d_v, a.ldq, a.ld_kv, a.ldo, a.splits) == (4, 16, 576, 512, 577, 577, 512, 12)
    assert not a.out_bf16 and a.ldob == 0


@pytest.mark.parametrize("M,K,N,want", [
    (1, 1536, 24576, "gemv"), (2, 1536, 24576, "mfma"), (2, 16384, 7168, "gemv"), (2, 7168, 2112, "gemv"),
    (3, 7168, 2112, "mfma"), (4, 16384, 7168, "mfma"), (1, 16384, 7168, "gemv")])
def test_auto_path_per_shape(M, K, N, want):
    # the measured crossovers: matrix cores from 3 rows, and at 2 rows where their plan has a
    # single K-slice; the choice depends on the shape alone
    code = {"gemv": nmm.NMM_PATH_GEMV, "mfma": nmm.NMM_PATH_MFMA}[want]
    assert nmm.nmm_gemv_plan(M, K, N)["path"] == code
