#!/usr/bin/env python3
"""Benchmark: one DeepSeek-V3 MLA single-token decode step on one MI355X.

A step is one pass of the whole hot path over one token: the narrow-MatMul chain
(x[1,7168] -> down-projection [7168,2112] -> W_UQ [1536,24576] -> per-head W_UK [128 x 128x512]
-> per-head W_UV [128 x 512x128] -> W_O [16384,7168], bf16 hand-offs fused into each gather) and,
concurrently, latent attention (128 heads over a 4096-position latent cache, d_qk 576, d_v 512)
-- the paper's overlap of narrow MatMul with independent matrix-unit work.  The step is one call
of nmm_mla_decode_step on one stream: attention's workgroups share W_O's launch, so the overlap
is fixed by the launch.  Steps are issued back to back (one C call each); the graph-replay form
and the earlier two-stream form (chain and attention on two streams, fork / join per step) are
timed beside it.

Inputs are seeded synthetic tensors at the model's shapes (trained weights are not available).
`--copies` weight sets (3 x 380 MB by default, > 1 GiB) are rotated step by step so that W comes
from HBM, not from the 256 MB Infinity Cache.  Every input is resident in HBM before timing.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time


ATTN_OVERLAP_SPLITS = 8


def mean_gain(t_opt: float, t_base: float) -> float:
    """The paper's mean gain G = 1 - E[T_opt] / E[T_base] (Section IV-F, Evaluation)."""
    return 1.0 - float(t_opt) / float(t_base)


METRIC = "narrow MatMul achieved HBM GB/s (% of peak) at M=1; MLA decode-chain µs"
HBM_PEAK_GBPS = 8000.0        # MI355X HBM3E peak


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def chain_bytes(d: dict) -> dict:
    """Algorithmic bytes per step: each matmul reads x (bf16) and W (bf16) once and writes y (fp32)."""
    n_down = d["q_lora"] + d["kv_lora"] + d["rope"]
    qk = d["nope"] + d["rope"]
    H = d["heads"]
    b = lambda batch, M, K, N: batch * (M * K * 2 + K * N * 2 + M * N * 4)
    steps = {
        "down": b(1, 1, d["hidden"], n_down),
        "w_uq": b(1, 1, d["q_lora"], H * qk),
        "w_uk": b(H, 1, d["nope"], d["kv_lora"]),
        "w_uv": b(H, 1, d["kv_lora"], d["v_head"]),
        "w_o": b(1, 1, H * d["v_head"], d["hidden"]),
    }
    return steps


def attention_bytes(heads, seq, dqk, dv) -> int:
    """q read once, the latent cache [seq, dqk] read once (V is a view of it), out written."""
    return heads * dqk * 2 + seq * dqk * 2 + heads * dv * 4


TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                            "gemv_kernel_bf16_m1_w_o_traffic.txt")
TRAFFIC_SOURCES = ("paper_2609_16009_amd/csrc/gemv.hip", "paper_2609_16009_amd/csrc/plan.cpp",
                   "paper_2609_16009_amd/csrc/api.cpp")


def kernel_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    root = os.path.dirname(os.path.abspath(__file__))
    for rel in TRAFFIC_SOURCES:
        with open(os.path.join(root, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def chain_traffic():
    """HBM bytes per launch of the roofline's kernel (the W_O launch), as the FETCH_SIZE and
    WRITE_SIZE counters read them (scaled by a plain copy of known size), from the stored counter
    summary -- or None when the kernel sources have changed since those counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            fields = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith(" "))
    except OSError:
        return None
    fields = {k.strip(): v.strip() for k, v in fields.items()}
    if fields.get("kernel_source_digest") != kernel_source_digest():
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def graph_time_us(torch, fn, reps: int = 20, iters: int = 5, mean: bool = False) -> float:
    """Best (or mean) of `iters` replays of one HIP graph holding `reps` calls of fn(r), timed
    with events on the replay stream; us per call."""
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for r in range(3):
            fn(r)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for r in range(reps):
                fn(r)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    with torch.cuda.stream(s):
        for _ in range(iters):
            e0.record(s)
            g.replay()
            e1.record(s)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e3 / reps)
    return sum(times) / len(times) if mean else min(times)


def crossover_sweep(nmm, torch, dev) -> dict:
    """The narrow-to-dense crossover: x[M,1536] . W_UQ[1536,24576] bf16 on both kernel families,
    M in {1,2,4,8,16,32}; W rotated over copies totalling > 1 GiB so it streams from HBM."""
    import numpy as np
    import synthetic as syn
    case = syn.uq_sweep(32)
    K, N = case.K, case.N
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    Ws = [up(case.W) for _ in range(14)]
    x = up(case.x)
    out = {}
    for M in (1, 2, 4, 8, 16, 32):
        y = torch.empty((M, N), dtype=torch.float32, device=dev)
        nbytes = M * K * 2 + K * N * 2 + M * N * 4
        row = {"bytes": nbytes, "auto": "mfma" if nmm.nmm_gemv_plan(M, K, N)["path"] == nmm.NMM_PATH_MFMA else "gemv"}
        for name, path in (("gemv", nmm.NMM_PATH_GEMV), ("mfma", nmm.NMM_PATH_MFMA)):
            ws = nmm.Workspace(dev)
            t = graph_time_us(torch, lambda r: nmm.nmm_gemv(x[:M], Ws[r % len(Ws)], y, path=path, workspace=ws))
            row[name + "_us"] = round(t, 2)
            row[name + "_gbps"] = round(nbytes / t / 1e3, 1)
        out[f"M={M}"] = row
        log(f"[bench] crossover M={M}: gemv {row['gemv_us']} us, mfma {row['mfma_us']} us, auto -> {row['auto']}")
    return out


def matmul2_section(nmm, torch, dev) -> dict:
    """The paper's MatMul 2 alone, x[1,7168] . (W^DKV | W^KR)^T [7168, 576] bf16: the plain fp32
    product, the bf16 output, and the product with its cache entry (RMSNorm, RoPE, one bf16 row
    of a 4097-row latent cache) in one launch; W rotated over copies totalling > 1 GiB."""
    import numpy as np
    import synthetic as syn
    c = syn.kv_update_case()
    K, n = c.w.shape[0], c.kv_lora + c.rope
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    nbytes = K * 2 + K * n * 2 + n * 4
    Ws = [up(c.w) for _ in range(max(2, int(1.2e9 // (K * n * 2))))]
    h, gamma = up(c.h), up(c.gamma)
    y = torch.empty((1, n), dtype=torch.float32, device=dev)
    yb = torch.empty((1, n), dtype=torch.bfloat16, device=dev)
    cache = torch.zeros((c.position + 1, n), dtype=torch.bfloat16, device=dev)
    ws = nmm.Workspace(dev)
    nw = len(Ws)
    t_plain = graph_time_us(torch, lambda r: nmm.nmm_gemv(h, Ws[r % nw], y, workspace=ws))
    t_bf16 = graph_time_us(torch, lambda r: nmm.nmm_gemv_bf16(h, Ws[r % nw], yb, workspace=ws))
    t_kv = graph_time_us(torch, lambda r: nmm.nmm_mla_kv_update(
        h, Ws[r % nw], gamma, y.view(-1), cache, kv_lora=c.kv_lora, rope=c.rope, eps=c.eps, theta=c.theta,
        position=c.position, workspace=ws))
    log(f"[bench] MatMul 2 [{K},{n}]: fp32 {t_plain:.2f} us, bf16 out {t_bf16:.2f} us, "
        f"with RMSNorm + RoPE + cache entry {t_kv:.2f} us")
    return {"bytes": nbytes, "fp32_us": round(t_plain, 2), "bf16_out_us": round(t_bf16, 2),
            "with_cache_entry_us": round(t_kv, 2), "fp32_gbps": round(nbytes / t_plain / 1e3, 1)}


def mla_step_section(nmm, torch, dev, step, copies, up, args) -> dict:
    """One MLA single-token decode step in its real dependency order (the paper's overlap): the
    query path (x . W_DQ -> W_UQ -> [q_nope . W_UK | RoPE(q_pe)]) on stream A beside MatMul 2 and
    its cache entry on stream B, then attention over the t + 1 cache rows, W_UV and W_O on A.
    W_DQ and (W_DKV | W_KR) are the column blocks of the down-projection.  Timed as HIP graph
    replays: one stream, two streams, and each branch alone."""
    import synthetic as syn
    d = step.dims
    H, ql, kvl, rp, nope = d["heads"], d["q_lora"], d["kv_lora"], d["rope"], d["nope"]
    qk = nope + rp
    seq = step.kv.shape[0]
    kvc = syn.kv_update_case()
    gamma = up(kvc.gamma)
    caches = []
    for c in range(args.copies):
        cache = torch.zeros((seq + 1, kvl + rp), dtype=torch.bfloat16, device=dev)
        cache[:seq] = copies[c][2]
        caches.append(cache)
    f32 = lambda *shape: torch.zeros(shape, dtype=torch.float32, device=dev)
    b16 = lambda *shape: torch.zeros(shape, dtype=torch.bfloat16, device=dev)
    b = dict(cq=f32(1, ql), cq_b=b16(1, ql), q=f32(1, H * qk), q_b=b16(1, H * qk), qlat=f32(H, kvl),
             query=b16(H, kvl + rp), kv=f32(kvl + rp), att=f32(H, kvl), att_b=b16(H, kvl), o=f32(H, d["v_head"]),
             o_b=b16(H, d["v_head"]), y=f32(1, d["hidden"]))
    sa, sb = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    ws_a, ws_b = nmm.Workspace(dev), nmm.Workspace(dev)

    def q_path(c, st):
        w = copies[c][0]
        nmm.nmm_gemv_bf16(w["x"].view(1, -1), w["w_down"].view(d["hidden"], -1)[:, :ql], b["cq_b"], y=b["cq"],
                          workspace=ws_a, stream=st)
        nmm.nmm_gemv_bf16(b["cq_b"], w["w_uq"].view(ql, -1), b["q_b"], y=b["q"], workspace=ws_a, stream=st)
        nmm.nmm_mla_query(b["q"], b["q_b"], w["w_uk"].view(H, nope, kvl), b["qlat"], b["query"], nope=nope, rope=rp,
                          position=seq, theta=syn.ROPE_THETA, workspace=ws_a, stream=st)

    def kv_path(c, st):
        w = copies[c][0]
        nmm.nmm_mla_kv_update(w["x"].view(1, -1), w["w_down"].view(d["hidden"], -1)[:, ql:], gamma, b["kv"],
                              caches[c], kv_lora=kvl, rope=rp, eps=syn.KV_EPS, theta=syn.ROPE_THETA, position=seq,
                              workspace=ws_b, stream=st)

    def tail(c, st):
        w = copies[c][0]
        nmm.nmm_latent_attention_bf16(b["query"], caches[c], b["att"], b["att_b"], step.scale, d_v=kvl,
                                      workspace=ws_a, stream=st)
        nmm.nmm_batched_gemv_bf16(b["att_b"].view(H, 1, kvl), w["w_uv"].view(H, kvl, -1), b["o_b"].view(H, 1, -1),
                                  y=b["o"].view(H, 1, -1), workspace=ws_a, stream=st)
        nmm.nmm_gemv(b["o_b"].view(1, -1), w["w_o"].view(H * d["v_head"], -1), b["y"], workspace=ws_a, stream=st)

    def one_stream(c):
        st = torch.cuda.current_stream()
        kv_path(c, st)
        q_path(c, st)
        tail(c, st)

    def two_streams(c):
        st = torch.cuda.current_stream()
        fork = torch.cuda.Event()
        fork.record(st)
        sb.wait_event(fork)
        kv_path(c, sb)
        q_path(c, st)
        join = torch.cuda.Event()
        join.record(sb)
        st.wait_event(join)
        tail(c, st)

    # MI355X's form: W_DQ and (W_DKV | W_KR) as one GEMV over the down-projection, the cache entry
    # on a spare workgroup of W_UQ, then the query: one stream, three launches
    down = torch.zeros((1, ql + kvl + rp), dtype=torch.float32, device=dev)
    qpaths = [nmm.PreparedQueryPath(d, dict(x=copies[c][0]["x"], w_down=copies[c][0]["w_down"],
                                            w_uq=copies[c][0]["w_uq"], w_uk=copies[c][0]["w_uk"], kv_gamma=gamma,
                                            kv_cache=caches[c], down_f32=down, cq_bf16=b["cq_b"], q_f32=b["q"],
                                            q_bf16=b["q_b"], qlat_f32=b["qlat"], query=b["query"]),
                                    eps=syn.KV_EPS, theta=syn.ROPE_THETA, position=seq, workspace=ws_a)
              for c in range(args.copies)]

    def fused(c):
        st = torch.cuda.current_stream()
        qpaths[c].launch(stream=st)
        tail(c, st)

    nc = args.copies
    out = {}
    for name, fn in (("one_stream", one_stream), ("two_streams", two_streams), ("fused_query_path", fused),
                     ("fused_query_path_only", lambda c: qpaths[c].launch(stream=torch.cuda.current_stream())),
                     ("query_path", lambda c: q_path(c, torch.cuda.current_stream())),
                     ("kv_path", lambda c: kv_path(c, torch.cuda.current_stream())),
                     ("attention_and_output", lambda c: tail(c, torch.cuda.current_stream()))):
        out[name + "_us"] = round(graph_time_us(torch, lambda r: fn(r % nc), reps=6, iters=max(3, args.steps // 20),
                                                mean=True), 2)
    out["overlap_gain"] = round(1.0 - out["two_streams_us"] / out["one_stream_us"], 4)
    log(f"[bench] MLA step in dependency order: one stream {out['one_stream_us']} us, two streams "
        f"{out['two_streams_us']} us, fused query path {out['fused_query_path_us']} us (query path "
        f"{out['query_path_us']}, MatMul 2 + entry {out['kv_path_us']}, fused both {out['fused_query_path_only_us']}, "
        f"attention + W_UV + W_O {out['attention_and_output_us']})")
    return out


def transposed_weights(nmm, torch, dev) -> dict:
    """The decode shapes with W stored transposed, Wt[N, K] (a torch Linear weight's layout), on
    nmm_gemv_nt, beside nmm_gemv on the same product with W [K, N]; M = 1, bf16, W rotated over
    copies totalling > 1 GiB."""
    import numpy as np
    import synthetic as syn
    out = {}
    for name, K, N in (("w_o", 16384, 7168), ("down", 7168, 2112), ("w_uq", 1536, 24576), ("matmul2", 7168, 576)):
        c = syn.gemv_case(900 + K % 97, 1, K, N, syn.BF16, name=name)
        up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        nw = max(2, int(1.2e9 // (K * N * 2)))
        W = up(c.W)
        Ws = [W.clone() for _ in range(nw)]
        Wts = [W.t().contiguous() for _ in range(nw)]
        x = up(c.x)
        y = torch.empty((1, N), dtype=torch.float32, device=dev)
        ws = nmm.Workspace(dev)
        t_rm = graph_time_us(torch, lambda r: nmm.nmm_gemv(x, Ws[r % nw], y, workspace=ws))
        t_nt = graph_time_us(torch, lambda r: nmm.nmm_gemv_nt(x, Wts[r % nw], y, workspace=ws))
        nbytes = K * 2 + K * N * 2 + N * 4
        out[name] = {"K": K, "N": N, "row_major_us": round(t_rm, 2), "transposed_us": round(t_nt, 2),
                     "transposed_gbps": round(nbytes / t_nt / 1e3, 1)}
        del Ws, Wts
        log(f"[bench] {name} [{K},{N}] with W as [N,K]: {t_nt:.2f} us (as [K,N]: {t_rm:.2f} us)")
    return out


def remnant_split(nmm, torch, dev) -> dict:
    """The paper's remnant split (Condition 4): for M = 16q + r, the first 16q rows on the matrix
    cores and the r remnant rows on the streaming GEMV at the same time (two streams forked and
    joined inside one HIP graph), against one matrix-core launch over all M rows.  W_UQ's shape,
    W rotated over copies totalling > 1 GiB."""
    import numpy as np
    import synthetic as syn
    case = syn.uq_sweep(32)
    K, N = case.K, case.N
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    Ws = [up(case.W) for _ in range(14)]
    x = up(case.x)
    sa, sb = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    ws_a, ws_b = nmm.Workspace(dev), nmm.Workspace(dev)
    out = {}
    for M in (17, 18, 20, 24):
        q16 = M // 16 * 16
        y = torch.empty((M, N), dtype=torch.float32, device=dev)
        t_one = graph_time_us(torch, lambda r: nmm.nmm_gemv(x[:M], Ws[r % len(Ws)], y, path=nmm.NMM_PATH_MFMA,
                                                            workspace=ws_a))

        def split(r):
            cur = torch.cuda.current_stream()
            start = torch.cuda.Event()
            start.record(cur)
            sa.wait_event(start)
            sb.wait_event(start)
            nmm.nmm_gemv(x[:q16], Ws[r % len(Ws)], y[:q16], path=nmm.NMM_PATH_MFMA, workspace=ws_a, stream=sa)
            nmm.nmm_gemv(x[q16:M], Ws[r % len(Ws)], y[q16:], path=nmm.NMM_PATH_GEMV, workspace=ws_b, stream=sb)
            cur.wait_stream(sa)
            cur.wait_stream(sb)
        t_split = graph_time_us(torch, split)
        out[f"M={M}"] = {"mfma_all_rows_us": round(t_one, 2), "split_us": round(t_split, 2),
                         "split_rows": f"{q16} on MFMA + {M - q16} on GEMV"}
        log(f"[bench] remnant split M={M}: one MFMA launch {t_one:.2f} us, "
            f"{q16} rows MFMA + {M - q16} rows GEMV concurrently {t_split:.2f} us")
    return out


def cpu_baseline(step, target_s: float, bytes_per_step: int) -> dict:
    import oracle
    threads = oracle.max_threads()
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.mla_chain(step)
        oracle.latent_attention(step.q, step.kv, step.scale)
        reps += 1
        el = time.perf_counter() - t0
        if el >= target_s or reps >= 50:
            break
    per = el / reps
    return {"value": round(bytes_per_step / per / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full decode step(s) (chain + attention) on the host, fp64, "
                      f"{per * 1e3:.1f} ms per step"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--copies", type=int, default=3, help="weight sets rotated across steps")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-crossover", action="store_true", help="skip the GEMV/MFMA crossover sweep")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch
    import paper_2609_16009_amd as nmm
    import synthetic as syn

    nmm.lib()                                   # fails loudly if the HIP library is not built
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"[bench] device: {torch.cuda.get_device_name(0)}")

    t = time.perf_counter()
    step = syn.decode_step()
    d = step.dims
    log(f"[bench] synthetic inputs generated in {time.perf_counter() - t:.1f}s")
    seq, dqk, dv = step.kv.shape[0], step.kv.shape[1], syn.ATTN_DV
    cb = chain_bytes(d)
    chain_total = sum(cb.values())
    attn_total = attention_bytes(d["heads"], seq, dqk, dv)

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    n_down = d["q_lora"] + d["kv_lora"] + d["rope"]
    qk = d["nope"] + d["rope"]
    f32 = lambda n: torch.zeros(n, dtype=torch.float32, device=dev)
    b16 = lambda n: torch.zeros(n, dtype=torch.bfloat16, device=dev)
    inter = dict(down_f32=f32(n_down), q_f32=f32(d["heads"] * qk), lat_f32=f32(d["heads"] * d["kv_lora"]),
                 o_f32=f32(d["heads"] * d["v_head"]), y=f32(d["hidden"]), cq_bf16=b16(d["q_lora"]),
                 qnope_bf16=b16(d["heads"] * d["nope"]), lat_bf16=b16(d["heads"] * d["kv_lora"]),
                 o_bf16=b16(d["heads"] * d["v_head"]))
    copies = []
    for _ in range(args.copies):
        w = dict(x=up(step.x), w_down=up(step.w_down), w_uq=up(step.w_uq), w_uk=up(step.w_uk),
                 w_uv=up(step.w_uv), w_o=up(step.w_o))
        copies.append((w, up(step.q), up(step.kv)))
    att_out = torch.zeros((d["heads"], dv), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    log(f"[bench] {args.copies} weight copies resident ({args.copies * (chain_total + attn_total) / 2**30:.2f} GiB)")

    sa, sb = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    cap = torch.cuda.Stream(device=dev)        # capture / replay stream
    ws_a, ws_b, ws_s = nmm.Workspace(dev), nmm.Workspace(dev), nmm.Workspace(dev)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    K, W = args.steps, args.warmup
    chains = [nmm.PreparedChain(d, {**copies[c][0], **inter}, workspace=ws_a) for c in range(args.copies)]

    # attention beside the chain: 12 position spans requested per head block (11 result, of 6
    # chunks each: 22 workgroups beside W_O's 224 in the decode step's shared launch).  Fewer spans
    # write fewer partial outputs into the HBM-bound launch: 77.4-77.7 us per step against
    # 78.0-78.3 with 16 spans (32 workgroups), 81.9 with 32 and 85.0 with 8, measured on one MI355X
    def attention(s, stream, splits=ATTN_OVERLAP_SPLITS):
        _, q, kv = copies[s % args.copies]
        nmm.nmm_latent_attention_ex(q, kv, att_out, step.scale, splits=splits, d_qk=dqk, d_v=dv, workspace=ws_b,
                                    stream=stream)

    # the decode step: one call, attention's workgroups in W_O's launch
    steps_one = [nmm.PreparedStep(d, {**copies[c][0], **inter},
                                  dict(q=copies[c][1], kv=copies[c][2], out=att_out, scale=step.scale,
                                       splits=ATTN_OVERLAP_SPLITS, d_qk=dqk, d_v=dv), workspace=ws_s)
                 for c in range(args.copies)]

    def one_launch(s):
        steps_one[s % args.copies].launch(stream=cap)

    def decode_step(s):
        # the two-stream form: stream A runs the narrow chain, stream B the latent attention; fork,
        # then join
        start = torch.cuda.Event()
        start.record(cap)
        sa.wait_event(start)
        sb.wait_event(start)
        chains[s % args.copies].launch(stream=sa)
        attention(s, sb)
        cap.wait_stream(sa)
        cap.wait_stream(sb)

    def chain_only(s):
        chains[s % args.copies].launch(stream=cap)

    def attn_only(s):
        attention(s, cap)

    def serial(s):
        chain_only(s)
        attn_only(s)

    def capture(fn, s):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            fn(s)
        return g

    # eager pass first: sizes the workspaces and gives the reference result for the graphs
    with torch.cuda.stream(cap):
        decode_step(0)
    torch.cuda.synchronize()
    y_eager, att_eager = inter["y"].clone(), att_out.clone()
    t = time.perf_counter()
    two_stream_graphs = [capture(decode_step, s) for s in range(args.copies)]
    one_launch_graphs = [capture(one_launch, s) for s in range(args.copies)]
    alone = {name: [capture(fn, s) for s in range(args.copies)]
             for name, fn in (("chain", chain_only), ("attention", attn_only), ("serial", serial))}
    log(f"[bench] captured {5 * args.copies} HIP graphs in {time.perf_counter() - t:.1f}s")

    def timed(graphs, n):
        """Mean time per replay of n replays (graphs rotated), events on the replay stream."""
        a, b = ev(), ev()
        with torch.cuda.stream(cap):
            a.record(cap)
            for s in range(n):
                graphs[s % len(graphs)].replay()
            b.record(cap)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    def issued(fn, n):
        """Mean time per step of n steps issued back to back on the replay stream (events on it),
        and the host's issue time per step."""
        a, b = ev(), ev()
        torch.cuda.synchronize()
        with torch.cuda.stream(cap):
            a.record(cap)
            h0 = time.perf_counter()
            for s in range(n):
                fn(s)
            h1 = time.perf_counter()
            b.record(cap)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n, (h1 - h0) / n * 1e3

    # ---- warmup, then exactly K timed decode steps (one nmm_mla_decode_step call each)
    issued(one_launch, W)
    step_ms, host_ms = issued(one_launch, K)
    assert torch.equal(inter["y"], y_eager) and torch.equal(att_out, att_eager), \
        "the one-launch decode step must reproduce the two-stream step bit for bit"
    # ---- the same step as graph replays, and the two-stream form (graph replays, and issued on
    # the two streams with a fork / join per step)
    timed(one_launch_graphs, W)
    graph_ms = timed(one_launch_graphs, K)
    timed(two_stream_graphs, W)
    two_graph_ms = timed(two_stream_graphs, K)
    assert torch.equal(inter["y"], y_eager) and torch.equal(att_out, att_eager), \
        "graph replays must reproduce the eager decode step bit for bit"
    issued(decode_step, W)
    two_eager_ms, _ = issued(decode_step, K)
    assert torch.equal(inter["y"], y_eager) and torch.equal(att_out, att_eager), \
        "two-stream steps must reproduce the first step bit for bit"
    # the step's segments from the chain's event hook (events before each launch and after the
    # merge; a separate pass, since the events add work between the launches)
    ev_slots = [[ev() for _ in range(6)] for _ in range(K)]
    steps_ev = [nmm.PreparedStep(d, {**copies[c][0], **inter},
                                 dict(q=copies[c][1], kv=copies[c][2], out=att_out, scale=step.scale,
                                      splits=ATTN_OVERLAP_SPLITS, d_qk=dqk, d_v=dv), workspace=ws_s, events=ev_slots)
                for c in range(args.copies)]
    with torch.cuda.stream(cap):
        for i in range(K):
            steps_ev[i % args.copies].launch(slot=i, stream=cap)
    torch.cuda.synchronize()
    seg = (("down", 0, 1), ("w_uq", 1, 2), ("w_uk_w_uv_pair", 2, 4), ("w_o_with_attention_and_merge", 4, 5))
    segments = {n: round(sum(ev_slots[i][a].elapsed_time(ev_slots[i][b]) for i in range(K)) / K * 1e3, 2)
                for n, a, b in seg}
    assert torch.equal(inter["y"], y_eager) and torch.equal(att_out, att_eager)
    log(f"[bench] decode step (one launch for W_O + attention): {step_ms * 1e3:.1f} us issued back to back "
        f"(host {host_ms * 1e3:.1f} us per call), {graph_ms * 1e3:.1f} us as graph replays; two streams: "
        f"{two_graph_ms * 1e3:.1f} us graph replays, {two_eager_ms * 1e3:.1f} us issued")

    # ---- the overlap experiment: each stream alone, then both serially on one stream
    timed(alone["chain"], W)
    t_a = timed(alone["chain"], K)
    timed(alone["attention"], W)
    t_b = timed(alone["attention"], K)
    att_default = [capture(lambda s: attention(s, cap, splits=0), s) for s in range(args.copies)]
    timed(att_default, W)
    t_b_default = timed(att_default, K)
    timed(alone["serial"], W)
    t_serial = timed(alone["serial"], K)
    # chain alone and chain then attention, issued like the decode step (the overlap's baseline)
    issued(chain_only, W)
    t_a_issued, _ = issued(chain_only, K)
    issued(serial, W)
    t_serial_issued, _ = issued(serial, K)
    # the chain with the cache entry behind its down-projection (RMSNorm, RoPE, one row of a
    # latent cache), timed right after the chain alone
    kvc = syn.kv_update_case()
    kv_cache = torch.zeros((seq + 1, syn.ATTN_DQK), dtype=torch.bfloat16, device=dev)
    kv_args = dict(gamma=up(kvc.gamma), cache=kv_cache, eps=kvc.eps, theta=kvc.theta, position=seq)
    chains_kv = [nmm.PreparedChain(d, {**copies[c][0], **inter}, workspace=ws_a, kv=kv_args) for c in range(args.copies)]
    with torch.cuda.stream(cap):
        chains_kv[0].launch(stream=cap)
    torch.cuda.synchronize()
    kv_graphs = [capture(lambda s: chains_kv[s % args.copies].launch(stream=cap), s) for s in range(args.copies)]
    timed(kv_graphs, W)
    t_a_kv = timed(kv_graphs, K)
    log(f"[bench] chain with the cache entry {t_a_kv * 1e3:.1f} us (without: {t_a * 1e3:.1f} us)")
    gain = mean_gain(step_ms, t_serial_issued)
    bound = 1.0 - max(t_a, t_b) / (t_a + t_b)
    log(f"[bench] chain alone {t_a * 1e3:.1f} us (issued {t_a_issued * 1e3:.1f} us), attention alone "
        f"{t_b * 1e3:.1f} us, serial {t_serial * 1e3:.1f} us (issued {t_serial_issued * 1e3:.1f} us), decode step "
        f"{step_ms * 1e3:.1f} us: gain {100 * gain:.1f}% (bound {100 * bound:.1f}%)")
    assert torch.isfinite(inter["y"]).all() and torch.isfinite(att_out).all()

    # ---- each MatMul of the chain alone (same shapes and plans, its own graph)
    H = d["heads"]
    shapes = {
        "down": lambda c, y: nmm.nmm_gemv(c["x"].view(1, -1), c["w_down"].view(d["hidden"], -1), y.view(1, -1), workspace=ws_a),
        "w_uq": lambda c, y: nmm.nmm_gemv(inter["cq_bf16"].view(1, -1), c["w_uq"].view(d["q_lora"], -1), y.view(1, -1), workspace=ws_a),
        "w_uk": lambda c, y: nmm.nmm_batched_gemv(inter["qnope_bf16"].view(H, 1, -1), c["w_uk"].view(H, d["nope"], -1),
                                                  y.view(H, 1, -1), workspace=ws_a),
        "w_uv": lambda c, y: nmm.nmm_batched_gemv(inter["lat_bf16"].view(H, 1, -1), c["w_uv"].view(H, d["kv_lora"], -1),
                                                  y.view(H, 1, -1), workspace=ws_a),
        "w_o": lambda c, y: nmm.nmm_gemv(inter["o_bf16"].view(1, -1), c["w_o"].view(H * d["v_head"], -1), y.view(1, -1), workspace=ws_a),
    }
    outs = {"down": torch.empty(n_down, device=dev), "w_uq": torch.empty(H * qk, device=dev),
            "w_uk": torch.empty(H * d["kv_lora"], device=dev), "w_uv": torch.empty(H * d["v_head"], device=dev),
            "w_o": torch.empty(d["hidden"], device=dev)}
    per_matmul = {}
    for name, fn in shapes.items():
        per_matmul[name] = graph_time_us(torch, lambda r: fn(copies[r % args.copies][0], outs[name]))
    log("[bench] each MatMul alone: " + ", ".join(f"{n} {t:.1f} us" for n, t in per_matmul.items()))
    # the roofline's kernel: the W_O launch, the chain's largest (mean over K launches)
    wo_us = graph_time_us(torch, lambda r: shapes["w_o"](copies[r % args.copies][0], outs["w_o"]),
                          reps=20, iters=max(1, K // 20), mean=True)
    wo_plan = nmm.nmm_gemv_plan(1, H * d["v_head"], d["hidden"])

    # ---- the practical read ceiling: the GEMV's load instruction streaming 2 GiB
    probe_buf = torch.empty(2 << 30, dtype=torch.uint8, device=dev)
    probe_out = torch.empty(4096, dtype=torch.int32, device=dev)
    probe = {}
    for unroll, grid in ((8, 256), (4, 512), (2, 1024), (1, 2048)):
        t_us = graph_time_us(torch, lambda r: nmm.nmm_read_probe(probe_buf, probe_out, grid, unroll), reps=5, iters=3)
        probe[f"U{unroll}x{grid}"] = round(probe_buf.numel() / t_us / 1e3, 1)
    read_ceiling = max(probe.values())
    log(f"[bench] read-probe ceiling {read_ceiling:.0f} GB/s ({probe})")
    # a plain device copy of known size: the calibration point for the HBM byte counters
    half = probe_buf.numel() // 2
    copy_us = graph_time_us(torch, lambda r: probe_buf[half:].copy_(probe_buf[:half]), reps=5, iters=3)
    copy_gbps = 2 * half / copy_us / 1e3
    del probe_buf
    log(f"[bench] device copy of {half >> 20} MiB: {copy_gbps:.0f} GB/s (read + write)")
    achieved = cb["w_o"] / (wo_us * 1e-6) / 1e9
    chain_gbps = chain_total / (t_a * 1e-3) / 1e9

    matmul2 = matmul2_section(nmm, torch, dev)
    mla_step = mla_step_section(nmm, torch, dev, step, copies, up, args)

    crossover = None if args.no_crossover else crossover_sweep(nmm, torch, dev)
    split = None if args.no_crossover else remnant_split(nmm, torch, dev)
    nt = None if args.no_crossover else transposed_weights(nmm, torch, dev)

    value = (chain_total + attn_total) / (step_ms * 1e-3) / 1e9
    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(step_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 operands, fp32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": "DeepSeek-V3 MLA single-token decode step: narrow chain x[1,7168] . "
                        "down[7168,2112] . W_UQ[1536,24576] . 128 x W_UK[128,512] . 128 x W_UV[512,128] . "
                        "W_O[16384,7168], with latent attention 128 heads x 4096 positions (d_qk 576, "
                        "d_v 512) beside W_O in one launch (nmm_mla_decode_step, one stream, steps issued "
                        "back to back)",
            "tokens": 1, "heads": d["heads"], "kv_len": seq, "weight_copies_rotated": args.copies,
            "bytes_per_step": chain_total + attn_total, "parallelism": "single GPU, one HIP stream",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": f"gemv_kernel<bf16, 1-row tile, {wo_plan['unroll']} row-steps in flight>: the W_O launch "
                      "x[1,16384].W[16384,7168], the decode chain's largest kernel (mean over "
                      f"{20 * max(1, K // 20)} launches timed on their stream)",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "algorithmic_bytes_per_launch": cb["w_o"],
            "avg_launch_us": round(wo_us, 3),
            "traffic": chain_traffic(),
        },
        "detail": {
            "chain_us": round(t_a * 1e3, 2),
            "chain_gbps": round(chain_gbps, 1),
            "chain_frac_of_peak": round(chain_gbps / HBM_PEAK_GBPS, 4),
            "chain_roofline_us_at_peak": round(chain_total / (HBM_PEAK_GBPS * 1e3), 2),
            "attention_us": round(t_b * 1e3, 2),
            "attention_splits": ATTN_OVERLAP_SPLITS,
            "attention_default_partition_us": round(t_b_default * 1e3, 2),
            "serial_us": round(t_serial * 1e3, 2),
            "chain_issued_us": round(t_a_issued * 1e3, 2),
            "serial_issued_us": round(t_serial_issued * 1e3, 2),
            "concurrent_us": round(step_ms * 1e3, 2),
            "decode_step_host_us_per_call": round(host_ms * 1e3, 2),
            "decode_step_graph_us": round(graph_ms * 1e3, 2),
            "decode_step_segments_with_events_us": segments,
            "two_streams_graph_us": round(two_graph_ms * 1e3, 2),
            "two_streams_issued_us": round(two_eager_ms * 1e3, 2),
            "overlap_gain": round(gain, 4),
            "overlap_gain_bound": round(bound, 4),
            "per_matmul_us": {n: round(t, 2) for n, t in per_matmul.items()},
            "chain_with_cache_entry_us": round(t_a_kv * 1e3, 2),
            "matmul2": matmul2,
            "mla_step_dependency_order": mla_step,
            "per_matmul_gbps": {n: round(cb[n] / t / 1e3, 1) for n, t in per_matmul.items()},
            "hbm_read_probe_gbps": probe,
            "hbm_copy_gbps": round(copy_gbps, 1),
            "w_o_frac_of_read_probe": round(achieved / read_ceiling, 4),
            "chain_frac_of_read_probe": round(chain_gbps / read_ceiling, 4),
        },
    }
    if crossover is not None:
        result["detail"]["crossover"] = crossover
        result["detail"]["remnant_split"] = split
        result["detail"]["transposed_weights"] = nt
    if not args.no_cpu_baseline:
        log(f"[bench] timing the oracle on the host (~{args.cpu_seconds:.0f}s)")
        result["cpu_baseline"] = cpu_baseline(step, args.cpu_seconds, chain_total + attn_total)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
