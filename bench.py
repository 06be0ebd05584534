#!/usr/bin/env python3
"""Benchmark: one DeepSeek-V3 MLA single-token decode step on one MI355X.

A step is one pass of the whole hot path over one token: the narrow-MatMul chain
(x[1,7168] -> down-projection [7168,2112] -> W_UQ [1536,24576] -> per-head W_UK [128 x 128x512]
-> per-head W_UV [128 x 512x128] -> W_O [16384,7168], bf16 hand-offs fused into each gather) on
stream A, concurrently with latent attention (128 heads over a 4096-position latent cache,
d_qk 576, d_v 512) on stream B -- the paper's overlap of narrow MatMul with independent
matrix-unit work, on two HIP streams.

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


def mean_gain(t_opt: float, t_base: float) -> float:
    """The paper's mean gain G = 1 - E[T_opt] / E[T_base] (Section IV-G, Evaluation)."""
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
    ws_a, ws_b = nmm.Workspace(dev), nmm.Workspace(dev)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    K, W = args.steps, args.warmup
    n_slots = W + K
    chain_ev = [[ev() for _ in range(6)] for _ in range(n_slots)]
    att_ev = [[ev(), ev()] for _ in range(n_slots)]
    chains = [nmm.PreparedChain(d, {**copies[c][0], **inter}, workspace=ws_a,
                                events=[chain_ev[s] for s in range(n_slots) if s % args.copies == c])
              for c in range(args.copies)]
    slot_of = lambda s: s // args.copies        # the slot index inside chain copy s % copies

    def attention(s, stream):
        _, q, kv = copies[s % args.copies]
        nmm.nmm_latent_attention(q, kv, att_out, step.scale, d_qk=dqk, d_v=dv, workspace=ws_b, stream=stream)

    def decode_step(s):
        # fork: stream A runs the narrow chain, stream B the latent attention; then join
        start = torch.cuda.Event()
        start.record(cap)
        sa.wait_event(start)
        sb.wait_event(start)
        chains[s % args.copies].launch(slot_of(s), stream=sa)
        att_ev[s][0].record(sb)
        attention(s, sb)
        att_ev[s][1].record(sb)
        cap.wait_stream(sa)
        cap.wait_stream(sb)

    def chain_only(s):
        chains[s % args.copies].launch(slot_of(s), stream=cap)

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

    for e in (x for pair in att_ev for x in pair):   # create the HIP events before any capture
        e.record(cap)
    # eager pass first: sizes the workspaces and gives the reference result for the graphs
    with torch.cuda.stream(cap):
        decode_step(0)
    torch.cuda.synchronize()
    y_eager, att_eager = inter["y"].clone(), att_out.clone()
    t = time.perf_counter()
    step_graphs = [capture(decode_step, s) for s in range(n_slots)]
    alone = {name: [capture(fn, s) for s in range(args.copies)]
             for name, fn in (("chain", chain_only), ("attention", attn_only), ("serial", serial))}
    log(f"[bench] captured {n_slots + 3 * args.copies} HIP graphs in {time.perf_counter() - t:.1f}s")

    # ---- warmup, then exactly K timed steps (graph replays on one stream)
    t0, t1 = ev(), ev()
    with torch.cuda.stream(cap):
        for s in range(W):
            step_graphs[s].replay()
        torch.cuda.synchronize()
        t0.record(cap)
        for s in range(W, W + K):
            step_graphs[s].replay()
        t1.record(cap)
    torch.cuda.synchronize()
    step_ms = t0.elapsed_time(t1) / K
    same = torch.equal(inter["y"], y_eager) and torch.equal(att_out, att_eager)
    assert same, "graph replays must reproduce the eager decode step bit for bit"
    names = list(cb)
    per_launch = {n: [] for n in names}
    for s in range(W, W + K):
        for i, n in enumerate(names):
            per_launch[n].append(chain_ev[s][i].elapsed_time(chain_ev[s][i + 1]))
    chain_ms_in_step = float(np.mean([chain_ev[s][0].elapsed_time(chain_ev[s][5]) for s in range(W, W + K)]))
    attn_ms_in_step = float(np.mean([att_ev[s][0].elapsed_time(att_ev[s][1]) for s in range(W, W + K)]))
    gemv_ms_total = sum(sum(v) for v in per_launch.values())
    achieved = chain_total * K / (gemv_ms_total * 1e-3) / 1e9
    log(f"[bench] step {step_ms * 1e3:.1f} us (chain {chain_ms_in_step * 1e3:.1f} us, attention "
        f"{attn_ms_in_step * 1e3:.1f} us on stream B); GEMV launches {achieved:.0f} GB/s")

    # ---- the overlap experiment: each stream alone, then both serially on one stream
    def timed(graphs):
        for s in range(len(graphs)):
            graphs[s].replay()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(cap)
        for s in range(K):
            graphs[s % len(graphs)].replay()
        b.record(cap)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    with torch.cuda.stream(cap):
        t_a = timed(alone["chain"])
        t_b = timed(alone["attention"])
        t_serial = timed(alone["serial"])
    gain = mean_gain(step_ms, t_serial)
    bound = 1.0 - max(t_a, t_b) / (t_a + t_b)
    log(f"[bench] chain alone {t_a * 1e3:.1f} us, attention alone {t_b * 1e3:.1f} us, serial "
        f"{t_serial * 1e3:.1f} us, concurrent {step_ms * 1e3:.1f} us: gain {100 * gain:.1f}% "
        f"(bound {100 * bound:.1f}%)")
    assert torch.isfinite(inter["y"]).all() and torch.isfinite(att_out).all()

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
                        "W_O[16384,7168] on stream A, concurrent latent attention 128 heads x 4096 "
                        "positions (d_qk 576, d_v 512) on stream B",
            "tokens": 1, "heads": d["heads"], "kv_len": seq, "weight_copies_rotated": args.copies,
            "bytes_per_step": chain_total + attn_total, "parallelism": "single GPU, two HIP streams",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "gemv_kernel<bf16, M tile 1> (the chain's five launches)",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": None,
        },
        "detail": {
            "chain_us": round(t_a * 1e3, 2),
            "chain_gbps": round(chain_total / (t_a * 1e-3) / 1e9, 1),
            "chain_pct_of_hbm_peak": round(100 * chain_total / (t_a * 1e-3) / 1e9 / HBM_PEAK_GBPS, 1),
            "attention_us": round(t_b * 1e3, 2),
            "serial_us": round(t_serial * 1e3, 2),
            "concurrent_us": round(step_ms * 1e3, 2),
            "overlap_gain": round(gain, 4),
            "overlap_gain_bound": round(bound, 4),
            "per_launch_us": {n: round(1e3 * float(np.mean(v)), 2) for n, v in per_launch.items()},
            "per_launch_gbps": {n: round(cb[n] / (1e-3 * float(np.mean(v))) / 1e9, 1) for n, v in per_launch.items()},
        },
    }
    if not args.no_cpu_baseline:
        log(f"[bench] timing the oracle on the host (~{args.cpu_seconds:.0f}s)")
        result["cpu_baseline"] = cpu_baseline(step, args.cpu_seconds, chain_total + attn_total)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
