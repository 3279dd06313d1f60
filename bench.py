#!/usr/bin/env python3
"""Benchmark of the ABFT-protected attention layer on one MI355X.

One step = the protected forward and backward of one attention layer at
the GPT-2 shape (B8 S1024 H768, 12 heads x 64, causal, bf16 storage, fp32
accumulation) on seeded synthetic inputs already resident in HBM, with
the workload's fault schedule: 1 to 4 extreme faults (INF, NaN, +-1e10)
in one step out of ten, spread over forward and backward GEMM outputs.

Printed (one JSON line): protected-layer TFLOP/s (useful GEMM flops only;
checksum work is overhead), the ABFT overhead against the same kernels
unprotected, the dominant kernel's roofline fraction measured with HIP
events, and the CPU oracle timed on a bounded sample on the host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def useful_flops(B, S, H, nh, causal, backward=True):
    d = H // nh
    P = S * (S + 1) // 2 if causal else S * S
    fwd = 8 * B * S * H * H + 4 * B * nh * d * P
    return fwd * (3 if backward else 1)


def stage_table(B, S, H, nh, causal, es=2):
    """Algorithmic work of each stage: (name, is_bwd, mask, kind, amount)
    with kind 'flop' (GEMM) or 'byte' (HBM-bound). Masked products count
    only the unmasked pairs."""
    d, T = H // nh, B * S
    P = S * (S + 1) // 2 if causal else S * S
    sq = B * nh * P            # unmasked score entries
    return [
        ("encode", False, 0x001, "byte", (T * H + 3 * H * H) * es + (B * S // 128 * 2 * H + 4 * T * nh) * 4),
        ("qkv", False, 0x002, "flop", 2 * T * H * 3 * H),
        ("score", False, 0x004, "flop", 2 * sq * d),
        ("softmax", False, 0x008, "byte", 2 * sq * es),
        ("context", False, 0x010, "flop", 2 * sq * d),
        ("out", False, 0x020, "flop", 2 * T * H * H),
        ("encode_dO", True, 0x001, "byte", T * H * es),
        ("dCL", True, 0x002, "flop", 2 * T * H * H),
        ("dWo", True, 0x004, "flop", 2 * T * H * H),
        ("dAP", True, 0x008, "flop", 2 * sq * d),
        ("dV", True, 0x010, "flop", 2 * sq * d),
        ("softmax_bwd", True, 0x020, "byte", 3 * sq * es),
        ("dQ", True, 0x040, "flop", 2 * sq * d),
        ("dK", True, 0x080, "flop", 2 * sq * d),
        ("dWqkv", True, 0x100, "flop", 2 * T * H * 3 * H),
        ("dX", True, 0x200, "flop", 2 * T * H * 3 * H),
    ]


def cpu_baseline(shape, seed):
    """The oracle, as it stands, on two batch elements of the workload
    (forward + backward with one injected fault); throughput in the
    metric's unit."""
    import workloads as W
    from oracle import OracleParams, forward, backward
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    sample = W.make_shape(2, shape.seq, shape.hidden, shape.heads, causal=shape.causal,
                          dtype=shape.dtype, block_rows=shape.block_rows)
    inp = W.make_inputs(sample, seed)
    faults = W.draw_faults(sample, seed + 1, 1, W.ALL_OPS, ["inf"])
    p = OracleParams(heads=sample.heads, causal=sample.causal, dtype=sample.dtype,
                     block_rows=sample.block_rows)
    t0 = time.perf_counter()
    f = forward(inp["X"], inp["Wqkv"], inp["Wo"], p, faults)
    b = backward(f, inp["dO"], p, faults)
    dt = time.perf_counter() - t0
    assert len(f["events"]) + len(b["events"]) == 1
    fl = useful_flops(2, sample.seq, sample.hidden, sample.heads, sample.causal)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"2 of {shape.batch} batch elements ({sample.name}), fwd+bwd with one "
                      f"injected fault, float64 numpy; {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stage-reps", type=int, default=20)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the protected layer has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    from paper_2410_11720_amd import abft

    key = args.config
    shape = W.CONFIGS[key]
    B, S, H, nh = shape.batch, shape.seq, shape.hidden, shape.heads
    dev = "cuda"
    torch.cuda.set_device(0)
    inp = W.make_inputs(shape, W.data_seed(key))
    tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    X, Wqkv, Wo, dO = (torch.from_numpy(inp[k]).to(dev).to(tdt) for k in ("X", "Wqkv", "Wo", "dO"))

    def make(protect):
        cfg = abft.LayerConfig(B, S, H, nh, dtype=shape.dtype, causal=shape.causal,
                               block_rows=shape.block_rows, protect=protect)
        return cfg, abft.ProtectedAttention(cfg, dev)

    cfg_p, lay_p = make(True)
    cfg_u, lay_u = make(False)
    O = torch.empty((B, S, H), dtype=tdt, device=dev)
    dX = torch.empty_like(O)
    dWqkv = torch.empty((H, 3 * H), dtype=torch.float32, device=dev)
    dWo = torch.empty((H, H), dtype=torch.float32, device=dev)

    # fault schedule: 1-4 faults in one step of every ten, prepared on device
    sched = []
    n_faulty = 0
    for k in range(args.steps):
        if k % 10 == 0:
            rng = np.random.default_rng(W.fault_seed(key, k))
            fl = W.draw_faults(shape, W.fault_seed(key, k), int(rng.integers(1, 5)), W.ALL_OPS,
                               ["inf", "nan", "+1e10", "-1e10"])
            sched.append((abft.faults_to_device(fl, dev), len(fl)))
            n_faulty += 1
        else:
            sched.append(((None, 0), 0))

    def step(lay, faults):
        lay.forward(X, Wqkv, Wo, faults, O=O)
        lay.backward(dO, X, Wqkv, Wo, faults, dX=dX, dWqkv=dWqkv, dWo=dWo)

    def timed(lay, schedule):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for f, _ in schedule:
            step(lay, f)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / len(schedule) * 1e3

    for _ in range(args.warmup):
        step(lay_p, (None, 0))
        step(lay_u, (None, 0))
    clean = [((None, 0), 0)] * args.steps
    ms = timed(lay_p, sched)                       # the workload: faults 1 step in 10
    ms_clean = timed(lay_p, clean)
    ms_unprot = timed(lay_u, clean)

    # every fault of a faulty step is detected and corrected
    f0, n0 = sched[0]
    step(lay_p, f0)
    torch.cuda.synchronize()
    rf, rb = abft.read_report(lay_p.report), abft.read_report(lay_p.report_bwd)
    corrected = rf["n_corrected"] + rb["n_corrected"]
    uncorrectable = rf["n_uncorrectable"] + rb["n_uncorrectable"]

    # per-stage kernel durations with HIP events on the launch stream
    stream = torch.cuda.current_stream()
    stages = []
    for name, is_bwd, mask, kind, amount in stage_table(B, S, H, nh, shape.causal):
        def run_once(mask=mask, is_bwd=is_bwd):
            if is_bwd:
                abft.attn_abft_backward_stages(cfg_p, dO, X, Wqkv, Wo, lay_p.workspace, dX, dWqkv,
                                               dWo, None, 0, lay_p.report_bwd, mask, stream,
                                               append=True)
            else:
                abft.attn_abft_forward_stages(cfg_p, X, Wqkv, Wo, O, lay_p.workspace, None, 0,
                                              lay_p.report, mask, stream, append=True)
        run_once()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.stage_reps):
            run_once()
        e1.record(stream)
        e1.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.stage_reps
        stages.append((name, kind, amount, us))
    # restore a consistent workspace after the stage runs
    step(lay_p, (None, 0))
    torch.cuda.synchronize()

    dom = max(stages, key=lambda s: s[3])
    name, kind, amount, us = dom
    if kind == "flop":
        achieved = amount / (us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    else:
        achieved = amount / (us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof.update({"traffic": None, "kernel": name, "avg_us": round(us, 2),
                 "algorithmic": amount, "per_launch": "one call of the stage"})

    flops = useful_flops(B, S, H, nh, shape.causal)
    value = flops / (ms * 1e-3) / 1e12
    out = {
        "metric": "protected attn-layer TFLOP/s + ABFT overhead % vs unprotected, GPT-2 shape",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if shape.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) activations, N(0,0.02^2) random-init weights)",
        "config": {"workload": f"{shape.name} fwd+bwd, faults in 1 of 10 steps",
                   "batch": B, "seq": S, "hidden": H, "heads": nh, "head_dim": H // nh,
                   "causal": shape.causal, "block_rows": shape.block_rows,
                   "parallelism": "single GPU"},
        "abft_overhead_pct": round((ms_clean - ms_unprot) / ms_unprot * 100, 2),
        "ms_per_step_protected_fault_free": round(ms_clean, 4),
        "ms_per_step_unprotected": round(ms_unprot, 4),
        "unprotected_tflops": round(flops / (ms_unprot * 1e-3) / 1e12, 3),
        "mfma_frac_layer": round(value / PEAK_BF16_TFLOPS, 4),
        "faulty_steps": n_faulty,
        "check": {"faults_injected": n0, "corrected": corrected, "uncorrectable": uncorrectable},
        "roofline": roof,
        "stages_us": {s[0]: round(s[3], 2) for s in stages},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, W.data_seed(key))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
