"""Benchmark of batched monotonic alignment search on one MI355X.

One step = one full alignment of a synthetic TTS-shaped batch already resident
in HBM: the forward sweep with backtrack (mas_search) and the dense path
writer (mas_expand_path) — the two launches mas_forward_ex makes.  Timing
follows the paper's protocol (warm-up steps, then the mean over timed steps).

Prints ONE JSON line.  Metric: MAS cells per second (sum over items of
t_x * t_y) for the whole batch; plus the roofline of the dominant kernel,
measured with HIP events on the launch stream, and the CPU oracle timed on
the host's cores as a reported baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, public spec


def algorithmic_bytes(tx, ty, B, T, S):
    """Bytes one step must move, per kernel (the HBM floor of the method).

    search: value read over each item's extent (4 B/cell), one decision bit
    per cell packed into 64-row words per column (8 B per 64 rows per column),
    the row_start table written (4 B per entry).
    path:   every byte of the [B, T, S] u8 path written, row_start read.
    """
    import numpy as np

    tx = tx.astype(np.int64)
    ty = ty.astype(np.int64)
    cells = int((tx * ty).sum())
    dec = int((((tx + 63) // 64) * 8 * ty).sum())
    rs = 4 * B * (T + 1)
    search = 4 * cells + dec + rs
    path = B * T * S + rs
    metric = 4 * cells + B * T * S + dec
    return cells, search, path, metric


def cpu_oracle_rate(value, tx, ty, budget_s: float):
    """Oracle cells/s on the host (single thread), full batch repeated."""
    import numpy as np

    import oracle

    cells = int((tx.astype(np.int64) * ty).sum())
    reps, t = 0, 0.0
    out = None
    while reps == 0 or t < budget_s:
        t0 = time.perf_counter()
        out = oracle.mas(value, tx, ty)
        t += time.perf_counter() - t0
        reps += 1
    return cells * reps / t, reps, t, out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle timing")
    ap.add_argument("--no-cpu", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU; --gpus {args.gpus} is not supported "
              "(items are independent, so more GPUs would each run their own share of the batch)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2409_07704_amd as mas
    import synth

    wname = args.workload or synth.BENCH_WORKLOAD
    value, tx, ty = synth.generate(wname)
    B, T, S = value.shape
    cells, bytes_search, bytes_path, bytes_metric = algorithmic_bytes(tx, ty, B, T, S)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    v = torch.from_numpy(value).to(dev)
    x = torch.from_numpy(tx).to(dev)
    y = torch.from_numpy(ty).to(dev)
    path = torch.empty((B, T, S), dtype=torch.uint8, device=dev)
    rs = torch.empty((B, T + 1), dtype=torch.int32, device=dev)
    score = torch.empty(B, dtype=torch.float32, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    ws = mas.Workspace(B, T, S, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        mas.mas_search(v, x, y, rs, score, status, workspace=ws, stream=stream)
        mas.mas_expand_path(rs, S, path, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for k in range(K):
        ev[k][0].record(stream)
        mas.mas_search(v, x, y, rs, score, status, workspace=ws, stream=stream)
        ev[k][1].record(stream)
        mas.mas_expand_path(rs, S, path, stream=stream)
        ev[k][2].record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0

    t_search = float(np.mean([ev[k][0].elapsed_time(ev[k][1]) for k in range(K)])) * 1e-3
    t_path = float(np.mean([ev[k][1].elapsed_time(ev[k][2]) for k in range(K)])) * 1e-3
    t_step_ev = float(np.mean([ev[k][0].elapsed_time(ev[k][2]) for k in range(K)])) * 1e-3

    # Parity of the timed outputs against the oracle (and the CPU baseline).
    gpu_path = path.cpu().numpy()
    gpu_score = score.cpu().numpy()
    if args.no_cpu:
        cpu = None
        _, _, _, (op, os_, _) = cpu_oracle_rate(value, tx, ty, 0.0)
    else:
        rate, reps, tcpu, (op, os_, _) = cpu_oracle_rate(value, tx, ty, args.cpu_budget)
        cpu = {"value": rate, "unit": "cells/s", "cores": 1, "kind": "oracle",
               "sample": f"full {wname} batch ({cells} cells) x {reps} reps, {tcpu:.1f} s, single thread"}
    parity = bool(np.array_equal(gpu_path, op) and gpu_score.tobytes() == os_.tobytes())

    if t_search >= t_path:
        dom, t_dom, b_dom = "mas_search_kernel", t_search, bytes_search
    else:
        dom, t_dom, b_dom = "mas_path_kernel16", t_path, bytes_path
    achieved = b_dom / t_dom / 1e9
    out = {
        "metric": "MAS cells/s (sum t_x*t_y per second), 1 GPU",
        "value": cells * K / wall,
        "unit": "cells/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": wall / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wname, "B": B, "T": T, "S": S, "cells": cells,
                   "metric_bytes": bytes_metric,
                   "metric_gbs": bytes_metric / (wall / K) / 1e9,
                   "metric_frac_of_hbm_peak": bytes_metric / (wall / K) / 1e9 / HBM_PEAK_GBS,
                   "search_us": t_search * 1e6, "path_us": t_path * 1e6, "step_us_events": t_step_ev * 1e6},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes": b_dom},
        "cpu_baseline": cpu,
        "parity": "bit-exact" if parity else "MISMATCH",
    }
    print(json.dumps(out), flush=True)
    if not parity:
        sys.exit(1)


if __name__ == "__main__":
    main()
