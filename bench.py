"""Benchmark of batched monotonic alignment search on one MI355X.

One step = one full alignment of a synthetic TTS-shaped batch already resident
in HBM: one ``mas_forward_ex`` call, i.e. one launch of the fused kernel that
clears the path, runs the forward sweep, walks the decisions back and writes
the path (workspace preallocated).  Timing follows the paper's protocol
(warm-up calls, then the mean over timed calls; Section 4).

Prints ONE JSON line.  Metric: MAS cells per second (sum over items of
t_x * t_y) for the whole batch; plus the roofline of the kernel, whose
per-launch duration is measured with HIP events on the launch stream, and the
CPU oracle timed on the host as a reported baseline.

Two extra modes serve the HBM-traffic measurement:
  --copy-probe      after the timed region, also run a few device-to-device
                    copies of a known size, so that one rocprofv3 --pmc pass
                    sees the copy kernel beside the MAS kernel;
  --pmc-summary F   (no GPU) reduce rocprofv3 counter_collection.csv files
                    (one per counter pass) into the traffic summary that
                    later bench runs read back.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, public spec
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix peak, public spec
KERNEL = "mas_kernel"  # the fused kernel one mas_forward_ex call launches
COPY_BYTES = 1 << 30  # copy-probe size (read once, written once)
COPY_REPS = 4
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "mas_kernel_tts-b64-t1024-s4096_traffic.json")
KERNEL_SOURCES = ("mas_kernels.hip", "mas_api.hip", "mas_layout.h", "mas_internal.h")


def kernel_source_hash() -> str:
    """SHA-256 over the sources of the kernel, to tell stale counters apart."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2409_07704_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def algorithmic_bytes(tx, ty, B, T, S):
    """Bytes one call must move (the HBM floor of the method), per launch.

    value read over each item's extent (4 B per cell), one decision bit per
    cell packed into 64-row words per column (8 B per 64 rows per column),
    every byte of the [B, T, S] u8 path written.  Also the smaller band-only
    read (cells that can lie on a path: t_x * (t_y - t_x + 1) per item).
    """
    import numpy as np

    tx = tx.astype(np.int64)
    ty = ty.astype(np.int64)
    ok = (tx >= 1) & (ty >= tx)
    cells = int((tx * ty).sum())
    dec = int((((tx + 63) // 64) * 8 * ty).sum())
    metric = 4 * cells + B * T * S + dec
    band = int(np.where(ok, tx * (ty - tx + 1), 0).sum())
    return cells, metric, 4 * band + B * T * S + dec


def host_description():
    """CPU model and thread counts of the host the CPU baselines ran on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def oracle_threads():
    """Threads for the all-core oracle run: the CPUs this process may use,
    at most 16 (the host share of one GPU on a shared GPU machine)."""
    return max(1, min(16, host_description()["usable_cpus"]))


def oracle_batch(value, tx, ty, threads: int):
    """The CPU oracle over the batch, items split into `threads` contiguous
    slices run concurrently (the oracle's C code runs without the GIL), as a
    batch-parallel CPU implementation runs one item per core."""
    import numpy as np

    import oracle

    B = value.shape[0]
    if threads <= 1 or B == 1:
        return oracle.mas(value, tx, ty)
    from concurrent.futures import ThreadPoolExecutor

    cuts = np.linspace(0, B, min(threads, B) + 1).astype(int)
    parts = [(a, b) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
    with ThreadPoolExecutor(len(parts)) as ex:
        outs = list(ex.map(lambda ab: oracle.mas(value[ab[0]:ab[1]], tx[ab[0]:ab[1]], ty[ab[0]:ab[1]]), parts))
    return tuple(np.concatenate([o[i] for o in outs]) for i in range(3))


def cpu_oracle_rate(value, tx, ty, budget_s: float, threads: int = 1, around=None):
    """Oracle cells/s on the host, the full batch repeated for about budget_s
    seconds.  `around`, if given, is a pair of callables run before and after
    each oracle pass inside the timed region (device copies)."""
    import numpy as np

    cells = int((tx.astype(np.int64) * ty).sum())
    reps, t = 0, 0.0
    out = None
    while reps == 0 or t < budget_s:
        t0 = time.perf_counter()
        v = around[0]() if around else value
        out = oracle_batch(v, tx, ty, threads)
        if around:
            around[1](out[0])
        t += time.perf_counter() - t0
        reps += 1
    return cells * reps / t, reps, t, out


def read_counter_csv(path):
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            rows.append((r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"]), int(r["Dispatch_Id"])))
    return rows


def pmc_summary(paths, out_path):
    """Per-launch HBM bytes of the MAS kernel from FETCH_SIZE / WRITE_SIZE.

    Each counter is in KiB per dispatch.  The copy kernel of the same run
    moved COPY_BYTES in and out per dispatch, so its counter readings give the
    scale factor that turns a counter reading into bytes.
    """
    acc = {}
    for p in paths:
        for kname, cname, val, _ in read_counter_csv(p):
            base = cname.replace("_sum", "")
            if base not in ("FETCH_SIZE", "WRITE_SIZE"):
                continue
            if KERNEL in kname:
                key = "mas"
            elif "copyBuffer" in kname or "copy" in kname.lower():
                key = "copy"
            else:
                continue
            acc.setdefault((key, base), []).append(val)
    need = [("mas", "FETCH_SIZE"), ("mas", "WRITE_SIZE"), ("copy", "FETCH_SIZE"), ("copy", "WRITE_SIZE")]
    missing = [k for k in need if k not in acc]
    if missing:
        raise SystemExit(f"pmc-summary: no readings for {missing}")
    import numpy as np

    def stats(k):
        v = np.array(acc[k])
        return float(np.median(v)), len(v)

    # Copy dispatches can include small ones (warm-up copies of other sizes):
    # the calibration uses the largest readings, one per COPY_BYTES dispatch.
    cf = sorted(acc[("copy", "FETCH_SIZE")])[-COPY_REPS:]
    cw = sorted(acc[("copy", "WRITE_SIZE")])[-COPY_REPS:]
    f_fetch = float(np.median(cf)) * 1024.0 / COPY_BYTES
    f_write = float(np.median(cw)) * 1024.0 / COPY_BYTES
    mf, nf = stats(("mas", "FETCH_SIZE"))
    mw, nw = stats(("mas", "WRITE_SIZE"))
    fetch_b = mf * 1024.0 / f_fetch
    write_b = mw * 1024.0 / f_write
    out = {
        "kernel": KERNEL,
        "workload": "tts-b64-t1024-s4096",
        "kernel_source_sha256": kernel_source_hash(),
        "fetch_kib_per_dispatch": mf,
        "write_kib_per_dispatch": mw,
        "dispatches": [nf, nw],
        "copy_bytes_per_dispatch": COPY_BYTES,
        "copy_fetch_kib": float(np.median(cf)),
        "copy_write_kib": float(np.median(cw)),
        "scale_fetch": f_fetch,
        "scale_write": f_write,
        "fetch_bytes": fetch_b,
        "write_bytes": write_b,
        "traffic_bytes_per_launch": fetch_b + write_b,
    }
    with open(out_path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out))


def load_traffic(wname):
    """Counter-derived bytes per launch, or None when absent or stale."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("workload") != wname or t.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return t


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle timing per CPU variant")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the secondary lines (path-less call, the smaller workloads)")
    ap.add_argument("--secondary-steps", type=int, default=200)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle timing (parity still checked)")
    ap.add_argument("--copy-probe", action="store_true", help="run copies of a known size after the timed region")
    ap.add_argument("--pmc-summary", nargs="+", default=None, metavar="CSV")
    ap.add_argument("--trace", default=None, metavar="OUT",
                    help="instead of timing: record the launch timeline with the debug build libmas_trace.so "
                         "(full batch with and without the path, and the last-finishing item alone) into OUT")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(args.pmc_summary, TRAFFIC_FILE)
        return
    if args.gpus != 1:
        print(f"bench.py: only the one-GPU path is built and measured; --gpus {args.gpus} is not supported "
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
    cells, bytes_metric, bytes_band = algorithmic_bytes(tx, ty, B, T, S)
    if args.trace:
        timeline(args.trace, wname, value, tx, ty)
        return

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    v = torch.from_numpy(value).to(dev)
    x = torch.from_numpy(tx).to(dev)
    y = torch.from_numpy(ty).to(dev)
    path = torch.empty((B, T, S), dtype=torch.uint8, device=dev)
    score = torch.empty(B, dtype=torch.float32, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    ws = mas.Workspace(B, T, S, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        mas.mas_forward_ex(v, x, y, path, score, status, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)

    K = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    ev[0].record(stream)
    for k in range(K):
        step()
        ev[k + 1].record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    per_launch = np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(K)]) * 1e-3  # seconds
    t_mean = float(per_launch.mean())

    if args.copy_probe:
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(COPY_REPS):
            dst.copy_(src)
        torch.cuda.synchronize(dev)
        del src, dst

    # Parity of the timed outputs against the oracle (and the CPU baselines).
    gpu_path = path.cpu().numpy()
    gpu_score = score.cpu().numpy()
    gpu_status = status.cpu().numpy()
    host = host_description()
    nthr = oracle_threads()
    if args.no_cpu:
        cpu, variants = None, None
        op, os_, ost = oracle_batch(value, tx, ty, nthr)
    else:
        rate, reps, tcpu, (op, os_, ost) = cpu_oracle_rate(value, tx, ty, args.cpu_budget, threads=nthr)
        cpu = {"value": rate, "unit": "cells/s", "cores": nthr, "kind": "oracle",
               "sample": f"full {wname} batch ({cells} cells) x {reps} reps, {tcpu:.1f} s, items split over "
                         f"{nthr} threads", **host}
        r1, reps1, t1, _ = cpu_oracle_rate(value, tx, ty, args.cpu_budget, threads=1)
        # The same all-core oracle with the copies a CPU implementation called
        # from a GPU training step makes: value device-to-host before, the
        # path host-to-device after.
        vdev = v

        def d2h():
            return vdev.cpu().numpy()

        def h2d(p):
            torch.from_numpy(p).to(dev)
            torch.cuda.synchronize(dev)

        rc, repsc, tc, _ = cpu_oracle_rate(value, tx, ty, args.cpu_budget, threads=nthr, around=(d2h, h2d))
        variants = [
            {"value": r1, "unit": "cells/s", "cores": 1, "kind": "oracle",
             "sample": f"full batch x {reps1} reps, {t1:.1f} s, one thread"},
            {"value": rc, "unit": "cells/s", "cores": nthr, "kind": "oracle+copies",
             "sample": f"full batch x {repsc} reps, {tc:.1f} s, {nthr} threads, including the value "
                       f"device-to-host copy and the path host-to-device copy"},
        ]
    parity = bool(np.array_equal(gpu_path, op) and gpu_score.tobytes() == os_.tobytes()
                  and np.array_equal(gpu_status, ost))

    secondary = None
    if not args.no_secondary:
        secondary = secondary_lines(mas, synth, dev, stream, wname, v, x, y, ws, op, tx, ty, cells,
                                    args.secondary_steps, max(3, args.warmup // 5), t_mean)
        parity = parity and all(s["parity"] for s in secondary.values())

    achieved = bytes_metric / t_mean / 1e9
    tr = load_traffic(wname)
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
                   "launch_us_mean": t_mean * 1e6,
                   "launch_us_median": float(np.median(per_launch)) * 1e6,
                   "launch_us_min": float(per_launch.min()) * 1e6,
                   "band_bytes": bytes_band,
                   "band_gbs": bytes_band / t_mean / 1e9},
        "roofline": {"bound": "hbm", "kernel": KERNEL, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": None if tr is None else tr["traffic_bytes_per_launch"],
                     "traffic_unit": "bytes/launch",
                     "algorithmic_bytes": bytes_metric},
        "cpu_baseline": cpu,
        "cpu_baseline_variants": variants,
        "secondary": secondary,
        "parity": "bit-exact" if parity else "MISMATCH",
    }
    print(json.dumps(out), flush=True)
    if not parity:
        sys.exit(1)


def timeline(out_path, wname, value, tx, ty):
    """Timeline summaries from the debug build (see paper_2409_07704_amd/trace.py)."""
    import numpy as np
    import torch

    from paper_2409_07704_amd import trace

    dev = torch.device("cuda:0")
    v, x, y = (torch.from_numpy(a).to(dev) for a in (value, tx, ty))
    parts = [f"Timeline of one launch on {wname} from the debug build (libmas_trace.so, MAS_TRACE: 100 MHz "
             f"wall-clock stamps; the product build has none).",
             f"Command: python bench.py --trace {os.path.relpath(out_path, ROOT)}"
             + (f" --workload {wname}" if wname != "tts-b64-t1024-s4096" else ""),
             f"kernel sources sha256 {kernel_source_hash()}", ""]
    lay, st = trace.run(v, x, y, with_path=True)
    s_full = trace.summary(lay, st, tx, ty, with_path=True)
    print(f"trace: full batch with path {s_full['launch_us']:.1f} us", flush=True)
    parts += [trace.format_summary(s_full, "== full batch, mas_forward_ex (dense path)"), ""]
    lay, st = trace.run(v, x, y, with_path=False)
    s_np = trace.summary(lay, st, tx, ty, with_path=False)
    print(f"trace: full batch without path {s_np['launch_us']:.1f} us", flush=True)
    parts += [trace.format_summary(s_np, "== full batch, mas_search (no dense path)"), ""]
    b = s_full["longest"][0]["b"]
    va, xa, ya = (torch.from_numpy(np.ascontiguousarray(a[b:b + 1])).to(dev) for a in (value, tx, ty))
    lay, st = trace.run(va, xa, ya, with_path=True)
    s_one = trace.summary(lay, st, tx[b:b + 1], ty[b:b + 1], with_path=True)
    print(f"trace: item {b} alone {s_one['launch_us']:.1f} us", flush=True)
    parts += [trace.format_summary(s_one, f"== item {b} alone (B=1), mas_forward_ex"), ""]
    with open(out_path, "w") as f:
        f.write("\n".join(parts))
    print("\n".join(parts), flush=True)


def time_launches(fn, stream, steps, warmup):
    """Per-launch seconds of `fn` (one library call), HIP events on `stream`."""
    import numpy as np
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record(stream)
    for k in range(steps):
        fn()
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    return np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(steps)]) * 1e-3


def secondary_lines(mas, synth, dev, stream, wname, v, x, y, ws, op, tx, ty, cells, steps, warmup, forward_s):
    """Secondary measurements reported beside the headline: the path-less call
    (mas_search: row_start, durations and score, no dense path) on the headline
    workload, and one mas_forward_ex line per smaller workload.  Each checks
    its outputs against the oracle."""
    import numpy as np
    import torch

    import oracle

    out = {}
    B, T, S = v.shape
    rs = torch.empty((B, T + 1), dtype=torch.int32, device=dev)
    du = torch.empty((B, T), dtype=torch.int32, device=dev)
    sc = torch.empty(B, dtype=torch.float32, device=dev)
    st = torch.empty(B, dtype=torch.int32, device=dev)
    pl = time_launches(lambda: mas.mas_search(v, x, y, rs, sc, st, workspace=ws, stream=stream, durations_out=du),
                       stream, steps, warmup)
    ok = bool(np.array_equal(rs.cpu().numpy(), oracle.row_start(op, tx, ty))
              and np.array_equal(du.cpu().numpy(), oracle.durations(op)))
    out["path_less"] = {"call": "mas_search", "workload": wname, "launch_us_mean": float(pl.mean()) * 1e6,
                        "launch_us_median": float(np.median(pl)) * 1e6, "cells_per_s": cells / float(pl.mean()),
                        "parity": ok}
    out["text_grid"] = text_grid_line(mas, synth, dev, stream, rs, op, tx, ty, float(pl.mean()), forward_s,
                                       steps, warmup)
    out["loglik"] = loglik_line(mas, synth, dev, stream, wname, ws, forward_s, steps, warmup, 0.2)
    out["loglik_unit_variance"] = loglik_line(mas, synth, dev, stream, wname, ws, forward_s, steps, warmup, None)
    for name in synth.WORKLOADS:
        if name == wname or name.startswith("tiny"):
            continue
        value, a, b = synth.generate(name)
        Bn, Tn, Sn = value.shape
        cn, metric, _ = algorithmic_bytes(a, b, Bn, Tn, Sn)
        vv, xx, yy = (torch.from_numpy(t).to(dev) for t in (value, a, b))
        pth = torch.empty((Bn, Tn, Sn), dtype=torch.uint8, device=dev)
        scn = torch.empty(Bn, dtype=torch.float32, device=dev)
        wsn = mas.Workspace(Bn, Tn, Sn, device=dev)
        tl = time_launches(lambda: mas.mas_forward_ex(vv, xx, yy, pth, scn, None, workspace=wsn, stream=stream),
                           stream, steps, warmup)
        o_path, o_score, _ = oracle.mas(value, a, b)
        ok = bool(np.array_equal(pth.cpu().numpy(), o_path) and scn.cpu().numpy().tobytes() == o_score.tobytes())
        t = float(tl.mean())
        out[name] = {"call": "mas_forward_ex", "launch_us_mean": t * 1e6, "launch_us_median": float(np.median(tl)) * 1e6,
                     "cells": cn, "cells_per_s": cn / t, "metric_bytes": metric, "gbs": metric / t / 1e9,
                     "frac": metric / t / 1e9 / HBM_PEAK_GBS, "parity": ok}
        del vv, pth, wsn
    return out


def text_grid_line(mas, synth, dev, stream, rs, op, tx, ty, search_s, forward_s, steps, warmup):
    """The aligned text grid on the headline workload: mas_expand_text from
    mas_search's row_start, 192 fp32 channels.  Beside it, for context, the
    dense product it replaces (torch.bmm of the 0/1 path, transposed, with the
    text features) and the two pipelines end to end."""
    import numpy as np
    import torch

    import oracle

    B, T1 = rs.shape
    T, S, C = T1 - 1, op.shape[2], synth.TEXT_CHANNELS
    h = synth.text_batch(B, T, C, seed=0)
    hd = torch.from_numpy(h).to(dev)
    grid = torch.empty((B, S, C), dtype=torch.float32, device=dev)
    tg = time_launches(lambda: mas.mas_expand_text(hd, rs, S, grid, stream=stream), stream, steps, warmup)
    ok = bool(np.array_equal(grid.cpu().numpy().view(np.uint32), oracle.expand_text(op, h).view(np.uint32)))
    t = float(tg.mean())
    valid = (tx >= 1) & (tx <= ty) & (tx <= T) & (ty <= S)
    moved = B * S * C * 4 + int(tx[valid].astype(np.int64).sum()) * C * 4 + B * (T + 1) * 4
    # The dense product, timed on a few launches (it is slow and only context).
    pt = torch.from_numpy(op).to(dev).transpose(1, 2).to(torch.float32).contiguous()
    dense = torch.empty_like(grid)
    td = time_launches(lambda: torch.bmm(pt, hd, out=dense), stream, 5, 2)
    dense_equal = bool(torch.equal(dense, grid))
    del pt, dense
    return {"call": "mas_expand_text", "channels": C, "dtype": "f32", "launch_us_mean": t * 1e6,
            "launch_us_median": float(np.median(tg)) * 1e6, "algorithmic_bytes": moved,
            "gbs": moved / t / 1e9, "frac": moved / t / 1e9 / HBM_PEAK_GBS,
            "dense_bmm_us_mean": float(td.mean()) * 1e6, "dense_bmm_equal": dense_equal,
            "search_plus_grid_us": (search_s + t) * 1e6,
            "forward_ex_plus_dense_us": (forward_s + float(td.mean())) * 1e6, "parity": ok}


def loglik_line(mas, synth, dev, stream, wname, ws, forward_s, steps, warmup, ls_scale):
    """The Gaussian log-likelihood producer on the headline workload's
    Gaussians (D = 80; log-sigmas ls_scale N(0,1), or unit variance as the
    headline values have): mas_loglik alone, then the producer and the
    alignment back to back, beside the same values formed with torch (the
    row constants plus batched fp32 products over the whole padded
    [B, T, S] grid, the usual way of writing it)."""
    import numpy as np
    import torch

    import oracle

    mu, ls, z, tx, ty = synth.gauss_inputs(wname, log_sigma_scale=ls_scale)
    B, T, D = mu.shape
    S = z.shape[1]
    dm, dz = (torch.from_numpy(a).to(dev) for a in (mu, z))
    dl = None if ls is None else torch.from_numpy(ls).to(dev)
    lsz = np.zeros_like(mu) if ls is None else ls
    dx, dy = (torch.from_numpy(a).to(dev) for a in (tx, ty))
    val = torch.full((B, T, S), float("nan"), dtype=torch.float32, device=dev)
    tl = time_launches(lambda: mas.mas_loglik(dm, dl, dz, dx, dy, val, stream=stream), stream, steps, warmup)
    path = torch.empty((B, T, S), dtype=torch.uint8, device=dev)
    sc = torch.empty(B, dtype=torch.float32, device=dev)

    def both():
        mas.mas_loglik(dm, dl, dz, dx, dy, val, stream=stream)
        mas.mas_forward_ex(val, dx, dy, path, sc, None, workspace=ws, stream=stream)

    tb = time_launches(both, stream, steps, warmup)
    # Parity: sampled band cells against the oracle (fp32-level bounds as in
    # the tests), the alignment against the oracle's on the same values.
    value = val.cpu().numpy()
    valid = (tx >= 1) & (tx <= ty)
    cells = []
    rng = np.random.default_rng(1)
    for b in np.flatnonzero(valid):
        i = rng.integers(0, tx[b], 2000)
        j = i + rng.integers(0, ty[b] - tx[b] + 1, 2000)
        cells.append(np.stack([np.full(2000, b), i, j], 1))
    cells = np.concatenate(cells)
    want = oracle.gauss_loglik(mu, ls, z, cells)
    m = mu[cells[:, 0], cells[:, 1]].astype(np.float64)
    r = np.exp(-2.0 * lsz[cells[:, 0], cells[:, 1]].astype(np.float64))
    x = z[cells[:, 0], cells[:, 2]].astype(np.float64)
    M = (0.5 * np.log(2 * np.pi) + np.abs(lsz[cells[:, 0], cells[:, 1]]) + 0.5 * m * m * r).sum(-1) \
        + (np.abs(m * r * x) + 0.5 * r * x * x).sum(-1)
    rel = np.abs(value[cells[:, 0], cells[:, 1], cells[:, 2]] - want) / (2.0 ** -24 * M)
    Kp = (2 * D + 31) // 32 * 32
    bound = 3 * Kp + D + 20 + 4.0 * float(np.abs(lsz).max())
    ok_values = bool(rel.max() <= bound and np.sqrt(np.mean(rel ** 2)) <= 4 * np.sqrt(3 * Kp))
    op, os_, _ = oracle.mas(value, tx, ty)
    ok_path = bool(np.array_equal(path.cpu().numpy(), op) and sc.cpu().numpy().tobytes() == os_.tobytes())
    # The torch formulation (context only; fp32 batched products, contiguous operands).
    dlz = torch.zeros_like(dm) if dl is None else dl
    r_t = torch.exp(-2.0 * dlz)
    c_t = (-0.5 * np.log(2 * np.pi) - dlz - 0.5 * dm * dm * r_t).sum(-1, keepdim=True)
    f1, f2 = (dm * r_t).contiguous(), (-0.5 * r_t).contiguous()
    g1, g2 = dz.transpose(1, 2).contiguous(), (dz * dz).transpose(1, 2).contiguous()
    ref = torch.empty((B, T, S), dtype=torch.float32, device=dev)

    def torch_values():
        torch.bmm(f1, g1, out=ref)
        ref.baddbmm_(f2, g2)
        ref.add_(c_t)

    tt = time_launches(torch_values, stream, 5, 2)
    del ref, f1, f2, g1, g2
    band_cells = int(sum(int(a) * (int(b2) - int(a) + 1) for a, b2 in zip(tx[valid], ty[valid])))
    moved = band_cells * 4 + int(tx[valid].astype(np.int64).sum()) * D * (4 if ls is None else 8) + B * S * D * 4
    t = float(tl.mean())
    flops = 2.0 * (D if ls is None else 2 * D) * band_cells
    return {"call": "mas_loglik", "D": D, "log_sigma": "none (unit variance)" if ls is None else f"{ls_scale} N(0,1)",
            "band_cells": band_cells,
            "launch_us_mean": t * 1e6, "launch_us_median": float(np.median(tl)) * 1e6,
            "algorithmic_bytes": moved, "gbs": moved / t / 1e9, "frac_hbm": moved / t / 1e9 / HBM_PEAK_GBS,
            "product_tflops": flops / t / 1e12,
            "mfma_frac": 3 * flops / t / 1e12 / MFMA_F16_PEAK_TFLOPS,
            "value_err_max_uM": float(rel.max()), "value_err_rms_uM": float(np.sqrt(np.mean(rel ** 2))),
            "loglik_plus_forward_ex_us": float(tb.mean()) * 1e6, "forward_ex_us": forward_s * 1e6,
            "torch_values_us_mean": float(tt.mean()) * 1e6,
            "parity": ok_values and ok_path}


if __name__ == "__main__":
    main()
