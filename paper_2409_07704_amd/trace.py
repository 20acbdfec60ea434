"""Timeline of one launch, from the debug build libmas_trace.so.

That build (MAS_TRACE) is the same kernel with 100 MHz wall-clock stamps at
every wave's milestones: each sweep wave after every eighth 32-column chunk,
the walker after every 32nd chunk, the item's walk start/end and row_start
publication, each path tile's start/end, each workgroup's start/end (layout:
TraceLayout in csrc/mas_internal.h).  The product library libmas.so carries
none of it.

run() times nothing itself: it runs a few warm-up calls, then one traced
mas_forward_ex (or mas_search) call, and returns the stamps; summary() turns
them into the per-item and per-chunk figures used to find where a launch's
time goes.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

from . import _native

_PKG = os.path.dirname(os.path.abspath(__file__))
TRACE_LIB_PATH = os.path.join(_PKG, "libmas_trace.so")
TICK_US = 0.01  # s_memrealtime runs at 100 MHz

ROWS_PER_WAVE, WAVES_PER_BLOCK, CHUNK, PATH_TILE_ROWS, PATH_WORKGROUPS = 63, 4, 32, 32, 192

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(TRACE_LIB_PATH):
            raise RuntimeError(f"{TRACE_LIB_PATH} is missing: build it with paper_2409_07704_amd/build.py")
        L = ctypes.CDLL(TRACE_LIB_PATH)
        for name, (args, res) in _native.SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes, fn.restype = args, res
        L.mas_trace_set.argtypes, L.mas_trace_set.restype = [ctypes.c_void_p], ctypes.c_int
        _lib = L
    return _lib


def layout(B, T, S, with_path: bool):
    """Index ranges of the stamp buffer (the same arithmetic as TraceLayout)."""
    NW = (T + ROWS_PER_WAVE - 1) // ROWS_PER_WAVE
    NB = (NW + WAVES_PER_BLOCK - 1) // WAVES_PER_BLOCK
    NC = (S + CHUNK - 1) // CHUNK
    ntile = (T + PATH_TILE_ROWS - 1) // PATH_TILE_ROWS
    grid = B * NB + (min(B * ntile, PATH_WORKGROUPS) if with_path else 0)
    t = {"wg": 0}
    t["chunk"] = t["wg"] + 2 * grid
    t["walk"] = t["chunk"] + B * NW * 64
    t["item"] = t["walk"] + B * 64
    t["tile"] = t["item"] + 8 * B
    t["win"] = t["tile"] + 2 * B * ntile
    t["total"] = t["win"] + B * 4 * 2 * 64
    return dict(NW=NW, NB=NB, NC=NC, ntile=ntile, grid=grid, **t)


def run(value, t_x, t_y, with_path: bool = True, warmup: int = 5):
    """Stamps of one traced launch on the current device: (layout, int64 array)."""
    L = lib()
    B, T, S = value.shape
    lay = layout(B, T, S, with_path)
    buf = torch.zeros(lay["total"], dtype=torch.int64, device=value.device)
    n = L.mas_workspace_bytes(B, T, S)
    wbuf = torch.empty(n + 256, dtype=torch.uint8, device=value.device)
    ws = wbuf.data_ptr() + (-wbuf.data_ptr()) % 256
    stream = torch.cuda.current_stream(value.device).cuda_stream
    assert L.mas_workspace_init(ws, n, stream) == 0
    path = torch.empty((B, T, S), dtype=torch.uint8, device=value.device)
    rs = torch.empty((B, T + 1), dtype=torch.int32, device=value.device)

    def call():
        if with_path:
            rc = L.mas_forward_ex(value.data_ptr(), t_x.data_ptr(), t_y.data_ptr(), path.data_ptr(), B, T, S,
                                  None, None, ws, n, stream)
        else:
            rc = L.mas_search(value.data_ptr(), t_x.data_ptr(), t_y.data_ptr(), B, T, S, rs.data_ptr(), None, None,
                              None, ws, n, stream)
        assert rc == 0, rc

    assert L.mas_trace_set(None) == 0
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    assert L.mas_trace_set(buf.data_ptr()) == 0
    call()
    torch.cuda.synchronize()
    assert L.mas_trace_set(None) == 0
    return lay, buf.cpu().numpy()


def _rel(a, t0):
    return (a.astype(np.int64) - t0) * TICK_US


def summary(lay, st, t_x, t_y, with_path: bool = True, top: int = 3):
    """Per-item and per-chunk figures of one traced launch (times in us from
    the first workgroup's start)."""
    B = len(t_x)
    grid, NW, NC, ntile = lay["grid"], lay["NW"], lay["NC"], lay["ntile"]
    wg = st[lay["wg"]:lay["chunk"]].reshape(grid, 2)
    t0 = int(wg[:, 0][wg[:, 0] > 0].min())
    chunk = st[lay["chunk"]:lay["walk"]].reshape(B, NW, 64)  # slot k: chunk 8k+7 (or the wave's last) done
    walk = st[lay["walk"]:lay["item"]].reshape(B, 64)         # slot k: chunks >= 32k walked
    item = st[lay["item"]:lay["tile"]].reshape(B, 8)
    tile = st[lay["tile"]:lay["win"]].reshape(B * ntile, 2)
    win = st[lay["win"]:lay["total"]].reshape(B, 4, 2, 64)  # loader k, issue/staged, n-th window
    out = {"launch_us": float(_rel(wg[:, 1].max(), t0))}
    items = []
    for b in range(B):
        tx, ty = int(t_x[b]), int(t_y[b])
        if not (1 <= tx <= ty):
            continue
        g_last = (tx - 1) // ROWS_PER_WAVE
        C = (ty + CHUNK - 1) // CHUNK
        cs = chunk[b, :g_last + 1].astype(np.int64)
        seen = cs > 0
        sweep_end = float(_rel(cs[seen].max(), t0)) if seen.any() else float("nan")
        # per-chunk step and hand-off lag from the full 8-chunk groups (a
        # wave's last group may be partial)
        full = seen.copy()
        for g in range(g_last + 1):
            ks = np.flatnonzero(seen[g])
            if len(ks):
                full[g, ks[-1]] = False
        steps, lags = [], []
        for g in range(g_last + 1):
            ks = np.flatnonzero(full[g])
            ks = ks[np.isin(ks + 1, ks)]
            steps += list((cs[g][ks + 1] - cs[g][ks]) * TICK_US / 8.0)
            if g > 0:
                both = full[g] & full[g - 1]
                lags += list((cs[g][both] - cs[g - 1][both]) * TICK_US)
        steps = np.array(steps) if steps else np.array([0.0])
        wk = walk[b].astype(np.int64)
        ks = [kk for kk in range((C - 1) // 32) if wk[kk] > 0 and wk[kk + 1] > 0]
        wk_chunk = float(np.median([(wk[kk] - wk[kk + 1]) * TICK_US / 32.0 for kk in ks])) if ks else 0.0
        rec = {"b": b, "t_x": tx, "t_y": ty, "waves": g_last + 1, "chunks": C,
               "sweep_end_us": sweep_end,
               "windows_ready_us": float(_rel(item[b, 0], t0)), "walk_start_us": float(_rel(item[b, 1], t0)),
               "walk_end_us": float(_rel(item[b, 2], t0)), "published_us": float(_rel(item[b, 3], t0)),
               "hand_lag_us_median": float(np.median(lags)) if lags else 0.0,
               "step_us_median": float(np.median(steps)), "step_us_p90": float(np.percentile(steps, 90)),
               "walk_us_per_chunk": wk_chunk, "walk_waited_us": float(item[b, 4]) * TICK_US}
        # window staging: latency of each window (issue to staged) and how
        # long before the walk start the first ones were staged
        w_iss, w_rdy = win[b, :, 0, :].astype(np.int64), win[b, :, 1, :].astype(np.int64)
        ok = (w_iss > 0) & (w_rdy > 0)
        lat = (w_rdy[ok] - w_iss[ok]) * TICK_US
        rec["win_lat_us_median"] = float(np.median(lat)) if lat.size else 0.0
        rec["win_lat_us_p90"] = float(np.percentile(lat, 90)) if lat.size else 0.0
        rec["windows"] = int(ok.sum())
        rec["walk_us"] = rec["walk_end_us"] - rec["walk_start_us"]
        items.append(rec)
    items.sort(key=lambda r: -r["published_us"])
    out["items"] = items
    out["longest"] = items[:top]
    if with_path:
        te = tile[:, 1][tile[:, 1] > 0]
        ts = tile[:, 0][tile[:, 0] > 0]
        out["path_first_tile_us"] = float(_rel(ts.min(), t0)) if len(ts) else float("nan")
        out["path_last_tile_end_us"] = float(_rel(te.max(), t0)) if len(te) else float("nan")
        out["last_publish_us"] = max(r["published_us"] for r in items)
        out["path_tail_us"] = out["path_last_tile_end_us"] - out["last_publish_us"]
    return out


def format_summary(s, title: str) -> str:
    lines = [title, f"launch (first workgroup start to last workgroup end): {s['launch_us']:.1f} us"]
    if "path_tail_us" in s:
        lines.append(f"path: first tile starts {s['path_first_tile_us']:.1f} us, last tile ends "
                     f"{s['path_last_tile_end_us']:.1f} us; last row_start published {s['last_publish_us']:.1f} us; "
                     f"path tail {s['path_tail_us']:.1f} us")
    lines.append("items finishing last (times from the first workgroup's start, us):")
    lines.append("   b   t_x   t_y waves chunks  sweep_end  win_ready walk_start  walk_end  published  walk_us "
                 "walk/chunk  step_med  step_p90  hand_lag  win_wait win_lat win_lat90")
    for r in s["longest"]:
        lines.append(f"{r['b']:4d} {r['t_x']:5d} {r['t_y']:5d} {r['waves']:5d} {r['chunks']:6d} {r['sweep_end_us']:10.1f} "
                     f"{r['windows_ready_us']:10.1f} {r['walk_start_us']:10.1f} {r['walk_end_us']:9.1f} "
                     f"{r['published_us']:10.1f} {r['walk_us']:8.1f} {r['walk_us_per_chunk']:10.3f} "
                     f"{r['step_us_median']:9.3f} {r['step_us_p90']:9.3f} {r['hand_lag_us_median']:9.2f} {r['walk_waited_us']:9.1f}"
                     f" {r['win_lat_us_median']:7.2f} {r['win_lat_us_p90']:9.2f}")
    lats = [r["win_lat_us_median"] for r in s["items"] if r["windows"]]
    if lats:
        lines.append(f"walk windows (issue to staged): median over items of the per-item median {np.median(lats):.2f} us")
    allsteps = np.array([r["step_us_median"] for r in s["items"]])
    lines.append(f"median per-chunk sweep step over all items: {np.median(allsteps):.3f} us; "
                 f"median walk per chunk: {np.median([r['walk_us_per_chunk'] for r in s['items']]):.3f} us")
    return "\n".join(lines)
