"""The timeline decoder (paper_2409_07704_amd.trace) on hand-made stamps.

The debug build's stamps are decoded on the host; these tests fix what each
slot means (sweep slot k: chunk 8k+7 done; walk slot k: chunks >= 32k
walked; per-item milestones; window issue/staged pairs) by building a stamp
buffer whose figures are known and checking the summary against them.
"""
import numpy as np
import pytest

from paper_2409_07704_amd import trace

TICK = 100  # stamp ticks per microsecond (100 MHz)


def fake_launch():
    """One item, t_x = 126 (two sweep waves), t_y = 2048 (64 chunks)."""
    B, T, S = 1, 126, 2048
    lay = trace.layout(B, T, S, with_path=True)
    st = np.zeros(lay["total"], dtype=np.int64)
    t0 = 1000
    wg = st[lay["wg"]:lay["chunk"]].reshape(lay["grid"], 2)
    wg[:, 0] = t0 + np.arange(lay["grid"])          # first start: t0
    wg[:, 1] = t0 + 30000 - np.arange(lay["grid"])  # last end: t0 + 300 us
    chunk = st[lay["chunk"]:lay["walk"]].reshape(B, lay["NW"], 64)
    for g in range(2):
        for k in range(8):  # chunk 8k+7 done at 1 us per chunk, wave g 0.5 us behind wave g-1
            chunk[0, g, k] = t0 + TICK * (8 * k + 7) + 50 * g
    walk = st[lay["walk"]:lay["item"]].reshape(B, 64)
    walk[0, 1] = 20000                # chunks >= 32 walked
    walk[0, 0] = 20000 + 32 * 12      # chunks >= 0 walked: 0.12 us per chunk
    item = st[lay["item"]:lay["tile"]].reshape(B, 8)
    item[0, :5] = [19000, 19100, 21000, 21200, 300]  # windows ready, walk start/end, published, ticks waited
    tile = st[lay["tile"]:lay["win"]].reshape(B * lay["ntile"], 2)
    tile[:, 0] = 21300 + 10 * np.arange(lay["ntile"])
    tile[:, 1] = tile[:, 0] + 200
    win = st[lay["win"]:lay["total"]].reshape(B, 4, 2, 64)
    for k in range(4):
        win[0, k, 0, :8] = 19000 + 10 * np.arange(8)  # issued
        win[0, k, 1, :8] = win[0, k, 0, :8] + 250     # staged 2.5 us later
    return lay, st, np.array([T], np.int32), np.array([S], np.int32), t0


def test_layout_offsets():
    lay = trace.layout(1, 126, 2048, with_path=True)
    assert (lay["NW"], lay["NB"], lay["NC"], lay["ntile"]) == (2, 1, 64, 4)
    assert lay["grid"] == 1 + 4  # one sweep workgroup, min(B * ntile, 192) path writers
    assert lay["chunk"] == 2 * lay["grid"]
    assert lay["walk"] == lay["chunk"] + 1 * 2 * 64
    assert lay["total"] == lay["win"] + 1 * 4 * 2 * 64
    assert trace.layout(1, 126, 2048, with_path=False)["grid"] == 1


def test_summary_figures():
    lay, st, tx, ty, t0 = fake_launch()
    s = trace.summary(lay, st, tx, ty, with_path=True)
    assert s["launch_us"] == pytest.approx(300.0)
    (r,) = s["items"]
    assert (r["t_x"], r["t_y"], r["waves"], r["chunks"]) == (126, 2048, 2, 64)
    assert r["step_us_median"] == pytest.approx(1.0)
    assert r["hand_lag_us_median"] == pytest.approx(0.5)
    assert r["sweep_end_us"] == pytest.approx((TICK * 63 + 50) / TICK)
    assert r["walk_us_per_chunk"] == pytest.approx(0.12)
    assert r["walk_waited_us"] == pytest.approx(3.0)
    assert r["windows_ready_us"] == pytest.approx((19000 - t0) / TICK)
    assert r["walk_us"] == pytest.approx((21000 - 19100) / TICK)
    assert r["published_us"] == pytest.approx((21200 - t0) / TICK)
    assert r["win_lat_us_median"] == pytest.approx(2.5) and r["windows"] == 32
    assert s["path_first_tile_us"] == pytest.approx((21300 - t0) / TICK)
    assert s["path_tail_us"] == pytest.approx((21300 + 10 * 3 + 200 - 21200) / TICK)  # last of 4 tiles
    text = trace.format_summary(s, "fake")
    assert "0.120" in text and "1.000" in text


def test_invalid_items_are_skipped():
    lay, st, tx, ty, _ = fake_launch()
    s = trace.summary(lay, st, np.array([0], np.int32), ty, with_path=False)
    assert s["items"] == []
