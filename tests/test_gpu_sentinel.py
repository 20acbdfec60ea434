"""GPU parity of the legacy-sentinel mode (mas_forward_sentinel) against the
CPU oracle run with the same finite sentinel, through the C ABI.

The mode is Algorithm 1 with every masked cell at a finite max_neg_val
instead of -inf (Sec. 2, issue 4: -1e9 is not small enough).  Paths, scores
and statuses must equal the oracle's bit for bit; the hand-derived case from
tests/golden/hand_cases.json checks the mode against values worked out on
paper, and a large-magnitude batch checks that the sentinel really changes
alignments the way Algorithm 1 with that sentinel does.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import _pins

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def mas():
    import paper_2409_07704_amd as m

    m.lib()  # raises when the HIP library is missing
    return m


def run_sentinel(mas, value, tx, ty, sentinel, value_dev=None, workspace=None):
    B, T, S = value.shape
    v = torch.from_numpy(np.ascontiguousarray(value)).cuda() if value_dev is None else value_dev
    x = torch.from_numpy(np.asarray(tx, np.int32)).cuda()
    y = torch.from_numpy(np.asarray(ty, np.int32)).cuda()
    path = torch.full((B, T, S), 0xA5, dtype=torch.uint8, device="cuda")
    score = torch.full((B,), 3.0, dtype=torch.float32, device="cuda")
    status = torch.full((B,), 99, dtype=torch.int32, device="cuda")
    mas.mas_forward_sentinel(v, x, y, sentinel, path, score, status, workspace=workspace)
    torch.cuda.synchronize()
    return path.cpu().numpy(), score.cpu().numpy(), status.cpu().numpy()


def assert_sentinel_parity(mas, value, tx, ty, sentinel, label, **kw):
    _say(f"{label} sentinel={sentinel:g} shape={value.shape}")
    gp, gs, gst = run_sentinel(mas, value, tx, ty, sentinel, **kw)
    op, os_, ost = oracle.mas(value, tx, ty, neg=sentinel)
    assert np.array_equal(gst, ost), f"{label}: status {gst} vs {ost}"
    bad = np.argwhere(gp != op)
    assert bad.size == 0, f"{label}: {len(bad)} path bytes differ, first at {bad[:5].tolist()}"
    assert gs.tobytes() == os_.tobytes(), f"{label}: scores differ {gs} vs {os_}"
    return gp, gs


def test_hand_case(mas):
    """The golden case worked out on paper: with -1e9 the masked predecessor
    of cell (1, 1) wins and the path steps at column 1."""
    case = next(c for c in json.load(open(GOLDEN))["cases"] if "legacy_neg" in c)
    v = np.array(case["value"], dtype=np.float32)[None]
    tx, ty = [case["t_x"]], [case["t_y"]]
    _say(f"{case['name']} sentinel={case['legacy_neg']:g}")
    gp, gs, gst = run_sentinel(mas, v, tx, ty, case["legacy_neg"])
    assert gst[0] == oracle.ITEM_OK
    assert _pins.alignment_of(gp[0], tx[0], ty[0]) == tuple(case["legacy_rows"])
    assert np.float32(gs[0]).tobytes() == np.float32(case["legacy_score"]).tobytes()


@pytest.mark.parametrize("sentinel", [-1e9, -1e32])
@pytest.mark.parametrize("name", ["iid-b4-t32-s128", "tts-b16-t128-s512", "tts-b32-t256-s1024"])
def test_workloads(mas, name, sentinel):
    """On the synthetic workloads every partial sum stays far above both
    sentinels, so the mode must also agree with the -inf results."""
    value, tx, ty = synth.generate(name)
    gp, gs = assert_sentinel_parity(mas, value, tx, ty, sentinel, name)
    ip, is_, _ = oracle.mas(value, tx, ty)
    assert np.array_equal(gp, ip) and gs.tobytes() == is_.tobytes()


def test_large_magnitudes_change_alignments(mas):
    """Values of order -5e7 drive partial sums below -1e9 within a few dozen
    columns: with -1e9 the masked diagonal predecessors win (the mismatch the
    paper reports), and the library must reproduce Algorithm 1 with that
    sentinel exactly; with -1e32 it must match the -inf results."""
    B, T, S = 8, 96, 640
    tx = np.array([96, 90, 70, 64, 40, 33, 96, 1], np.int32)
    ty = np.array([640, 600, 500, 640, 300, 250, 96, 40], np.int32)
    value, tx, ty = synth.normal_batch(B, T, S, tx, ty, seed=1234)
    value = (value * np.float32(1e7) - np.float32(5e7)).astype(np.float32)
    gp, gs = assert_sentinel_parity(mas, value, tx, ty, -1e9, "large-magnitude")
    ip, _, _ = oracle.mas(value, tx, ty)
    assert not np.array_equal(gp, ip), "the -1e9 sentinel should change some alignment here"
    gp32, gs32 = assert_sentinel_parity(mas, value, tx, ty, -1e32, "large-magnitude")
    ip32, is32, _ = oracle.mas(value, tx, ty)
    assert np.array_equal(gp32, ip32) and gs32.tobytes() == is32.tobytes()


def test_odd_shapes_and_unaligned_value(mas):
    """A shape that is no multiple of the wave or chunk sizes, through the
    16-byte and the 4-byte loaders (the second from a value pointer that is
    not 16-byte aligned)."""
    B, T, S = 5, 131, 419
    tx = np.array([131, 64, 63, 2, 100], np.int32)
    ty = np.array([419, 300, 63, 5, 101], np.int32)
    value, tx, ty = synth.normal_batch(B, T, S, tx, ty, seed=77)
    value = (value * np.float32(1e7) - np.float32(3e7)).astype(np.float32)
    gp, _ = assert_sentinel_parity(mas, value, tx, ty, -1e9, "odd-shape")
    ip, _, _ = oracle.mas(value, tx, ty)
    assert not np.array_equal(gp, ip), "the -1e9 sentinel should change some alignment here"
    flat = torch.empty(B * T * S + 1, dtype=torch.float32, device="cuda")
    flat[1:].copy_(torch.from_numpy(value.reshape(-1)).cuda())
    v = flat[1:].view(B, T, S)
    assert v.data_ptr() % 16 != 0
    assert_sentinel_parity(mas, value, tx, ty, -1e9, "odd-shape-unaligned", value_dev=v)


def test_invalid_lengths_and_mode_switches(mas):
    """Invalid items in the mode, and the same workspace alternating between
    the sentinel mode and the -inf mode."""
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    tx = tx.copy()
    ty = ty.copy()
    tx[0], ty[1], tx[2], ty[2] = 0, 0, 100, 50
    ws = mas.Workspace(*value.shape)
    for k in range(2):
        assert_sentinel_parity(mas, value, tx, ty, -1e9, f"invalid-lengths-{k}", workspace=ws)
        v = torch.from_numpy(value).cuda()
        path = mas.mas_forward_ex(v, torch.from_numpy(tx).cuda(), torch.from_numpy(ty).cuda(), workspace=ws)
        torch.cuda.synchronize()
        op, _, _ = oracle.mas(value, tx, ty)
        assert np.array_equal(path.cpu().numpy(), op)
