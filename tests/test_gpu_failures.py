"""Failure handling of libmas on the GPU, through the C ABI.

Every kernel in these tests still ends normally: the conditions are set from
the host (an uninitialised workspace; a tiny bound on the device-side waits
through the MAS_WAIT_BOUND diagnostic), never by a fault or a hang.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def mas():
    import paper_2409_07704_amd as m

    m.lib()  # raises when the HIP library is missing
    return m


def _inputs(name):
    value, tx, ty = synth.generate(name)
    return value, tx, ty, torch.from_numpy(value).cuda(), torch.from_numpy(tx).cuda(), torch.from_numpy(ty).cuda()


def _call(mas, v, x, y, ws):
    B, T, S = v.shape
    path = torch.full((B, T, S), 0xA5, dtype=torch.uint8, device="cuda")
    score = torch.full((B,), 3.0, dtype=torch.float32, device="cuda")
    status = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    mas.mas_forward_ex(v, x, y, path, score, status, workspace=ws)
    torch.cuda.synchronize()
    return path.cpu().numpy(), score.cpu().numpy(), status.cpu().numpy()


def test_uninitialised_workspace_is_reported(mas):
    """A workspace that never went through mas_workspace_init: the call
    computes nothing and every item reports MAS_ITEM_BAD_WORKSPACE; once
    initialised, the same buffer gives the oracle's results."""
    value, tx, ty, v, x, y = _inputs("tts-b16-t128-s512")
    B, T, S = value.shape
    _say("uninitialised workspace tts-b16-t128-s512")
    ws = mas.Workspace.__new__(mas.Workspace)
    ws.shape, ws.nbytes = (B, T, S), mas.mas_workspace_bytes(B, T, S)
    ws._buf = torch.zeros(ws.nbytes + 256, dtype=torch.uint8, device="cuda")
    ws.ptr = ws._buf.data_ptr() + (-ws._buf.data_ptr()) % 256
    ws.device = ws._buf.device
    path, score, status = _call(mas, v, x, y, ws)
    assert (status == mas.ITEM_BAD_WORKSPACE).all()
    assert (path == 0xA5).all() and (score == 3.0).all()  # nothing else touched
    mas.mas_workspace_init(ws.ptr, ws.nbytes)
    path, score, status = _call(mas, v, x, y, ws)
    op, os_, ost = oracle.mas(value, tx, ty)
    assert np.array_equal(status, ost) and np.array_equal(path, op) and score.tobytes() == os_.tobytes()


def test_tiny_wait_bound_reports_timeouts(mas, monkeypatch):
    """With the bound of every device-side wait lowered to 2 polls, waves give
    up, the launch still ends, no item is reported OK unless its outputs are
    the oracle's, and the next call with the normal bound is exact again."""
    value, tx, ty, v, x, y = _inputs("tts-b32-t256-s1024")
    B, T, S = value.shape
    ws = mas.Workspace(B, T, S)
    op, os_, ost = oracle.mas(value, tx, ty)
    _say("MAS_WAIT_BOUND=2 tts-b32-t256-s1024")
    monkeypatch.setenv("MAS_WAIT_BOUND", "2")
    path, score, status = _call(mas, v, x, y, ws)
    monkeypatch.delenv("MAS_WAIT_BOUND")
    assert set(np.unique(status).tolist()) <= {mas.ITEM_OK, mas.ITEM_SYNC_TIMEOUT}
    assert (status == mas.ITEM_SYNC_TIMEOUT).any()
    ok = np.flatnonzero(status == mas.ITEM_OK)
    for b in ok:
        assert np.array_equal(path[b], op[b]) and score[b].tobytes() == os_[b].tobytes(), f"item {b} reported OK"
    _say("normal bound after a timed-out call")
    path, score, status = _call(mas, v, x, y, ws)
    assert np.array_equal(status, ost) and np.array_equal(path, op) and score.tobytes() == os_.tobytes()
