"""The entry point that allocates nothing (mas_forward_static), through the
C ABI: its outputs must equal mas_forward_ex's bit for bit, on two calls in a
row, the second with a smaller batch (the static scratch keeps the first
call's state), and both must equal the oracle's."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


def _run(mas, name):
    value, tx, ty = synth.generate(name)
    B, T, S = value.shape
    print(f"[gpu-case] no-alloc {name} shape={value.shape}", flush=True)
    v, x, y = (torch.from_numpy(a).cuda() for a in (value, tx, ty))
    outs = []
    for fn in ("static", "ex"):
        path = torch.full((B, T, S), 0xA5, dtype=torch.uint8, device="cuda")
        score = torch.full((B,), 3.0, dtype=torch.float32, device="cuda")
        status = torch.full((B,), -1, dtype=torch.int32, device="cuda")
        if fn == "static":
            mas.mas_forward_static(v, x, y, path, score, status)
        else:
            mas.mas_forward_ex(v, x, y, path, score, status)
        torch.cuda.synchronize()
        outs.append((path.cpu().numpy(), score.cpu().numpy(), status.cpu().numpy()))
    (ps, ss, sts), (pe, se, ste) = outs
    assert np.array_equal(ps, pe) and ss.tobytes() == se.tobytes() and np.array_equal(sts, ste), name
    op, os_, ost = oracle.mas(value, tx, ty)
    assert np.array_equal(ps, op) and ss.tobytes() == os_.tobytes() and np.array_equal(sts, ost), name


def test_static_scratch_matches_mas_forward_ex():
    import paper_2409_07704_amd as mas

    mas.lib()
    for _ in range(2):
        _run(mas, "tts-b64-t1024-s4096")  # the largest workload: 72 MiB of the 80 MiB scratch
        _run(mas, "tts-b16-t128-s512")    # then smaller batches on the same scratch
        _run(mas, "tts-b32-t256-s1024")
        _run(mas, "tts-b32-t512-s2048")
