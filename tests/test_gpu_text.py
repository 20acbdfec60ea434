"""GPU parity of the aligned text grid (mas_expand_text) against the oracle.

The grid of an item is its MAS path multiplied with its text features (Sec.
5, Conclusion).  The library gathers it from the row_start table that
mas_search produced on the GPU; the oracle selects rows by its own dense path.
Both must agree byte for byte, for every element width and alignment, for
padding and invalid items, and at the full benchmark size.
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


def gpu_row_start(mas, value, tx, ty):
    B, T, S = value.shape
    v = torch.from_numpy(np.ascontiguousarray(value)).cuda()
    x = torch.from_numpy(np.asarray(tx, np.int32)).cuda()
    y = torch.from_numpy(np.asarray(ty, np.int32)).cuda()
    rs = mas.mas_search(v, x, y, workspace=mas.Workspace(B, T, S))
    torch.cuda.synchronize()
    return rs


def _to_device(h):
    """h on the GPU; 2-byte elements go as bfloat16 (the bits are what count)."""
    if h.dtype.itemsize == 2:
        return torch.from_numpy(np.ascontiguousarray(h).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(h)).cuda()


def check_grid(mas, path, rs, h, label, text_dev=None, out=None):
    """mas_expand_text on the GPU against oracle.expand_text, byte for byte."""
    B, T, S = path.shape
    C = h.shape[2]
    _say(f"{label} text={h.dtype}x{C} shape={path.shape}")
    t = _to_device(h) if text_dev is None else text_dev
    if out is None:  # filled with a pattern no frame holds
        out = torch.full((B * S * C * h.dtype.itemsize,), 0x5A, dtype=torch.uint8, device="cuda")
        out = out.view(t.dtype).view(B, S, C)
    mas.mas_expand_text(t, rs, S, out)
    torch.cuda.synchronize()
    got = out.contiguous().view(torch.uint8).cpu().numpy().reshape(B, S, -1)
    want = oracle.expand_text(path, h).view(np.uint8).reshape(B, S, -1)
    bad = np.argwhere(got != want)
    assert bad.size == 0, f"{label}: {len(bad)} bytes differ, first at {bad[:5].tolist()}"


@pytest.mark.parametrize("name", ["iid-b4-t32-s128", "tts-b16-t128-s512", "tts-b32-t256-s1024", "tts-b32-t512-s2048"])
def test_workloads_fp32_192(mas, name):
    value, tx, ty = synth.generate(name)
    path, _, _ = oracle.mas(value, tx, ty)
    rs = gpu_row_start(mas, value, tx, ty)
    assert np.array_equal(rs.cpu().numpy(), oracle.row_start(path, tx, ty))
    h = synth.text_batch(len(tx), value.shape[1], seed=1)
    check_grid(mas, path, rs, h, name)


def test_benchmark_size(mas):
    """B=64, T=1024, S=4096 with 192 fp32 channels (201 MB of grid),
    including the t_x = t_y and t_x = 1 items of that batch."""
    name = synth.BENCH_WORKLOAD
    value, tx, ty = synth.generate(name)
    path, _, _ = oracle.mas(value, tx, ty)
    rs = gpu_row_start(mas, value, tx, ty)
    assert np.array_equal(rs.cpu().numpy(), oracle.row_start(path, tx, ty))
    h = synth.text_batch(len(tx), value.shape[1], seed=2)
    check_grid(mas, path, rs, h, name)


@pytest.mark.parametrize("dtype,C", [(np.float32, 1), (np.float32, 7), (np.uint16, 192), (np.uint16, 7),
                                     (np.uint8, 3), (np.uint8, 48), (np.float64, 5), (np.float64, 2)])
def test_element_widths(mas, dtype, C):
    """1, 2, 4 and 8-byte elements with row sizes that take every word width
    (16, 8, 4, 2 and 1 bytes); 2-byte elements stand for bf16 and fp16."""
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    path, _, _ = oracle.mas(value, tx, ty)
    rs = gpu_row_start(mas, value, tx, ty)
    rng = np.random.default_rng(C)
    h = rng.integers(1, 250, size=(16, 128, C)).astype(dtype)
    check_grid(mas, path, rs, h, f"width-{np.dtype(dtype).itemsize}")


def test_unaligned_pointers(mas):
    """Text and grid 4 bytes off a 16-byte boundary: 4-byte words."""
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    path, _, _ = oracle.mas(value, tx, ty)
    rs = gpu_row_start(mas, value, tx, ty)
    B, T, S = value.shape
    h = synth.text_batch(B, T, 192, seed=3)
    flat = torch.zeros(B * T * 192 + 1, dtype=torch.float32, device="cuda")
    flat[1:].copy_(torch.from_numpy(h.reshape(-1)).cuda())
    t = flat[1:].view(B, T, 192)
    oflat = torch.zeros(B * S * 192 + 1, dtype=torch.float32, device="cuda")
    o = oflat[1:].view(B, S, 192)
    assert t.data_ptr() % 16 != 0 and o.data_ptr() % 16 != 0
    check_grid(mas, path, rs, h, "unaligned", text_dev=t, out=o)
    assert oflat[0].item() == 0.0


def test_invalid_items_padding_and_non_finite(mas):
    """Invalid items and padding frames are zero; -0, inf and NaN features
    are copied bit for bit."""
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    tx, ty = tx.copy(), ty.copy()
    tx[0], ty[1], tx[2], ty[2], tx[3] = 0, 0, 100, 50, 200
    path, _, _ = oracle.mas(value, tx, ty)
    rs = gpu_row_start(mas, value, tx, ty)
    h = synth.text_batch(16, 128, 8, seed=4)
    h[:, ::3, 0] = -0.0
    h[:, 1::5, 1] = np.inf
    h[:, 2::7, 2] = np.nan
    check_grid(mas, path, rs, h, "invalid-items")


def test_malformed_table_stays_inside_the_tensors(mas):
    """A row_start table that is not monotone and leaves [0, S]: frames are
    unspecified, but nothing outside the output tensor changes."""
    B, T, S, C = 3, 40, 300, 16
    rng = np.random.default_rng(5)
    rs = torch.from_numpy(rng.integers(-50, S + 50, size=(B, T + 1)).astype(np.int32)).cuda()
    h = torch.from_numpy(synth.text_batch(B, T, C, seed=5)).cuda()
    guard = torch.full((B * S * C + 2 * 64,), 7.0, dtype=torch.float32, device="cuda")
    out = guard[64:64 + B * S * C].view(B, S, C)
    _say("malformed row_start B=3 T=40 S=300 C=16")
    mas.mas_expand_text(h, rs, S, out)
    torch.cuda.synchronize()
    g = guard.cpu().numpy()
    assert (g[:64] == 7.0).all() and (g[64 + B * S * C:] == 7.0).all()
