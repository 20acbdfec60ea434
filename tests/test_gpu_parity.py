"""GPU parity of libmas against the CPU oracle, through the C ABI.

The bar is bit-exactness: every path byte, every row_start entry, every
per-item status and the bits of every exported score must equal the
oracle's.  Every case prints its name, shape and seed before touching the GPU.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import _pins

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def mas():
    import paper_2409_07704_amd as m

    m.lib()  # raises when the HIP library is missing
    return m


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda")


def run_gpu(mas, value, tx, ty, workspace=None, value_dev=None):
    """mas_forward_ex, then mas_search (no dense path) on the same workspace;
    every output back on the host."""
    B, T, S = value.shape
    v = _dev(value) if value_dev is None else value_dev
    x = _dev(np.asarray(tx, np.int32))
    y = _dev(np.asarray(ty, np.int32))
    ws = workspace or mas.Workspace(B, T, S)
    path = torch.empty((B, T, S), dtype=torch.uint8, device="cuda")
    score = torch.empty(B, dtype=torch.float32, device="cuda")
    status = torch.empty(B, dtype=torch.int32, device="cuda")
    mas.mas_forward_ex(v, x, y, path, score, status, workspace=ws)
    s_score = torch.full((B,), 7.0, dtype=torch.float32, device="cuda")
    s_status = torch.full((B,), 99, dtype=torch.int32, device="cuda")
    s_dur = torch.full((B, T), -5, dtype=torch.int32, device="cuda")
    rs = mas.mas_search(v, x, y, None, s_score, s_status, workspace=ws, durations_out=s_dur)
    torch.cuda.synchronize()
    return (path.cpu().numpy(), score.cpu().numpy(), status.cpu().numpy(), rs.cpu().numpy(),
            s_score.cpu().numpy(), s_status.cpu().numpy(), s_dur.cpu().numpy())


def assert_parity(mas, value, tx, ty, label, **kw):
    _say(f"{label} shape={value.shape}")
    gp, gs, gst, grs, sgs, sgst, sdur = run_gpu(mas, value, tx, ty, **kw)
    op, os_, ost = oracle.mas(value, tx, ty)
    assert np.array_equal(gst, ost), f"{label}: status {gst} vs {ost}"
    bad = np.argwhere(gp != op)
    assert bad.size == 0, f"{label}: {len(bad)} path bytes differ, first at {bad[:5].tolist()}"
    assert gs.tobytes() == os_.tobytes(), f"{label}: scores differ {gs} vs {os_}"
    # the path-less call: row_start, durations, score and status
    assert np.array_equal(grs, oracle.row_start(op, tx, ty)), f"{label}: row_start differs"
    assert np.array_equal(sdur, oracle.durations(op)), f"{label}: durations differ"
    assert sgs.tobytes() == os_.tobytes(), f"{label}: mas_search scores differ"
    assert np.array_equal(sgst, ost), f"{label}: mas_search status differs"
    return gp, gs


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_workload_parity(mas, name):
    value, tx, ty = synth.generate(name)
    assert_parity(mas, value, tx, ty, name)


def test_exhaustive_small_pairs(mas):
    pairs = [(a, c) for a in range(1, 6) for c in range(a, 11)]
    st = synth.Stream(4242)
    value = st.normal_f32(len(pairs) * 5 * 10).reshape(len(pairs), 5, 10)
    tx = [a for a, _ in pairs]
    ty = [c for _, c in pairs]
    gp, gs = assert_parity(mas, value, tx, ty, "exhaustive-40")
    for b, (a, c) in enumerate(pairs):
        best, arg = _pins.brute_force(value[b], a, c)
        assert gs[b].tobytes() == np.float32(best).tobytes()


def test_integer_ties(mas):
    st = synth.Stream(99)
    B, T, S = 24, 70, 200
    value = st.randint(-2, 2, B * T * S).astype(np.float32).reshape(B, T, S)
    tx = st.randint(1, T, B)
    ty = np.array([int(st.randint(int(a), S)[0]) for a in tx], np.int32)
    assert_parity(mas, value, tx, ty, "integer-ties")


def test_signed_zero_inputs(mas):
    """Integer values with both signs of zero: exact ties between -0 and +0
    partial sums, decided by the signed-zero order of the forward max."""
    st = synth.Stream(123)
    B, T, S = 16, 150, 260
    value = st.randint(-1, 1, B * T * S).astype(np.float32)
    neg = st.randint(0, 1, B * T * S).astype(bool)
    value[(value == 0) & neg] = np.float32(-0.0)
    value = value.reshape(B, T, S)
    tx = st.randint(1, T, B)
    ty = np.array([int(st.randint(int(a), S)[0]) for a in tx], np.int32)
    assert (np.signbit(value) & (value == 0)).any()
    assert_parity(mas, value, tx, ty, "signed-zeros")
    # the exhaustive small shapes, all zeros of random sign
    pairs = [(a, c) for a in range(1, 6) for c in range(a, 11)]
    z = np.where(st.randint(0, 1, 40 * 5 * 10).astype(bool), np.float32(-0.0), np.float32(0.0)).reshape(40, 5, 10)
    assert_parity(mas, z, np.array([a for a, _ in pairs], np.int32), np.array([c for _, c in pairs], np.int32), "zeros-40")


def test_subnormal_values_and_partial_sums(mas):
    """Integer multiples of 2^-140 (values and partial sums on both sides of
    the smallest normal, many subnormal), and values around 1e-40: bit-exact
    only if neither side flushes subnormals to zero."""
    st = synth.Stream(321)
    B, T, S = 12, 200, 700
    q = np.float32(2.0 ** -140)
    value = (st.randint(-40000, 40000, B * T * S).astype(np.float32) * q).reshape(B, T, S)
    value[6:] = (st.normal_f32(6 * T * S).reshape(6, T, S) * np.float32(2.0 ** -133)).astype(np.float32)
    tx = st.randint(1, T, B)
    ty = np.array([int(st.randint(int(a), S)[0]) for a in tx], np.int32)
    tx[0], ty[0] = T, S
    _, gs = assert_parity(mas, value, tx, ty, "subnormals")
    assert ((gs != 0) & (np.abs(gs) < np.float32(2.0 ** -126))).any()


@pytest.mark.parametrize(
    "B,T,S,seed",
    [(3, 33, 129, 1), (5, 65, 96, 2), (4, 257, 1001, 3), (2, 300, 301, 4), (6, 1, 77, 5), (3, 130, 4099, 6)],
)
def test_odd_shapes(mas, B, T, S, seed):
    st = synth.Stream(seed)
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(30.0)
    tx = st.randint(1, T, B)
    ty = np.array([int(st.randint(int(a), S)[0]) for a in tx], np.int32)
    tx[0], ty[0] = T, S                 # full extent
    if B > 1:
        ty[1] = tx[1]                   # forced diagonal
    if B > 2:
        tx[2] = 1                       # single text row
    assert_parity(mas, value, tx, ty, f"odd B={B} T={T} S={S} seed={seed}")


def test_many_waves_per_item(mas):
    """Items with thousands of text rows: many chained waves and workgroups."""
    st = synth.Stream(8)
    B, T, S = 3, 2100, 2400
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(10.0) - np.float32(150.0)
    tx = np.array([2100, 2000, 1500], np.int32)
    ty = np.array([2400, 2000, 2399], np.int32)
    assert_parity(mas, value, tx, ty, "many-waves")


def test_full_length_batch(mas):
    """Every item spans the whole padded extent (t_x = T, t_y = S) at the
    largest workload shape: every workgroup of the grid carries a sweep, so
    each one depends on a chain of others across the whole launch."""
    st = synth.Stream(77)
    B, T, S = 64, 1024, 4096
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(4.0) - np.float32(2.0)
    tx = np.full(B, T, np.int32)
    ty = np.full(B, S, np.int32)
    assert_parity(mas, value, tx, ty, "full-length-b64-t1024-s4096")


def test_long_items(mas):
    """Long speech axes: a backtrack over hundreds of chunks with banded
    decision windows (T above the window height), a path pinned to the last
    diagonal by a ridge of high values, and lengths around 1024 chunks with
    the walking wave last in its workgroup (t_x 190 and 252)."""
    st = synth.Stream(91)
    B, T, S = 3, 1500, 9000
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(4.0) - np.float32(2.0)
    assert_parity(mas, value, np.array([1500, 1200, 700], np.int32), np.array([9000, 8500, 6000], np.int32),
                  "long-banded")

    B, T, S = 2, 300, 5000
    tx = np.array([300, 250], np.int32)
    ty = np.array([5000, 4990], np.int32)
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(0.1)
    for b in range(B):
        i = np.arange(tx[b])
        value[b, i, i + (ty[b] - tx[b])] += np.float32(50.0)
    assert_parity(mas, value, tx, ty, "long-ridge")

    B, T, S = 6, 256, 32800
    tx = np.array([256, 190, 2, 1, 252, 200], np.int32)
    ty = np.array([32768, 32769, 992, 993, 1024, 32800], np.int32)
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(4.0) - np.float32(2.0)
    assert_parity(mas, value, tx, ty, "long-1024-chunks")


def test_banded_walk_windows(mas):
    """Items taller than the walk's whole-chunk windows allow (t_x above
    about 4350 rows at these shapes): the loaders stage banded windows, a
    row band around the walker plus the mid entries of its waves, and the
    walk crosses many wave boundaries through them.  T = 8192 is the largest
    height the library accepts."""
    st = synth.Stream(4242)
    B, T, S = 2, 6000, 7000
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(3.0) - np.float32(1.0)
    assert_parity(mas, value, np.array([6000, 4700], np.int32), np.array([7000, 6999], np.int32), "banded-t6000-s7000")
    B, T, S = 1, 8192, 8200
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(3.0) - np.float32(1.0)
    assert_parity(mas, value, np.array([8192], np.int32), np.array([8200], np.int32), "banded-t8192-s8200")


def test_mixed_batch_tall_items(mas):
    """A mixed batch with T above the walk's window height (banded windows),
    several workgroups per item (boundary rows handed on by the loaders, one
    storer per workgroup) and many path tiles per item, plus degenerate items
    (single row, diagonal, empty) in the same launch."""
    st = synth.Stream(123)
    B, T, S = 12, 2048, 3000
    value = st.normal_f32(B * T * S).reshape(B, T, S) * np.float32(3.0) - np.float32(1.0)
    tx = st.randint(1, T, B)
    ty = np.array([int(st.randint(int(a), S)[0]) for a in tx], np.int32)
    tx[0], ty[0] = T, S          # full extent
    tx[1], ty[1] = 1500, 1500    # diagonal
    tx[2], ty[2] = 1, 2999       # one row
    tx[3], ty[3] = 0, 100        # empty
    tx[4], ty[4] = 1100, 2999    # just above the window height
    assert_parity(mas, value, tx, ty, "mixed-tall-b12-t2048-s3000")


def test_unaligned_value_pointer(mas):
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    B, T, S = value.shape
    flat = torch.empty(B * T * S + 1, dtype=torch.float32, device="cuda")
    flat[1:].copy_(torch.from_numpy(value.reshape(-1)).cuda())
    v = flat[1:].view(B, T, S)  # 4-byte aligned, not 16-byte aligned
    assert v.data_ptr() % 16 != 0
    assert_parity(mas, value, tx, ty, "unaligned-value", value_dev=v)


def test_nan_poisoned_padding_triangle_and_band(mas):
    value, tx, ty = synth.generate("tts-b32-t256-s1024")
    B, T, S = value.shape
    ii = np.arange(T)[:, None]
    jj = np.arange(S)[None, :]
    poisoned = value.copy()
    for b in range(B):
        a, c = int(tx[b]), int(ty[b])
        poisoned[b][(ii >= a) | (jj >= c) | (ii > jj) | (ii < a - c + jj)] = np.nan
    gp0, gs0 = assert_parity(mas, value, tx, ty, "clean")
    gp1, gs1 = assert_parity(mas, poisoned, tx, ty, "poisoned")
    assert np.array_equal(gp0, gp1) and gs0.tobytes() == gs1.tobytes()


def test_invalid_lengths(mas):
    B, T, S = 7, 40, 90
    st = synth.Stream(11)
    value = st.normal_f32(B * T * S).reshape(B, T, S)
    tx = np.array([0, 3, 50, -1, 41, 3, 40], np.int32)
    ty = np.array([4, 0, 45, 5, 90, 91, 90], np.int32)
    gp, gs = assert_parity(mas, value, tx, ty, "invalid-lengths")
    assert not gp[:6].any()


def test_determinism_and_workspace_reuse(mas):
    v1, x1, y1 = synth.generate("tts-b32-t512-s2048")
    v0, x0, y0 = synth.generate("iid-b4-t32-s128")
    ws = mas.Workspace(*v1.shape)
    _say("determinism x10 tts-b32-t512-s2048")
    ref = run_gpu(mas, v1, x1, y1, workspace=ws)
    for _ in range(9):
        out = run_gpu(mas, v1, x1, y1, workspace=ws)
        assert all(np.array_equal(a, b) for a, b in zip(ref, out))
    # a smaller batch in the same workspace, then the large one again
    assert_parity(mas, v0, x0, y0, "reuse-small", workspace=ws)
    assert_parity(mas, v1, x1, y1, "reuse-large", workspace=ws)


def test_shape_changes_on_one_workspace(mas):
    """Calls of different shapes, large to small and back, on one workspace:
    each call lays its regions out differently, over the previous call's data
    (step masks, row starts), which must never pass for this call's flags."""
    names = ["tts-b64-t1024-s4096", "tts-b16-t128-s512", "tts-b32-t256-s1024", "tts-b32-t512-s2048"]
    data = {n: synth.generate(n) for n in names}
    ws = mas.Workspace(64, 1024, 4096)
    for rnd in range(3):
        for n in names:
            value, tx, ty = data[n]
            assert_parity(mas, value, tx, ty, f"shape-change round {rnd} {n}", workspace=ws)


def test_canaries_and_nonnull_outputs(mas):
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    B, T, S = value.shape
    _say("canaries tts-b16-t128-s512")
    pad = 4096
    pbuf = torch.full((B * T * S + 2 * pad,), 0xA5, dtype=torch.uint8, device="cuda")
    path = pbuf[pad:pad + B * T * S].view(B, T, S)
    rbuf = torch.full((B * (T + 1) + 2 * pad,), -7, dtype=torch.int32, device="cuda")
    rs = rbuf[pad:pad + B * (T + 1)].view(B, T + 1)
    sbuf = torch.full((B + 2 * pad,), 3.0, dtype=torch.float32, device="cuda")
    score = sbuf[pad:pad + B]
    x, y, v = _dev(tx), _dev(ty), _dev(value)
    ws = mas.Workspace(B, T, S)
    mas.mas_forward_ex(v, x, y, path, score, None, workspace=ws)
    mas.mas_search(v, x, y, rs, None, None, workspace=ws)
    torch.cuda.synchronize()
    pb, rb, sb = pbuf.cpu().numpy(), rbuf.cpu().numpy(), sbuf.cpu().numpy()
    assert (pb[:pad] == 0xA5).all() and (pb[-pad:] == 0xA5).all()
    assert (rb[:pad] == -7).all() and (rb[-pad:] == -7).all()
    assert (sb[:pad] == 3.0).all() and (sb[-pad:] == 3.0).all()
    op, os_, _ = oracle.mas(value, tx, ty)
    assert np.array_equal(path.cpu().numpy(), op)
    assert score.cpu().numpy().tobytes() == os_.tobytes()


def test_side_stream_and_two_streams(mas):
    va, xa, ya = synth.generate("tts-b32-t256-s1024")
    vb, xb, yb = synth.generate("tts-b16-t128-s512")
    _say("two streams")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    wa, wb = mas.Workspace(*va.shape), mas.Workspace(*vb.shape)
    da, db = _dev(va), _dev(vb)
    pa = torch.empty(va.shape, dtype=torch.uint8, device="cuda")
    pb = torch.empty(vb.shape, dtype=torch.uint8, device="cuda")
    xa_, ya_, xb_, yb_ = _dev(xa), _dev(ya), _dev(xb), _dev(yb)
    torch.cuda.synchronize()
    for _ in range(3):
        mas.mas_forward_ex(da, xa_, ya_, pa, workspace=wa, stream=sa)
        mas.mas_forward_ex(db, xb_, yb_, pb, workspace=wb, stream=sb)
    torch.cuda.synchronize()
    assert np.array_equal(pa.cpu().numpy(), oracle.mas(va, xa, ya)[0])
    assert np.array_equal(pb.cpu().numpy(), oracle.mas(vb, xb, yb)[0])


def test_allocating_entry_point(mas):
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    _say("mas_forward (allocating)")
    path = mas.mas_forward(_dev(value), _dev(tx), _dev(ty))
    torch.cuda.synchronize()
    assert np.array_equal(path.cpu().numpy(), oracle.mas(value, tx, ty)[0])


def test_path_writer_alone(mas):
    """mas_expand_path from a row_start table, aligned and unaligned S."""
    st = synth.Stream(12)
    for S in (64, 100, 4096):
        B, T = 5, 37
        _say(f"expand_path S={S}")
        rs = np.zeros((B, T + 1), np.int32)
        for b in range(B):
            cuts = np.sort(st.randint(0, S, T + 1))
            rs[b] = cuts
        path = mas.mas_expand_path(_dev(rs), S)
        torch.cuda.synchronize()
        got = path.cpu().numpy()
        jj = np.arange(S)[None, None, :]
        want = ((rs[:, :-1, None] <= jj) & (jj < rs[:, 1:, None])).astype(np.uint8)
        assert np.array_equal(got, want)
