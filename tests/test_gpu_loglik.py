"""GPU parity of the Gaussian log-likelihood producer (mas_loglik).

The producer computes q[b][i][j] = log N(z_j; mu_i, sigma_i) on fp16 matrix
cores with split operands, so its values are checked against the oracle's
double-precision evaluation within bounds derived from that arithmetic (in
units of u = 2^-24 times M_ij, the sum of the absolute values of the cell's
terms):
  - every cell: |error| <= (3 Kp + D + 20 + 4 max|log_sigma|) u M_ij, the
    worst case of the 3 Kp fp32 accumulations of the product, the D-term
    row constant, the square roundings, the 2^-22 split error and the
    exp(-2 log_sigma) evaluation (hardware exp2 of a rounded product:
    about (1 + 3 |log_sigma|) u relative) (Kp = the padded contraction
    length 2 D rounded up to 32);
  - over all cells: rms(error / M) <= 4 u sqrt(3 Kp), which a dropped split
    part (an error of 2^-12 per product) exceeds many times.
The decisions MAS then takes over those values must be the oracle's on the
same fp32 values, bit for bit: paths, scores and statuses.  Cells outside
the feasible band must be left untouched.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu
U = 2.0 ** -24
HALF_LOG_TWO_PI = 0.5 * np.log(2.0 * np.pi)


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module")
def mas():
    import paper_2409_07704_amd as m

    m.lib()  # raises when the HIP library is missing
    return m


def band_mask(tx, ty, T, S):
    """Cells each valid item's MAS reads: i < t_x, i <= j < t_y, j - i <= t_y - t_x."""
    i = np.arange(T)[:, None]
    j = np.arange(S)[None, :]
    out = np.zeros((len(tx), T, S), bool)
    for b, (x, y) in enumerate(zip(tx, ty)):
        if 1 <= x <= y and x <= T and y <= S:
            out[b] = (i < x) & (j >= i) & (j < y) & (j - i <= y - x)
    return out


def magnitude(mu, ls, z, b, i, j):
    """M for cells (b, i, j): sum of |terms| of the row constant and the product."""
    m = mu[b, i].astype(np.float64)
    s = np.zeros_like(m) if ls is None else ls[b, i].astype(np.float64)
    r = np.exp(-2.0 * s)
    x = z[b, j].astype(np.float64)
    a_abs = (HALF_LOG_TWO_PI + np.abs(s) + 0.5 * m * m * r).sum(-1)
    return a_abs + (np.abs(m * r * x) + 0.5 * r * x * x).sum(-1)


def run_loglik(mas, mu, ls, z, tx, ty, S, z_dev=None):
    B, T, D = mu.shape
    v = torch.full((B, T, S), float("nan"), dtype=torch.float32, device="cuda")
    dm = torch.from_numpy(mu).cuda()
    dl = None if ls is None else torch.from_numpy(ls).cuda()
    dz = torch.from_numpy(z).cuda() if z_dev is None else z_dev
    dx = torch.from_numpy(np.asarray(tx, np.int32)).cuda()
    dy = torch.from_numpy(np.asarray(ty, np.int32)).cuda()
    mas.mas_loglik(dm, dl, dz, dx, dy, v)
    torch.cuda.synchronize()
    return v, dx, dy


def check_values(mu, ls, z, value, tx, ty, cells=None, label=""):
    B, T, D = mu.shape
    S = z.shape[1]
    Kp = (2 * ((D + 7) // 8 * 8) + 31) // 32 * 32
    bound = 3 * Kp + D + 20 + (0.0 if ls is None else 4.0 * float(np.abs(ls).max()))
    if cells is None:
        band = band_mask(tx, ty, T, S)
        assert np.isnan(value[~band]).all(), f"{label}: a cell outside the band was written"
        cells = np.argwhere(band)
    b, i, j = cells[:, 0], cells[:, 1], cells[:, 2]
    got = value[b, i, j].astype(np.float64)
    want = oracle.gauss_loglik(mu, ls, z, cells)
    M = magnitude(mu, ls, z, b, i, j)
    rel = np.abs(got - want) / (U * M)
    worst, rms = float(rel.max()), float(np.sqrt(np.mean(rel ** 2)))
    _say(f"{label}: {len(cells)} cells, max error {worst:.1f} u*M (bound {bound:.0f}), "
         f"rms {rms:.2f} u*M (bound {4 * np.sqrt(3 * Kp):.1f})")
    assert worst <= bound, f"{label}: cell error {worst:.1f} u*M"
    assert rms <= 4 * np.sqrt(3 * Kp), f"{label}: rms error {rms:.2f} u*M"


def check_alignment(mas, value_dev, dx, dy, tx, ty, label):
    """MAS over the producer's values: GPU against the oracle on the same values."""
    B, T, S = value_dev.shape
    path = torch.empty((B, T, S), dtype=torch.uint8, device="cuda")
    score = torch.empty(B, dtype=torch.float32, device="cuda")
    status = torch.empty(B, dtype=torch.int32, device="cuda")
    mas.mas_forward_ex(value_dev, dx, dy, path, score, status, workspace=mas.Workspace(B, T, S))
    torch.cuda.synchronize()
    op, os_, ost = oracle.mas(value_dev.cpu().numpy(), tx, ty)
    assert np.array_equal(status.cpu().numpy(), ost), label
    assert np.array_equal(path.cpu().numpy(), op), f"{label}: paths differ"
    assert score.cpu().numpy().tobytes() == os_.tobytes(), f"{label}: scores differ"


@pytest.mark.parametrize("ls_scale", [None, 0.3])
@pytest.mark.parametrize("name", ["tts-b16-t128-s512", "tts-b32-t256-s1024"])
def test_workloads(mas, name, ls_scale):
    mu, ls, z, tx, ty = synth.gauss_inputs(name, log_sigma_scale=ls_scale)
    S = z.shape[1]
    _say(f"{name} log_sigma_scale={ls_scale}")
    v, dx, dy = run_loglik(mas, mu, ls, z, tx, ty, S)
    check_values(mu, ls, z, v.cpu().numpy(), tx, ty, label=name)
    check_alignment(mas, v, dx, dy, tx, ty, name)


@pytest.mark.parametrize("unit", [False, True])
@pytest.mark.parametrize("D", [1, 7, 80, 100, 192])
def test_channel_counts(mas, D, unit):
    """Contractions of one k-step up to the largest (D = 192, as in VITS),
    channel counts that are no multiple of 8 (the 4-byte frame loads), and
    shapes that are no multiple of the tile sizes; large log-sigmas push
    the operands across many binades.  unit: no log_sigma (the contraction
    over D channels with a per-frame constant)."""
    rng = np.random.default_rng(D)
    B, T, S = 5, 150, 333
    tx = np.array([150, 1, 97, 33, 140], np.int32)
    ty = np.array([333, 40, 97, 300, 141], np.int32)
    mu = (3.0 * rng.standard_normal((B, T, D))).astype(np.float32)
    ls = (1.5 * rng.standard_normal((B, T, D))).astype(np.float32)
    z = (3.0 * rng.standard_normal((B, S, D))).astype(np.float32)
    if unit:
        ls = None
    _say(f"D={D} B={B} T={T} S={S} unit={unit}")
    v, dx, dy = run_loglik(mas, mu, ls, z, tx, ty, S)
    check_values(mu, ls, z, v.cpu().numpy(), tx, ty, label=f"D={D} unit={unit}")
    check_alignment(mas, v, dx, dy, tx, ty, f"D={D} unit={unit}")


def test_unaligned_frames_and_invalid_items(mas):
    """z 4 bytes off a 16-byte boundary (scalar frame loads) gives the same
    bits as the aligned call; invalid items are not written at all."""
    mu, ls, z, tx, ty = synth.gauss_inputs("tts-b16-t128-s512", log_sigma_scale=0.3)
    tx, ty = tx.copy(), ty.copy()
    tx[0], ty[1], tx[2], ty[2], tx[3] = 0, 0, 100, 50, 200
    B, S, D = z.shape
    _say("unaligned z, invalid items")
    v, dx, dy = run_loglik(mas, mu, ls, z, tx, ty, S)
    flat = torch.zeros(B * S * D + 1, dtype=torch.float32, device="cuda")
    flat[1:].copy_(torch.from_numpy(z.reshape(-1)).cuda())
    zu = flat[1:].view(B, S, D)
    assert zu.data_ptr() % 16 != 0
    vu, _, _ = run_loglik(mas, mu, ls, z, tx, ty, S, z_dev=zu)
    a, c = v.cpu().numpy(), vu.cpu().numpy()
    assert np.array_equal(a.view(np.uint32), c.view(np.uint32))
    for b in range(4):
        assert np.isnan(a[b]).all()
    check_values(mu, ls, z, a, tx, ty, label="invalid-items")


@pytest.mark.parametrize("ls_scale", [None, 0.2])
def test_benchmark_size(mas, ls_scale):
    """B=64, T=1024, S=4096, D=80, unit variance and with log-sigmas: 200k
    sampled band cells against the oracle, every alignment against the
    oracle's on the same values, and every cell outside the band untouched."""
    mu, ls, z, tx, ty = synth.gauss_inputs(synth.BENCH_WORKLOAD, log_sigma_scale=ls_scale)
    B, T, D = mu.shape
    S = z.shape[1]
    _say(f"{synth.BENCH_WORKLOAD} D={D} log_sigma_scale={ls_scale}")
    v, dx, dy = run_loglik(mas, mu, ls, z, tx, ty, S)
    value = v.cpu().numpy()
    band = band_mask(tx, ty, T, S)
    assert np.isnan(value[~band]).all()
    cells = np.argwhere(band)
    pick = np.random.default_rng(0).choice(len(cells), size=200_000, replace=False)
    check_values(mu, ls, z, value, tx, ty, cells=cells[np.sort(pick)], label=synth.BENCH_WORKLOAD)
    del cells, band
    check_alignment(mas, v, dx, dy, tx, ty, synth.BENCH_WORKLOAD)
