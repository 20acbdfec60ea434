"""Pins of the oracle's Gaussian log-likelihood (oracle.gauss_loglik).

q[i][j] = log N(z_j; mu_i, sigma_i) over D channels with a diagonal
covariance (Sec. 2).  The oracle evaluates it in double.  These pins hold it
to scipy's normal log-density (a library routine with its own arrangement of
the formula), to hand-derived values, to the closed form at z = mu, to the
unit-variance input generator, and to planted mistakes.
"""
from __future__ import annotations

import ctypes
import json
import os
import subprocess
import tempfile

import numpy as np
import pytest
from scipy.stats import norm

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "loglik_cases.json")
HALF_LOG_TWO_PI = 0.5 * np.log(2.0 * np.pi)


def _inputs(B, T, S, D, seed, ls_scale=0.3):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((B, T, D)).astype(np.float32)
    ls = None if ls_scale is None else (ls_scale * rng.standard_normal((B, T, D))).astype(np.float32)
    z = rng.standard_normal((B, S, D)).astype(np.float32)
    return mu, ls, z


def _scipy(mu, ls, z):
    m = mu[:, :, None, :].astype(np.float64)
    x = z[:, None, :, :].astype(np.float64)
    sd = 1.0 if ls is None else np.exp(ls[:, :, None, :].astype(np.float64))
    return norm.logpdf(x, loc=m, scale=sd).sum(axis=-1)


@pytest.mark.parametrize("B,T,S,D,ls_scale", [(2, 5, 9, 1, 0.3), (3, 7, 11, 80, 0.3), (2, 4, 6, 192, 1.0),
                                              (2, 6, 8, 80, None)])
def test_equals_scipy_normal_logpdf(B, T, S, D, ls_scale):
    mu, ls, z = _inputs(B, T, S, D, seed=D, ls_scale=ls_scale)
    q = oracle.gauss_loglik(mu, ls, z)
    ref = _scipy(mu, ls, z)
    assert np.abs(q - ref).max() <= 1e-12 * (1.0 + np.abs(ref).max())


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_derived_values(case):
    mu = np.array(case["mu"], np.float32)[None, None]
    ls = np.array(case["log_sigma"], np.float32)[None, None]
    z = np.array(case["z"], np.float32)[None, None]
    q = oracle.gauss_loglik(mu, ls, z)[0, 0, 0]
    assert abs(q - case["q"]) <= 1e-15 * abs(case["q"]) * 4


def test_frame_at_the_mean_is_the_normaliser():
    mu, ls, _ = _inputs(2, 6, 1, 80, seed=3)
    q = oracle.gauss_loglik(mu, ls, mu.copy())  # z_j = mu_j for j < T
    T = mu.shape[1]
    diag = q[:, np.arange(T), np.arange(T)]
    want = (-HALF_LOG_TWO_PI - ls.astype(np.float64)).sum(axis=-1)
    assert np.abs(diag - want).max() <= 1e-12 * np.abs(want).max()


def test_unit_variance_equals_the_input_generator():
    """The workload generator writes -sum (x - mu)^2 / 2 - D ln(2 pi) / 2 in
    double and rounds to fp32; the oracle rounded to fp32 agrees to 1 ulp
    (the two sum in different orders)."""
    mu, _, z, tx, ty = synth.gauss_inputs("tts-b16-t128-s512")
    q = oracle.gauss_loglik(mu[:2], None, z[:2]).astype(np.float32)
    for b in range(2):
        ref = np.empty(q.shape[1:], np.float32)
        synth.gauss_loglik(mu[b].astype(np.float64), z[b].astype(np.float64), ref)
        ulps = np.abs(q[b].view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
        assert ulps.max() <= 1


def test_cells_subset_and_bounds():
    mu, ls, z = _inputs(2, 5, 9, 8, seed=4)
    full = oracle.gauss_loglik(mu, ls, z)
    cells = np.array([[0, 0, 0], [1, 4, 8], [0, 2, 5]])
    assert np.array_equal(oracle.gauss_loglik(mu, ls, z, cells), full[cells[:, 0], cells[:, 1], cells[:, 2]])
    with pytest.raises(ValueError):
        oracle.gauss_loglik(mu, ls, z, np.array([[0, 5, 0]]))


# ------------------------------------------------------------- mutation check
_MUTATIONS = {
    "variance_not_squared": ("t * t / (2.0 * sigma * sigma)", "t * t / (2.0 * sigma)"),
    "half_dropped": ("t * t / (2.0 * sigma * sigma)", "t * t / (sigma * sigma)"),
    "log_sigma_sign": ("q += -half_log_two_pi - lsd -", "q += -half_log_two_pi + lsd -"),
    "normaliser_not_halved": ("q += -half_log_two_pi - lsd", "q += -2.0 * half_log_two_pi - lsd"),
    "frame_row_from_text_index": ("x = z + ((size_t)b * (size_t)S + (size_t)j) * (size_t)D;",
                                  "x = z + ((size_t)b * (size_t)S + (size_t)i) * (size_t)D;"),
}


def _variant(so):
    lib = ctypes.CDLL(so)
    P, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.oracle_gauss_loglik_cells.argtypes = [P, P, P, i32, i32, i32, i32, P, ctypes.c_int64, P]

    def gl(mu, ls, z):
        B, T, D = mu.shape
        S = z.shape[1]
        b, i, j = np.meshgrid(np.arange(B), np.arange(T), np.arange(S), indexing="ij")
        cells = np.ascontiguousarray(np.stack([b.ravel(), i.ravel(), j.ravel()], 1), dtype=np.int32)
        out = np.empty(len(cells))
        p = lambda a: None if a is None else a.ctypes.data_as(P)
        lib.oracle_gauss_loglik_cells(p(mu), p(ls), p(z), B, T, S, D, p(cells), len(cells), p(out))
        return out.reshape(B, T, S)

    return gl


def _pins_pass(gl) -> bool:
    for B, T, S, D, s in [(2, 5, 9, 1, 0.3), (2, 6, 8, 80, 0.3)]:
        mu, ls, z = _inputs(B, T, S, D, seed=D, ls_scale=s)
        ref = _scipy(mu, ls, z)
        if not np.abs(gl(mu, ls, z) - ref).max() <= 1e-12 * (1.0 + np.abs(ref).max()):
            return False
    return True


def test_pins_accept_the_oracle():
    assert _pins_pass(oracle.gauss_loglik)


@pytest.mark.parametrize("mutation", sorted(_MUTATIONS))
def test_pins_catch_planted_mistakes(mutation):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "mas_oracle.c")).read()
    old, new = _MUTATIONS[mutation]
    assert src.count(old) == 1, mutation
    with tempfile.TemporaryDirectory() as d:
        c, so = os.path.join(d, "variant.c"), os.path.join(d, "variant.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.check_call(["gcc", *oracle.CFLAGS, c, "-o", so, "-lm"])
        assert not _pins_pass(_variant(so)), f"pins did not detect mutation {mutation}"
