"""Seeded synthetic inputs for batched monotonic alignment search.

Shared by the HIP library's tests/benchmark and by the CPU oracle; holds none
of the alignment method's arithmetic.  The random streams and the Gaussian
log-likelihood live in ``synth.c`` (SplitMix64 + Box-Muller, double
precision, fixed summation order), compiled with gcc.

Workloads mirror the shapes of TTS training batches (speech frames about four
times the text length, ragged per-item lengths).  The paper benchmarks on a
random [B, T, S] tensor with S = 4T taken from LibriTTS statistics; LibriTTS
is not available here, so these synthetic tensors stand in for it.

Draw order for one workload from ``seed``:
  1. for every item b: its text length t_x, then its speech length t_y
     (items whose recipe fixes a length draw only the other one);
  2. for every item b: its values over the full padded [T, S] slab —
     i.i.d. workloads draw T*S normals row-major; log-likelihood workloads
     draw mu_b [T, D] then x_b [S, D] (row-major) and evaluate
     value[i, j] = -0.5 * sum_d (x_b[j, d] - mu_b[i, d])^2 - (D/2) ln(2 pi).
"""
from __future__ import annotations

import ctypes
import dataclasses
import hashlib
import os
import subprocess
from typing import Callable

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libmas_synth.so")
CFLAGS = ["-O3", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile ``synth.c`` into ``synth/libmas_synth.so`` with gcc."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        lib.synth_raw.argtypes = [P, P, sz]
        lib.synth_randint.argtypes = [P, i32, i32, P, sz]
        lib.synth_normal.argtypes = [P, P, sz]
        lib.synth_to_f32.argtypes = [P, P, sz]
        lib.synth_gauss_loglik.argtypes = [P, P, i32, i32, i32, P]
        lib.synth_gauss_loglik.restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


class Stream:
    """One SplitMix64 stream; every draw advances the shared state."""

    def __init__(self, seed: int):
        self.state = np.array([seed & 0xFFFFFFFFFFFFFFFF], dtype=np.uint64)

    def raw(self, n: int) -> np.ndarray:
        out = np.empty(n, dtype=np.uint64)
        _load().synth_raw(_p(self.state), _p(out), n)
        return out

    def randint(self, lo: int, hi: int, n: int = 1) -> np.ndarray:
        out = np.empty(n, dtype=np.int32)
        _load().synth_randint(_p(self.state), lo, hi, _p(out), n)
        return out

    def normal(self, n: int) -> np.ndarray:
        out = np.empty(n, dtype=np.float64)
        _load().synth_normal(_p(self.state), _p(out), n)
        return out

    def normal_f32(self, n: int) -> np.ndarray:
        d = self.normal(n)
        out = np.empty(n, dtype=np.float32)
        _load().synth_to_f32(_p(d), _p(out), n)
        return out


def gauss_loglik(mu: np.ndarray, x: np.ndarray, out: np.ndarray) -> None:
    """value[i, j] = -0.5 sum_d (x[j,d] - mu[i,d])^2 - (D/2) ln(2 pi), into out [T, S] f32."""
    mu = np.ascontiguousarray(mu, dtype=np.float64)
    x = np.ascontiguousarray(x, dtype=np.float64)
    T, D = mu.shape
    S, D2 = x.shape
    assert D == D2 and out.shape == (T, S) and out.dtype == np.float32 and out.flags.c_contiguous
    if _load().synth_gauss_loglik(_p(mu), _p(x), T, S, D, _p(out)) != 0:
        raise MemoryError("synth_gauss_loglik allocation failed")


# ---------------------------------------------------------------- workloads
LengthRecipe = Callable[[Stream, int], tuple]


def _fixed(tx: int, ty: int) -> LengthRecipe:
    return lambda st, b: (tx, ty)


def _ragged(tx_lo: int, tx_hi: int, ty_lo: int, ty_hi: int) -> LengthRecipe:
    """t_x ~ U[tx_lo, tx_hi], then t_y ~ U[max(t_x, ty_lo), ty_hi]."""

    def f(st: Stream, b: int):
        tx = int(st.randint(tx_lo, tx_hi)[0])
        ty = int(st.randint(max(tx, ty_lo), ty_hi)[0])
        return tx, ty

    return f


def _long_mix(st: Stream, b: int):
    """Items 0..55 ragged; 56..59 forced diagonal (t_y = t_x); 60..63 t_x = 1."""
    if b < 56:
        return _ragged(256, 1024, 1024, 4096)(st, b)
    if b < 60:
        tx = int(st.randint(256, 1024)[0])
        return tx, tx
    return 1, int(st.randint(1024, 4096)[0])


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    T: int
    S: int
    values: str  # "normal" | "loglik" | "int"
    lengths: LengthRecipe
    D: int = 80

    @property
    def shape(self):
        return (self.B, self.T, self.S)


WORKLOADS = {
    w.name: w
    for w in [
        # i.i.d. N(0,1) values, full lengths
        Workload("iid-b4-t32-s128", 4, 32, 128, "normal", _fixed(32, 128)),
        # tiny ragged batch for brute-force enumeration (t_x <= 5, t_y <= 10)
        Workload("tiny-b8-t5-s10", 8, 5, 10, "normal", _ragged(1, 5, 1, 10)),
        Workload("tiny-int-b8-t5-s10", 8, 5, 10, "int", _ragged(1, 5, 1, 10)),
        # Gaussian log-likelihood TTS-shaped batches (D = 80)
        Workload("tts-b16-t128-s512", 16, 128, 512, "loglik", _ragged(64, 128, 256, 512)),
        Workload("tts-b32-t256-s1024", 32, 256, 1024, "loglik", _ragged(128, 256, 512, 1024)),
        Workload("tts-b32-t512-s2048", 32, 512, 2048, "loglik", _ragged(256, 512, 1024, 2048)),
        Workload("tts-b64-t1024-s4096", 64, 1024, 4096, "loglik", _long_mix),
    ]
}

# Parity sizes (every workload above) and the one the benchmark times.
BENCH_WORKLOAD = "tts-b64-t1024-s4096"


def draw_lengths(w: Workload, st: Stream):
    tx = np.empty(w.B, dtype=np.int32)
    ty = np.empty(w.B, dtype=np.int32)
    for b in range(w.B):
        tx[b], ty[b] = w.lengths(st, b)
    return tx, ty


def generate(w: Workload | str, seed: int = 0):
    """(value f32 [B,T,S], t_x i32 [B], t_y i32 [B]) for a workload and seed."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    st = Stream(seed)
    tx, ty = draw_lengths(w, st)
    value = np.empty((w.B, w.T, w.S), dtype=np.float32)
    for b in range(w.B):
        if w.values == "normal":
            value[b] = st.normal_f32(w.T * w.S).reshape(w.T, w.S)
        elif w.values == "int":
            value[b] = st.randint(-2, 2, w.T * w.S).astype(np.float32).reshape(w.T, w.S)
        elif w.values == "loglik":
            mu = st.normal(w.T * w.D).reshape(w.T, w.D)
            x = st.normal(w.S * w.D).reshape(w.S, w.D)
            gauss_loglik(mu, x, value[b])
        else:
            raise ValueError(w.values)
    return value, tx, ty


def normal_batch(B: int, T: int, S: int, tx, ty, seed: int):
    """Ad-hoc i.i.d. N(0,1) batch with given lengths (odd shapes, edge cases)."""
    st = Stream(seed)
    value = st.normal_f32(B * T * S).reshape(B, T, S)
    return value, np.asarray(tx, dtype=np.int32).reshape(B), np.asarray(ty, dtype=np.int32).reshape(B)


def gauss_inputs(w: Workload | str, seed: int = 0, log_sigma_scale: float | None = None):
    """The Gaussian parameters behind a "loglik" workload, as fp32 tensors:
    (mu [B,T,D], log_sigma [B,T,D] or None, z [B,S,D], t_x [B], t_y [B]).

    mu and z are the draws generate() makes for the same workload and seed
    (in the same order), rounded to fp32.  With log_sigma_scale, log_sigma
    is log_sigma_scale * N(0,1) from a stream of its own; without it the
    variance is 1, as in generate()."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    if w.values != "loglik":
        raise ValueError(f"{w.name} is not a log-likelihood workload")
    st = Stream(seed)
    tx, ty = draw_lengths(w, st)
    mu = np.empty((w.B, w.T, w.D), dtype=np.float32)
    z = np.empty((w.B, w.S, w.D), dtype=np.float32)
    for b in range(w.B):
        mu[b] = st.normal(w.T * w.D).reshape(w.T, w.D)
        z[b] = st.normal(w.S * w.D).reshape(w.S, w.D)
    ls = None
    if log_sigma_scale is not None:
        ls = (np.float32(log_sigma_scale) * Stream(seed + 104729).normal_f32(w.B * w.T * w.D)).reshape(w.B, w.T, w.D)
    return mu, ls, z, tx, ty


# Text features per token for the aligned text grid: 192 channels, the hidden
# size of the text encoders whose outputs MAS aligns in TTS training.
TEXT_CHANNELS = 192


def text_batch(B: int, T: int, C: int = TEXT_CHANNELS, seed: int = 0) -> np.ndarray:
    """Seeded text features h f32 [B, T, C], i.i.d. N(0,1) (no exact zeros, so
    that a zero frame in a grid can only come from an uncovered column)."""
    st = Stream(seed + 7919)
    h = st.normal_f32(B * T * C).reshape(B, T, C)
    h[h == 0] = np.float32(1.0)
    return h


def sha256(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()
