"""Pins of the oracle's aligned text grid (oracle.expand_text).

The grid is the MAS path multiplied with the text features (Sec. 5,
Conclusion): out[b] = path[b]^T @ h[b].  The oracle computes it as a
selection (each speech column copies the text row its alignment picks); these
pins check that selection against the product itself, evaluated by numpy in
float64 where it is exact, against hand-derived grids, and against planted
mistakes.
"""
from __future__ import annotations

import ctypes
import json
import os
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")


def _product(path, h):
    """path^T @ h in float64 (exact here: one nonzero term per column)."""
    return np.matmul(path.transpose(0, 2, 1).astype(np.float64), h.astype(np.float64))


def _normal_text(B, T, C, seed):
    st = synth.Stream(seed)
    h = st.normal_f32(B * T * C).reshape(B, T, C)
    h[h == 0] = 1.0  # no signed zeros: the float64 product would turn -0 into +0
    return h


@pytest.mark.parametrize("name,C", [("iid-b4-t32-s128", 1), ("tts-b16-t128-s512", 192), ("tts-b32-t256-s1024", 7)])
def test_equals_path_times_text(name, C):
    value, tx, ty = synth.generate(name)
    path, _, _ = oracle.mas(value, tx, ty)
    h = _normal_text(len(tx), value.shape[1], C, seed=5)
    out = oracle.expand_text(path, h)
    assert out.dtype == np.float32 and out.shape == (len(tx), value.shape[2], C)
    assert np.array_equal(out, _product(path, h).astype(np.float32))


@pytest.mark.parametrize("dtype,hi", [(np.uint8, 256), (np.uint16, 1 << 16), (np.uint32, 1 << 32), (np.uint64, 1 << 53)])
def test_integer_elements_of_every_width(dtype, hi):
    """Integers below 2^53 are exact in float64, so the product pins the
    selection for every element width (2 bytes covers bf16 and fp16 bit
    patterns, 8 bytes fp64)."""
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    path, _, _ = oracle.mas(value, tx, ty)
    B, T, S = path.shape
    rng = np.random.default_rng(11)
    h = rng.integers(0, hi, size=(B, T, 5), dtype=np.uint64).astype(dtype)
    out = oracle.expand_text(path, h)
    assert out.dtype == dtype
    assert np.array_equal(out.astype(np.float64), _product(path, h))


@pytest.mark.parametrize("case", [c for c in json.load(open(GOLDEN))["cases"] if "text_grid" in c],
                         ids=lambda c: c["name"])
def test_hand_derived_grids(case):
    v = np.array([[np.nan if x == "nan" else float(x) for x in row] for row in case["value"]], dtype=np.float32)
    path, _, _ = oracle.mas(v[None], [case["t_x"]], [case["t_y"]])
    h = np.array(case["text"], dtype=np.float32)[None]
    out = oracle.expand_text(path, h)
    assert np.array_equal(out[0], np.array(case["text_grid"], dtype=np.float32))


def test_padding_and_invalid_items_are_zero():
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    tx, ty = tx.copy(), ty.copy()
    tx[0], ty[1], tx[2], ty[2] = 0, 0, 100, 50
    path, _, status = oracle.mas(value, tx, ty)
    h = _normal_text(16, 128, 3, seed=2)
    out = oracle.expand_text(path, h)
    for b in range(16):
        if status[b] != oracle.ITEM_OK:
            assert (out[b] == 0).all()
        else:
            assert (out[b, ty[b]:] == 0).all() and (out[b, :ty[b]] != 0).all()


def test_selection_copies_signed_zeros_and_non_finite_values():
    """The selection reading: a column takes its text row as it is, bit for
    bit, including -0, infinities and NaN (the float product would give +0
    and NaN there)."""
    v = np.zeros((1, 3, 5), np.float32)
    path, _, _ = oracle.mas(v, [3], [5])
    h = np.array([[[-0.0, np.inf], [np.nan, -np.inf], [1.0, -0.0]]], np.float32)
    out = oracle.expand_text(path, h)
    rows = path[0].argmax(axis=0)
    assert out.view(np.uint32)[0].tolist() == h.view(np.uint32)[0][rows].tolist()


def test_not_a_mas_path_is_refused():
    path = np.zeros((1, 2, 3), np.uint8)
    path[0, :, 1] = 1
    with pytest.raises(ValueError):
        oracle.expand_text(path, np.ones((1, 2, 4), np.float32))


# ------------------------------------------------------------- mutation check
_MUTATIONS = {
    "row_after_the_selected": ("src = i;\n", "src = i + 1 < T ? i + 1 : i;\n"),
    "first_one_instead_of_the_one": ("          src = i;\n          ++ones;", "          if (src < 0) src = i;\n          ones = 1;"),
    "uncovered_column_copies_row_0": ("if (src < 0)\n        memset(dst, 0, row);", "if (src < 0)\n        memcpy(dst, h + (size_t)b * (size_t)T * row, row);"),
    "transposed_item_stride": ("memcpy(dst, h + ((size_t)b * (size_t)T + (size_t)src) * row, row);",
                               "memcpy(dst, h + ((size_t)src * (size_t)B + (size_t)b) * row, row);"),
}


def _variant_expand(so):
    lib = ctypes.CDLL(so)
    P, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.oracle_expand_text.argtypes = [P, P, i32, i32, i32, i32, i32, P]
    lib.oracle_expand_text.restype = ctypes.c_int

    def expand(path, h):
        path = np.ascontiguousarray(path)
        h = np.ascontiguousarray(h)
        B, T, S = path.shape
        out = np.empty((B, S, h.shape[2]), h.dtype)
        p = lambda a: a.ctypes.data_as(P)
        if lib.oracle_expand_text(p(path), p(h), B, T, S, h.shape[2], h.dtype.itemsize, p(out)) != 0:
            raise ValueError("not a MAS path")
        return out

    return expand


def _pins_pass(expand) -> bool:
    try:
        value, tx, ty = synth.generate("tts-b16-t128-s512")
        path, _, _ = oracle.mas(value, tx, ty)
        h = _normal_text(16, 128, 6, seed=9)
        assert np.array_equal(expand(path, h), _product(path, h).astype(np.float32))
        bad = np.zeros((1, 2, 3), np.uint8)
        bad[0, :, 1] = 1
        try:
            expand(bad, np.ones((1, 2, 4), np.float32))
            return False
        except ValueError:
            pass
        return True
    except AssertionError:
        return False


def test_pins_accept_the_oracle():
    assert _pins_pass(oracle.expand_text)


@pytest.mark.parametrize("mutation", sorted(_MUTATIONS))
def test_pins_catch_planted_mistakes(mutation):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "mas_oracle.c")).read()
    old, new = _MUTATIONS[mutation]
    assert src.count(old) == 1, mutation
    with tempfile.TemporaryDirectory() as d:
        c, so = os.path.join(d, "variant.c"), os.path.join(d, "variant.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.check_call(["gcc", *oracle.CFLAGS, c, "-o", so, "-lm"])
        assert not _pins_pass(_variant_expand(so)), f"pins did not detect mutation {mutation}"
