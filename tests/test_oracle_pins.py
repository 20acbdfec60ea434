"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these compares the oracle with itself: brute-force enumeration of all
monotonic alignments, hand-derived cases, closed forms for the degenerate
shapes, exact-arithmetic characterisations of the tie rule, metamorphic
relations and masking invariances.  ``test_pins_catch_planted_mistakes``
recompiles the oracle with plausible mistakes and checks that these pins
reject each one.
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
from tests import _pins

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")


def _load_case(c):
    v = np.array([[np.nan if x == "nan" else float(x) for x in row] for row in c["value"]], dtype=np.float32)
    return v


def _one(v, tx, ty, neg=-np.inf, impl=None):
    T, S = v.shape
    fn = impl or oracle.mas
    path, score, status = fn(v[None], [tx], [ty], neg=neg)
    return path[0], score[0], status[0]


# ------------------------------------------------------------- golden cases
@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_derived_cases(case):
    v = _load_case(case)
    path, score, status = _one(v, case["t_x"], case["t_y"])
    assert status == oracle.ITEM_OK
    assert _pins.alignment_of(path, case["t_x"], case["t_y"]) == tuple(case["rows"])
    assert np.float32(score).tobytes() == np.float32(case["score"]).tobytes()
    assert not _pins.check_invariants(path[None], [case["t_x"]], [case["t_y"]])
    if "legacy_neg" in case:
        lp, ls, _ = _one(v, case["t_x"], case["t_y"], neg=case["legacy_neg"])
        assert _pins.alignment_of(lp, case["t_x"], case["t_y"]) == tuple(case["legacy_rows"])
        assert np.float32(ls) == np.float32(case["legacy_score"])


# ------------------------------------------------------------- row_start / durations
def _path_from_rows(rows, T, S):
    """The 0/1 alignment of one item built directly from A(j) (no oracle)."""
    p = np.zeros((1, T, S), np.uint8)
    for j, r in enumerate(rows):
        p[0, r, j] = 1
    return p


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_row_start_and_durations_hand_tables(case):
    """oracle.row_start and oracle.durations on paths built from the hand
    cases' rows, against tables counted by hand."""
    T, S = len(case["value"]), len(case["value"][0])
    p = _path_from_rows(case["rows"], T, S)
    rs = oracle.row_start(p, [case["t_x"]], [case["t_y"]])
    assert rs.shape == (1, T + 1) and rs[0].tolist() == case["row_start"]
    assert oracle.durations(p)[0].tolist() == case["durations"]


def test_row_start_invalid_items_and_padding():
    # invalid items: all-zero tables; a valid item in a wider padded slab
    p = np.zeros((3, 4, 9), np.uint8)
    for j, r in enumerate([0, 0, 1, 2, 2, 2]):
        p[2, r, j] = 1
    rs = oracle.row_start(p, [0, 5, 3], [4, 3, 6])
    assert rs[0].tolist() == [0] * 5 and rs[1].tolist() == [0] * 5
    assert rs[2].tolist() == [0, 2, 3, 6, 6]
    assert oracle.durations(p)[2].tolist() == [2, 1, 3, 0]


# ------------------------------------------------------------- brute force
def _all_pairs():
    return [(tx, ty) for tx in range(1, 6) for ty in range(tx, 11)]


def test_exhaustive_pair_count():
    assert len(_all_pairs()) == 40


def _check_bruteforce(v, tx, ty, impl=None):
    path, score, status = _one(v, tx, ty, impl=impl)
    assert status == oracle.ITEM_OK
    best, arg = _pins.brute_force(v, tx, ty)
    assert np.float32(score).tobytes() == np.float32(best).tobytes(), (tx, ty, score, best)
    a = _pins.alignment_of(path, tx, ty)
    assert _pins.path_sum_f32(v, a).tobytes() == np.float32(best).tobytes()
    assert a in arg
    if len(arg) == 1:
        assert a == arg[0]
    assert not _pins.check_invariants(path[None], [tx], [ty])


@pytest.mark.parametrize("seed", range(6))
def test_bruteforce_all_pairs_normal(seed):
    """All 40 (t_x <= 5, t_x <= t_y <= 10) pairs, N(0,1) values in a 5x10 slab."""
    st = synth.Stream(1000 + seed)
    for tx, ty in _all_pairs():
        v = st.normal_f32(50).reshape(5, 10)
        _check_bruteforce(v, tx, ty)


def test_bruteforce_tiny_workload():
    value, tx, ty = synth.generate("tiny-b8-t5-s10")
    path, score, status = oracle.mas(value, tx, ty)
    for b in range(value.shape[0]):
        if status[b] != oracle.ITEM_OK:
            continue
        best, arg = _pins.brute_force(value[b], int(tx[b]), int(ty[b]))
        assert score[b].tobytes() == np.float32(best).tobytes()
        assert _pins.alignment_of(path[b], int(tx[b]), int(ty[b])) in arg


def test_bruteforce_large_magnitudes():
    """Log-likelihood-scale values, where fp32 partial sums round."""
    st = synth.Stream(77)
    for tx, ty in _all_pairs():
        v = (st.normal_f32(50).reshape(5, 10) * np.float32(13.0) - np.float32(153.0)) * np.float32(1024.0)
        _check_bruteforce(v.astype(np.float32), tx, ty)


def test_bruteforce_subnormal_values():
    """Values on the subnormal scale (|v| ~ 1e-40): fp32 keeps them (no
    flush to zero), so the DP must still equal the brute force bit for bit."""
    st = synth.Stream(91)
    tiny = np.float32(2.0 ** -133)  # ~9.2e-41, subnormal
    for tx, ty in _all_pairs():
        v = (st.normal_f32(50).reshape(5, 10) * tiny).astype(np.float32)
        assert (np.abs(v[v != 0]) < np.float32(2.0 ** -126)).any()
        _check_bruteforce(v, tx, ty)


def test_bruteforce_partial_sums_cross_the_subnormal_range():
    """Integer multiples of 2^-140 up to about 3e-38: values on both sides of
    the smallest normal (2^-126), partial sums landing among the subnormals;
    every sum is exact, so the brute force is exact, and a flush to zero of
    any subnormal input or partial sum changes the result."""
    st = synth.Stream(92)
    q = np.float32(2.0 ** -140)
    hit = 0
    for tx, ty in _all_pairs():
        v = (st.randint(-40000, 40000, 50).astype(np.float32) * q).reshape(5, 10)
        _check_bruteforce(v, tx, ty)
        path, score, _ = _one(v, tx, ty)
        hit += bool(score != 0 and abs(score) < np.float32(2.0 ** -126))
    assert hit > 3  # some scores themselves are subnormal


# ------------------------------------------------------------- tie rule
@pytest.mark.parametrize("seed", range(4))
def test_tie_rule_lex_greatest_integer_inputs(seed):
    """Integer values in {-2..2}: sums are exact, ties are frequent, and the
    stay-on-tie backtrack must return the optimal alignment whose rows, read
    from the last column backwards, are lexicographically greatest."""
    st = synth.Stream(2000 + seed)
    n_ties = 0
    for tx, ty in _all_pairs():
        v = st.randint(-2, 2, 50).astype(np.float32).reshape(5, 10)
        path, score, _ = _one(v, tx, ty)
        best, arg = _pins.brute_force(v, tx, ty)
        n_ties += len(arg) > 1
        assert score == best
        assert _pins.alignment_of(path, tx, ty) == _pins.lex_greatest_reversed(arg), (tx, ty)
    assert n_ties > 5  # the rule was actually exercised


def test_tie_rule_workload_integer():
    value, tx, ty = synth.generate("tiny-int-b8-t5-s10")
    path, score, status = oracle.mas(value, tx, ty)
    for b in range(value.shape[0]):
        if status[b] != oracle.ITEM_OK:
            continue
        best, arg = _pins.brute_force(value[b], int(tx[b]), int(ty[b]))
        assert _pins.alignment_of(path[b], int(tx[b]), int(ty[b])) == _pins.lex_greatest_reversed(arg)


# ------------------------------------------------------------- closed forms
@pytest.mark.parametrize("n", [1, 2, 7, 64, 65, 300])
def test_square_is_identity(n):
    st = synth.Stream(n)
    v = st.normal_f32(n * (n + 3)).reshape(n, n + 3)
    path, score, _ = _one(v, n, n)
    assert _pins.alignment_of(path, n, n) == tuple(range(n))
    s = np.float32(v[0, 0])
    for i in range(1, n):
        s = np.float32(s + v[i, i])
    assert score.tobytes() == s.tobytes()


@pytest.mark.parametrize("ty", [1, 2, 33, 1000])
def test_single_text_row_is_prefix_sum(ty):
    st = synth.Stream(ty)
    v = st.normal_f32(2 * (ty + 1)).reshape(2, ty + 1)
    path, score, _ = _one(v, 1, ty)
    assert (path[0, :ty] == 1).all() and not path[0, ty:].any() and not path[1:].any()
    s = np.float32(v[0, 0])
    for j in range(1, ty):
        s = np.float32(s + v[0, j])
    assert score.tobytes() == s.tobytes()


def test_negative_zero_single_cell():
    v = np.array([[-0.0]], dtype=np.float32)
    _, score, _ = _one(v, 1, 1)
    assert score.tobytes() == np.float32(-0.0).tobytes()


def test_signed_zero_tie_takes_positive_zero():
    # t_x = 2, t_y = 3 has two alignments: rows [0,1,1] sums -0 + -0 + -0 = -0
    # and rows [0,0,1] sums -0 + +0 + -0 = +0.  In the order of IEEE 754-2019
    # maximum() +0 is the larger, so the forward max takes the diagonal at
    # (1, 2) (Q[1][1] = -0 below Q[0][1] = +0) and the backtrack steps there.
    v = np.array([[-0.0, 0.0, 7.0], [5.0, -0.0, -0.0]], dtype=np.float32)
    path, score, _ = _one(v, 2, 3)
    assert _pins.alignment_of(path, 2, 3) == (0, 0, 1)
    assert score.tobytes() == np.float32(0.0).tobytes()
    best, arg = _pins.brute_force(v, 2, 3)
    assert best.tobytes() == np.float32(0.0).tobytes() and arg == [(0, 0, 1)]


# ------------------------------------------------------------- metamorphic
def test_power_of_two_scaling():
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    p0, s0, _ = oracle.mas(value, tx, ty)
    for k in (-3, 5):
        scale = np.float32(2.0 ** k)
        p1, s1, _ = oracle.mas(value * scale, tx, ty)
        assert np.array_equal(p0, p1)
        assert (s0 * scale).tobytes() == s1.tobytes()


def test_integer_column_offsets():
    """Every alignment visits each column once, so adding c_j to column j
    shifts every path by sum(c_j): same path, score + sum(c_j) (exact ints)."""
    st = synth.Stream(5)
    B, T, S = 6, 24, 70
    v = st.randint(-3, 3, B * T * S).astype(np.float32).reshape(B, T, S)
    tx = st.randint(1, T, B)
    ty = np.array([int(st.randint(int(a), S)[0]) for a in tx], dtype=np.int32)
    c = st.randint(-50, 50, S).astype(np.float32)
    p0, s0, _ = oracle.mas(v, tx, ty)
    p1, s1, _ = oracle.mas(v + c[None, None, :], tx, ty)
    assert np.array_equal(p0, p1)
    for b in range(B):
        assert s1[b] == s0[b] + c[: ty[b]].sum()


# ------------------------------------------------------------- masking
def test_nan_poisoning_padding_triangle_and_band():
    value, tx, ty = synth.generate("tts-b16-t128-s512")
    p0, s0, st0 = oracle.mas(value, tx, ty)
    poisoned = value.copy()
    B, T, S = value.shape
    ii = np.arange(T)[:, None]
    jj = np.arange(S)[None, :]
    for b in range(B):
        a, c = int(tx[b]), int(ty[b])
        outside = (ii >= a) | (jj >= c)
        triangle = ii > jj
        band = ii < (a - c + jj)  # cannot reach (t_x-1, t_y-1)
        poisoned[b][outside | triangle | band] = np.nan
    p1, s1, st1 = oracle.mas(poisoned, tx, ty)
    assert np.array_equal(p0, p1) and s0.tobytes() == s1.tobytes() and np.array_equal(st0, st1)


def test_invalid_lengths_status_and_zero_slab():
    B, T, S = 7, 8, 12
    v = np.zeros((B, T, S), dtype=np.float32)
    tx = np.array([0, 3, 5, -1, 9, 3, 8], dtype=np.int32)
    ty = np.array([4, 0, 4, 5, 12, 13, 12], dtype=np.int32)
    path, score, status = oracle.mas(v, tx, ty)
    assert status.tolist() == [1, 1, 2, 3, 3, 3, 0]
    assert not path[:6].any()
    assert np.isneginf(score[:6]).all()
    assert not _pins.check_invariants(path, tx, ty)


# ------------------------------------------------------------- invariants at size
@pytest.mark.parametrize("name", ["iid-b4-t32-s128", "tts-b16-t128-s512", "tts-b32-t256-s1024"])
def test_invariants_at_workload_sizes(name):
    value, tx, ty = synth.generate(name)
    path, score, status = oracle.mas(value, tx, ty)
    assert (status == 0).all()
    assert not _pins.check_invariants(path, tx, ty)
    assert np.isfinite(score).all()
    dur = oracle.durations(path)
    assert (dur.sum(axis=1) == ty).all()


# ------------------------------------------------------------- mutation check
_MUTATIONS = {
    # (a tie flip in the forward select only swaps equal values, so it is not
    # a mistake; the tie that decides the path is the backtrack's)
    "backtrack_tie_flipped": ("below(QC(idx, j - 1), QC(idx - 1, j - 1))", "!below(QC(idx - 1, j - 1), QC(idx, j - 1))"),
    "dropped_value_term": ("QC(i, j) = (take_diag ? diag : stay) + QV(i, j);", "QC(i, j) = (take_diag ? diag : stay);"),
    "wrong_value_index": ("QC(i, j) = (take_diag ? diag : stay) + QV(i, j);", "QC(i, j) = (take_diag ? diag : stay) + QV(i, j - 1);"),
    "max_became_min": ("QC(i, j) = (take_diag ? diag : stay) + QV(i, j);", "QC(i, j) = (take_diag ? stay : diag) + QV(i, j);"),
    "first_row_not_summed": ("QC(0, j) = QC(0, j - 1) + QV(0, j);", "QC(0, j) = QV(0, j);"),
    "backtrack_compare_reversed": ("below(QC(idx, j - 1), QC(idx - 1, j - 1))", "below(QC(idx - 1, j - 1), QC(idx, j - 1))"),
    "signed_zero_order_dropped": ("return a < b || (a == 0.0f && b == 0.0f && signbit(a) && !signbit(b));", "return a < b;"),
    "diag_wrong_row": ("float diag = QC(i - 1, j - 1);", "float diag = QC(i - 1, j);"),
    "loop_bound_off_by_one": ("int32_t imax = j < tx - 1 ? j : tx - 1;", "int32_t imax = j - 1 < tx - 1 ? j - 1 : tx - 1;"),
    # what a flush-to-zero build (or a kernel compiled with denormals off) does
    "subnormals_flushed": ("QC(i, j) = (take_diag ? diag : stay) + QV(i, j);",
                           "{ float r_ = (take_diag ? diag : stay) + QV(i, j); "
                           "QC(i, j) = fabsf(r_) < 1.17549435e-38f ? 0.0f * r_ : r_; }"),
}


def _compile_variant(src: str, d: str) -> str:
    c = os.path.join(d, "variant.c")
    so = os.path.join(d, "variant.so")
    open(c, "w").write(src)
    subprocess.check_call(["gcc", *oracle.CFLAGS, c, "-o", so, "-lm"])
    return so


def _variant_mas(so):
    lib = ctypes.CDLL(so)
    P, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.oracle_mas_batch_neg.argtypes = [P, i32, i32, i32, P, P, ctypes.c_float, P, P, P]

    def mas(value, t_x, t_y, neg=-np.inf):
        value = np.ascontiguousarray(value, dtype=np.float32)
        B, T, S = value.shape
        tx = np.ascontiguousarray(t_x, dtype=np.int32)
        ty = np.ascontiguousarray(t_y, dtype=np.int32)
        path = np.empty((B, T, S), np.uint8)
        score = np.empty(B, np.float32)
        status = np.empty(B, np.int32)
        p = lambda a: a.ctypes.data_as(P)
        lib.oracle_mas_batch_neg(p(value), B, T, S, p(tx), p(ty), float(neg), p(path), p(score), p(status))
        return path, score, status

    return mas


def _pins_pass(mas) -> bool:
    """The brute-force, golden and tie-rule pins, run against an oracle build."""
    try:
        for case in json.load(open(GOLDEN))["cases"]:
            v = _load_case(case)
            path, score, _ = _one(v, case["t_x"], case["t_y"], impl=mas)
            assert _pins.alignment_of(path, case["t_x"], case["t_y"]) == tuple(case["rows"])
            assert np.float32(score).tobytes() == np.float32(case["score"]).tobytes()
        st = synth.Stream(31)
        q = np.float32(2.0 ** -140)
        for tx, ty in _all_pairs():
            v = st.normal_f32(50).reshape(5, 10)
            _check_bruteforce(v, tx, ty, impl=mas)
            vs = (st.randint(-40000, 40000, 50).astype(np.float32) * q).reshape(5, 10)
            _check_bruteforce(vs, tx, ty, impl=mas)
            vi = st.randint(-2, 2, 50).astype(np.float32).reshape(5, 10)
            path, score, _ = _one(vi, tx, ty, impl=mas)
            best, arg = _pins.brute_force(vi, tx, ty)
            assert score == best
            assert _pins.alignment_of(path, tx, ty) == _pins.lex_greatest_reversed(arg)
        return True
    except AssertionError:
        return False


def test_pins_accept_the_oracle():
    assert _pins_pass(lambda v, a, b, neg=-np.inf: oracle.mas(v, a, b, neg=neg))


@pytest.mark.parametrize("mutation", sorted(_MUTATIONS))
def test_pins_catch_planted_mistakes(mutation):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "mas_oracle.c")).read()
    old, new = _MUTATIONS[mutation]
    assert src.count(old) == 1, mutation
    with tempfile.TemporaryDirectory() as d:
        so = _compile_variant(src.replace(old, new), d)
        assert not _pins_pass(_variant_mas(so)), f"pins did not detect mutation {mutation}"
