"""Independent checks used to pin the oracle (and, through it, the GPU path).

Nothing here reuses the oracle's code: the brute force enumerates every
monotonic alignment directly from its definition (Super-MAS Sec. 2: one text
row per speech column, starting in the first row at the first column, ending
in the last row at the last column, the row never decreasing and growing by
at most one per column) and scores each one as the fp32 left-to-right sum of
its log-likelihoods.  Maximising that sum is what Algorithm 1 computes:
x -> fl(x + v) is monotone, so fl(max(a, b) + v) = max(fl(a + v), fl(b + v))
and by induction the dynamic programme's Q[t_x-1][t_y-1] equals the largest
fp32 path sum, bit for bit.  That also holds in the order IEEE 754-2019
maximum() uses (+0 above -0): fl(-0 + v) and fl(+0 + v) differ only for
v = -0, giving -0 and +0 in that same order.
"""
from __future__ import annotations

import itertools

import numpy as np


def enumerate_alignments(tx: int, ty: int):
    """Every monotonic alignment as a tuple A(0..ty-1) of row indices."""
    for steps in itertools.combinations(range(1, ty), tx - 1):
        a, row, k = [], 0, 0
        for j in range(ty):
            if k < len(steps) and steps[k] == j:
                row += 1
                k += 1
            a.append(row)
        yield tuple(a)


def path_sum_f32(v: np.ndarray, a) -> np.float32:
    """fp32 sum of v[a[j], j] over j ascending (round to nearest after each add)."""
    s = np.float32(v[a[0], 0])
    for j in range(1, len(a)):
        s = np.float32(s + np.float32(v[a[j], j]))
    return s


def above(a, b) -> bool:
    """a > b in the order IEEE 754-2019 maximum() uses: numeric, with +0
    above -0."""
    a, b = np.float32(a), np.float32(b)
    if a > b:
        return True
    return bool(a == 0 and b == 0 and not np.signbit(a) and np.signbit(b))


def brute_force(v: np.ndarray, tx: int, ty: int):
    """(best score, list of all maximising alignments), maximising in the
    order of `above` (ties: same numeric value and same sign of zero)."""
    best, arg = None, []
    for a in enumerate_alignments(tx, ty):
        s = path_sum_f32(v, a)
        if best is None or above(s, best):
            best, arg = s, [a]
        elif not above(best, s):
            arg.append(a)
    return best, arg


def lex_greatest_reversed(alignments):
    """The alignment whose row sequence read from the last column backwards is
    lexicographically greatest: the stay-on-tie backtrack picks exactly this
    one among exact-arithmetic optima."""
    return max(alignments, key=lambda a: tuple(reversed(a)))


def alignment_of(path_slab: np.ndarray, tx: int, ty: int):
    """Row index per column of a [T, S] 0/1 slab, for columns < ty."""
    return tuple(int(np.argmax(path_slab[:tx, j])) for j in range(ty))


def check_invariants(path: np.ndarray, t_x, t_y, status=None):
    """Path invariants of every item in a [B, T, S] u8 batch.

    Valid items: exactly one 1 per column j < t_y, none elsewhere; the row is
    non-decreasing in steps of 0 or 1; A(0) = 0 and A(t_y-1) = t_x-1; sum of
    ones = t_y.  Invalid items (0 < t_x <= t_y, t_x <= T, t_y <= S violated):
    an all-zero slab.  Returns a list of error strings (empty when valid).
    """
    B, T, S = path.shape
    errs = []
    for b in range(B):
        tx, ty = int(t_x[b]), int(t_y[b])
        slab = path[b]
        if not (0 < tx <= ty and tx <= T and ty <= S):
            if slab.any():
                errs.append(f"item {b}: invalid lengths but non-zero slab")
            continue
        if set(np.unique(slab).tolist()) - {0, 1}:
            errs.append(f"item {b}: values other than 0/1")
            continue
        if slab[tx:, :].any() or slab[:, ty:].any():
            errs.append(f"item {b}: ones outside the [t_x, t_y] extent")
        colsum = slab[:tx, :ty].sum(axis=0)
        if not (colsum == 1).all():
            errs.append(f"item {b}: column sums not all 1")
            continue
        rows = slab[:tx, :ty].argmax(axis=0)
        if rows[0] != 0 or rows[-1] != tx - 1:
            errs.append(f"item {b}: endpoints {rows[0]},{rows[-1]}")
        d = np.diff(rows)
        if ((d != 0) & (d != 1)).any():
            errs.append(f"item {b}: row steps outside {{0,1}}")
        if int(slab.sum()) != ty:
            errs.append(f"item {b}: {int(slab.sum())} ones, expected {ty}")
    return errs
