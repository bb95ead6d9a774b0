"""Independent numpy (fp64) checks used to pin the oracle.

Nothing here reuses oracle code: group membership is evaluated from the three
set definitions of Eq. 1 directly, code optimality by enumerating every level
of the group's grid, and order statistics by counting.
"""
from __future__ import annotations

import numpy as np


def eq1_membership(x: np.ndarray, thr) -> np.ndarray:
    """Group of each value from Eq. 1's three sets, asserting they partition x.

    Returns 0 (inner), 1 (middle), 2 (outer)."""
    lo_o, lo_i, hi_i, hi_o = (float(t) for t in thr)
    x = np.asarray(x, dtype=np.float64)
    g_o = (x < lo_o) | (hi_o < x)
    g_m = ((lo_o <= x) & (x < lo_i)) | ((hi_i < x) & (x <= hi_o))
    g_i = (lo_i <= x) & (x <= hi_i)
    hits = g_o.astype(int) + g_m.astype(int) + g_i.astype(int)
    assert np.all(hits == 1), "Eq. 1 sets must partition the values"
    return np.where(g_o, 2, np.where(g_m, 1, 0))


def shifted_magnitude(x: np.ndarray, grp: np.ndarray, thr) -> tuple[np.ndarray, np.ndarray]:
    """Eq. 4 shift (fp64): returns (|x - T_side|, side) with side 1 = upper."""
    lo_o, lo_i, hi_i, hi_o = (float(t) for t in thr)
    x = np.asarray(x, dtype=np.float64)
    side = np.where(grp == 2, x > hi_o, np.where(grp == 1, x > hi_i, x >= 0)).astype(int)
    shift = np.where(grp == 2, np.where(side == 1, hi_o, lo_o),
                     np.where(grp == 1, np.where(side == 1, hi_i, lo_i), 0.0))
    return np.abs(x - shift), side


def check_nearest_level(a: np.ndarray, c: np.ndarray, levels: int, rel_tol=2e-6):
    """c must select a level of the min-max grid over `a` that is nearest to each a.

    Ties within the fp32 rounding of the scale computation are accepted."""
    a = np.asarray(a, np.float64)
    if a.size == 0:
        return
    mn, mx = a.min(), a.max()
    if mx == mn:
        assert np.all(c == 0)
        return
    grid = mn + np.arange(levels + 1) * (mx - mn) / levels
    dist = np.abs(a[:, None] - grid[None, :])
    best = dist.min(axis=1)
    mine = dist[np.arange(a.size), c]
    assert np.all(mine <= best + rel_tol * (mx - mn)), (mine - best).max()
    assert c[np.argmin(a)] == 0 and c[np.argmax(a)] == levels


def order_stat_ok(values: np.ndarray, t: float, k: int, side: str) -> bool:
    """True iff t is the k-th (0-based) order statistic from `side` ('low' or 'high')."""
    v = np.asarray(values, np.float64)
    if side == "low":
        return (v < t).sum() <= k < (v <= t).sum()
    return (v > t).sum() <= k < (v >= t).sum()


# ---- group-count variants ----------------------------------------------------
def variant_membership(x: np.ndarray, thr8, n_out: int, n_in: int) -> np.ndarray:
    """Group of each value for the nested-interval variants, numbered from the inside
    out (0 = innermost, n_in = middle, n_in + n_out = outermost), from the interval
    definitions directly; asserts that the sets partition x.  Boundaries belong to the
    inner side, as in Eq. 1."""
    lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob = (float(t) for t in thr8)
    x = np.asarray(x, dtype=np.float64)
    inside = lambda lo, hi: (lo <= x) & (x <= hi)
    sets = []
    if n_in == 2:
        sets.append(inside(lo_ib, hi_ib))                            # innermost
        sets.append(inside(lo_ia, hi_ia) & ~inside(lo_ib, hi_ib))    # inner a
    elif n_in == 1:
        sets.append(inside(lo_ia, hi_ia))
    mid = inside(lo_oa, hi_oa) & (~inside(lo_ia, hi_ia) if n_in else True)
    sets.append(mid)
    if n_out == 2:
        sets.append(inside(lo_ob, hi_ob) & ~inside(lo_oa, hi_oa))    # outer a
        sets.append(~inside(lo_ob, hi_ob))                           # outer b
    else:
        sets.append(~inside(lo_oa, hi_oa))
    hits = sum(s.astype(int) for s in sets)
    assert np.all(hits == 1), "the variant's sets must partition the values"
    g = np.zeros(x.shape, int)
    for k, s in enumerate(sets):
        g[s] = k
    return g


def variant_shift(x: np.ndarray, grp: np.ndarray, thr8, n_out: int, n_in: int):
    """(|x - T|, side) with T the boundary on the value's side between its group and the
    next group inwards; the innermost group (and the middle without inner groups) is not
    shifted and its side is x >= 0."""
    lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob = (float(t) for t in thr8)
    x = np.asarray(x, dtype=np.float64)
    mid = n_in
    lo = np.zeros(x.shape)
    hi = np.zeros(x.shape)
    shifted = np.ones(x.shape, bool)
    for g in range(n_in + 1 + n_out):
        sel = grp == g
        if g == mid + 2:
            lo[sel], hi[sel] = lo_ob, hi_ob
        elif g == mid + 1:
            lo[sel], hi[sel] = lo_oa, hi_oa
        elif g == mid and n_in > 0:
            lo[sel], hi[sel] = lo_ia, hi_ia
        elif g == 1 and n_in == 2:
            lo[sel], hi[sel] = lo_ib, hi_ib
        else:
            shifted[sel] = False
    side = np.where(shifted, x > hi, x >= 0).astype(int)
    t = np.where(shifted, np.where(side == 1, hi, lo), 0.0)
    return np.abs(x - t), side
