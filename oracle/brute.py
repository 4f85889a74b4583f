"""Oracle: exact-rational brute force over candidate splits (test infrastructure only).

For tiny inputs only.  Each candidate split (feature f, threshold b) of a leaf
R is evaluated straight from the definition of the scoring function
(Section 2, eq. 4, with the single hessian column of Section 3's S_G): the
children are formed by the predicate bins[i, f] <= b over the rows themselves,
and S(child) = sum_t (sum_i GH[i,t])^2 / (sum_i h_i + lambda) is computed in
exact rational arithmetic from the stored (binary floating point) inputs.  No
histogram, prefix sum or floating-point rounding is involved, so this pins the
histogram path of ``split.py`` independently.
"""
from fractions import Fraction

import numpy as np


def _frac_matrix(GH):
    return [[Fraction(float(x)) for x in row] for row in np.asarray(GH)]


def exact_region_score(GHf, rows, lam):
    """S(R) in exact arithmetic; GHf is the Fraction matrix of GH."""
    if len(GHf) == 0:
        return Fraction(0)
    c = len(GHf[0])
    k = c - 1
    sums = [Fraction(0)] * c
    for i in rows:
        r = GHf[i]
        for t in range(c):
            sums[t] += r[t]
    num = sum((sums[t] * sums[t] for t in range(k)), Fraction(0))
    return num / (sums[k] + Fraction(lam))


def brute_best_split(bins, GH, rows, n_bins, lam, min_child_weight=0.0, GHf=None):
    """All candidate scores of one leaf and its best split, exactly.

    Returns (best, table) where table maps (f, b) -> (score Fraction, valid)
    and best = (f, b, score) chosen by (score desc, f asc, b asc), or
    (-1, -1, None) if no candidate is valid.
    """
    bins = np.asarray(bins)
    if GHf is None:
        GHf = _frac_matrix(GH)
    c = GH.shape[1]
    k = c - 1
    mcw = Fraction(float(min_child_weight))
    table = {}
    best = (-1, -1, None)
    for f in range(bins.shape[1]):
        for b in range(n_bins - 1):
            left = [i for i in rows if int(bins[i, f]) <= b]
            right = [i for i in rows if int(bins[i, f]) > b]
            hl = sum((GHf[i][k] for i in left), Fraction(0))
            hr = sum((GHf[i][k] for i in right), Fraction(0))
            s = exact_region_score(GHf, left, lam) + exact_region_score(GHf, right, lam)
            valid = hl > mcw and hr > mcw
            table[(f, b)] = (s, valid)
            if valid and (best[2] is None or s > best[2]):
                best = (f, b, s)
    return best, table


def brute_tree(bins, GH, depth, lam, n_bins, min_child_weight=0.0):
    """Depth-wise tree by brute force: per level the node list, exact best splits.

    Returns list over levels of lists of (rows, f, b, score) plus the final
    leaf row lists.  Terminal nodes send every row to the left child.
    """
    bins = np.asarray(bins)
    GHf = _frac_matrix(GH)
    segments = [list(range(bins.shape[0]))]
    levels = []
    for _ in range(depth):
        info = []
        nxt = []
        for rows in segments:
            (f, b, s), _ = brute_best_split(bins, GH, rows, n_bins, lam, min_child_weight, GHf)
            info.append((rows, f, b, s))
            if f < 0:
                nxt += [list(rows), []]
            else:
                nxt += [[i for i in rows if int(bins[i, f]) <= b], [i for i in rows if int(bins[i, f]) > b]]
        levels.append(info)
        segments = nxt
    return levels, segments
