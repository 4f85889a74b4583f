"""Pins for the leaf-value oracle (Section 2, "Finding the leaf values", eq. 3).

The expected values come from what the paper and mathematics fix, not from
the closed form the oracle implements:
- the leaf value minimises the leaf's second-order objective.  The objective
  is a convex quadratic, so a central difference gives its exact partial
  derivatives, and every one must vanish at the oracle's value;
- substituting the optimum back into the objective gives -S(R)/2, where S is
  the split-scoring function of eq. 4 (the derivation of eq. 4 in Section 2);
- d = 1 squared loss with lambda -> 0 is the textbook regression-tree leaf:
  the mean residual;
- the three hessian forms agree where they describe the same weights.
A mutation check plants plausible mistakes and shows the pins catch each.
"""
import numpy as np
import pytest

import oracle
from oracle import leaf as leaf_mod
from workloads import small_case


def _stationarity(G, rows, v, lam, hess=None, h=None, delta=0.5):
    """Largest |dQ/dv_j| at v, by central differences (exact for a quadratic up to rounding),
    relative to the scale of the objective's linear term."""
    worst = 0.0
    scale = np.abs(np.asarray(G, dtype=np.float64)[rows]).sum() + 1e-300
    for j in range(v.shape[0]):
        e = np.zeros_like(v)
        e[j] = delta
        dq = (oracle.leaf_objective(G, rows, v + e, lam, hess, h)
              - oracle.leaf_objective(G, rows, v - e, lam, hess, h)) / (2 * delta)
        worst = max(worst, abs(dq) / scale)
    return worst


def _leaves(n, n_leaves, seed, empty=()):
    """A random row grouping: row_idx groups rows by leaf (ascending inside a leaf)."""
    rng = np.random.default_rng(seed)
    leaf_of = rng.integers(0, n_leaves, n)
    for L in empty:
        leaf_of[leaf_of == L] = (L + 1) % n_leaves
    row_idx = np.argsort(leaf_of, kind="stable").astype(np.int32)
    leaf_off = np.zeros(n_leaves + 1, dtype=np.int32)
    leaf_off[1:] = np.cumsum(np.bincount(leaf_of, minlength=n_leaves))
    return row_idx, leaf_off


@pytest.mark.parametrize("form", ["per_element", "per_row", "none"])
def test_leaf_values_minimise_the_objective(form):
    rng = np.random.default_rng(11)
    case = small_case(300, 2, 4, 6, seed=3)
    G = case.G
    hess = rng.uniform(0.01, 0.3, G.shape).astype(np.float32) if form == "per_element" else None
    h = rng.uniform(0.05, 1.0, G.shape[0]).astype(np.float32) if form == "per_row" else None
    row_idx, leaf_off = _leaves(300, 8, seed=4)
    lam = 1.5
    V = oracle.leaf_values(G, row_idx, leaf_off, lam, hess=hess, h=h)
    for L, rows in enumerate(oracle.leaf_rows(row_idx, leaf_off)):
        assert _stationarity(G, rows, V[L], lam, hess, h) < 1e-12, L
        # convex: any move increases the objective
        q0 = oracle.leaf_objective(G, rows, V[L], lam, hess, h)
        for j in range(G.shape[1]):
            e = np.zeros(G.shape[1])
            e[j] = 1e-3
            assert oracle.leaf_objective(G, rows, V[L] + e, lam, hess, h) > q0
            assert oracle.leaf_objective(G, rows, V[L] - e, lam, hess, h) > q0


def test_optimum_gives_minus_half_the_split_score():
    # Substituting the leaf values into the objective yields eq. 4's S(R):
    # Q(v*) = -S(R) / 2 for the identity sketch with the same hessian weights.
    case = small_case(200, 2, 4, 5, seed=8, h_kind="random")
    row_idx, leaf_off = _leaves(200, 6, seed=9)
    lam = 1.0
    V = oracle.leaf_values(case.G, row_idx, leaf_off, lam, h=case.h)
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(5))
    for L, rows in enumerate(oracle.leaf_rows(row_idx, leaf_off)):
        q = oracle.leaf_objective(case.G, rows, V[L], lam, h=case.h)
        assert q == pytest.approx(-0.5 * oracle.sketch_score(GH, rows, lam), rel=1e-12, abs=1e-14)


def test_squared_loss_leaf_is_mean_residual():
    # d = 1, loss (a - y)^2 / 2: g = a - y, h = 1.  As lambda -> 0 the leaf value is
    # the mean of y - a over the leaf (least-squares regression tree).
    rng = np.random.default_rng(2)
    n = 1000
    a = rng.standard_normal(n)
    y = rng.standard_normal(n) * 3 + 1
    g = (a - y).astype(np.float32)[:, None]
    row_idx, leaf_off = _leaves(n, 5, seed=3)
    V = oracle.leaf_values(g, row_idx, leaf_off, 1e-12)
    for L, rows in enumerate(oracle.leaf_rows(row_idx, leaf_off)):
        mean_residual = float(np.mean(y[rows] - a[rows]))
        # g was stored in fp32: each residual carries up to 2^-24 relative rounding
        tol = 2.0 ** -23 * float(np.mean(np.abs(y[rows] - a[rows])))
        assert abs(V[L, 0] - mean_residual) <= tol + 1e-9 * abs(mean_residual)


def test_hessian_forms_agree_and_empty_leaf():
    case = small_case(120, 2, 4, 3, seed=5, h_kind="random")
    row_idx, leaf_off = _leaves(120, 7, seed=6, empty=(2, 5))
    assert leaf_off[3] == leaf_off[2] and leaf_off[6] == leaf_off[5]
    hess = np.repeat(case.h[:, None], 3, axis=1)
    V_row = oracle.leaf_values(case.G, row_idx, leaf_off, 2.0, h=case.h)
    V_el = oracle.leaf_values(case.G, row_idx, leaf_off, 2.0, hess=hess)
    assert np.array_equal(V_row, V_el)
    V_none = oracle.leaf_values(case.G, row_idx, leaf_off, 2.0)
    V_ones = oracle.leaf_values(case.G, row_idx, leaf_off, 2.0, h=np.ones(120, dtype=np.float32))
    assert np.array_equal(V_none, V_ones)
    assert np.all(V_none[2] == 0) and np.all(V_none[5] == 0)


def test_leaves_of_a_grown_tree():
    # the leaves of an oracle tree cover every row once; the weighted leaf values
    # give back the total gradient: sum_L (H_L + lambda) v_L = -sum_i g_i
    case = small_case(400, 4, 8, 4, seed=12)
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(4))
    tree = oracle.grow_tree(case.bins, GH, 3, 1.0, 8)
    segs = tree["segments"]
    row_idx = np.concatenate([np.asarray(s, dtype=np.int32) for s in segs])
    leaf_off = np.concatenate([[0], np.cumsum([len(s) for s in segs])]).astype(np.int32)
    assert np.array_equal(np.sort(row_idx), np.arange(400))
    V = oracle.leaf_values(case.G, row_idx, leaf_off, 1.0)
    counts = np.diff(leaf_off).astype(np.float64)
    tot = ((counts + 1.0)[:, None] * V).sum(axis=0)
    assert np.allclose(tot, -case.G.astype(np.float64).sum(axis=0), rtol=1e-12, atol=1e-12)


def test_leaf_pins_catch_planted_mistakes():
    """Plausible mistakes in the leaf values; the stationarity pin must fail for each."""
    rng = np.random.default_rng(13)
    case = small_case(200, 2, 4, 4, seed=14)
    hess = rng.uniform(0.01, 0.3, case.G.shape).astype(np.float32)
    row_idx, leaf_off = _leaves(200, 5, seed=15)
    lam = 1.0
    good = leaf_mod.leaf_values(case.G, row_idx, leaf_off, lam, hess=hess)

    def sign_flip():
        return -good

    def no_lambda():
        return leaf_mod.leaf_values(case.G, row_idx, leaf_off, 0.0, hess=hess)

    def row_count_instead_of_hessian():
        return leaf_mod.leaf_values(case.G, row_idx, leaf_off, lam)

    def transposed_hessian_columns():
        return leaf_mod.leaf_values(case.G, row_idx, leaf_off, lam, hess=hess[:, ::-1])

    def off_by_one_segments():
        off = leaf_off.copy()
        off[1:-1] += 1
        return leaf_mod.leaf_values(case.G, row_idx, off, lam, hess=hess)

    rows_of = oracle.leaf_rows(row_idx, leaf_off)
    for bad in (sign_flip, no_lambda, row_count_instead_of_hessian, transposed_hessian_columns,
                off_by_one_segments):
        V = bad()
        worst = max(_stationarity(case.G, rows, V[L], lam, hess) for L, rows in enumerate(rows_of))
        assert worst > 1e-6, bad.__name__
