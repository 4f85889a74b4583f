"""Pins for the CPU oracle: values and properties fixed by the paper or by mathematics.

None of these tests compares the oracle with itself: each expected value is
hand-derived (tests/golden), exact rational brute force, a textbook identity,
a closed form, or a statistical property of the sketch distribution.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import brute
from workloads import small_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _gh(g, h=None):
    g = np.asarray(g, dtype=np.float32)
    h = np.ones(g.shape[0], dtype=np.float32) if h is None else np.asarray(h, dtype=np.float32)
    return np.concatenate([g, h[:, None]], axis=1)


# ---------------------------------------------------------------- worked examples
@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_worked_examples(case):
    bins = np.array(case["bins"], dtype=np.uint8)
    GH = _gh(case["g"])
    rows = np.arange(bins.shape[0])
    H = oracle.node_histograms(bins, GH, rows, case["n_bins"])
    S, valid = oracle.split_scores(H, 1.0)
    for f in range(bins.shape[1]):
        for b in range(case["n_bins"] - 1):
            want = case["scores"][f][b]
            if want is None:
                assert not valid[f, b]
            else:
                assert valid[f, b]
                assert S[f, b] == pytest.approx(float(Fraction(want)), rel=1e-15)
    f, b, s1, s2 = oracle.best_split(S, valid)
    assert (f, b) == tuple(case["best"][:2])
    assert s1 == pytest.approx(float(Fraction(case["best"][2])), rel=1e-15)
    if case["runner_up"] is None:
        assert s2 == -np.inf
    else:
        assert s2 == pytest.approx(float(Fraction(case["runner_up"])), rel=1e-15)
    # the brute force agrees exactly with the hand values
    (bf, bb, bs), table = brute.brute_best_split(bins, GH, list(rows), case["n_bins"], 1.0)
    assert (bf, bb) == tuple(case["best"][:2]) and bs == Fraction(case["best"][2])


# ---------------------------------------------------------------- sketch pins
def test_norms_match_exact_sum():
    rng = np.random.default_rng(5)
    G = (rng.standard_normal((300, 7)) * np.exp(rng.uniform(-20, 20, (300, 7)))).astype(np.float32)
    n2 = oracle.column_norms2(G)
    for j in range(7):
        exact = sum((Fraction(float(x)) ** 2 for x in G[:, j]), Fraction(0))
        assert abs(Fraction(n2[j]) - exact) <= exact * Fraction(1, 2 ** 50)


def test_norms_closed_form():
    G = np.empty((1000, 3), dtype=np.float32)
    G[:, 0] = 0.5
    G[:, 1] = -3.0
    G[:, 2] = 0.0
    assert list(oracle.column_norms2(G)) == [250.0, 9000.0, 0.0]


def test_top_outputs_order_and_ties():
    cols, scales = oracle.top_outputs(np.array([3.0, 5.0, 5.0, 1.0, 0.0]), 3)
    assert list(cols) == [1, 2, 0]
    assert list(scales) == [1.0, 1.0, 1.0]


def test_random_sampling_hand_example():
    # C = [1, 1, 4], total 4; x = u*4 = 0, 0.8, 1.0, 2.0, 3.96
    # i = first j with C_j > x: 0, 0, 2, 2, 2 (column 1 has zero norm: never drawn)
    n2 = np.array([1.0, 0.0, 3.0])
    cols, scales = oracle.random_sampling(n2, 5, np.array([0.0, 0.2, 0.25, 0.5, 0.99]))
    assert list(cols) == [0, 0, 2, 2, 2]
    s0 = np.float32(math.sqrt(4.0 / 5.0))      # 1/sqrt(k p_0), p_0 = 1/4
    s2 = np.float32(math.sqrt(4.0 / 15.0))     # 1/sqrt(k p_2), p_2 = 3/4
    assert list(scales) == [s0, s0, s2, s2, s2]


def test_random_sampling_all_zero():
    cols, scales = oracle.random_sampling(np.zeros(4), 3, np.array([0.1, 0.5, 0.9]))
    assert list(cols) == [-1, -1, -1] and list(scales) == [0.0, 0.0, 0.0]


def test_random_sampling_frequencies_chi2():
    rng = np.random.default_rng(11)
    n2 = rng.uniform(0, 5, 6)
    n2[3] = 0.0
    u = rng.random(30000)
    cols, _ = oracle.random_sampling(n2, len(u), u)
    counts = np.bincount(cols, minlength=6)
    p = n2 / n2.sum()
    assert counts[3] == 0
    keep = p > 0
    chi = stats.chisquare(counts[keep], p[keep] * len(u))
    assert chi.pvalue > 1e-4


def _region_score_sketch(GH, rows, lam=1.0):
    return oracle.sketch_score(GH, rows, lam)


def test_random_sampling_unbiased():
    # E[||G_k^T v||^2] = ||G^T v||^2 (Section 3.2): Monte Carlo over draws
    case = small_case(40, 1, 2, 6, seed=3)
    G, h = case.G, case.h
    rng = np.random.default_rng(4)
    rows = np.flatnonzero(rng.random(40) < 0.5)
    exact = _region_score_sketch(oracle.materialise(G, h, *oracle.identity_sketch(6)), rows)
    n2 = oracle.column_norms2(G)
    k = 2
    vals = []
    for _ in range(6000):
        cols, scales = oracle.random_sampling(n2, k, rng.random(k))
        vals.append(_region_score_sketch(oracle.materialise(G, h, cols, scales), rows))
    vals = np.array(vals)
    se = vals.std() / math.sqrt(len(vals))
    assert abs(vals.mean() - exact) < 5 * se + 1e-6 * exact


def test_random_projection_identity_pi():
    case = small_case(50, 1, 2, 4, seed=8)
    GH = oracle.random_projection(case.G, case.h, np.eye(4, dtype=np.float32))
    assert np.array_equal(GH[:, :4], np.asarray(case.G, dtype=np.float64))
    assert np.array_equal(GH[:, 4], case.h.astype(np.float64))


def test_random_projection_unbiased():
    # E[Pi Pi^T] = I for N(0, 1/k) entries, so E[S_{G Pi}(R)] = S_G(R) (Section 3.3)
    case = small_case(30, 1, 2, 5, seed=9)
    rows = np.arange(0, 30, 2)
    exact = _region_score_sketch(oracle.materialise(case.G, case.h, *oracle.identity_sketch(5)), rows)
    rng = np.random.default_rng(10)
    k = 3
    vals = np.array([_region_score_sketch(
        oracle.random_projection(case.G, case.h, rng.standard_normal((5, k)) / math.sqrt(k)), rows)
        for _ in range(6000)])
    se = vals.std() / math.sqrt(len(vals))
    assert abs(vals.mean() - exact) < 5 * se


def _all_subsets_errors(GH_full, GH_sk, n, lam=1.0):
    worst = 0.0
    for mask in range(1, 1 << n):
        rows = [i for i in range(n) if mask >> i & 1]
        worst = max(worst, abs(_region_score_sketch(GH_full, rows, lam) - _region_score_sketch(GH_sk, rows, lam)))
    return worst


@pytest.mark.parametrize("kind", ["top_outputs", "random_sampling", "random_projection"])
def test_lemma_a1_and_prop_a3(kind):
    # Lemma A.1: sup_R |S_G(R) - S_Gk(R)| <= ||G G^T - G_k G_k^T||_2 (unit hessian);
    # Prop. A.3: for Top Outputs the right side is <= sum of the dropped squared norms.
    n, d, k = 11, 6, 2
    case = small_case(n, 1, 2, d, seed=21)
    G64 = np.asarray(case.G, dtype=np.float64)
    GH_full = oracle.materialise(case.G, case.h, *oracle.identity_sketch(d))
    if kind == "random_projection":
        GH_sk = oracle.random_projection(case.G, case.h, case.Pi[:, :k] * math.sqrt(d / k))
    else:
        n2 = oracle.column_norms2(case.G)
        cols, scales = (oracle.top_outputs(n2, k) if kind == "top_outputs"
                        else oracle.random_sampling(n2, k, case.u[:k]))
        GH_sk = oracle.materialise(case.G, case.h, cols, scales)
    Gk = np.asarray(GH_sk[:, :k], dtype=np.float64)
    op = np.linalg.norm(G64 @ G64.T - Gk @ Gk.T, 2)
    err = _all_subsets_errors(GH_full, GH_sk, n)
    assert err <= op * (1 + 1e-9) + 1e-12
    if kind == "top_outputs":
        n2 = np.sort(oracle.column_norms2(case.G))[::-1]
        assert op <= n2[k:].sum() * (1 + 1e-9)


def test_top_outputs_k_equals_d_is_exact():
    # Prop. A.3 with k = d: the bound is an empty sum, so every split score is
    # unchanged (exact rational arithmetic over all candidates).
    case = small_case(24, 2, 5, 4, seed=2)
    rows = list(range(24))
    n2 = oracle.column_norms2(case.G)
    GH_to = oracle.materialise(case.G, case.h, *oracle.top_outputs(n2, 4))
    GH_id = oracle.materialise(case.G, case.h, *oracle.identity_sketch(4))
    _, t_to = brute.brute_best_split(case.bins, GH_to, rows, 5, 1.0)
    _, t_id = brute.brute_best_split(case.bins, GH_id, rows, 5, 1.0)
    assert t_to == t_id


def test_single_output_textbook_gain():
    # d = 1: S(b) = GL^2/(HL+lam) + GR^2/(HR+lam), the classic second-order gain.
    rng = np.random.default_rng(1)
    n, B = 60, 7
    bins = rng.integers(0, B, (n, 1), dtype=np.uint8)
    g = rng.standard_normal(n).astype(np.float32)
    hh = rng.uniform(0.5, 2.0, n).astype(np.float32)
    GH = _gh(g[:, None], hh)
    S, valid = oracle.split_scores(oracle.node_histograms(bins, GH, np.arange(n), B), 2.5)
    for b in range(B - 1):
        L = bins[:, 0] <= b
        GL, HL = math.fsum(g[L].astype(float)), math.fsum(hh[L].astype(float))
        GR, HR = math.fsum(g[~L].astype(float)), math.fsum(hh[~L].astype(float))
        assert S[0, b] == pytest.approx(GL * GL / (HL + 2.5) + GR * GR / (HR + 2.5), rel=1e-12)


# ---------------------------------------------------------------- histogram pins
def test_histogram_totals_and_subtraction_exact():
    # integer-valued inputs make fp64 sums exact, so the identities hold exactly
    rng = np.random.default_rng(3)
    n, m, B = 500, 4, 16
    bins = rng.integers(0, B, (n, m), dtype=np.uint8)
    GH = rng.integers(-50, 50, (n, 4)).astype(np.float32)
    GH[:, 3] = rng.integers(1, 4, n)
    rows = np.flatnonzero(rng.random(n) < 0.6)
    H = oracle.node_histograms(bins, GH, rows, B)
    tot = GH[rows].astype(np.float64).sum(axis=0)
    for f in range(m):
        assert np.array_equal(H[f].sum(axis=0), tot)
    left, right = oracle.partition(bins, rows, 2, 7)
    HL = oracle.node_histograms(bins, GH, left, B)
    HR = oracle.node_histograms(bins, GH, right, B)
    assert np.array_equal(HL + HR, H)


def test_histogram_matches_row_loop():
    case = small_case(80, 3, 5, 2, seed=6, h_kind="random")
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(2))
    rows = np.arange(0, 80, 3)
    H = oracle.node_histograms(case.bins, GH, rows, 5)
    for f in range(3):
        for b in range(5):
            for t in range(3):
                want = sum((Fraction(float(GH[i, t])) for i in rows if case.bins[i, f] == b), Fraction(0))
                assert abs(Fraction(H[f, b, t]) - want) <= Fraction(1, 2 ** 45)


# ---------------------------------------------------------------- scores / split search
@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_scores_match_brute_force(seed):
    case = small_case(40, 3, 6, 3, seed=seed, h_kind="random" if seed % 2 else "ones")
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(3))
    rows = np.arange(40)
    S, valid = oracle.split_scores(oracle.node_histograms(case.bins, GH, rows, 6), 1.0)
    (bf, bb, bs), table = brute.brute_best_split(case.bins, GH, list(rows), 6, 1.0)
    for (f, b), (s, v) in table.items():
        assert bool(valid[f, b]) == v
        assert S[f, b] == pytest.approx(float(s), rel=1e-12)
    f, b, s1, s2 = oracle.best_split(S, valid)
    assert (f, b) == (bf, bb)
    assert s2 == pytest.approx(float(brute_runner_up(table)), rel=1e-12)


def brute_runner_up(table):
    """Second-best valid exact score of a brute-force table (the best removed once; -inf if none)."""
    vals = sorted((s for s, v in table.values() if v), reverse=True)
    return vals[1] if len(vals) > 1 else -math.inf


def _runner_up_pins_hold(best_split):
    """The runner-up pins (hand-worked cases and exact brute force) for a given best_split."""
    for case in json.load(open(GOLDEN))["cases"]:
        bins = np.array(case["bins"], dtype=np.uint8)
        GH = _gh(case["g"])
        S, valid = oracle.split_scores(oracle.node_histograms(bins, GH, np.arange(bins.shape[0]), case["n_bins"]), 1.0)
        s2 = best_split(S, valid)[3]
        want = -math.inf if case["runner_up"] is None else float(Fraction(case["runner_up"]))
        if not (s2 == want or (math.isfinite(want) and abs(s2 - want) <= 1e-15 * abs(want))):
            return False
    for seed in (0, 1):
        case = small_case(40, 3, 6, 3, seed=seed, h_kind="random" if seed % 2 else "ones")
        GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(3))
        rows = np.arange(40)
        S, valid = oracle.split_scores(oracle.node_histograms(case.bins, GH, rows, 6), 1.0)
        _, table = brute.brute_best_split(case.bins, GH, list(rows), 6, 1.0)
        if best_split(S, valid)[3] != pytest.approx(float(brute_runner_up(table)), rel=1e-12):
            return False
    return True


def test_runner_up_pins_catch_planted_mistakes():
    """Plausible mistakes in the runner-up score of best_split each fail a runner-up pin."""
    assert _runner_up_pins_hold(oracle.best_split)

    def unmasked(S, valid):           # runner-up taken over invalid candidates too
        f, b, s1, _ = oracle.best_split(S, valid)
        rest = S.astype(np.float64).ravel().copy()
        if f >= 0:
            rest[f * S.shape[1] + b] = -np.inf
        return f, b, s1, float(rest.max()) if rest.size else -np.inf

    def ties_dropped(S, valid):       # every candidate equal to the best removed, not just the best one
        f, b, s1, _ = oracle.best_split(S, valid)
        flat = np.where(valid, S, -np.inf).ravel()
        rest = flat[flat < s1]
        return f, b, s1, float(rest.max()) if rest.size else -np.inf

    def same_feature_only(S, valid):  # runner-up searched within the best feature only
        f, b, s1, _ = oracle.best_split(S, valid)
        if f < 0:
            return f, b, s1, -np.inf
        row = np.where(valid[f], S[f], -np.inf).copy()
        row[b] = -np.inf
        return f, b, s1, float(row.max())

    def best_twice(S, valid):         # the best itself reported as runner-up
        f, b, s1, _ = oracle.best_split(S, valid)
        return f, b, s1, s1

    for bad in (unmasked, ties_dropped, same_feature_only, best_twice):
        assert not _runner_up_pins_hold(bad), bad.__name__


def test_partition_stable_and_terminal():
    case = small_case(50, 2, 4, 1, seed=7)
    rows = np.array([3, 9, 10, 22, 23, 31, 40, 49])
    left, right = oracle.partition(case.bins, rows, 1, 1)
    assert list(left) == [i for i in rows if case.bins[i, 1] <= 1]
    assert list(right) == [i for i in rows if case.bins[i, 1] > 1]
    l2, r2 = oracle.partition(case.bins, rows, -1, -1)
    assert list(l2) == list(rows) and len(r2) == 0


@pytest.mark.parametrize("seed,h_kind", [(0, "ones"), (1, "random")])
def test_tree_matches_brute_force(seed, h_kind):
    case = small_case(36, 3, 5, 2, seed=seed, h_kind=h_kind)
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(2))
    tree = oracle.grow_tree(case.bins, GH, 3, 1.0, 5)
    levels, leaves = brute.brute_tree(case.bins, GH, 3, 1.0, 5)
    for l, info in enumerate(levels):
        for j, (rows, f, b, s) in enumerate(info):
            assert list(tree["levels"][l][j]) == rows
            assert (tree["feature"][l][j], tree["bin"][l][j]) == (f, b)
            if s is not None:
                assert tree["score"][l][j] == pytest.approx(float(s), rel=1e-12)
    assert [list(s) for s in tree["segments"]] == leaves


# ---------------------------------------------------------------- mutation checks
def test_pins_catch_planted_mistakes(monkeypatch):
    """Plant plausible mistakes in the oracle; the brute-force pin must fail for each."""
    case = small_case(40, 3, 6, 3, seed=0)
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(3))
    rows = np.arange(40)
    _, table = brute.brute_best_split(case.bins, GH, list(rows), 6, 1.0)
    split_mod = oracle.split
    good = split_mod.split_scores

    def strict_prefix(H, lam, mcw=0.0):      # left = bins < b (off by one)
        Hs = np.concatenate([np.zeros_like(H[:, :1]), H[:, :-1]], axis=1)
        return good(Hs, lam, mcw)

    def no_lambda(H, lam, mcw=0.0):
        return good(H, 0.0 * lam + 1e-300, mcw)

    def swapped_sides(H, lam, mcw=0.0):       # right child takes its own hessian wrong
        k = H.shape[2] - 1
        H2 = H.copy()
        H2[:, :, k] = H[:, ::-1, k]
        return good(H2, lam, mcw)

    for bad in (strict_prefix, no_lambda, swapped_sides):
        S, valid = bad(oracle.node_histograms(case.bins, GH, rows, 6), 1.0)
        mismatch = any(abs(S[f, b] - float(s)) > 1e-9 * abs(float(s)) for (f, b), (s, v) in table.items())
        assert mismatch, bad.__name__
