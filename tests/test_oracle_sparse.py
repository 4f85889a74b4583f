"""Pins for the sparse projections (Section 3.3 with other entry distributions;
sparse JL transforms named at the end of the proof of Prop. A.5).

- A signed permutation (k = d, one +-1 per row) reproduces G's columns exactly.
- E[Pi Pi^T] = I for both generators, so the sketched score is unbiased:
  Monte-Carlo mean of S_{G Pi}(R) against the exact S_G(R), as for the
  Gaussian projection.
- The generators: a sparse JL row has s distinct columns of +-1/sqrt(s)
  (squared row norm exactly 1); Achlioptas entries take 0 and +-sqrt(3/k)
  with frequencies 2/3, 1/6, 1/6 (chi-square).
- The row-sparse form: padding columns (-1) and repeated columns.
"""
import math

import numpy as np
from scipy import stats

import oracle
from workloads import achlioptas_pi, small_case, sparse_jl_pi


def _score(GH, rows, lam=1.0):
    k = GH.shape[1] - 1
    W = np.asarray(GH[rows], dtype=np.float64)
    g = W[:, :k].sum(axis=0)
    return float(g @ g / (W[:, k].sum() + lam))


def test_signed_permutation_is_exact():
    case = small_case(40, 1, 2, 6, seed=3)
    perm = np.array([3, 0, 5, 1, 4, 2])
    sign = np.array([1, -1, -1, 1, 1, -1], dtype=np.float32)
    GH = oracle.sparse_projection(case.G, case.h, 6, perm[:, None], sign[:, None])
    for j in range(6):
        assert np.array_equal(GH[:, perm[j]], sign[j] * case.G[:, j].astype(np.float64))
    assert np.array_equal(GH[:, 6], case.h.astype(np.float64))


def test_row_sparse_form_padding_and_repeats():
    pi_col = np.array([[0, -1], [2, 2], [1, 7]])
    pi_val = np.array([[0.5, 9.0], [1.0, 2.0], [-1.0, 4.0]])
    want = np.array([[0.5, 0, 0], [0, 0, 3.0], [0, -1.0, 0]])
    assert np.array_equal(oracle.sparse_pi_matrix(3, 3, pi_col, pi_val), want)


def test_sparse_jl_generator():
    pi_col, pi_val = sparse_jl_pi(50, 12, 3, seed=1)
    for j in range(50):
        assert len(set(pi_col[j])) == 3 and np.all((0 <= pi_col[j]) & (pi_col[j] < 12))
    P = oracle.sparse_pi_matrix(50, 12, pi_col, pi_val)
    assert np.allclose((P * P).sum(axis=1), 1.0, rtol=1e-7)
    assert set(np.round(np.abs(pi_val.ravel()) * math.sqrt(3), 6)) == {1.0}


def test_achlioptas_generator_frequencies():
    k = 30
    pi_col, pi_val = achlioptas_pi(400, k, seed=2, s_max=30)
    P = oracle.sparse_pi_matrix(400, k, pi_col, pi_val)
    a = math.sqrt(3.0 / k)
    vals = np.round(P.ravel() / a).astype(int)
    counts = np.array([(vals == 1).sum(), (vals == 0).sum(), (vals == -1).sum()])
    assert counts.sum() == P.size
    _, p = stats.chisquare(counts, P.size * np.array([1 / 6, 2 / 3, 1 / 6]))
    assert p > 1e-3


def _unbiased(make_pi):
    case = small_case(30, 1, 2, 5, seed=9)
    rows = np.arange(0, 30, 2)
    exact = _score(oracle.materialise(case.G, case.h, *oracle.identity_sketch(5)), rows)
    vals = np.array([_score(oracle.sparse_projection(case.G, case.h, 3, *make_pi(r)), rows) for r in range(6000)])
    se = vals.std() / math.sqrt(len(vals))
    assert abs(vals.mean() - exact) < 5 * se


def test_sparse_jl_is_unbiased():
    _unbiased(lambda r: sparse_jl_pi(5, 3, 1, seed=r))


def test_achlioptas_is_unbiased():
    _unbiased(lambda r: achlioptas_pi(5, 3, seed=r, s_max=3))


def test_planted_scale_mistake_is_caught():
    # a sparse JL without the 1/sqrt(s) scale is biased by a factor s
    case = small_case(30, 1, 2, 5, seed=9)
    rows = np.arange(0, 30, 2)
    exact = _score(oracle.materialise(case.G, case.h, *oracle.identity_sketch(5)), rows)
    vals = []
    for r in range(3000):
        c, v = sparse_jl_pi(5, 3, 2, seed=r)
        vals.append(_score(oracle.sparse_projection(case.G, case.h, 3, c, v * math.sqrt(2)), rows))
    vals = np.array(vals)
    assert abs(vals.mean() - exact) > 5 * vals.std() / math.sqrt(len(vals))
