"""Parity of sb_sketch_sparse_projection (Section 3.3 with a sparse Pi) with the oracle.

fp32 accumulation against the exact product, term by term in the order
(j, q): Higham's dot-product bound |fl(sum) - sum| <= gamma_c sum |terms|
with c = d * s terms at most and gamma_c = c u / (1 - c u), u = 2^-24, plus
one rounding of the stored value.  The hessian channel and the row padding
are exact; the exponents follow the documented rule on the stored sketch.
Rows of Pi with s = 1 entry take the sparse kernel, s = 2, 4 and 8 the
assembled dense Pi; both routes are covered.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import achlioptas_pi, small_case, sparse_jl_pi

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from paper_2211_12858_amd import _lib as L  # noqa: E402
from paper_2211_12858_amd.driver import workspace  # noqa: E402


def run_sparse(G_T, h, k, pi_col, pi_val, ld_gh=None):
    d, n = G_T.shape
    s = pi_col.shape[1]
    ld_gh = (k + 1 + 7) // 8 * 8 if ld_gh is None else ld_gh
    GH = torch.full((n, ld_gh), float("nan"), dtype=torch.float32, device=gu.DEV)
    qexp = torch.zeros(k + 1, dtype=torch.int32, device=gu.DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=k), gu.DEV)
    L.sb_sketch_sparse_projection(gu.up(G_T), n, d, n, gu.up(h), k, s, gu.up(np.ascontiguousarray(pi_col)),
                                  gu.up(np.ascontiguousarray(pi_val)), GH, ld_gh, qexp, ws, ws.numel())
    gu.sync()
    g = GH.cpu().numpy()
    return g[:, :k + 1], g[:, k + 1:], qexp.cpu().numpy()


def check(G_T, h, k, pi_col, pi_val, ld_gh=None):
    d, n = G_T.shape
    s = pi_col.shape[1]
    print("sparse case: n=%d d=%d k=%d s=%d" % (n, d, k, s), flush=True)
    GH, pad, qexp = run_sparse(G_T, h, k, pi_col, pi_val, ld_gh)
    G = G_T.T
    GH_o = oracle.sparse_projection(G, h, k, pi_col, pi_val)
    P = np.abs(oracle.sparse_pi_matrix(d, k, pi_col, pi_val))
    absprod = np.abs(G.astype(np.float64)) @ P
    u = 2.0 ** -24
    c = d * s
    gamma = c * u / (1 - c * u)
    err = np.abs(GH[:, :k].astype(np.float64) - GH_o[:, :k])
    assert np.all(err <= gamma * absprod + u * np.abs(GH_o[:, :k]) + 1e-30), float((err / (gamma * absprod + 1e-30)).max())
    assert np.array_equal(GH[:, k], h)
    assert not pad.any()
    assert np.array_equal(qexp, gu.qexp_rule(GH))


@pytest.mark.parametrize("s", [1, 2, 4, 8])
def test_sparse_jl(s):
    case = small_case(3 * 1024 + 333, 1, 2, 37, seed=s)
    pi_col, pi_val = sparse_jl_pi(37, 20, s, seed=s)
    check(case.G_T, case.h, 20, pi_col, pi_val)


def test_achlioptas_padded_rows():
    case = small_case(2500, 1, 2, 50, seed=5, h_kind="random")
    pi_col, pi_val = achlioptas_pi(50, 9, seed=5, s_max=8)
    assert (pi_col < 0).any()          # padding entries are present
    check(case.G_T, case.h, 9, pi_col, pi_val)


def test_two_passes_over_k_and_odd_stride():
    # k = 40 needs two 32-column passes; ld_gh = 41 leaves no padding
    case = small_case(1500, 1, 2, 70, seed=6)
    pi_col, pi_val = sparse_jl_pi(70, 40, 2, seed=6)
    check(case.G_T, case.h, 40, pi_col, pi_val, ld_gh=44)


def test_signed_permutation_is_exact_on_device():
    case = small_case(5000, 1, 2, 12, seed=7)
    perm = np.random.default_rng(7).permutation(12).astype(np.int32)
    sign = np.where(np.arange(12) % 3 == 0, -1.0, 1.0).astype(np.float32)
    GH, _, _ = run_sparse(case.G_T, case.h, 12, perm[:, None], sign[:, None])
    for j in range(12):
        assert np.array_equal(GH[:, perm[j]], sign[j] * case.G_T[j])


def test_repeated_columns_add_dense_route():
    # s = 4 goes through the assembled dense Pi (so does s = 2 below)
    case = small_case(3000, 1, 2, 5, seed=9)
    pi_col = np.array([[0, 0, 1, -1], [1, 1, 1, 2], [2, -1, -1, -1], [0, 2, 0, 2], [1, 0, 1, 0]], dtype=np.int32)
    pi_val = np.array([[0.5, 0.25, 1, 3], [1, 1, 2, -1], [2, 7, 7, 7], [1, 1, -0.5, 0.5], [-1, 0.5, 0.25, 2]],
                      dtype=np.float32)
    check(case.G_T, case.h, 3, pi_col, pi_val)


def test_repeated_columns_add():
    case = small_case(3000, 1, 2, 6, seed=8)
    pi_col = np.array([[0, 0], [1, 1], [2, -1], [0, 2], [1, 1], [2, 2]], dtype=np.int32)
    pi_val = np.array([[0.5, 0.25], [1, 1], [2, 7], [1, 1], [-1, 0.5], [0.125, 0.125]], dtype=np.float32)
    check(case.G_T, case.h, 3, pi_col, pi_val)
