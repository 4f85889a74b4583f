"""Full-size parity of the boosting-step calls and the projections, at the shapes bench.py times.

- Gradient pass, 2,000,000 rows x 100 softmax outputs: G and the hessians on
  2000 sampled rows (softmax is row-local) within the fp32 bound of
  tests/test_gpu_boost.py, and all 100 column norms against the oracle's.
- Update: bit-exact on the sampled rows.
- Leaf values with hessians formed from G and the labels, on a grown
  full-size tree: eight sampled leaves.
- Random Projections at 2,000,000 x 1000 -> 20: the dense product (matrix-core
  kernel) and sparse JL with s = 1 on 2000 sampled rows, against the exact
  product with the dot-product bound.
Inputs: seeded, generated on the host in parallel chunks.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from oracle import boost as ob
from workloads import make_inputs, sparse_jl_pi, workload

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from paper_2211_12858_amd import _lib as L  # noqa: E402
from paper_2211_12858_amd.driver import SplitSearch, workspace  # noqa: E402
from test_gpu_boost import grad_tolerances  # noqa: E402

U = 2.0 ** -24


def normal_cols(d, n, seed, scale=1.0):
    """(d, n) float32 N(0, scale^2), column by column from per-column generators."""
    out = np.empty((d, n), dtype=np.float32)

    def one(j):
        out[j] = np.random.default_rng([seed, 21, j]).standard_normal(n, dtype=np.float32) * np.float32(scale)
    with ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0)))) as pool:
        list(pool.map(one, range(d)))
    return out


@pytest.fixture(scope="module")
def scores():
    n, d = 2_000_000, 100
    F_T = normal_cols(d, n, seed=31, scale=2.0)
    y = np.random.default_rng(32).integers(0, d, n).astype(np.int32)
    return F_T, y


def test_fullsize_gradient_pass(scores):
    F_T, y = scores
    d, n = F_T.shape
    print("full-size gradients: n=%d d=%d" % (n, d), flush=True)
    Fd = gu.up(F_T)
    G = torch.empty((d, n), dtype=torch.float32, device=gu.DEV)
    H = torch.empty((d, n), dtype=torch.float32, device=gu.DEV)
    n2 = torch.empty(d, dtype=torch.float64, device=gu.DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_GRADIENTS, n=n, d=d), gu.DEV)
    L.sb_gradients(L.SB_LOSS_SOFTMAX_CE, Fd, n, d, n, gu.up(y), None, n, G, n, H, n, None, n2, ws, ws.numel())
    gu.sync()
    rows = np.sort(np.random.default_rng(33).choice(n, 2000, replace=False))
    Fs = np.ascontiguousarray(F_T[:, rows])
    G_o, H_o, _, _ = ob.gradients("softmax", Fs.T, y[rows])
    _, _, tg, th = grad_tolerances("softmax", Fs, y[rows])
    Gs = G[:, torch.from_numpy(rows).to(gu.DEV)].cpu().numpy().T
    Hs = H[:, torch.from_numpy(rows).to(gu.DEV)].cpu().numpy().T
    assert np.all(np.abs(Gs - G_o) <= tg), float((np.abs(Gs - G_o) / tg).max())
    assert np.all(np.abs(Hs - H_o) <= th), float((np.abs(Hs - H_o) / th).max())
    # the norms of the device's G against the oracle's norms of its own G: the
    # per-element bound summed over all rows (p <= 1, so |g| <= 1 and
    # |g_dev - g| <= (d + 20 + 2R) 2^-24 + 2^-23)
    G_all = ob.softmax_ce_derivatives(F_T.T, y)[0].astype(np.float32)
    n2_o = oracle.column_norms2(G_all)
    R = np.abs(F_T - F_T.max(axis=0, keepdims=True)).max()
    tol = 2 * (d + 20 + 2 * float(R)) * U + 2 * U
    bound = 2 * np.abs(G_all.astype(np.float64)).sum(axis=0) * tol + 1e-12 * n2_o
    assert np.all(np.abs(n2.cpu().numpy() - n2_o) <= bound)


def test_fullsize_update_bit_exact(scores):
    F_T, _ = scores
    d, n = F_T.shape
    rng = np.random.default_rng(34)
    leaf_of = rng.integers(0, 64, n)
    row_idx = np.argsort(leaf_of, kind="stable").astype(np.int32)
    leaf_off = np.concatenate([[0], np.cumsum(np.bincount(leaf_of, minlength=64))]).astype(np.int32)
    V = rng.standard_normal((64, d))
    Fd = gu.up(F_T)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_UPDATE_PREDICTIONS, n=n), gu.DEV)
    L.sb_update_predictions(Fd, n, d, n, gu.up(row_idx), gu.up(leaf_off), 64, gu.up(V), d, 0.01, ws, ws.numel())
    gu.sync()
    rows = np.sort(rng.choice(n, 2000, replace=False))
    got = Fd[:, torch.from_numpy(rows).to(gu.DEV)].cpu().numpy().T
    want = (F_T[:, rows].T.astype(np.float64) + 0.01 * V[leaf_of[rows]]).astype(np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_fullsize_leaf_values_from_loss():
    wl = workload("mc2m_rs5")
    inp = make_inputs(wl)
    ss = SplitSearch(inp.bins, wl.n_bins, wl.k, wl.depth, wl.lam, device=gu.DEV)
    G_T = gu.up(inp.G_T)
    ss.step(wl.kind, G_T, gu.up(inp.h), u=gu.up(inp.u, torch.float64))
    V = ss.leaf_values_from_loss("softmax", G_T, labels=gu.up(inp.y)).cpu().numpy()
    gu.sync()
    tree = ss.tree()
    off = tree["leaf_off"]
    sizes = np.diff(off)
    rng = np.random.default_rng(35)
    pick = sorted({int(np.argmax(sizes))} | set(int(x) for x in rng.choice(len(sizes), 7, replace=False)))
    col_max = np.abs(inp.G_T).max(axis=1)
    for Lf in pick:
        rows = tree["row_idx"][off[Lf]:off[Lf + 1]].astype(np.int64)
        if rows.size == 0:
            assert np.all(V[Lf] == 0)
            continue
        G = inp.G[rows]
        p = G.astype(np.float64)
        p[np.arange(rows.size), inp.y[rows]] += 1.0
        Hd = (p * (1.0 - p)).astype(np.float32)
        idx = np.arange(rows.size, dtype=np.int32)
        Vo = oracle.leaf_values(G, idx, np.array([0, rows.size]), wl.lam, hess=Hd)
        ok, worst = gu.leaf_value_error_ok(V[Lf:Lf + 1], Vo, G, [idx.astype(np.int64)], wl.lam, hess=Hd,
                                           col_max=col_max, hess_err=2.0 ** -22)
        assert ok, (Lf, worst)


@pytest.fixture(scope="module")
def projection_input():
    n, d, k = 2_000_000, 1000, 20
    return normal_cols(d, n, seed=41), n, d, k


def _check_projection_rows(GH, G_T, rows, Pi64, terms):
    Gs = G_T[:, rows].T.astype(np.float64)
    exact = Gs @ Pi64
    absprod = np.abs(Gs) @ np.abs(Pi64)
    gamma = terms * U / (1 - terms * U)
    err = np.abs(GH[:, :Pi64.shape[1]].astype(np.float64) - exact)
    assert np.all(err <= gamma * absprod + U * np.abs(exact) + 1e-30), float((err / (gamma * absprod)).max())


def test_fullsize_dense_projection(projection_input):
    G_T, n, d, k = projection_input
    print("full-size dense projection: n=%d d=%d k=%d" % (n, d, k), flush=True)
    Pi = (np.random.default_rng(42).standard_normal((d, k)) / np.sqrt(k)).astype(np.float32)
    ld_gh = 24
    GH = torch.empty((n, ld_gh), dtype=torch.float32, device=gu.DEV)
    qexp = torch.empty(k + 1, dtype=torch.int32, device=gu.DEV)
    h = np.ones(n, dtype=np.float32)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=k), gu.DEV)
    Gd = gu.up(G_T)
    L.sb_sketch(L.SB_SKETCH_RANDOM_PROJECTION, Gd, n, d, n, gu.up(h), k, None, gu.up(Pi), GH, ld_gh, None, None,
                None, qexp, ws, ws.numel())
    gu.sync()
    rows = np.sort(np.random.default_rng(43).choice(n, 2000, replace=False))
    GHs = GH[torch.from_numpy(rows).to(gu.DEV)].cpu().numpy()
    _check_projection_rows(GHs, G_T, rows, Pi.astype(np.float64), d)
    assert np.all(GHs[:, k] == 1.0) and not GHs[:, k + 1:].any()


def test_fullsize_sparse_projection(projection_input):
    G_T, n, d, k = projection_input
    pc, pv = sparse_jl_pi(d, k, 1, seed=44)
    ld_gh = 24
    GH = torch.empty((n, ld_gh), dtype=torch.float32, device=gu.DEV)
    qexp = torch.empty(k + 1, dtype=torch.int32, device=gu.DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=k), gu.DEV)
    L.sb_sketch_sparse_projection(gu.up(G_T), n, d, n, gu.up(np.ones(n, dtype=np.float32)), k, 1, gu.up(pc),
                                  gu.up(pv), GH, ld_gh, qexp, ws, ws.numel())
    gu.sync()
    rows = np.sort(np.random.default_rng(45).choice(n, 2000, replace=False))
    GHs = GH[torch.from_numpy(rows).to(gu.DEV)].cpu().numpy()
    _check_projection_rows(GHs, G_T, rows, oracle.sparse_pi_matrix(d, k, pc, pv), d)
