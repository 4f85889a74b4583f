"""Parity of the boosting-step calls with the oracle (Section 2, eq. 2 and the update).

- sb_gradients (softmax / sigmoid cross-entropy) against oracle.boost.gradients:
  G, the per-element hessians, the row means and the column norms, each within
  a bound derived from fp32 arithmetic (below); ragged tiles, chunks of
  columns, more tiles than blocks, extreme scores.
- sb_update_predictions against oracle.boost.update_predictions: bit-exact
  (both compute lr * v and the sum in fp64 and round once).
- sb_sketch_given_norms: bit-identical to sb_sketch when handed sb_sketch's
  own norms.
- The Booster loop against oracle.boost.boost for several rounds: the same
  trees (the split-identity rule, with the oracle following a near-tied
  device choice), leaf values and final scores within tolerance.

fp32 bound for the gradient pass.  Per row, p_j = exp(a_j - m) / sum_l exp(a_l - m)
is formed from fp32 differences (relative error 2^-24 of |a_j - m|), fp32
exponentials (a few ulp), and a sum of d terms with one rescale per 8
columns, so |p - p_exact| <= (d + 20 + 2 R) 2^-24 p with R = max_j |a_j - m|;
g and h add one rounding each, and the oracle's stored values one more.
Sigmoid: |s - s_exact| <= (|a| + 6) 2^-24 s (1 - s) + 2^-23 s.
Values in fp32's subnormal range carry an absolute error of a few 2^-149.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import boost as ob
from workloads import scores_and_targets

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from paper_2211_12858_amd import _lib as L  # noqa: E402
from paper_2211_12858_amd.driver import Booster, SplitSearch, workspace  # noqa: E402

U = 2.0 ** -24
SUB = 4 * 2.0 ** -149  # values below fp32's normal range carry absolute, not relative, rounding


def run_gradients(loss, F_T, target, want_hess=True, want_row=True, want_norms=True):
    d, n = F_T.shape
    Fd = gu.up(F_T)
    G = torch.full((d, n), float("nan"), dtype=torch.float32, device=gu.DEV)
    H = torch.full((d, n), float("nan"), dtype=torch.float32, device=gu.DEV) if want_hess else None
    hr = torch.full((n,), float("nan"), dtype=torch.float32, device=gu.DEV) if want_row else None
    n2 = torch.full((d,), float("nan"), dtype=torch.float64, device=gu.DEV) if want_norms else None
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_GRADIENTS, n=n, d=d), gu.DEV)
    labels = gu.up(target) if loss == "softmax" else None
    Y = gu.up(target) if loss == "sigmoid" else None
    L.sb_gradients(L.LOSS[loss], Fd, n, d, n, labels, Y, n, G, n, H, n, hr, n2, ws, ws.numel())
    gu.sync()
    out = [G.cpu().numpy()]
    out.append(H.cpu().numpy() if want_hess else None)
    out.append(hr.cpu().numpy() if want_row else None)
    out.append(n2.cpu().numpy() if want_norms else None)
    return out


def grad_tolerances(loss, F_T, target):
    """Per-element bounds for g and h, from the oracle's fp64 values and the scores."""
    F = F_T.T.astype(np.float64)
    if loss == "softmax":
        g, h = ob.softmax_ce_derivatives(F, target)
        z = F - F.max(axis=1, keepdims=True)
        p = np.exp(z) / np.exp(z).sum(axis=1, keepdims=True)
        R = np.abs(z).max(axis=1, keepdims=True)
        d = F.shape[1]
        tp = (d + 20 + 2 * R) * U * p
        tg = tp + 2 * U * np.abs(g) + SUB
        th = tp + 2 * U * h + SUB
    else:
        g, h = ob.sigmoid_bce_derivatives(F, target.T)
        s = 1.0 / (1.0 + np.exp(-F))
        ts = (np.abs(F) + 6) * U * s * (1 - s) + 2 * U * s
        tg = ts + 2 * U * np.abs(g) + SUB
        th = ts + 2 * U * h + SUB
    return g, h, tg, th


def check_gradients(loss, F_T, target):
    d, n = F_T.shape
    print("gradients case: %s d=%d n=%d" % (loss, d, n), flush=True)
    G, H, hr, n2 = run_gradients(loss, F_T, target)
    tgt = target if loss == "softmax" else target.T
    G_o, H_o, hr_o, n2_o = ob.gradients(loss, F_T.T, tgt)
    _, _, tg, th = grad_tolerances(loss, F_T, target)
    eg = np.abs(G.T.astype(np.float64) - G_o) / tg
    eh = np.abs(H.T.astype(np.float64) - H_o) / th
    assert eg.max() <= 1.0, ("G", eg.max())
    assert eh.max() <= 1.0, ("hess", eh.max())
    thr = th.mean(axis=1) + (d + 4) * U * hr_o
    assert np.all(np.abs(hr.astype(np.float64) - hr_o) <= thr), "row means"
    Gd = G_o.astype(np.float64)
    tn = ((2 * np.abs(Gd) + tg) * tg).sum(axis=0) + 1e-12 * n2_o
    assert np.all(np.abs(n2 - n2_o) <= tn), ("norms", np.abs(n2 - n2_o).max())
    return G, H, hr, n2


# d at and around each kernel boundary: rows held in registers for d <= 16,
# 32, 64, 104, the two-pass kernel above (ragged last column chunks)
@pytest.mark.parametrize("d", [1, 5, 16, 17, 32, 64, 100, 104, 105, 130, 257])
def test_softmax_gradients(d):
    F_T, y = scores_and_targets(3 * 256 + 77, d, "softmax", seed=d, scale=2.0)
    G, H, _, _ = check_gradients("softmax", F_T, y)
    if d > 1:
        assert np.abs(G.astype(np.float64).sum(axis=0)).max() < (d + 24) * U


@pytest.mark.parametrize("d", [1, 8, 33, 130])
def test_sigmoid_gradients(d):
    F_T, Y = scores_and_targets(5 * 256 + 3, d, "sigmoid", seed=100 + d, scale=3.0)
    check_gradients("sigmoid", F_T, Y)


def test_gradients_many_tiles_per_block():
    # more 256-row tiles than the 2048 blocks of the grid: blocks loop over tiles
    F_T, y = scores_and_targets(2048 * 256 + 1000, 3, "softmax", seed=7)
    check_gradients("softmax", F_T, y)


def test_gradients_extreme_scores():
    F_T, y = scores_and_targets(1000, 6, "softmax", seed=8, scale=40.0)
    check_gradients("softmax", F_T, y)
    F_T, y = scores_and_targets(1000, 120, "softmax", seed=11, scale=40.0)
    check_gradients("softmax", F_T, y)
    F_T, Y = scores_and_targets(1000, 6, "sigmoid", seed=9, scale=40.0)
    check_gradients("sigmoid", F_T, Y)


def test_gradients_optional_outputs_and_determinism():
    F_T, y = scores_and_targets(3000, 12, "softmax", seed=10)
    G1, _, _, n1 = run_gradients("softmax", F_T, y, want_hess=False, want_row=False)
    G2, H2, _, n2 = run_gradients("softmax", F_T, y)
    assert np.array_equal(G1.view(np.uint32), G2.view(np.uint32))
    assert np.array_equal(n1.view(np.uint64), n2.view(np.uint64))
    G3, _, _, n3 = run_gradients("softmax", F_T, y, want_norms=False)
    assert np.array_equal(G3.view(np.uint32), G2.view(np.uint32))


@pytest.mark.parametrize("n_leaves,d", [(64, 100), (8, 3), (4096, 2), (300, 17)])
def test_update_predictions_bit_exact(n_leaves, d):
    rng = np.random.default_rng(n_leaves + d)
    n = 20000
    F_T = rng.standard_normal((d, n)).astype(np.float32)
    leaf_of = rng.integers(0, n_leaves, n)
    row_idx = np.argsort(leaf_of, kind="stable").astype(np.int32)
    leaf_off = np.concatenate([[0], np.cumsum(np.bincount(leaf_of, minlength=n_leaves))]).astype(np.int32)
    V = rng.standard_normal((n_leaves, d)) * 3.0
    Fd = gu.up(F_T)
    Vd = gu.up(np.ascontiguousarray(V))
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_UPDATE_PREDICTIONS, n=n), gu.DEV)
    L.sb_update_predictions(Fd, n, d, n, gu.up(row_idx), gu.up(leaf_off), n_leaves, Vd, d, 0.1, ws, ws.numel())
    gu.sync()
    want = ob.update_predictions(F_T.T, row_idx, leaf_off, V, 0.1)
    assert np.array_equal(Fd.cpu().numpy().T.view(np.uint32), want.view(np.uint32))


# The fused update + derivatives against the two calls it stands for, bit for
# bit: the one-pass kernel (softmax, d <= 104, <= 256 leaves whose lr * V
# table fits 64 KB) at each register-kernel width and ragged tiles, and the
# two-call route (sigmoid, d > 104, wider tables, more leaves).
@pytest.mark.parametrize("loss,d,n_leaves,n", [
    ("softmax", 1, 1, 1000), ("softmax", 5, 64, 3 * 256 + 77), ("softmax", 17, 3, 2000), ("softmax", 33, 64, 2500),
    ("softmax", 64, 100, 1500), ("softmax", 100, 64, 2048 * 256 + 1000), ("softmax", 104, 78, 5000),
    ("softmax", 100, 82, 3000), ("softmax", 105, 64, 3000), ("softmax", 16, 300, 3000), ("sigmoid", 8, 64, 3000),
])
def test_update_and_gradients_bit_exact(loss, d, n_leaves, n):
    print("update+gradients case: %s d=%d leaves=%d n=%d" % (loss, d, n_leaves, n), flush=True)
    rng = np.random.default_rng(d * 1000 + n_leaves)
    F_T = (rng.standard_normal((d, n)) * 2.0).astype(np.float32)
    tgt = rng.integers(0, d, n).astype(np.int32) if loss == "softmax" else \
        (rng.random((d, n)) < 0.3).astype(np.uint8)
    leaf_of = rng.integers(0, n_leaves, n)
    row_idx = np.argsort(leaf_of, kind="stable").astype(np.int32)
    leaf_off = np.concatenate([[0], np.cumsum(np.bincount(leaf_of, minlength=n_leaves))]).astype(np.int32)
    V = np.ascontiguousarray(rng.standard_normal((n_leaves, d)) * 3.0)
    lr = 0.1
    labels = gu.up(tgt) if loss == "softmax" else None
    Y = gu.up(tgt) if loss == "sigmoid" else None
    ri, lo, Vd = gu.up(row_idx), gu.up(leaf_off), gu.up(V)

    def outputs():
        G = torch.full((d, n), float("nan"), dtype=torch.float32, device=gu.DEV)
        H = torch.full((d, n), float("nan"), dtype=torch.float32, device=gu.DEV)
        hr = torch.full((n,), float("nan"), dtype=torch.float32, device=gu.DEV)
        n2 = torch.full((d,), float("nan"), dtype=torch.float64, device=gu.DEV)
        return G, H, hr, n2

    # the two calls
    F1 = gu.up(F_T)
    G1, H1, hr1, n21 = outputs()
    wu = workspace(L.sb_workspace_bytes(L.SB_CALL_UPDATE_PREDICTIONS, n=n), gu.DEV)
    wg = workspace(L.sb_workspace_bytes(L.SB_CALL_GRADIENTS, n=n, d=d), gu.DEV)
    L.sb_update_predictions(F1, n, d, n, ri, lo, n_leaves, Vd, d, lr, wu, wu.numel())
    L.sb_gradients(L.LOSS[loss], F1, n, d, n, labels, Y, n, G1, n, H1, n, hr1, n21, wg, wg.numel())
    # the fused call, twice (its workspace keeps nothing between calls)
    wf = workspace(L.sb_workspace_bytes(L.SB_CALL_UPDATE_AND_GRADIENTS, n=n, d=d), gu.DEV)
    for _ in range(2):
        F2 = gu.up(F_T)
        G2, H2, hr2, n22 = outputs()
        L.sb_update_and_gradients(L.LOSS[loss], F2, n, d, n, ri, lo, n_leaves, Vd, d, lr, labels, Y, n, G2, n, H2, n,
                                  hr2, n22, wf, wf.numel())
        gu.sync()
        for a, b in ((F1, F2), (G1, G2), (H1, H2), (hr1, hr2)):
            assert np.array_equal(a.cpu().numpy().view(np.uint32), b.cpu().numpy().view(np.uint32))
        assert np.array_equal(n21.cpu().numpy().view(np.uint64), n22.cpu().numpy().view(np.uint64))
    # and the update itself is the oracle's
    want = ob.update_predictions(F_T.T, row_idx, leaf_off, V, lr)
    assert np.array_equal(F2.cpu().numpy().T.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("kind", ["top_outputs", "random_sampling"])
def test_sketch_given_norms_matches_sketch(kind):
    from workloads import small_case
    case = small_case(5000, 4, 16, 12, seed=11, k=4)
    ss = SplitSearch(case.bins, 16, 4, 2, device=gu.DEV)
    G, h, u = gu.up(case.G_T), gu.up(case.h), gu.up(case.u, torch.float64)
    ss.sketch(kind, G, h, u=u)
    gu.sync()
    GH1, cols1, n2 = ss.gh(), ss.cols.cpu().numpy(), ss.norm2.clone()
    ss.GH.zero_()
    ss.sketch(kind, G, h, u=u, norm2_in=n2)
    gu.sync()
    assert np.array_equal(ss.cols.cpu().numpy(), cols1)
    assert np.array_equal(ss.gh().view(np.uint32), GH1.view(np.uint32))


@pytest.mark.parametrize("loss,kind,k", [("softmax", "random_sampling", 3), ("softmax", "identity", 5),
                                         ("sigmoid", "top_outputs", 2)])
def test_boosting_loop_matches_oracle(loss, kind, k):
    n, m, B, d, depth, rounds, lr = 6000, 5, 16, 5, 3, 4, 0.5
    rng = np.random.default_rng(12)
    bins = rng.integers(0, B, (n, m), dtype=np.uint8)
    if loss == "softmax":
        target = ((bins[:, 0] // 4 + (bins[:, 1] > 9)) % d).astype(np.int32)
        tgt_dev = gu.up(target)
    else:
        target = np.stack([(bins[:, j % m] > 5 + j) for j in range(d)], axis=0).astype(np.uint8)  # (d, n)
        tgt_dev = gu.up(target)
    u_rounds = rng.random((rounds, k))
    bst = Booster(bins, B, d, loss, kind, k, depth, lam=1.0, lr=lr, device=gu.DEV)
    bst.set_target(tgt_dev)
    trees, Vs = [], []
    for r in range(rounds):
        bst.step(u=gu.up(u_rounds[r], torch.float64))
        gu.sync()
        trees.append(bst.ss.tree())
        Vs.append(bst.ss.V.cpu().numpy())
    F_gpu = bst.F.cpu().numpy().T

    def follow(r, level, j, f, b, s1, s2, S, valid):
        gf, gb = int(trees[r]["feature"][level][j]), int(trees[r]["bin"][level][j])
        if f < 0:
            assert gf == -1, (r, level, j)
            return f, b
        assert gf >= 0 and valid[gf, gb], (r, level, j)
        if (gf, gb) != (f, b):
            assert S[gf, gb] >= s1 * (1 - gu.TOL), (r, level, j, (gf, gb), (f, b))
        return gf, gb

    tgt_o = target if loss == "softmax" else target.T
    F_o, hist = ob.boost(bins, B, np.zeros((n, d), np.float32), tgt_o, loss, rounds, lr, kind, k, depth, 1.0,
                         u_rounds=u_rounds, choose=follow)
    for r in range(rounds):
        assert np.array_equal(trees[r]["row_idx"], hist[r]["row_idx"]), r
        assert np.array_equal(trees[r]["leaf_off"], hist[r]["leaf_off"]), r
        Vo = hist[r]["V"]
        assert np.allclose(Vs[r], Vo, rtol=1e-4, atol=1e-5 * np.abs(Vo).max()), (r, np.abs(Vs[r] - Vo).max())
    assert np.allclose(F_gpu, F_o, rtol=1e-4, atol=1e-5 * np.abs(F_o).max()), np.abs(F_gpu - F_o).max()
