"""Full-size parity on the headline workload, in the configuration bench.py times.

Workload mc2m_rs5:
- 2,000,000 rows, 100 features, 256 quantile bins;
- d = 100 softmax outputs;
- Random Sampling, k = 5;
- depth 6, lambda = 1.

The oracle cannot grow this tree within a test's time, so the checks are:
- the sketch, bit for bit, on all 2M x 6 values;
- properties of the row partition that hold at any size:
  - the leaves hold a permutation of the rows;
  - every leaf keeps ascending row order (stable partitions from the identity order);
  - each node's left child holds exactly its rows with bin <= threshold of the split feature, and the right child the others;
  - terminal nodes send everything left;
- the root and two sampled nodes per level, against the oracle on that node's own rows (which the properties above show are the right rows):
  - the chosen split by the split-identity rule;
  - its score within 1e-4;
- the root histograms of four sampled features from the histogram call, against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import make_inputs, workload

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from paper_2211_12858_amd import _lib as L  # noqa: E402
from paper_2211_12858_amd.driver import SplitSearch, workspace  # noqa: E402


@pytest.fixture(scope="module")
def grown():
    wl = workload("mc2m_rs5")
    inp = make_inputs(wl)
    ss = SplitSearch(inp.bins, wl.n_bins, wl.k, wl.depth, wl.lam, wl.min_child_weight, device=gu.DEV)
    ss.step(wl.kind, gu.up(inp.G_T), gu.up(inp.h), u=gu.up(inp.u, torch.float64))
    gu.sync()
    GH_o, cols_o, _, _ = oracle.sketch(wl.kind, inp.G, inp.h, wl.k, u=inp.u)
    return wl, inp, ss, ss.tree(), GH_o, cols_o


def node_rows(tree, depth, level, j):
    span = 1 << (depth - level)
    off = tree["leaf_off"]
    return tree["row_idx"][off[j * span]:off[(j + 1) * span]]


def test_fullsize_sketch_bit_exact(grown):
    wl, inp, ss, tree, GH_o, cols_o = grown
    assert np.array_equal(ss.cols.cpu().numpy(), cols_o)
    assert np.array_equal(ss.gh().view(np.uint32), GH_o.view(np.uint32))
    assert not ss.gh_padding().any()


def test_fullsize_partition_properties(grown):
    wl, inp, ss, tree, GH_o, _ = grown
    n, depth = wl.n, wl.depth
    off = tree["leaf_off"]
    rows = tree["row_idx"]
    assert off[0] == 0 and off[-1] == n and np.all(np.diff(off) >= 0)
    assert np.array_equal(np.sort(rows), np.arange(n, dtype=np.int32))
    for j in range(1 << depth):  # stable partitions from the identity order: every leaf ascending
        assert np.all(np.diff(node_rows(tree, depth, depth, j)) > 0), j
    for level in range(depth):
        for j in range(1 << level):
            r = node_rows(tree, depth, level, j)
            f, b = int(tree["feature"][level][j]), int(tree["bin"][level][j])
            left, right = node_rows(tree, depth, level + 1, 2 * j), node_rows(tree, depth, level + 1, 2 * j + 1)
            if f < 0:
                assert right.size == 0 and np.array_equal(left, r), (level, j)
                continue
            col = inp.bins[:, f]
            assert np.all(col[left] <= b) and np.all(col[right] > b), (level, j)
            assert left.size + right.size == r.size


def sampled_nodes(tree, depth, rng):
    out = [(0, 0)]
    for level in range(1, depth):
        sizes = [node_rows(tree, depth, level, j).size for j in range(1 << level)]
        big = int(np.argmax(sizes))
        other = int(rng.integers(0, 1 << level))
        out += [(level, big)] + ([(level, other)] if other != big else [])
    return out


def test_fullsize_sampled_splits(grown):
    wl, inp, ss, tree, GH_o, _ = grown
    rng = np.random.default_rng(7)
    for level, j in sampled_nodes(tree, wl.depth, rng):
        r = node_rows(tree, wl.depth, level, j)
        H = oracle.node_histograms(inp.bins, GH_o, r, wl.n_bins)
        S, valid = oracle.split_scores(H, wl.lam, wl.min_child_weight)
        f, b, s1, s2 = oracle.best_split(S, valid)
        gf, gb, gs = int(tree["feature"][level][j]), int(tree["bin"][level][j]), float(tree["score"][level][j])
        if f < 0:
            assert (gf, gb) == (-1, -1) and gs == -np.inf, (level, j)
            continue
        assert gf >= 0 and valid[gf, gb], (level, j)
        if s1 - s2 > gu.TOL * s1:
            assert (gf, gb) == (f, b), (level, j, (gf, gb), (f, b), s1, s2)
        else:
            assert S[gf, gb] >= s1 * (1 - gu.TOL), (level, j)
        assert abs(gs - S[gf, gb]) <= gu.TOL * s1, (level, j, gs, S[gf, gb])


def test_fullsize_root_histograms_sampled_features(grown):
    wl, inp, ss, tree, GH_o, _ = grown
    n, m, B, k, c = wl.n, wl.m, wl.n_bins, wl.k, wl.k + 1
    H = torch.full((1, m, c, B), float("nan"), dtype=torch.float64, device=gu.DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=n, m=m, n_bins=B, k=k, n_nodes=1), gu.DEV)
    off = gu.up(np.array([0, n], dtype=np.int32))
    L.sb_build_histograms(ss.bins4, n, None, 0, n, m, B, ss.GH, ss.ld_gh, k, ss.qexp, None, off, 1, None, 1, H, ws,
                          ws.numel())
    gu.sync()
    Hg = gu.host_layout(H.cpu().numpy())[0]
    qexp = ss.qexp.cpu().numpy()
    chan_max = np.abs(GH_o.astype(np.float64)).max(axis=0)
    ones = np.ones((n, 1), dtype=np.float32)
    for f in (0, 37, 64, 99):
        sub = np.ascontiguousarray(inp.bins[:, f:f + 1])
        rows = np.arange(n)
        Ho = oracle.node_histograms(sub, GH_o, rows, B)[0]
        counts = oracle.node_histograms(sub, ones, rows, B)[0][:, 0]
        mass = oracle.node_histograms(sub, np.abs(GH_o), rows, B)[0]
        ok1, ok2, worst = gu.hist_tolerance_ok(Hg[f], Ho, counts, qexp, mass, chan_max)
        assert ok1 and ok2, (f, worst)


def test_fullsize_leaf_values_sampled_leaves(grown):
    # leaf values of the full-size tree from the full G (eq. 3), in the
    # configuration bench.py times: unit hessians, all 64 leaves computed,
    # eight leaves (the largest, the smallest non-empty, six random) checked
    wl, inp, ss, tree, GH_o, _ = grown
    G_T = gu.up(inp.G_T)
    V = ss.leaf_values(G_T).cpu().numpy()
    gu.sync()
    off = tree["leaf_off"]
    sizes = np.diff(off)
    rng = np.random.default_rng(11)
    nonempty = np.flatnonzero(sizes > 0)
    pick = {int(np.argmax(sizes)), int(nonempty[np.argmin(sizes[nonempty])])}
    pick |= set(int(x) for x in rng.choice(len(sizes), 6, replace=False))
    assert np.all(V[sizes == 0] == 0)
    G = inp.G
    col_max = np.abs(inp.G_T).max(axis=1)
    for Lf in sorted(pick):
        rows = tree["row_idx"][off[Lf]:off[Lf + 1]].astype(np.int64)
        sub_idx = np.arange(rows.size, dtype=np.int32)
        Vo = oracle.leaf_values(G[rows], sub_idx, np.array([0, rows.size]), wl.lam)
        ok, worst = gu.leaf_value_error_ok(V[Lf:Lf + 1], Vo, G[rows], [sub_idx.astype(np.int64)], wl.lam,
                                           col_max=col_max)
        assert ok, (Lf, worst)


def _hist_report(label, Hg, Ho, counts, qexp, mass, chan_max):
    """Errors of one node's histograms against the oracle's: the fixed-point bound, the 1e-4 bar
    relative to max(|H|, cell mass) with and without the channel-maximum floor, and the plain
    relative error of the cells well above the quantisation noise."""
    half_q = np.ldexp(1.0, -(qexp.astype(np.int64) + 1))
    noise = counts[..., None] * half_q
    err = np.abs(Hg - Ho)
    fixed_ok = err <= noise + 1e-12 * mass
    scale = np.maximum(np.abs(Ho), mass)
    unfloored = err <= gu.TOL * scale
    floored = err <= gu.TOL * np.maximum(scale, chan_max)
    big = np.abs(Ho) > 1e4 * np.maximum(noise, 1e-300)
    rel_big = float((err[big] / np.abs(Ho[big])).max()) if big.any() else 0.0
    cells = err.size
    print("hist %-22s cells %8d | fixed-point bound %d | 1e-4 of max(|H|, mass): %d (%.4f%%) | with the "
          "channel-max floor: %d | max rel. error where |H| > 1e4 x noise: %.2e (%d cells)"
          % (label, cells, int(fixed_ok.sum()), int(unfloored.sum()), 100.0 * unfloored.mean(), int(floored.sum()),
             rel_big, int(big.sum())), flush=True)
    return fixed_ok.all(), floored.all(), unfloored


def test_fullsize_histograms_unfloored_report(grown):
    """All 100 root features, and the largest and a random node of levels 3
    and 5 built through sb_build_histograms on the tree's own rows, against
    the oracle: every cell within the fixed-point bound and the 1e-4 bar with
    the channel-maximum floor; the count of cells meeting 1e-4 of
    max(|H|, cell mass) without that floor is printed (run with -s)."""
    wl, inp, ss, tree, GH_o, _ = grown
    n, m, B, k, c = wl.n, wl.m, wl.n_bins, wl.k, wl.k + 1
    qexp = ss.qexp.cpu().numpy()
    chan_max = np.abs(GH_o.astype(np.float64)).max(axis=0)
    ones = np.ones((n, 1), dtype=np.float32)
    absGH = np.abs(GH_o)
    rng = np.random.default_rng(23)
    cases = [("root", 0, 0)]
    for level in (3, 5):
        sizes = [node_rows(tree, wl.depth, level, j).size for j in range(1 << level)]
        big = int(np.argmax(sizes))
        other = int(rng.choice([j for j in range(1 << level) if j != big and sizes[j] > 0]))
        cases += [("level %d node %d" % (level, big), level, big), ("level %d node %d" % (level, other), level, other)]
    total, passed = 0, 0
    for label, level, j in cases:
        H = torch.full((1, m, c, B), float("nan"), dtype=torch.float64, device=gu.DEV)
        ws = workspace(L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=n, m=m, n_bins=B, k=k, n_nodes=1), gu.DEV)
        if level == 0:
            rows = np.arange(n, dtype=np.int32)
            off = gu.up(np.array([0, n], dtype=np.int32))
            L.sb_build_histograms(ss.bins4, n, None, 0, n, m, B, ss.GH, ss.ld_gh, k, ss.qexp, None, off, 1, None, 1, H,
                                  ws, ws.numel())
        else:
            rows = node_rows(tree, wl.depth, level, j)
            off = gu.up(np.array([0, rows.size], dtype=np.int32))
            L.sb_build_histograms(None, 0, ss.rec, ss.ld_rec, n, m, B, ss.GH, ss.ld_gh, k, ss.qexp,
                                  gu.up(rows, torch.int32), off, 1, None, 1, H, ws, ws.numel())
        gu.sync()
        Hg = gu.host_layout(H.cpu().numpy())[0]
        Ho = oracle.node_histograms(inp.bins, GH_o, rows, B)
        counts = oracle.node_histograms(inp.bins, ones, rows, B)[..., 0]
        mass = oracle.node_histograms(inp.bins, absGH, rows, B)
        fixed_ok, floored_ok, unfloored = _hist_report(label, Hg, Ho, counts, qexp, mass, chan_max)
        assert fixed_ok and floored_ok, label
        total += unfloored.size
        passed += int(unfloored.sum())
    print("hist all sampled nodes: %d of %d cells (%.4f%%) within 1e-4 of max(|H|, mass) without the floor"
          % (passed, total, 100.0 * passed / total), flush=True)
