"""Full-size parity on the Random Projections workload (Section 3.3).

Workload mc2m_d1000_rp20:
- 2,000,000 rows, 100 features, 256 quantile bins;
- d = 1000 softmax outputs, Pi ~ N(0, 1/20) given as an input;
- Random Projections, k = 20 (21 channels: the row-per-lane histogram kernel);
- depth 6, lambda = 1.

G.Pi is accumulated in fp32 in the hardware's order, so the sketch is checked
against the exact product within the dot-product bound on a sample of
200,000 rows (all 2M rows hold h exactly).  The tree is then checked given the
device's own sketch, which fixes every split: partition properties at full
size, and the root and the largest node of every level against the oracle on
that node's rows and that sketch (split identity, score within 1e-4).
"""
import numpy as np
import pytest

import oracle
from workloads import make_inputs, workload

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from paper_2211_12858_amd.driver import SplitSearch  # noqa: E402


@pytest.fixture(scope="module")
def grown():
    wl = workload("mc2m_d1000_rp20")
    inp = make_inputs(wl)
    ss = SplitSearch(inp.bins, wl.n_bins, wl.k, wl.depth, wl.lam, wl.min_child_weight, device=gu.DEV)
    ss.step(wl.kind, gu.up(inp.G_T), gu.up(inp.h), Pi=gu.up(inp.Pi))
    gu.sync()
    return wl, inp, ss, ss.tree(), ss.gh()


def node_rows(tree, depth, level, j):
    span = 1 << (depth - level)
    off = tree["leaf_off"]
    return tree["row_idx"][off[j * span]:off[(j + 1) * span]]


def test_fullsize_rp_sketch_within_dot_product_bound(grown):
    wl, inp, ss, tree, GH_g = grown
    k, d = wl.k, wl.d
    assert np.array_equal(GH_g[:, k], inp.h)
    rows = np.sort(np.random.default_rng(21).choice(wl.n, 200_000, replace=False))
    G_rows = np.ascontiguousarray(inp.G_T[:, rows].T)
    GH_o = oracle.random_projection(G_rows, inp.h[rows], inp.Pi)
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    absprod = np.abs(G_rows.astype(np.float64)) @ np.abs(inp.Pi.astype(np.float64))
    err = np.abs(GH_g[rows, :k].astype(np.float64) - GH_o[:, :k])
    assert np.all(err <= gamma * absprod + u * np.abs(GH_o[:, :k]) + 1e-30)


def test_fullsize_rp_partition_properties(grown):
    wl, inp, ss, tree, GH_g = grown
    n, depth = wl.n, wl.depth
    off = tree["leaf_off"]
    rows = tree["row_idx"]
    assert off[0] == 0 and off[-1] == n and np.all(np.diff(off) >= 0)
    assert np.array_equal(np.sort(rows), np.arange(n, dtype=np.int32))
    for j in range(1 << depth):
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


def test_fullsize_rp_sampled_splits(grown):
    wl, inp, ss, tree, GH_g = grown
    for level in range(wl.depth):
        sizes = [node_rows(tree, wl.depth, level, j).size for j in range(1 << level)]
        j = int(np.argmax(sizes))
        r = node_rows(tree, wl.depth, level, j)
        H = oracle.node_histograms(inp.bins, GH_g, r, wl.n_bins)
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
