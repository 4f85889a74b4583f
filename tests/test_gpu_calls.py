"""Per-call parity of the HIP path against the CPU oracle (through the C ABI).

Bars: sketch columns, scales, GH (Top Outputs, Random Sampling, identity),
partitions and build lists bit-exact; histograms within the fixed-point
bound and 1e-4 of the cell mass; chosen splits identical wherever the
oracle's top-two gap exceeds 1e-4 of the best score.
"""
import math

import numpy as np
import pytest

import oracle
from workloads import small_case, make_inputs, workload

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402


# ---------------------------------------------------------------- sketch
SKETCH_CASES = [
    # (n, d, k, kind, seed)
    (1, 3, 3, "identity", 0),
    (1000, 5, 5, "identity", 1),
    (4097, 20, 5, "top_outputs", 2),
    (4097, 20, 20, "top_outputs", 3),
    (70001, 100, 5, "random_sampling", 4),
    (5000, 7, 1, "random_sampling", 5),
    (33333, 50, 10, "top_outputs", 6),
    # more outputs than the selection holds in LDS (4096): norms read from
    # global memory; Top Outputs over 79 blocks of 64 columns
    (1000, 5000, 7, "top_outputs", 7),
    (1000, 5000, 3, "random_sampling", 8),
]


@pytest.mark.parametrize("n,d,k,kind,seed", SKETCH_CASES)
def test_sketch_bit_exact(n, d, k, kind, seed):
    case = small_case(n, 1, 2, d, seed=seed, h_kind="random", k=k)
    GH_g, cols_g, sc_g, n2_g, qexp_g, pad = gu.run_sketch(kind, case.G_T, case.h, k, u=case.u)
    GH_o, cols_o, sc_o, n2_o = oracle.sketch(kind, case.G, case.h, k, u=case.u)
    assert np.array_equal(cols_g, cols_o)
    assert np.array_equal(sc_g.view(np.uint32), sc_o.view(np.uint32))
    assert np.array_equal(GH_g.view(np.uint32), GH_o.view(np.uint32))
    np.testing.assert_allclose(n2_g, n2_o, rtol=1e-12, atol=0)
    assert np.array_equal(qexp_g, gu.qexp_rule(GH_o))
    assert not pad.any()  # the rows are written whole: padding floats are 0


@pytest.mark.parametrize("k", range(1, 24))
def test_sketch_every_width(k):
    # every sketch width the histogram calls take (k + 1 <= 24): the packing
    # kernel's per-width instantiations, odd row counts, bit for bit
    case = small_case(1031, 1, 2, 30, seed=200 + k, h_kind="random", k=k)
    GH_g, cols_g, sc_g, _, qexp_g, pad = gu.run_sketch("top_outputs", case.G_T, case.h, k)
    GH_o, cols_o, sc_o, _ = oracle.sketch("top_outputs", case.G, case.h, k)
    assert np.array_equal(cols_g, cols_o)
    assert np.array_equal(GH_g.view(np.uint32), GH_o.view(np.uint32))
    assert np.array_equal(qexp_g, gu.qexp_rule(GH_o))
    assert not pad.any()


def test_sketch_random_sampling_zero_gradients():
    n, d, k = 3000, 6, 4
    G_T = np.zeros((d, n), dtype=np.float32)
    h = np.ones(n, dtype=np.float32)
    GH_g, cols_g, sc_g, _, _, _ = gu.run_sketch("random_sampling", G_T, h, k, u=np.array([0.1, 0.5, 0.7, 0.99]))
    assert list(cols_g) == [-1] * k and list(sc_g) == [0.0] * k
    assert not GH_g[:, :k].any() and np.all(GH_g[:, k] == 1.0)


@pytest.mark.parametrize("kind,k,ld_gh", [("top_outputs", 5, 6), ("identity", 12, 16), ("random_projection", 3, 4),
                                         ("random_projection", 9, 11)])
def test_sketch_row_strides(kind, k, ld_gh):
    # tight, padded and odd row strides; padding floats are written as 0
    d = 12
    case = small_case(2049, 1, 2, d, seed=9, k=k)
    GH_g, _, _, _, _, pad = gu.run_sketch(kind, case.G_T, case.h, k, Pi=case.Pi, u=case.u, ld_gh=ld_gh)
    assert not pad.any()
    if kind != "random_projection":
        GH_o, _, _, _ = oracle.sketch(kind, case.G, case.h, k)
        assert np.array_equal(GH_g.view(np.uint32), GH_o.view(np.uint32))
    else:
        assert np.array_equal(GH_g[:, k], case.h)


# k = 13 leaves a partial group of four columns and d = 300 a second, partial
# block of staged Pi rows; k = 33 takes a second pass of one column
@pytest.mark.parametrize("n,d,k,seed", [(5000, 40, 5, 0), (20001, 200, 20, 1), (777, 3, 8, 2), (3001, 300, 13, 3),
                                        (2000, 40, 33, 4)])
def test_random_projection_error_bound(n, d, k, seed):
    # fp32 accumulation against the exact product: Higham's dot-product bound
    # |fl(x.y) - x.y| <= gamma_d |x|.|y| with gamma_d = d u / (1 - d u), u = 2^-24,
    # plus the final rounding u |x.y|.
    case = small_case(n, 1, 2, d, seed=seed, k=k)
    GH_g, _, _, _, qexp_g, _ = gu.run_sketch("random_projection", case.G_T, case.h, k, Pi=case.Pi)
    GH_o = oracle.random_projection(case.G, case.h, case.Pi)
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    absprod = np.abs(np.asarray(case.G, dtype=np.float64)) @ np.abs(case.Pi.astype(np.float64))
    err = np.abs(GH_g[:, :k].astype(np.float64) - GH_o[:, :k])
    assert np.all(err <= gamma * absprod + u * np.abs(GH_o[:, :k]) + 1e-30)
    assert np.array_equal(GH_g[:, k], case.h)
    assert np.array_equal(qexp_g, gu.qexp_rule(GH_g))


@pytest.mark.parametrize("k", range(1, 34))
def test_random_projection_every_width(k):
    # every column count of one 32-column pass and a second pass of one: the
    # vector kernel below 8 columns, the matrix-core kernel with 1 to 8 groups
    # of four columns (partial last groups), within the dot-product bound
    d = 37
    case = small_case(1500, 1, 2, d, seed=300 + k, k=k)
    GH_g, _, _, _, qexp_g, pad = gu.run_sketch("random_projection", case.G_T, case.h, k, Pi=case.Pi)
    GH_o = oracle.random_projection(case.G, case.h, case.Pi)
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    absprod = np.abs(np.asarray(case.G, dtype=np.float64)) @ np.abs(case.Pi.astype(np.float64))
    err = np.abs(GH_g[:, :k].astype(np.float64) - GH_o[:, :k])
    assert np.all(err <= gamma * absprod + u * np.abs(GH_o[:, :k]) + 1e-30)
    assert np.array_equal(GH_g[:, k], case.h)
    assert np.array_equal(qexp_g, gu.qexp_rule(GH_g))
    assert not pad.any()


# ---------------------------------------------------------------- histograms
def _segments(rng, n, n_nodes, empty_every=0):
    perm = rng.permutation(n).astype(np.int32)
    cuts = np.sort(rng.integers(0, n + 1, n_nodes - 1))
    off = np.concatenate([[0], cuts, [n]]).astype(np.int32)
    if empty_every:
        for j in range(0, n_nodes, empty_every):
            off[j + 1] = off[j]
        off = np.maximum.accumulate(off)
        off[-1] = n
    # rows inside each node sorted, as a stable partition leaves them
    for j in range(n_nodes):
        perm[off[j]:off[j + 1]] = np.sort(perm[off[j]:off[j + 1]])
    return perm, off


HIST_CASES = [
    # (n, m, B, k, n_nodes, build, seed)
    (1, 1, 2, 1, 1, False, 0),
    (10000, 10, 256, 5, 1, False, 1),       # tiny multiclass root
    (20000, 50, 64, 5, 1, False, 2),        # 50 features / 64 bins root
    (20000, 50, 64, 5, 8, True, 3),         # deeper level, smaller children only
    (30011, 100, 256, 5, 4, True, 4),       # five 20-feature slices, ragged tail
    (9000, 13, 256, 20, 16, True, 5),       # k=20 (21 channels)
    (12000, 31, 256, 10, 32, True, 6),      # k=10, many nodes, some empty
    (5000, 3, 7, 2, 2, False, 7),           # odd bins, m not a multiple of 4
    (7001, 100, 256, 5, 1, False, 8),       # five slices, root read straight from the data
    (20011, 24, 256, 5, 4, True, 9),        # a 16-feature slice and a thin slice of 8 (two cell copies)
    (6000, 7, 32, 3, 2, False, 10),         # only a thin slice of 8 features, root
    (9001, 40, 256, 4, 8, True, 11),        # two full slices and a thin slice of 8, odd channel count
    (4000, 2, 256, 5, 1, False, 12),        # thin slice of 2 features (eight copies)
    # channel groups of six: every group count and the partial last groups
    (6000, 17, 64, 6, 4, True, 13),         # k=6: two groups, the last of one channel
    (6000, 17, 64, 11, 1, False, 14),       # k=11: two full groups, root
    (5000, 9, 32, 12, 2, False, 15),        # k=12: three groups, the last of one channel
    (9000, 13, 256, 15, 8, True, 16),       # k=15: three groups, the last of four channels
    (7000, 20, 64, 17, 4, True, 17),        # k=17: three full groups
    (6000, 18, 128, 18, 2, True, 18),       # k=18: four groups, the last of one channel
    (6000, 18, 256, 23, 1, False, 19),      # k=23: 24 channels, the widest sketch taken
    # more slices than an XCD has CUs (one row group per XCD)
    (5000, 1000, 256, 5, 2, True, 20),      # 62 full slices and a padded one
    (3000, 333, 64, 15, 1, False, 21),      # 20 full slices and a padded one of 13 features, three channel groups
]


@pytest.mark.parametrize("n,m,B,k,n_nodes,build,seed", HIST_CASES)
def test_histograms(n, m, B, k, n_nodes, build, seed):
    rng = np.random.default_rng(seed)
    case = small_case(n, m, B, max(k, 2), seed=seed, h_kind="random" if seed % 2 else "ones", k=k)
    n2 = oracle.column_norms2(case.G)
    GH = oracle.materialise(case.G, case.h, *oracle.top_outputs(n2, k))
    qexp = gu.qexp_rule(GH)
    rows, off = _segments(rng, n, n_nodes, empty_every=3 if n_nodes >= 16 else 0)
    if build:
        build_list = np.array([2 * p + int(rng.integers(0, 2)) for p in range(n_nodes // 2)], dtype=np.int32)
        if n_nodes == 1:
            build_list = np.array([0], dtype=np.int32)
    else:
        build_list = None
    if seed == 8:  # positions are the rows (no row_idx), leading dimension padded
        rows = np.arange(n, dtype=np.int32)
        Hg = gu.host_layout(gu.run_hist(case.bins, GH, qexp, B, None, off, build_list, ld_pad=19).cpu().numpy())
    else:
        Hg = gu.host_layout(gu.run_hist(case.bins, GH, qexp, B, rows, off, build_list).cpu().numpy())
    todo = range(n_nodes) if build_list is None else build_list
    chan_max = np.abs(GH.astype(np.float64)).max(axis=0)
    ones = np.ones((n, 1), dtype=np.float32)
    for j in todo:
        node_rows = rows[off[j]:off[j + 1]]
        Ho = oracle.node_histograms(case.bins, GH, node_rows, B)
        counts = oracle.node_histograms(case.bins, ones, node_rows, B)[..., 0]
        mass = oracle.node_histograms(case.bins, np.abs(GH), node_rows, B)
        ok1, ok2, worst = gu.hist_tolerance_ok(Hg[j], Ho, counts, qexp, mass, chan_max)
        assert ok1 and ok2, (j, worst)
    if build_list is not None:  # untouched nodes keep their contents
        others = sorted(set(range(n_nodes)) - set(build_list.tolist()))
        assert np.isnan(Hg[others]).all()


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5, 6, 11, 12, 15, 17, 23])
@pytest.mark.parametrize("gathered", [False, True])
def test_histograms_quantised_extremes(k, gathered):
    # values whose fixed-point images reach the largest magnitude, 2^18
    # (1 - 2^-24 with exponent 18), mixed with both signs of small values, on
    # every channel count one 16-byte quantised row holds (c = 2 .. 6) and on
    # one, two, three and four such words per row with full and partial last
    # words (c = 7 .. 24)
    rng = np.random.default_rng(100 + k)
    n, m, B = 3001, 9, 16
    c = k + 1
    top = np.float32(1.0) - np.float32(2.0 ** -24)
    pool = np.array([top, -top, top / 2, -top / 2, 2.0 ** -19, -(2.0 ** -19), 0.0, 3e-5, -7e-6], dtype=np.float32)
    GH = pool[rng.integers(0, len(pool), size=(n, c))]
    GH[0, :] = top
    GH[1, :] = -top
    bins = rng.integers(0, B, size=(n, m), dtype=np.uint8)
    qexp = gu.qexp_rule(GH)
    assert (qexp == 18).all()
    rows = np.sort(rng.permutation(n)[: n - 500]).astype(np.int32) if gathered else np.arange(n, dtype=np.int32)
    off = np.array([0, len(rows)], dtype=np.int32)
    Hg = gu.host_layout(gu.run_hist(bins, GH, qexp, B, rows if gathered else None, off).cpu().numpy())
    Ho = oracle.node_histograms(bins, GH, rows, B)
    counts = oracle.node_histograms(bins, np.ones((n, 1), dtype=np.float32), rows, B)[..., 0]
    mass = oracle.node_histograms(bins, np.abs(GH), rows, B)
    ok1, ok2, worst = gu.hist_tolerance_ok(Hg[0], Ho, counts, qexp, mass, np.abs(GH.astype(np.float64)).max(axis=0))
    assert ok1 and ok2, worst


def test_histograms_identity_row_order_and_determinism():
    case = small_case(50000, 20, 256, 5, seed=11)
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(5))
    qexp = gu.qexp_rule(GH)
    off = np.array([0, 50000], dtype=np.int32)
    H1 = gu.run_hist(case.bins, GH, qexp, 256, None, off).cpu().numpy()
    H2 = gu.run_hist(case.bins, GH, qexp, 256, np.arange(50000, dtype=np.int32), off).cpu().numpy()
    assert np.array_equal(H1, H2)  # fixed-point sums do not depend on the order of the atomics


def test_subtraction_is_exact():
    rng = np.random.default_rng(12)
    n, m, B, k = 40000, 24, 128, 5
    case = small_case(n, m, B, k, seed=12, h_kind="random")
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(k))
    qexp = gu.qexp_rule(GH)
    rows, off = _segments(rng, n, 4)
    parent_off = off[[0, 2, 4]]
    Hp = gu.run_hist(case.bins, GH, qexp, B, rows, parent_off)
    build = np.array([1, 2], dtype=np.int32)
    Hc = gu.run_hist(case.bins, GH, qexp, B, rows, off, build)
    from paper_2211_12858_amd import _lib as L
    L.sb_subtract_histograms(Hp, Hc, 2, m, B, k, gu.up(build))
    gu.sync()
    Hdirect = gu.run_hist(case.bins, GH, qexp, B, rows, off).cpu().numpy()
    assert np.array_equal(Hc.cpu().numpy(), Hdirect)


# ---------------------------------------------------------------- scores
@pytest.mark.parametrize("seed,m,B,k,nodes", [(0, 10, 256, 5, 1), (1, 50, 64, 5, 8), (2, 7, 5, 3, 4),
                                               (3, 100, 256, 5, 2), (4, 3, 2, 1, 3)])
def test_score_from_oracle_histograms(seed, m, B, k, nodes):
    rng = np.random.default_rng(seed)
    n = 3000
    case = small_case(n, m, B, k, seed=seed, h_kind="random" if seed % 2 else "ones")
    GH = oracle.materialise(case.G, case.h, *oracle.identity_sketch(k))
    rows, off = _segments(rng, n, nodes)
    if nodes > 2:
        off[2] = off[1]  # one empty node
    Hs = np.stack([oracle.node_histograms(case.bins, GH, rows[off[j]:off[j + 1]], B) for j in range(nodes)])
    bf, bb, bs = gu.run_score(Hs, B, k, lam=1.0)
    for j in range(nodes):
        S, valid = oracle.split_scores(Hs[j], 1.0)
        f, b, s1, s2 = oracle.best_split(S, valid)
        if f < 0:
            assert (bf[j], bb[j]) == (-1, -1) and bs[j] == -np.inf
            continue
        if s1 - s2 > gu.TOL * s1:
            assert (bf[j], bb[j]) == (f, b)
        else:
            assert valid[bf[j], bb[j]] and S[bf[j], bb[j]] >= s1 * (1 - gu.TOL)
        assert bs[j] == pytest.approx(S[bf[j], bb[j]], rel=1e-12)


def test_score_ties_and_min_child_weight():
    # two identical features and a constant one: lower feature wins, the
    # constant feature is never valid; min_child_weight removes light children
    n, B, k = 64, 8, 2
    rng = np.random.default_rng(3)
    col = rng.integers(0, B, n).astype(np.uint8)
    bins = np.stack([np.zeros(n, np.uint8), col, col], axis=1)
    GH = np.concatenate([rng.standard_normal((n, k)).astype(np.float32), np.ones((n, 1), np.float32)], axis=1)
    H = oracle.node_histograms(bins, GH, np.arange(n), B)[None]
    bf, bb, bs = gu.run_score(H, B, k)
    S, valid = oracle.split_scores(H[0], 1.0)
    f, b, _, _ = oracle.best_split(S, valid)
    assert (bf[0], bb[0]) == (f, b) and f == 1
    bf2, bb2, _ = gu.run_score(H, B, k, mcw=10.0)
    S2, valid2 = oracle.split_scores(H[0], 1.0, 10.0)
    f2, b2, _, _ = oracle.best_split(S2, valid2)
    assert (bf2[0], bb2[0]) == (f2, b2)
    bf3, bb3, bs3 = gu.run_score(H, B, k, mcw=1e9)
    assert (bf3[0], bb3[0], bs3[0]) == (-1, -1, -np.inf)


# ---------------------------------------------------------------- partition
# 2048 nodes: the largest level whose node table the flags and scatter blocks
# stage in LDS; 3000: the same kernels reading it from global memory; from
# 1536 tiles of 1024 rows the scatter blocks take two tiles each (1537 tiles:
# the last block has one)
@pytest.mark.parametrize("n,m,n_nodes,seed", [(1, 1, 1, 0), (4095, 3, 1, 1), (4097, 5, 2, 2), (100003, 20, 16, 3),
                                               (50000, 7, 64, 4), (60000, 4, 2048, 5), (70001, 6, 3000, 6),
                                               (1536 * 1024 + 1, 3, 32, 7), (2_000_000, 2, 1, 8),
                                               (1536 * 1024 + 5000, 2, 2048, 9)])
def test_partition_bit_exact(n, m, n_nodes, seed):
    rng = np.random.default_rng(seed)
    bins = rng.integers(0, 256, (n, m), dtype=np.uint8)
    rows, off = _segments(rng, n, n_nodes, empty_every=5 if n_nodes > 8 else 0)
    bf = rng.integers(0, m, n_nodes).astype(np.int32)
    bb = rng.integers(0, 255, n_nodes).astype(np.int32)
    bf[::3] = -1  # terminal nodes
    bb[::3] = -1
    row_in = None if n_nodes == 1 and seed % 2 == 0 else rows
    if row_in is None:
        rows = np.arange(n, dtype=np.int32)
    row_g, off_g, bl_g = gu.run_partition(bins, row_in, off, bf, bb)
    want_rows, want_off, want_bl = [], [0], []
    for j in range(n_nodes):
        left, right = oracle.partition(bins, rows[off[j]:off[j + 1]], bf[j], bb[j])
        want_rows += [left, right]
        want_off += [want_off[-1] + len(left), want_off[-1] + len(left) + len(right)]
        want_bl.append(2 * j if len(left) <= len(right) else 2 * j + 1)
    assert np.array_equal(row_g, np.concatenate(want_rows).astype(np.int32))
    assert np.array_equal(off_g, np.array(want_off, dtype=np.int32))
    assert np.array_equal(bl_g, np.array(want_bl, dtype=np.int32))


@pytest.mark.parametrize("gathered", [False, True])
def test_histograms_int32_partials_escape(gathered):
    """A workgroup's partial sum of one bin leaves int32 past 8192 rows of
    full-scale values: a constant feature puts every row of a workgroup in one
    bin, with channels of +-(1 - 2^-24), whose
    fixed-point images are +-2^18.  Those cells take the exact int64 overflow
    slot; every cell must still match the oracle within the fixed-point bound.
    With 100 features a slice has 32 (gathered) to 40 (root) row groups, so a
    workgroup holds 12,500 to 15,000 rows."""
    rng = np.random.default_rng(321)
    n, m, B, k = 600_000, 100, 8, 5
    bins = rng.integers(0, B, size=(n, m), dtype=np.uint8)
    bins[:, 0] = 3                       # constant feature
    bins[:, 1] = (np.arange(n) % 2).astype(np.uint8)
    top = np.float32(1.0) - np.float32(2.0 ** -24)
    GH = np.empty((n, k + 1), dtype=np.float32)
    GH[:, 0] = top
    GH[:, 1] = -top
    GH[:, 2] = np.where(rng.random(n) < 0.5, top, -top)
    GH[:, 3] = rng.standard_normal(n).astype(np.float32) * np.float32(0.25)
    GH[:, 4] = np.float32(0.5)
    GH[:, 5] = np.float32(1.0)
    qexp = gu.qexp_rule(GH)
    if gathered:
        rows = np.sort(rng.permutation(n)[: n - 1000]).astype(np.int32)
        cut = len(rows) // 3
        off = np.array([0, cut, len(rows)], dtype=np.int32)
        build_list = np.array([1], dtype=np.int32)
        nodes = [1]
    else:
        rows = np.arange(n, dtype=np.int32)
        off = np.array([0, n], dtype=np.int32)
        build_list = None
        nodes = [0]
    Hg = gu.host_layout(gu.run_hist(bins, GH, qexp, B, rows if gathered else None, off, build_list).cpu().numpy())
    chan_max = np.abs(GH.astype(np.float64)).max(axis=0)
    for j in nodes:
        node_rows = rows[off[j]:off[j + 1]]
        Ho = oracle.node_histograms(bins, GH, node_rows, B)
        counts = oracle.node_histograms(bins, np.ones((n, 1), dtype=np.float32), node_rows, B)[..., 0]
        mass = oracle.node_histograms(bins, np.abs(GH), node_rows, B)
        assert np.abs(Ho[0, 3, 0]) > 2.0 ** 14  # the constant feature's cell exceeds int32 per workgroup
        ok1, ok2, worst = gu.hist_tolerance_ok(Hg[j], Ho, counts, qexp, mass, chan_max)
        assert ok1 and ok2, worst
