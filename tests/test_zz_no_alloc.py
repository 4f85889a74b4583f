"""The allocation-free partition (sb_partition_rows_noalloc) against sb_partition_rows.

Both calls run the same kernels; the allocation-free one takes its scratch
from the library's static device array instead of a caller workspace.  Two
calls in a row on the same GPU (the second on a smaller level than the
first) must each give bit for bit the rows, child offsets and build list of
sb_partition_rows on the same inputs, and the stable partition that the
oracle defines.
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from gpu_util import DEV, L, sync, up  # noqa: E402


def _level(rng, n, m, n_nodes):
    bins = rng.integers(0, 256, (n, m), dtype=np.uint8)
    rows = rng.permutation(n).astype(np.int32)
    cuts = np.sort(rng.integers(0, n + 1, n_nodes - 1))
    off = np.concatenate([[0], cuts, [n]]).astype(np.int32)
    for j in range(n_nodes):
        rows[off[j]:off[j + 1]] = np.sort(rows[off[j]:off[j + 1]])
    bf = rng.integers(0, m, n_nodes).astype(np.int32)
    bb = rng.integers(0, 255, n_nodes).astype(np.int32)
    bf[1::4] = -1  # terminal nodes: every row goes left
    bb[1::4] = -1
    return bins, rows, off, bf, bb


def _noalloc(bins, rows, off, bf, bb):
    n, m = bins.shape
    n_nodes = len(off) - 1
    bins_cm = up(np.ascontiguousarray(bins.T))
    row_out = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    off_out = torch.full((2 * n_nodes + 1,), -1, dtype=torch.int32, device=DEV)
    bl_out = torch.full((n_nodes,), -1, dtype=torch.int32, device=DEV)
    L.sb_partition_rows_noalloc(bins_cm, n, m, n, up(rows, torch.int32), up(off, torch.int32), n_nodes,
                                up(bf, torch.int32), up(bb, torch.int32), row_out, off_out, bl_out)
    sync()
    return row_out.cpu().numpy(), off_out.cpu().numpy(), bl_out.cpu().numpy()


@pytest.mark.parametrize("sizes", [((300_007, 100, 16), (4_099, 30, 3)), ((2_000_000, 20, 32), (1, 4, 1))])
def test_noalloc_partition_matches_the_workspace_call(sizes):
    rng = np.random.default_rng(11)
    for n, m, n_nodes in sizes:
        print("case: noalloc partition n=%d m=%d nodes=%d" % (n, m, n_nodes), flush=True)
        bins, rows, off, bf, bb = _level(rng, n, m, n_nodes)
        got = _noalloc(bins, rows, off, bf, bb)
        want = gu.run_partition(bins, rows, off, bf, bb)
        for g, w in zip(got, want):
            assert np.array_equal(g, w)
        # and the oracle's stable partition of every node
        parts, offs = [], [0]
        for j in range(n_nodes):
            left, right = oracle.partition(bins, rows[off[j]:off[j + 1]], bf[j], bb[j])
            parts += [left, right]
            offs += [offs[-1] + len(left), offs[-1] + len(left) + len(right)]
        assert np.array_equal(got[0], np.concatenate(parts).astype(np.int32))
        assert np.array_equal(got[1], np.array(offs, dtype=np.int32))
