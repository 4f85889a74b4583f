"""A whole tree (sketch plus level loop) captured in a HIP graph and replayed.

The library launches only kernels on the caller's stream (no host
synchronisation, no allocation, no memset nodes), so a caller that grows many
small trees can capture one step and replay it.  Each replay here follows a
different eager step on the same buffers, and every replay's tree (splits,
scores, leaf rows and offsets) must equal, bit for bit, the eager tree grown
from the same uniforms.
"""
import numpy as np
import pytest
import torch

from workloads import make_inputs, workload

pytestmark = pytest.mark.gpu

import gpu_util as gu  # noqa: E402
from paper_2211_12858_amd.driver import SplitSearch  # noqa: E402


def tree_bits(t):
    return (np.concatenate([np.asarray(x) for x in t["feature"]]), np.concatenate([np.asarray(x) for x in t["bin"]]),
            np.concatenate([np.asarray(x, dtype=np.float64) for x in t["score"]]).view(np.uint64),
            np.asarray(t["row_idx"]).copy(), np.asarray(t["leaf_off"]).copy())


@pytest.mark.parametrize("kind,depth", [("random_sampling", 4), ("top_outputs", 6)])
def test_graph_replay_equals_eager(kind, depth):
    wl = workload("mc2m_rs5", n=30_000, m=20, d=12, depth=depth)
    inp = make_inputs(wl)
    print("graph case: %s depth %d n %d" % (kind, depth, wl.n), flush=True)
    ss = SplitSearch(inp.bins, wl.n_bins, wl.k, wl.depth, wl.lam, device=gu.DEV)
    G_T, h = gu.up(inp.G_T), gu.up(inp.h)
    U = gu.up(np.random.default_rng(7).random((3, wl.k)), torch.float64)
    ref = []
    for i in range(3):
        ss.step(kind, G_T, h, u=U[i])
        gu.sync()
        ref.append(tree_bits(ss.tree()))
    u_static = U[0].clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ss.step(kind, G_T, h, u=u_static)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    gu.sync()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ss.step(kind, G_T, h, u=u_static)
    gu.sync()
    for rep in range(2):
        for i in range(3):
            u_static.copy_(U[i])
            g.replay()
            gu.sync()
            got = tree_bits(ss.tree())
            for a, b in zip(got, ref[i]):
                assert np.array_equal(a, b), (rep, i)
            # eager work on the same buffers between replays
            ss.step(kind, G_T, h, u=U[(i + 1) % 3])
            gu.sync()
