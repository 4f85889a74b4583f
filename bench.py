#!/usr/bin/env python3
"""Benchmark of the sketched split-search hot path on one MI355X.

One step is one tree: the sketch of the gradient matrix (taken once per tree)
followed by the depth-wise level loop (histograms of the built nodes, sibling
subtraction, scoring, partition) for every level.  Workload: 2,000,000 rows,
100 features quantile-binned to 256 bins, 100 softmax outputs, Random
Sampling sketch with k = 5, depth 6, lambda = 1 (the shape of the paper's
synthetic timing experiment, Appendix B.7).  Inputs are generated on the
host, uploaded once, and resident in HBM when timing starts; each tree uses
its own k uniforms.

Prints one JSON line on stdout.  Besides seconds per tree it reports the
histogram kernel's algorithmic bandwidth against the 8 TB/s HBM peak
(``roofline``) and the CPU oracle timed on this host (``cpu_baseline``).

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0
# LDS roof of the histogram kernel: the LDS data path moves 128 bytes per
# clock per CU; a 64-bit add carries two 32-bit channel sums, so the path
# takes at most 128 / 4 = 32 channel-adds per clock per CU; 256 CUs at 2.4 GHz.
LDS_BYTES_PER_CLK_CU = 128
LDS_ADDS_PER_CLK_CU = LDS_BYTES_PER_CLK_CU // 4
LDS_PEAK_GADDS = LDS_ADDS_PER_CLK_CU * 256 * 2.4
METRIC = "sec per tree (depth 6) + histogram-build HBM GB/s (% of peak)"
TRAFFIC_FILE = os.path.join(HERE, "profiles", "hist_traffic.json")
HIST_SRCS = [os.path.join(HERE, "paper_2211_12858_amd", "csrc", f) for f in ("sb_hist.hip", "sb_hist_plan.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def level_sizes(leaf_off, depth):
    """Node sizes of every level, from the leaf offsets of the finished tree."""
    leaf_off = np.asarray(leaf_off, dtype=np.int64)
    out = []
    for l in range(depth):
        span = 1 << (depth - l)
        edges = leaf_off[::span]
        out.append(np.diff(edges))
    return out


def hist_algorithmic_bytes(leaf_off, depth, m, n_bins, c):
    """Algorithmic bytes of the histogram kernel over one tree, per launch.

    Per level: every built row is read once (m bin bytes + 4c sketch bytes)
    and every built node's histogram is written once (m * n_bins * c * 4).
    Level 0 builds the root; level l >= 1 builds the smaller child of each
    pair (ties: left), the other child coming from subtraction.
    """
    sizes = level_sizes(leaf_off, depth)
    per_launch = []
    for l in range(depth):
        s = sizes[l]
        if l == 0:
            rows, nodes = int(s.sum()), 1
        else:
            left, right = s[0::2], s[1::2]
            rows, nodes = int(np.minimum(left, right).sum()), len(left)
        per_launch.append(rows * (m + 4 * c) + nodes * m * n_bins * c * 4)
    return per_launch


def hist_rows_built(leaf_off, depth):
    """Rows whose histograms are built at each level (all at the root, the smaller child of each pair below)."""
    sizes = level_sizes(leaf_off, depth)
    return [int(s.sum()) if l == 0 else int(np.minimum(s[0::2], s[1::2]).sum()) for l, s in enumerate(sizes)]


def leaf_algorithmic_bytes(n, d, n_leaves):
    """Leaf values: G read once (n*d*4), the row order once (4n), the values written (n_leaves*d*8)."""
    return n * d * 4 + 4 * n + n_leaves * d * 8


def boost_leg(wl, inp, dev, L, warm=100, timed=100):
    """The whole boosting step on the workload (Section 2), timed as in Appendix B.7:
    iterations warm+1 .. warm+timed, so that set-up costs drop out.  Starts from
    zero scores with the workload's labels; learning rate 0.01."""
    import torch
    from paper_2211_12858_amd.driver import Booster
    if wl.loss != "softmax":
        return None
    bst = Booster(inp.bins, wl.n_bins, wl.d, "softmax", wl.kind, wl.k, wl.depth, wl.lam, lr=0.01, device=dev)
    bst.set_target(torch.from_numpy(inp.y).to(dev))
    Pi = torch.from_numpy(inp.Pi).to(dev)
    rng = np.random.default_rng(wl.seed + 2000)
    u_all = torch.from_numpy(rng.random((warm + timed, wl.k))).to(dev)
    for s in range(warm):
        bst.step(u=u_all[s], Pi=Pi)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for s in range(timed):
        bst.step(u=u_all[warm + s], Pi=Pi)
    b.record()
    torch.cuda.synchronize()
    it_ms = a.elapsed_time(b) / timed
    # the gradient pass on its own (scores and labels in; G and the norms out),
    # after the last tree's held update
    bst.flush()
    torch.cuda.synchronize()
    a.record()
    for _ in range(10):
        bst.gradients()
    b.record()
    torch.cuda.synchronize()
    g_ms = a.elapsed_time(b) / 10
    n, d = wl.n, wl.d
    g_bytes = 2 * n * d * 4 + 4 * n  # scores read, G written, labels read
    log("bench: boosting iteration %.3f ms (gradient pass %.3f ms)" % (it_ms, g_ms))
    return {
        "ms_per_iteration": it_ms,
        "iterations": "%d-%d (the difference protocol of the synthetic experiment)" % (warm + 1, warm + timed),
        "what": "softmax-CE gradients with column norms, sketch from those norms, tree, leaf values with the "
                "full G and per-element hessians formed from G and the labels, score update; lr 0.01, zero "
                "initial scores; each tree's update runs in one pass with the next iteration's gradients",
        "gradient_pass_ms": g_ms,
        "gradient_pass_bytes": g_bytes,
        "gradient_pass_GBps": g_bytes / (g_ms * 1e-3) / 1e9,
    }


def projection_leg(dev, L, n=2_000_000, d=1000, k=20, reps=5):
    """Random Projections at the 2M x 1000, k = 20 shape (Section 3.3): the dense
    Gaussian Pi against row-sparse Pi with s = 1, 2, 4, 8 entries per row (sparse
    JL).  G is drawn on the device (the kernels' speed does not depend on its
    values); each call reads G once (n*d*4 bytes) and writes the sketch."""
    import torch
    from paper_2211_12858_amd.driver import workspace
    from workloads import sparse_jl_pi
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    G = torch.randn((d, n), device=dev, dtype=torch.float32, generator=g)
    h = torch.ones(n, device=dev, dtype=torch.float32)
    ld_gh = (k + 1 + 7) // 8 * 8
    GH = torch.empty((n, ld_gh), device=dev, dtype=torch.float32)
    qexp = torch.empty(k + 1, device=dev, dtype=torch.int32)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=k), dev)
    Pi = (torch.randn((d, k), device=dev, generator=g) / k ** 0.5).float()
    alg = n * d * 4 + n * ld_gh * 4
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    out = {"shape": "n=%d, d=%d, k=%d" % (n, d, k), "bytes": alg}
    ms = timed(lambda: L.sb_sketch(L.SB_SKETCH_RANDOM_PROJECTION, G, n, d, n, h, k, None, Pi, GH, ld_gh, None, None,
                                   None, qexp, ws, ws.numel()))
    out["dense_ms"] = ms
    for s in (1, 2, 4, 8):
        pc, pv = sparse_jl_pi(d, k, s, seed=s)
        pcd, pvd = torch.from_numpy(pc).to(dev), torch.from_numpy(pv).to(dev)
        out["sparse_s%d_ms" % s] = timed(lambda: L.sb_sketch_sparse_projection(G, n, d, n, h, k, s, pcd, pvd, GH, ld_gh,
                                                                                qexp, ws, ws.numel()))
    best = min(out["sparse_s1_ms"], out["sparse_s2_ms"])
    out["sparse_s1_GBps"] = alg / (out["sparse_s1_ms"] * 1e-3) / 1e9
    out["dense_GBps"] = alg / (ms * 1e-3) / 1e9
    log("bench: projection 2M x 1000 -> 20: dense %.3f ms, sparse s=1 %.3f ms (best of s=1,2: %.3f)"
        % (ms, out["sparse_s1_ms"], best))
    del G, GH
    torch.cuda.empty_cache()
    return out


def hist_source_hash():
    """sha256 over the histogram kernel's source files (the traffic record is tied to it)."""
    h = hashlib.sha256()
    for f in HIST_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def traffic_for_current_kernel(wl_name):
    """Counter-measured HBM bytes per histogram launch, if taken on this kernel source and workload."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    try:
        rec = json.load(open(TRAFFIC_FILE))
        src = hist_source_hash()
        if rec.get("kernel_source_sha256") != src or rec.get("workload") != wl_name:
            return None
        return rec.get("bytes_per_launch")
    except (OSError, ValueError):
        return None


_POOL = {}


def _pool_hist(task):
    """One (node, feature range) histogram by the oracle, in a pool worker."""
    import oracle
    j, f0, f1 = task
    return j, f0, oracle.node_histograms(_POOL["bins"][:, f0:f1], _POOL["GH"], _POOL["segments"][j], _POOL["n_bins"])


def oracle_tree_pooled(bins, GH, depth, lam, n_bins, min_child_weight, workers):
    """oracle.grow_tree with its histogram step over a process pool.

    Level by level, every node's histograms are computed by oracle.node_histograms
    on feature ranges in `workers` processes (fork), then scored, chosen and
    partitioned by the oracle's own split_scores / best_split / partition, in the
    order of oracle.grow_tree.  Returns (features, bins, leaf segments)."""
    import multiprocessing as mp
    import oracle
    n, m = bins.shape
    step = max(1, -(-m // workers))
    ranges = [(f0, min(m, f0 + step)) for f0 in range(0, m, step)]
    segments = [np.arange(n, dtype=np.int64)]
    feats, bs = [], []
    ctx = mp.get_context("fork")
    for _ in range(depth):
        _POOL.update(bins=bins, GH=GH, segments=segments, n_bins=n_bins)
        with ctx.Pool(workers) as pool:
            parts = pool.map(_pool_hist, [(j, f0, f1) for j in range(len(segments)) for f0, f1 in ranges], chunksize=1)
        H = [np.zeros((m, n_bins, GH.shape[1])) for _ in segments]
        for j, f0, h in parts:
            H[j][f0:f0 + h.shape[0]] = h
        lf, lb, nxt = [], [], []
        for j, rows in enumerate(segments):
            S, valid = oracle.split_scores(H[j], lam, min_child_weight)
            f, b, _, _ = oracle.best_split(S, valid)
            left, right = oracle.partition(bins, rows, f, b)
            lf.append(f)
            lb.append(b)
            nxt += [left, right]
        feats.append(lf)
        bs.append(lb)
        segments = nxt
    _POOL.clear()
    return feats, bs, segments


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline_worker(path):
    """Runs in a child process that never touches the GPU: the oracle timed on the
    workload's inputs (dumped by the parent): one tree with the histogram step
    over a pool of all host cores and, where asked, the same tree on all rows
    with one thread."""
    import oracle
    meta = json.load(open(os.path.join(path, "meta.json")))
    bins = np.load(os.path.join(path, "bins.npy"), mmap_mode="r")
    G_T = np.load(os.path.join(path, "G_T.npy"), mmap_mode="r")
    h = np.load(os.path.join(path, "h.npy"))
    u = np.load(os.path.join(path, "u.npy"))
    Pi = np.load(os.path.join(path, "Pi.npy")) if meta["kind"] == "random_projection" else None
    bins = np.ascontiguousarray(bins)
    G = np.asarray(G_T).T
    cores = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    GH, _, _, _ = oracle.sketch(meta["kind"], G, h, meta["k"], u=u[:meta["k"]], Pi=Pi)
    t_sketch = time.perf_counter() - t0
    print("cpu baseline: sketch %.1f s" % t_sketch, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    feats, bs, segs = oracle_tree_pooled(bins, GH, meta["depth"], meta["lam"], meta["n_bins"], meta["mcw"], cores)
    t_pool = time.perf_counter() - t0
    print("cpu baseline: pooled tree %.1f s" % t_pool, file=sys.stderr, flush=True)
    t_one, same = None, None
    if meta["one_core"]:
        t0 = time.perf_counter()
        tree = oracle.grow_tree(bins, GH, meta["depth"], meta["lam"], meta["n_bins"], meta["mcw"])
        t_one = time.perf_counter() - t0
        same = all(list(tree["feature"][l]) == feats[l] and list(tree["bin"][l]) == bs[l]
                   for l in range(meta["depth"]))
    print(json.dumps({"sketch_s": t_sketch, "tree_1core_s": t_one, "tree_pool_s": t_pool, "cores": cores,
                      "cpu_model": cpu_model(), "pool_tree_equal": same}), flush=True)


# The one-thread oracle tree is timed where rows x features x channels is at
# most this (the 10,000-, 200,000- and 2,000,000-row softmax workloads); the
# wider two take minutes on one core and are timed with the pool only.
ONE_CORE_MAX_CELLS = 1_500_000_000


def cpu_baseline(inp, wl):
    """The oracle timed on this host in a child process (which never touches the GPU)."""
    import shutil
    import subprocess
    import tempfile
    one_core = wl.n * wl.m * (wl.k + 1) <= ONE_CORE_MAX_CELLS
    path = tempfile.mkdtemp(prefix="sb_cpu_")
    try:
        np.save(os.path.join(path, "bins.npy"), inp.bins)
        np.save(os.path.join(path, "G_T.npy"), inp.G_T)
        np.save(os.path.join(path, "h.npy"), inp.h)
        np.save(os.path.join(path, "u.npy"), inp.u)
        if wl.kind == "random_projection":
            np.save(os.path.join(path, "Pi.npy"), np.ascontiguousarray(inp.Pi[:, :wl.k]))
        json.dump({"kind": wl.kind, "k": wl.k, "depth": wl.depth, "lam": wl.lam, "n_bins": wl.n_bins,
                   "mcw": wl.min_child_weight, "one_core": one_core}, open(os.path.join(path, "meta.json"), "w"))
        env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1", MKL_NUM_THREADS="1")
        res = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-baseline-worker", path],
                             capture_output=True, text=True, env=env, timeout=900)
        if res.returncode != 0:
            log("bench: cpu baseline worker failed: " + res.stderr[-2000:])
            return None
        r = json.loads(res.stdout.strip().splitlines()[-1])
    finally:
        shutil.rmtree(path, ignore_errors=True)
    total_pool = r["sketch_s"] + r["tree_pool_s"]
    total_one = r["sketch_s"] + r["tree_1core_s"] if one_core else None
    # the faster of the two runs (the pool's start-up outweighs its work on the
    # small workloads)
    pooled = total_one is None or total_pool <= total_one
    return {
        "value": total_pool if pooled else total_one,
        "unit": "s/tree",
        "cores": r["cores"] if pooled else 1,
        "kind": "oracle",
        "sample": "one whole tree (sketch + %d levels) on all %d rows of workload %s; value is the faster of "
                  "the oracle.grow_tree run on one thread and the same tree with the oracle's histogram step "
                  "over a process pool of %d workers (feature ranges per node), here the %s; same tree in "
                  "both runs: %s"
                  % (wl.depth, wl.n, wl.name, r["cores"], "pool" if pooled else "one thread",
                     r["pool_tree_equal"] if one_core else "one-thread tree not timed at this size"),
        "value_pool": total_pool,
        "value_1core": total_one,
        "sketch_s": r["sketch_s"],
        "cpu_model": r["cpu_model"],
    }


def cold_mall_leg(ss, wl, G_T, h, u_all, Pi, L, trees=3):
    """Histogram kernel with warm and with cold caches, on trees grown level by
    level through the per-step calls (SplitSearch.grow_levelwise).  Cold: 1 GiB
    is read and written between levels, more than the 256 MB Infinity Cache, so
    each level's rows, records and sketch words come from HBM.  Returns the
    histogram GB/s of both (algorithmic bytes over the kernel's event time)."""
    import torch
    flush = torch.empty(1 << 28, dtype=torch.float32, device=ss.device)  # 1 GiB
    flush.fill_(1.0)

    def run(cold):
        alg, ms = 0, 0.0
        for t in range(trees):
            ss.sketch(wl.kind, G_T, h, u=u_all[t], Pi=Pi)
            L.sb_profile_begin()
            ss.grow_levelwise(before_histograms=(lambda l: flush.mul_(1.0)) if cold else None)
            torch.cuda.synchronize()
            hist_ms, _ = L.sb_profile_end()
            ms += hist_ms
            alg += sum(hist_algorithmic_bytes(ss.leaf_off.cpu().numpy(), wl.depth, wl.m, wl.n_bins, wl.k + 1))
        return alg / (ms * 1e-3) / 1e9, ms / trees

    run(False)  # warm-up of the level-wise buffers
    warm_gbps, warm_ms = run(False)
    cold_gbps, cold_ms = run(True)
    del flush
    torch.cuda.empty_cache()
    log("bench: histogram kernel warm %.0f GB/s (%.3f ms/tree), cold %.0f GB/s (%.3f ms/tree)"
        % (warm_gbps, warm_ms, cold_gbps, cold_ms))
    return {"warm_GBps": warm_gbps, "warm_ms_per_tree": warm_ms, "cold_GBps": cold_gbps,
            "cold_ms_per_tree": cold_ms, "cold_frac_hbm_peak": cold_gbps / HBM_PEAK_GBPS,
            "what": "trees grown level by level through sb_build_histograms / sb_subtract_histograms / "
                    "sb_score_splits / sb_partition_rows; cold: 1 GiB streamed before every histogram launch"}


def copy_probe(nbytes):
    """A plain device copy of known size, the reference for scaling HBM counters."""
    import torch
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes}))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mc2m_rs5")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache histogram leg")
    ap.add_argument("--cpu-baseline-worker", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--no-boost", action="store_true", help="skip the boosting-loop leg")
    ap.add_argument("--no-projection", action="store_true", help="skip the projection leg")
    ap.add_argument("--copy-probe", type=int, default=0, help="only run a plain copy of this many bytes")
    ap.add_argument("--projection-only", action="store_true",
                    help="only the projection leg (2M x 1000 -> 20), for profiling its kernels")
    args = ap.parse_args()
    if args.cpu_baseline_worker:
        sys.path.insert(0, HERE)
        cpu_baseline_worker(args.cpu_baseline_worker)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build measures one GPU; --gpus %d is not supported (multi-GPU is design only)"
              % max(args.gpus, world), file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.projection_only:
        import torch
        sys.path.insert(0, HERE)
        from paper_2211_12858_amd import _lib as L
        L.load()
        print(json.dumps(projection_leg(torch.device("cuda:0"), L)), flush=True)
        return

    import torch
    sys.path.insert(0, HERE)
    from workloads import make_inputs, workload
    from paper_2211_12858_amd import _lib as L
    from paper_2211_12858_amd.driver import SplitSearch

    L.load()  # fails loudly if the HIP library is not built
    wl = workload(args.workload)
    t0 = time.perf_counter()
    log("bench: generating %s (n=%d m=%d d=%d)" % (wl.name, wl.n, wl.m, wl.d))
    inp = make_inputs(wl)
    log("bench: inputs ready in %.1f s" % (time.perf_counter() - t0))

    dev = torch.device("cuda:0")
    ss = SplitSearch(inp.bins, wl.n_bins, wl.k, wl.depth, wl.lam, wl.min_child_weight, device=dev)
    G_T = torch.from_numpy(inp.G_T).to(dev)
    h = torch.from_numpy(inp.h).to(dev)
    Pi = torch.from_numpy(inp.Pi).to(dev)
    K, W = args.steps, args.warmup
    rng = np.random.default_rng(wl.seed + 1000)
    u_all = torch.from_numpy(rng.random((K + W, wl.k))).to(dev)
    torch.cuda.synchronize()
    log("bench: resident in HBM; %d warmup + %d timed trees" % (W, K))

    for s in range(W):
        ss.step(wl.kind, G_T, h, u=u_all[s], Pi=Pi)
    torch.cuda.synchronize()

    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    # the timed trees run without instrumentation beyond one event between
    # trees: the per-launch events of the histogram profile add a pipeline
    # drain around every histogram kernel
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    start.record()
    for s in range(K):
        marks[s].record()
        ss.step(wl.kind, G_T, h, u=u_all[W + s], Pi=Pi)
    marks[K].record()
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    tree_ms = np.array([marks[s].elapsed_time(marks[s + 1]) for s in range(K)])
    # the same K trees again with HIP events around every histogram launch
    L.sb_profile_begin()
    for s in range(K):
        ss.step(wl.kind, G_T, h, u=u_all[W + s], Pi=Pi)
    torch.cuda.synchronize()
    hist_ms, launches = L.sb_profile_end()
    log("bench: %d trees in %.3f ms (median %.3f ms per tree); histogram kernel %.3f ms over %d launches"
        % (K, total_ms, float(np.median(tree_ms)), hist_ms, launches))

    # algorithmic bytes of every timed histogram launch (trees are deterministic
    # in their uniforms, so replaying one reproduces its node sizes)
    alg, rows_built = [], []
    for s in range(K):
        ss.step(wl.kind, G_T, h, u=u_all[W + s], Pi=Pi)
        torch.cuda.synchronize()
        alg += hist_algorithmic_bytes(ss.leaf_off.cpu().numpy(), wl.depth, wl.m, wl.n_bins, wl.k + 1)
        rows_built += hist_rows_built(ss.leaf_off.cpu().numpy(), wl.depth)
    assert len(alg) == launches, (len(alg), launches)
    bytes_per_launch = float(np.mean(alg))
    adds_per_launch = float(np.mean(rows_built)) * wl.m * (wl.k + 1)
    lds_gadds = adds_per_launch / (hist_ms / launches * 1e-3) / 1e9
    hist_kernel = "k_hist_rot"
    ms_per_launch = hist_ms / launches
    achieved = bytes_per_launch / (ms_per_launch * 1e-3) / 1e9
    traffic = traffic_for_current_kernel(wl.name)

    # leaf values of the last tree from the full G (eq. 3), timed on their own
    for _ in range(2):
        ss.leaf_values(G_T)
    torch.cuda.synchronize()
    start.record()
    for _ in range(K):
        ss.leaf_values(G_T)
    stop.record()
    torch.cuda.synchronize()
    leaf_ms = start.elapsed_time(stop) / K
    leaf_bytes = leaf_algorithmic_bytes(wl.n, wl.d, 1 << wl.depth)
    log("bench: leaf values %.3f ms per tree" % leaf_ms)

    cold = None if args.no_cold else cold_mall_leg(ss, wl, G_T, h, u_all, Pi, L)
    boost = None if args.no_boost else boost_leg(wl, inp, dev, L)
    proj = None if args.no_projection else projection_leg(dev, L)

    med_ms = float(np.median(tree_ms))
    sec_per_tree = med_ms / 1e3
    out = {
        "metric": METRIC,
        "value": sec_per_tree,
        "unit": "s/tree",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": med_ms,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 sketch, i32 fixed-point histogram accumulation, f64 scores",
        "data": "synthetic",
        "config": {
            "workload": "%s: n=%d rows, m=%d features, %d quantile bins, d=%d softmax outputs, %s sketch k=%d, "
                        "depth %d, lambda=%g" % (wl.name, wl.n, wl.m, wl.n_bins, wl.d, wl.kind.replace("_", " "),
                                                 wl.k, wl.depth, wl.lam),
        },
        "tree_ms": {"median": med_ms, "p10": float(np.percentile(tree_ms, 10)),
                    "p90": float(np.percentile(tree_ms, 90)), "mean": float(tree_ms.mean()),
                    "mean_bracketed": total_ms / K, "trees": K,
                    "what": "HIP events between consecutive trees on the stream; value is the median"},
        "hist_GBps": achieved,
        "hist_pct_peak": 100.0 * achieved / HBM_PEAK_GBPS,
        "hist_ms_per_tree": hist_ms / K,
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "kernel": hist_kernel,
            "bytes_per_launch": bytes_per_launch,
            "ms_per_launch": ms_per_launch,
        },
        # the roof that binds the histogram kernel: its useful channel-adds
        # (rows built x m features x c channels) per second against the LDS
        # data path (128 bytes per clock per CU, 4 bytes per channel-add)
        "lds_roofline": {
            "achieved": lds_gadds,
            "peak": LDS_PEAK_GADDS,
            "unit": "G channel-adds/s",
            "frac": lds_gadds / LDS_PEAK_GADDS,
            "adds_per_launch": adds_per_launch,
        },
    }
    out["next"] = {
        "leaf_values": {
            "ms_per_tree": leaf_ms,
            "bytes": leaf_bytes,
            "GBps": leaf_bytes / (leaf_ms * 1e-3) / 1e9,
            "frac_hbm_peak": leaf_bytes / (leaf_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "what": "sb_leaf_values over the last tree's %d leaves, full d=%d, unit hessians; not inside value"
                    % (1 << wl.depth, wl.d),
        },
    }
    if cold is not None:
        out["hist_cold_cache"] = cold
    if boost is not None:
        out["next"]["boosting"] = boost
    if proj is not None:
        out["next"]["projection"] = proj
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle (one tree on all rows: one thread, then a pool of all cores)")
        cb = cpu_baseline(inp, wl)
        if cb is not None:
            out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
