"""Seeded synthetic inputs for the split-search hot path.

Serves both the device path and the oracle; holds none of the method's
arithmetic (no sketching, histograms, scores or partitions).  It produces
what a boosting step hands to split search: the binned feature matrix, the
gradient matrix G (stored column-major, as ``G_T`` with shape (d, n)), the
hessian column h, and the random numbers a sketch draws (k uniforms for
Random Sampling, the d x k matrix Pi for Random Projections).

Workloads (shapes of the paper's synthetic timing experiment, Appendix B.7,
and of its multiclass / multilabel datasets, Table 5; the public datasets
themselves are not used):

===================  =========  ====  ===  ====  =====================  =====
name                 n          m     B    d     sketch                 depth
===================  =========  ====  ===  ====  =====================  =====
tiny_multiclass      10,000     10    256  5     identity (k = d)       3
mc200k_top5          200,000    50    64   20    top outputs, k=5       6
mc2m_rs5             2,000,000  100   256  100   random sampling, k=5   6
mc2m_d1000_rp20      2,000,000  100   256  1000  random projection k=20 6
ml1m_top10           1,000,000  200   256  500   top outputs, k=10      8
===================  =========  ====  ===  ====  =====================  =====

Recipes: multiclass gradients are softmax(z) - onehot(y) with logits
z ~ N(0,1) and unit hessian; tiny_multiclass / mc200k_top5 draw bins
uniformly and labels uniformly; the 2M-row workloads draw raw features
X ~ N(0,1), quantile-bin each feature into 256 bins (edges at the empirical
t/256 quantiles, t = 1..255, bin = number of edges below the value) and take
labels y = argmax(X W + eps), W ~ N(0,1)/sqrt(m), eps ~ N(0,1).  The
multilabel workload has Y ~ Bernoulli(0.05), g = sigmoid(z) - y and
h_i = mean_j sigmoid(z_ij)(1 - sigmoid(z_ij)).  Gradients are formed in
fp64 and stored as fp32.  lambda = 1 everywhere.
"""
import os
from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    m: int
    n_bins: int
    d: int
    k: int
    kind: str          # identity | top_outputs | random_sampling | random_projection
    depth: int
    lam: float
    seed: int
    loss: str          # softmax | sigmoid
    binning: str       # uniform | quantile
    min_child_weight: float = 0.0


WORKLOADS = {
    "tiny_multiclass": Workload("tiny_multiclass", 10_000, 10, 256, 5, 5, "identity", 3, 1.0, 0,
                                "softmax", "uniform"),
    "mc200k_top5": Workload("mc200k_top5", 200_000, 50, 64, 20, 5, "top_outputs", 6, 1.0, 1,
                            "softmax", "uniform"),
    "mc2m_rs5": Workload("mc2m_rs5", 2_000_000, 100, 256, 100, 5, "random_sampling", 6, 1.0, 2,
                         "softmax", "quantile"),
    "mc2m_d1000_rp20": Workload("mc2m_d1000_rp20", 2_000_000, 100, 256, 1000, 20, "random_projection", 6,
                                1.0, 3, "softmax", "quantile"),
    "ml1m_top10": Workload("ml1m_top10", 1_000_000, 200, 256, 500, 10, "top_outputs", 8, 1.0, 4,
                           "sigmoid", "quantile"),
}


def workload(name, **overrides):
    """A named workload, optionally with fields replaced (e.g. a smaller n)."""
    return replace(WORKLOADS[name], **overrides)


def quantile_bin(x, n_bins):
    """Bins of one raw feature column: number of empirical quantile edges below x.

    Edges sit at the t/n_bins quantiles (t = 1..n_bins-1) with linear
    interpolation between order statistics.
    """
    xs = np.sort(x)
    n = xs.shape[0]
    pos = np.arange(1, n_bins, dtype=np.float64) / n_bins * (n - 1)
    lo = np.floor(pos).astype(np.int64)
    hi = np.minimum(lo + 1, n - 1)
    frac = pos - lo
    edges = xs[lo].astype(np.float64) + frac * (xs[hi].astype(np.float64) - xs[lo].astype(np.float64))
    return np.searchsorted(edges, x.astype(np.float64), side="left").astype(np.uint8)


@dataclass
class Inputs:
    bins: np.ndarray      # (n, m) uint8, row-major
    G_T: np.ndarray       # (d, n) float32: column j of G is G_T[j]
    h: np.ndarray         # (n,) float32
    u: np.ndarray         # (k,) float64 uniforms in [0, 1) for random sampling
    Pi: np.ndarray        # (d, k) float32, N(0, 1/k), for random projections
    wl: Workload
    y: np.ndarray = None  # (n,) int32 class labels (softmax workloads)
    Y: np.ndarray = None  # (d, n) uint8 0/1 targets, column-major (sigmoid workloads)

    @property
    def G(self):
        """The n x d gradient matrix as a (non-contiguous) view."""
        return self.G_T.T


def _softmax_grad_cols(z_T, y):
    """Column-major softmax-CE gradient block: z_T is (d, rows) fp64 logits."""
    z_T = z_T - z_T.max(axis=0, keepdims=True)
    p = np.exp(z_T)
    p /= p.sum(axis=0, keepdims=True)
    p[y, np.arange(z_T.shape[1])] -= 1.0
    return p.astype(np.float32)


def _softmax_grad_T(z, y):
    """Row-major logits (rows, d) -> column-major fp32 gradient block (d, rows)."""
    return _softmax_grad_cols(np.ascontiguousarray(np.asarray(z, dtype=np.float64).T), y)


def _pool():
    from concurrent.futures import ThreadPoolExecutor
    return ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0))))


def make_inputs(wl, chunk=65_536):
    """Generate the inputs of workload ``wl``.

    Deterministic in wl.seed and independent of the thread count: every
    feature column and every row chunk draws from its own child generator
    (numpy SeedSequence keyed by (seed, stream, index)).
    """
    n, m, d, k, B = wl.n, wl.m, wl.d, wl.k, wl.n_bins
    rng = np.random.default_rng(wl.seed)
    chunks = [(r0, min(n, r0 + chunk)) for r0 in range(0, n, chunk)]
    bins = np.empty((n, m), dtype=np.uint8)
    X_cm = None
    with _pool() as pool:
        if wl.binning == "uniform":
            def one_bins(f):
                bins[:, f] = np.random.default_rng([wl.seed, 1, f]).integers(0, B, size=n, dtype=np.uint8)
            list(pool.map(one_bins, range(m)))
        else:
            X_cm = np.empty((m, n), dtype=np.float32)

            def one_feature(f):
                X_cm[f] = np.random.default_rng([wl.seed, 2, f]).standard_normal(n, dtype=np.float32)
                bins[:, f] = quantile_bin(X_cm[f], B)
            list(pool.map(one_feature, range(m)))
        G_T = np.empty((d, n), dtype=np.float32)
        h = np.ones(n, dtype=np.float32)
        labels = np.empty(n, dtype=np.int32) if wl.loss == "softmax" else None
        Yt = np.empty((d, n), dtype=np.uint8) if wl.loss == "sigmoid" else None
        if wl.loss == "softmax":
            W = (rng.standard_normal((m, d)) / np.sqrt(m)).astype(np.float32) if X_cm is not None else None

            def one_chunk(ci):
                r0, r1 = chunks[ci]
                g = np.random.default_rng([wl.seed, 3, ci])
                if X_cm is None:
                    y = g.integers(0, d, size=r1 - r0)
                else:
                    logits = W.T @ X_cm[:, r0:r1] + g.standard_normal((d, r1 - r0), dtype=np.float32)
                    y = np.argmax(logits, axis=0)
                labels[r0:r1] = y
                G_T[:, r0:r1] = _softmax_grad_cols(g.standard_normal((d, r1 - r0)), y)
            list(pool.map(one_chunk, range(len(chunks))))
        elif wl.loss == "sigmoid":
            def one_chunk(ci):
                r0, r1 = chunks[ci]
                g = np.random.default_rng([wl.seed, 4, ci])
                y = g.random((d, r1 - r0)) < 0.05
                Yt[:, r0:r1] = y
                sg = 1.0 / (1.0 + np.exp(-g.standard_normal((d, r1 - r0))))
                G_T[:, r0:r1] = (sg - y).astype(np.float32)
                h[r0:r1] = np.mean(sg * (1.0 - sg), axis=0).astype(np.float32)
            list(pool.map(one_chunk, range(len(chunks))))
        else:
            raise ValueError(wl.loss)
    u = rng.random(k)
    Pi = (rng.standard_normal((d, k)) / np.sqrt(k)).astype(np.float32)
    return Inputs(bins=bins, G_T=G_T, h=h, u=u, Pi=Pi, wl=wl, y=labels, Y=Yt)


def scores_and_targets(n, d, loss, seed, scale=1.0):
    """Raw scores F (d, n) fp32 ~ N(0, scale^2), column-major, and targets: labels (n,)
    int32 uniform over d classes for softmax, a (d, n) uint8 Bernoulli(0.3) matrix for sigmoid."""
    rng = np.random.default_rng([seed, 7])
    F_T = (rng.standard_normal((d, n)) * scale).astype(np.float32)
    if loss == "softmax":
        return F_T, rng.integers(0, d, n).astype(np.int32)
    return F_T, (rng.random((d, n)) < 0.3).astype(np.uint8)


def sparse_jl_pi(d, k, s, seed):
    """A sparse JL projection in row-sparse form: every row j of Pi (d x k) has
    s nonzeros in distinct random columns, each +-1/sqrt(s) with a random
    sign (Kane and Nelson's construction with s nonzeros per input
    coordinate).  Returns pi_col (d, s) int32 and pi_val (d, s) float32."""
    rng = np.random.default_rng([seed, 11])
    pi_col = np.stack([rng.choice(k, size=s, replace=False) for _ in range(d)]).astype(np.int32)
    pi_val = (rng.choice([-1.0, 1.0], size=(d, s)) / np.sqrt(s)).astype(np.float32)
    return pi_col, pi_val


def achlioptas_pi(d, k, seed, s_max=8):
    """Achlioptas' sparse projection in row-sparse form: entries sqrt(3/k) * {+1, 0, -1}
    with probabilities {1/6, 2/3, 1/6}.  Rows with more than s_max nonzeros keep
    their first s_max columns (rare for k <= 12); shorter rows are padded with
    column -1 and value 0."""
    rng = np.random.default_rng([seed, 12])
    draw = rng.choice([1.0, 0.0, -1.0], size=(d, k), p=[1 / 6, 2 / 3, 1 / 6])
    pi_col = np.full((d, s_max), -1, dtype=np.int32)
    pi_val = np.zeros((d, s_max), dtype=np.float32)
    scale = np.sqrt(3.0 / k)
    for j in range(d):
        nz = np.flatnonzero(draw[j])[:s_max]
        pi_col[j, :nz.size] = nz
        pi_val[j, :nz.size] = draw[j, nz] * scale
    return pi_col, pi_val


def small_case(n, m, n_bins, d, seed, h_kind="ones", k=None):
    """A small random case for unit and parity tests (uniform bins, softmax-like G)."""
    rng = np.random.default_rng(seed)
    bins = rng.integers(0, n_bins, size=(n, m), dtype=np.uint8)
    y = rng.integers(0, d, size=n)
    z = rng.standard_normal((n, d))
    G_T = _softmax_grad_T(z, y) if d > 1 else rng.standard_normal((1, n)).astype(np.float32)
    if h_kind == "ones":
        h = np.ones(n, dtype=np.float32)
    else:
        h = rng.uniform(0.05, 0.25, size=n).astype(np.float32)
    k = d if k is None else k
    u = rng.random(k)
    Pi = (rng.standard_normal((d, k)) / np.sqrt(k)).astype(np.float32)
    wl = Workload("small", n, m, n_bins, d, k, "identity", 3, 1.0, seed, "softmax", "uniform")
    return Inputs(bins=bins, G_T=G_T, h=h, u=u, Pi=Pi, wl=wl)
