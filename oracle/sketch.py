"""Oracle: gradient sketches of Section 3 (test infrastructure only).

Notation follows the paper: G is the n x d gradient matrix with columns
g_1..g_d, k is the sketch dimension, h is the hessian column used as the
denominator weight of the scoring function.  A sketch is returned as the
packed matrix GH = [G_k, h] (n x (k+1)): the k sketch columns followed by h.

The random numbers a sketch draws are inputs here, never generated inside:
Random Sampling takes k uniforms u_t in [0, 1); Random Projections takes the
d x k matrix Pi.
"""
import math

import numpy as np


def column_norms2(G):
    """Squared Euclidean norms ||g_j||^2 of the columns of G, in fp64.

    Section 3.1 ranks columns by ||g_j||; Section 3.2 samples with
    p_j = ||g_j||^2 / sum_l ||g_l||^2.  Each column is summed separately in
    fp64 (the square of an fp32 value is exact in fp64).
    """
    G = np.asarray(G)
    n2 = np.empty(G.shape[1], dtype=np.float64)
    for j in range(G.shape[1]):
        col = np.asarray(G[:, j], dtype=np.float64)
        n2[j] = np.sum(col * col)
    return n2


def top_outputs(n2, k):
    """Top Outputs (Section 3.1): the k columns of largest norm, unscaled.

    Columns are ordered by decreasing norm; equal norms keep the lower column
    index first (the paper leaves ties open).  Returns (cols, scales) with
    scales all 1.
    """
    d = len(n2)
    if not 1 <= k <= d:
        raise ValueError("top outputs needs 1 <= k <= d")
    order = sorted(range(d), key=lambda j: (-float(n2[j]), j))
    cols = np.array(order[:k], dtype=np.int32)
    return cols, np.ones(k, dtype=np.float32)


def random_sampling(n2, k, u):
    """Random Sampling (Section 3.2) by inverse-CDF draws from given uniforms.

    p_j = n2_j / sum(n2).  Draw t picks i_t = min{ j : C_j > u_t * C_total }
    where C_j = n2_0 + ... + n2_j is accumulated left to right in fp64; the
    draws are i.i.d. with replacement and each picked column is scaled by
    1 / sqrt(k p_{i_t}) = sqrt(C_total / (k n2_{i_t})), rounded once to fp32.
    A column of zero norm is never drawn.  If every column is zero the sketch
    is all zero: cols = -1 and scales = 0.
    """
    d = len(n2)
    u = np.asarray(u, dtype=np.float64)
    if k < 1 or u.shape != (k,):
        raise ValueError("random sampling needs k >= 1 uniforms")
    C = np.empty(d, dtype=np.float64)
    acc = 0.0
    for j in range(d):
        acc = acc + float(n2[j])
        C[j] = acc
    total = acc
    cols = np.full(k, -1, dtype=np.int32)
    scales = np.zeros(k, dtype=np.float32)
    if total == 0.0:
        return cols, scales
    for t in range(k):
        x = float(u[t]) * total
        i = 0
        while not C[i] > x:
            i += 1
        cols[t] = i
        scales[t] = np.float32(math.sqrt(total / (float(k) * float(n2[i]))))
    return cols, scales


def identity_sketch(d):
    """Full-output scoring: every column once, unscaled (k = d)."""
    return np.arange(d, dtype=np.int32), np.ones(d, dtype=np.float32)


def materialise(G, h, cols, scales):
    """GH[:, t] = fp32(G[:, cols[t]] * scales[t]); GH[:, k] = h.

    One fp32 multiply per element (the sketch column times its scale).  A
    column index of -1 gives an all-zero column.
    """
    G = np.asarray(G)
    n = G.shape[0]
    k = len(cols)
    GH = np.zeros((n, k + 1), dtype=np.float32)
    for t in range(k):
        if cols[t] >= 0:
            GH[:, t] = np.asarray(G[:, cols[t]], dtype=np.float32) * np.float32(scales[t])
    GH[:, k] = np.asarray(h, dtype=np.float32)
    return GH


def random_projection(G, h, Pi):
    """Random Projections (Section 3.3): G_k = G Pi, exact product in fp64.

    Pi is the d x k matrix of i.i.d. N(0, 1/k) entries, passed in.  Returns
    GH in fp64 (n x (k+1)), the last column being h.
    """
    G64 = np.asarray(G, dtype=np.float64)
    Pi64 = np.asarray(Pi, dtype=np.float64)
    n = G64.shape[0]
    k = Pi64.shape[1]
    GH = np.empty((n, k + 1), dtype=np.float64)
    GH[:, :k] = G64 @ Pi64
    GH[:, k] = np.asarray(h, dtype=np.float64)
    return GH


def sparse_pi_matrix(d, k, pi_col, pi_val):
    """The d x k matrix of a row-sparse projection: row j holds pi_val[j, q] in
    column pi_col[j, q] for q < s (repeated columns add; columns outside
    [0, k) hold nothing, which lets rows be padded).  fp64."""
    pi_col = np.asarray(pi_col).reshape(d, -1)
    pi_val = np.asarray(pi_val, dtype=np.float64).reshape(d, -1)
    Pi = np.zeros((d, k), dtype=np.float64)
    for j in range(d):
        for q in range(pi_col.shape[1]):
            c = int(pi_col[j, q])
            if 0 <= c < k:
                Pi[j, c] += pi_val[j, q]
    return Pi


def sparse_projection(G, h, k, pi_col, pi_val):
    """Random Projections (Section 3.3) with a sparse Pi: the entries of Pi may
    follow distributions other than the normal one (Achlioptas), and sparse
    JL transforms (Dasgupta, Kumar and Sarlos 2010; Kane and Nelson 2014) make
    G Pi cheaper (the end of the proof of Prop. A.5).  G_k = G Pi exactly in
    fp64, with Pi assembled from its row-sparse form."""
    d = np.asarray(G).shape[1]
    return random_projection(G, h, sparse_pi_matrix(d, k, pi_col, pi_val))


def sketch(kind, G, h, k, u=None, Pi=None):
    """Dispatch on the sketch kind; returns (GH, cols, scales, norm2).

    kind: "identity", "top_outputs", "random_sampling", "random_projection".
    For random_projection GH is fp64 and cols/scales are None.
    """
    if kind == "random_projection":
        return random_projection(G, h, Pi), None, None, None
    n2 = column_norms2(G)
    if kind == "identity":
        if k != n2.shape[0]:
            raise ValueError("identity sketch needs k == d")
        cols, scales = identity_sketch(k)
    elif kind == "top_outputs":
        cols, scales = top_outputs(n2, k)
    elif kind == "random_sampling":
        cols, scales = random_sampling(n2, k, u)
    else:
        raise ValueError(kind)
    return materialise(G, h, cols, scales), cols, scales, n2
