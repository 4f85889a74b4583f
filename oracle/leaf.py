"""Oracle: leaf values of a grown tree from the full gradient matrix (test infrastructure only).

Section 2, "Finding the leaf values": once the leaves R_1..R_J are fixed,
each leaf's value v in R^d minimises, over the leaf's rows,

    Q(v) = sum_i ( g_i^T v + 1/2 v^T H_i v ) + lambda/2 ||v||^2,

and with diagonal Hessians H_i = diag(h_i^1 .. h_i^d) (eq. 3) the minimiser
is, output by output,

    v_j = - sum_{i in R} g_ij / ( sum_{i in R} h_ij + lambda ).

Section 3: the sketch only serves the search for the tree structure; the
leaf values use all d columns of G.

Three hessian forms are accepted:
* ``hess`` (n, d): the per-element diagonal h_ij of eq. 3;
* ``h`` (n,): one weight per row shared by every output (h_ij = h_i);
* neither: h_ij = 1, so the denominator is the leaf's row count plus lambda
  (the weight of the hessian-free score S_G of Section 3).

A leaf is the row segment row_idx[leaf_off[L] : leaf_off[L+1]] of the grown
tree (empty segments give v = -0/lambda = 0).  fp64 throughout.
"""
import numpy as np


def leaf_rows(row_idx, leaf_off):
    """The rows of every leaf, as a list of int64 arrays."""
    row_idx = np.asarray(row_idx, dtype=np.int64)
    leaf_off = np.asarray(leaf_off, dtype=np.int64)
    return [row_idx[leaf_off[L]:leaf_off[L + 1]] for L in range(leaf_off.shape[0] - 1)]


def _hess_sums(rows, d, hess, h):
    if hess is not None:
        return np.asarray(hess, dtype=np.float64)[rows].sum(axis=0)
    if h is not None:
        return np.full(d, np.asarray(h, dtype=np.float64)[rows].sum())
    return np.full(d, float(rows.shape[0]))


def leaf_values(G, row_idx, leaf_off, lam, hess=None, h=None):
    """V[L, j] = -sum_{i in leaf L} G[i, j] / (sum_{i in leaf L} h_ij + lam)  (eq. 3).

    G: (n, d) gradients (any float dtype, read as fp64).  Returns (n_leaves, d) fp64.
    """
    G = np.asarray(G, dtype=np.float64)
    d = G.shape[1]
    rows_of = leaf_rows(row_idx, leaf_off)
    V = np.zeros((len(rows_of), d), dtype=np.float64)
    for L, rows in enumerate(rows_of):
        gs = G[rows].sum(axis=0)
        hs = _hess_sums(rows, d, hess, h)
        V[L] = -gs / (hs + lam)
    return V


def leaf_objective(G, rows, v, lam, hess=None, h=None):
    """Q(v) of one leaf (Section 2, the objective minimised by the leaf value), with
    diagonal Hessians: sum_i sum_j (g_ij v_j + 1/2 h_ij v_j^2) + lam/2 sum_j v_j^2."""
    G = np.asarray(G, dtype=np.float64)[rows]
    v = np.asarray(v, dtype=np.float64)
    if hess is not None:
        Hd = np.asarray(hess, dtype=np.float64)[rows]
    elif h is not None:
        Hd = np.repeat(np.asarray(h, dtype=np.float64)[rows][:, None], G.shape[1], axis=1)
    else:
        Hd = np.ones_like(G)
    return float((G * v).sum() + 0.5 * (Hd * v * v).sum() + 0.5 * lam * (v * v).sum())
