"""Oracle: loss derivatives, prediction update and the boosting loop (test infrastructure only).

Section 2: boosting step t fits a tree to the first derivatives g_i and the
(diagonal) second derivatives of the loss at the current predictions
a_{t-1}(x_i) (eq. 2), then updates the model a_t = a_{t-1} + eps * f_t, where
f_t(x) is the value of the leaf that x falls in.  The experiments use the
cross-entropy: softmax cross-entropy for multiclass tasks and per-output
binary cross-entropy for multilabel tasks (Section 4; Appendix B).

Losses, for one row with raw scores a in R^d:
* softmax cross-entropy, label y in {0..d-1}:
    l = -log p_y,  p = softmax(a);  g_j = p_j - [j = y];  h_j = p_j (1 - p_j)
  (h_j is the diagonal of the Hessian diag(p) - p p^T, the simplification of
  Section 2 for losses whose Hessian is not diagonal);
* sigmoid binary cross-entropy, labels Y_j in {0, 1}:
    l = -sum_j [Y_j log s_j + (1 - Y_j) log(1 - s_j)],  s = sigmoid(a);
    g_j = s_j - Y_j;  h_j = s_j (1 - s_j).

Arithmetic: fp64, then one rounding to fp32 for what is stored (G, the
hessians, the predictions), as the device stores them.
"""
import numpy as np

from .leaf import leaf_rows, leaf_values
from .sketch import column_norms2, sketch
from .split import grow_tree


# ---------------------------------------------------------------- losses
def softmax_ce_loss(F, y):
    """Per-row -log softmax(F_i)[y_i] (fp64), for the pins."""
    F = np.asarray(F, dtype=np.float64)
    z = F - F.max(axis=1, keepdims=True)
    lse = np.log(np.exp(z).sum(axis=1))
    return lse - z[np.arange(F.shape[0]), np.asarray(y)]


def sigmoid_bce_loss(F, Y):
    """Per-row binary cross-entropy summed over outputs (fp64), for the pins."""
    F = np.asarray(F, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    # log(1 + exp(-|a|)) form: log s = -softplus(-a), log(1 - s) = -softplus(a)
    sp_pos = np.logaddexp(0.0, F)
    sp_neg = np.logaddexp(0.0, -F)
    return (Y * sp_neg + (1.0 - Y) * sp_pos).sum(axis=1)


def softmax_ce_derivatives(F, y):
    """(g, h) in fp64: g = softmax(F) - onehot(y), h = p (1 - p), both (n, d)."""
    F = np.asarray(F, dtype=np.float64)
    z = F - F.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    g = p.copy()
    g[np.arange(F.shape[0]), np.asarray(y)] -= 1.0
    return g, p * (1.0 - p)


def sigmoid_bce_derivatives(F, Y):
    """(g, h) in fp64: g = sigmoid(F) - Y, h = s (1 - s), both (n, d)."""
    F = np.asarray(F, dtype=np.float64)
    s = 1.0 / (1.0 + np.exp(-F))
    return s - np.asarray(Y, dtype=np.float64), s * (1.0 - s)


def gradients(loss, F, target):
    """What one gradient pass stores: G and the per-element hessians rounded to
    fp32, the per-row mean hessian (fp32), and the fp64 column norms of the
    stored G (Section 3.1, 3.2).  loss: 'softmax' (target = labels) or
    'sigmoid' (target = 0/1 matrix)."""
    if loss == "softmax":
        g, h = softmax_ce_derivatives(F, target)
    elif loss == "sigmoid":
        g, h = sigmoid_bce_derivatives(F, target)
    else:
        raise ValueError(loss)
    G32 = g.astype(np.float32)
    H32 = h.astype(np.float32)
    h_row = h.mean(axis=1).astype(np.float32)
    return G32, H32, h_row, column_norms2(G32)


# ---------------------------------------------------------------- update
def leaf_of_rows(n, row_idx, leaf_off):
    """Leaf id of every row from the leaf segments of a grown tree."""
    ids = np.full(n, -1, dtype=np.int64)
    for L, rows in enumerate(leaf_rows(row_idx, leaf_off)):
        ids[rows] = L
    return ids


def update_predictions(F, row_idx, leaf_off, V, lr):
    """a_t = a_{t-1} + eps * f_t (Section 2): row i gets lr * V[leaf of i].

    fp64 arithmetic (lr * v, then the sum), rounded once to fp32."""
    F = np.asarray(F, dtype=np.float32)
    ids = leaf_of_rows(F.shape[0], row_idx, leaf_off)
    step = float(lr) * np.asarray(V, dtype=np.float64)[ids]
    return (F.astype(np.float64) + step).astype(np.float32)


# ---------------------------------------------------------------- loop
def boost(bins, n_bins, F0, target, loss, rounds, lr, kind, k, depth, lam, min_child_weight=0.0, u_rounds=None,
          Pi=None, choose=None):
    """`rounds` boosting steps from the predictions F0 (n, d).

    Each step, in the paper's order:
    1. derivatives at the current predictions (eq. 2);
    2. the sketch of G (Section 3) with the split-search weight h: 1 for
       softmax (the count weight of S_G), the row mean of the hessians for
       sigmoid;
    3. the tree structure by the histogram split search (Section 2, eq. 4);
    4. leaf values from the full G and the per-element hessians (eq. 3);
    5. the update a_t = a_{t-1} + lr * f_t.
    u_rounds[r]: Random Sampling uniforms of step r.  choose: the split-search
    hook of split.grow_tree (called with the step index first).
    Returns the final predictions and, per step, the tree and its leaf values.
    """
    F = np.asarray(F0, dtype=np.float32).copy()
    n = F.shape[0]
    history = []
    for r in range(rounds):
        G, Hd, h_row, _ = gradients(loss, F, target)
        h = np.ones(n, dtype=np.float32) if loss == "softmax" else h_row
        u = None if u_rounds is None else u_rounds[r]
        GH, _, _, _ = sketch(kind, G, h, k, u=u, Pi=Pi)
        hook = None if choose is None else (lambda *a, _r=r: choose(_r, *a))
        tree = grow_tree(bins, GH, depth, lam, n_bins, min_child_weight, choose=hook)
        segs = tree["segments"]
        row_idx = np.concatenate([np.asarray(s, dtype=np.int64) for s in segs]).astype(np.int32)
        leaf_off = np.concatenate([[0], np.cumsum([len(s) for s in segs])]).astype(np.int32)
        V = leaf_values(G, row_idx, leaf_off, lam, hess=Hd)
        F = update_predictions(F, row_idx, leaf_off, V, lr)
        history.append({"tree": tree, "row_idx": row_idx, "leaf_off": leaf_off, "V": V})
    return F, history
