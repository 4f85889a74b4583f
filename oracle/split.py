"""Oracle: histogram split search and depth-wise tree growth (test infrastructure only).

Scoring function (Section 2, "Finding the tree structure", eq. 4), with the
hessian weights of Section 3 collapsed to one column h as the sketched score
S_G uses it:

    S(R) = sum_t ( sum_{i in R} GH[i, t] )^2 / ( sum_{i in R} h_i + lambda )

over the k sketch columns t.  A split of leaf R into R_left / R_right is
scored by S(R_left) + S(R_right) and the best split maximises it over leaves,
features and thresholds (Section 2).  Thresholds come from the histogram
algorithm of Section 3.4: feature values are bins 0..B-1 and the candidate
split "bin <= b" is tried for b = 0..B-2.

Readings of points the paper leaves open:
* a candidate is valid when both children have hessian weight above
  ``min_child_weight`` (default 0, i.e. both children non-empty when h > 0);
* ties in score go to the lower feature, then the lower bin;
* a leaf with no valid candidate is terminal: it keeps all rows in its left
  child and its right child is empty (both children stay in the level arrays
  so that node numbering is the same at every level);
* node j of level l has children 2j (bin <= b) and 2j+1 (bin > b); rows keep
  their original relative order inside each child.

Every node histogram is computed directly from the node's rows; nothing here
uses the sibling-subtraction shortcut.
"""
import numpy as np


def node_histograms(bins, GH, rows, n_bins):
    """H[f, b, t] = sum over rows i of the node with bins[i, f] == b of GH[i, t].

    fp64 accumulation (np.bincount with weights).  Shape (m, n_bins, c).
    """
    bins = np.asarray(bins)
    rows = np.asarray(rows, dtype=np.int64)
    m = bins.shape[1]
    c = GH.shape[1]
    H = np.zeros((m, n_bins, c), dtype=np.float64)
    if rows.size == 0:
        return H
    W = np.asarray(GH[rows], dtype=np.float64)
    for f in range(m):
        b = np.asarray(bins[rows, f], dtype=np.int64)
        for t in range(c):
            H[f, :, t] = np.bincount(b, weights=W[:, t], minlength=n_bins)
    return H


def split_scores(H, lam, min_child_weight=0.0):
    """Scores S(left) + S(right) for every (feature, threshold) of one node.

    H has shape (m, B, k+1): k gradient channels then the hessian channel.
    Left of threshold b holds bins 0..b (inclusive prefix sums), right holds
    the rest (node total minus left).  Returns (S, valid), both (m, B-1).
    """
    k = H.shape[2] - 1
    cum = np.cumsum(H, axis=1)
    total = cum[:, -1, :]
    GL = cum[:, :-1, :k]
    HL = cum[:, :-1, k]
    GR = total[:, None, :k] - GL
    HR = total[:, None, k] - HL
    S = np.sum(GL * GL, axis=2) / (HL + lam) + np.sum(GR * GR, axis=2) / (HR + lam)
    valid = (HL > min_child_weight) & (HR > min_child_weight)
    return S, valid


def best_split(S, valid):
    """Best valid (feature, bin, score) and the runner-up score.

    Order: larger score first, then lower feature, then lower bin.  Returns
    (f, b, s1, s2) with (-1, -1, -inf, -inf) when nothing is valid and
    s2 = -inf when only one candidate is valid.
    """
    Sm = np.where(valid, S, -np.inf)
    flat = Sm.ravel()
    if flat.size == 0 or not np.isfinite(flat).any():
        return -1, -1, -np.inf, -np.inf
    idx = int(np.argmax(flat))  # first maximum in row-major (f, b) order
    f, b = divmod(idx, Sm.shape[1])
    s1 = float(flat[idx])
    rest = flat.copy()
    rest[idx] = -np.inf
    s2 = float(rest.max()) if rest.size > 1 else -np.inf
    return f, b, s1, s2


def partition(bins, rows, f, b):
    """Split a node's row list: left = rows with bins[:, f] <= b, right = rest.

    Stable (original relative order kept).  f < 0 marks a terminal node: all
    rows go left.
    """
    rows = np.asarray(rows, dtype=np.int64)
    if f < 0:
        return rows, rows[:0]
    go_left = np.asarray(bins)[rows, f] <= b
    return rows[go_left], rows[~go_left]


def sketch_score(GH, rows, lam):
    """S(R) of one region from its rows (used by the approximation-error pins)."""
    rows = np.asarray(rows, dtype=np.int64)
    k = GH.shape[1] - 1
    W = np.asarray(GH[rows], dtype=np.float64)
    g = W[:, :k].sum(axis=0)
    return float(np.dot(g, g) / (W[:, k].sum() + lam))


def grow_tree(bins, GH, depth, lam, n_bins, min_child_weight=0.0, choose=None):
    """Depth-wise growth of one tree structure (Section 2; Appendix B.1 depth-wise policy).

    For level l = 0..depth-1, every node of the level gets its histograms,
    scores and best split, and is partitioned.  ``choose(level, j, f, b, s1,
    s2, S, valid)`` may replace the chosen (f, b) of a node (used by tests to
    follow a device's choice between near-tied candidates); it returns (f, b).

    Returns a dict with, per level, arrays ``feature``, ``bin``, ``score``,
    ``runner_up``, ``count`` (rows per node), plus ``segments`` (list of row
    arrays of the 2^depth leaves) and ``levels`` (list of the per-level
    segment lists, level 0 first).
    """
    n = np.asarray(bins).shape[0]
    segments = [np.arange(n, dtype=np.int64)]
    out = {"feature": [], "bin": [], "score": [], "runner_up": [], "count": [], "levels": []}
    for level in range(depth):
        out["levels"].append(segments)
        feats, bs, s1s, s2s, cnts, nxt = [], [], [], [], [], []
        for j, rows in enumerate(segments):
            H = node_histograms(bins, GH, rows, n_bins)
            S, valid = split_scores(H, lam, min_child_weight)
            f, b, s1, s2 = best_split(S, valid)
            if choose is not None:
                f, b = choose(level, j, f, b, s1, s2, S, valid)
                s1 = float(S[f, b]) if f >= 0 else -np.inf
            left, right = partition(bins, rows, f, b)
            feats.append(f)
            bs.append(b)
            s1s.append(s1)
            s2s.append(s2)
            cnts.append(len(rows))
            nxt += [left, right]
        out["feature"].append(np.array(feats, dtype=np.int32))
        out["bin"].append(np.array(bs, dtype=np.int32))
        out["score"].append(np.array(s1s, dtype=np.float64))
        out["runner_up"].append(np.array(s2s, dtype=np.float64))
        out["count"].append(np.array(cnts, dtype=np.int64))
        segments = nxt
    out["segments"] = segments
    return out
