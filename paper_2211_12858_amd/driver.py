"""Device-side driver: torch allocates the buffers, libsketchboost computes.

``SplitSearch`` holds one binned dataset resident in HBM in the three
layouts the kernels read (built on the device by ``sb_layout_bins`` from
the row-major bins):

* quad-major words ``bins4[q, i]`` (features 4q..4q+3 of row i): the
  histogram kernel's lanes take consecutive rows and read contiguous words;
* column-major bytes ``bins_cm[f, i]``: the partition reads one run of the
  split feature's column per node;
* row records ``rec[i]`` of ``ld_rec`` bytes (one 128-byte line for up to
  128 features): the histograms of the deeper levels read one record per
  row.

The sketch lives row-major in ``GH[i, t]``, each row padded to a multiple of
8 floats so that it fills whole 32-byte sectors.  ``step()`` runs one
tree: the sketch (once per tree) and the depth-wise level loop, entirely on
the device; ``leaf_values()`` then gives the tree's leaf values from the
full gradient matrix.  No computation happens in Python.
"""
import numpy as np
import torch

from . import _lib as L


def _round_up(x, a):
    return (x + a - 1) // a * a


def workspace(nbytes, device):
    t = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert t.data_ptr() % 256 == 0
    return t


def record_stride(m):
    """Bytes per row record: a power of two up to 128 bytes (so that no
    record straddles a 128-byte line), else a multiple of 128."""
    need = _round_up(m, 16)
    if need <= 128:
        s = 16
        while s < need:
            s *= 2
        return s
    return _round_up(need, 128)


class SplitSearch:
    def __init__(self, bins, n_bins, k, depth, lam=1.0, min_child_weight=0.0, device="cuda", ld_rec=None):
        bins = np.ascontiguousarray(bins, dtype=np.uint8)
        self.n, self.m = bins.shape
        self.n_bins, self.k, self.c, self.depth = n_bins, k, k + 1, depth
        self.lam, self.mcw = float(lam), float(min_child_weight)
        self.device = dev = torch.device(device)
        n, m, c = self.n, self.m, self.c
        self.nq = (m + 3) // 4
        self.ld_rec = record_stride(m) if ld_rec is None else ld_rec
        self.ld_gh = _round_up(c, 8)
        self.bins4 = torch.empty((self.nq, n), dtype=torch.int32, device=dev)
        self.bins_cm = torch.empty((m, n), dtype=torch.uint8, device=dev)
        self.rec = torch.zeros((n, self.ld_rec), dtype=torch.uint8, device=dev)
        rm = torch.from_numpy(bins).to(dev)
        L.sb_layout_bins(rm, n, m, m, self.bins4, n, self.bins_cm, n, self.rec, self.ld_rec)
        torch.cuda.synchronize(dev)
        del rm
        self.GH = torch.zeros((n, self.ld_gh), dtype=torch.float32, device=dev)
        self.qexp = torch.zeros(c, dtype=torch.int32, device=dev)
        self.cols = torch.zeros(k, dtype=torch.int32, device=dev)
        self.scales = torch.zeros(k, dtype=torch.float32, device=dev)
        nt = (1 << depth) - 1
        self.tree_feature = torch.zeros(nt, dtype=torch.int32, device=dev)
        self.tree_bin = torch.zeros(nt, dtype=torch.int32, device=dev)
        self.tree_score = torch.zeros(nt, dtype=torch.float64, device=dev)
        self.row_idx = torch.zeros(n, dtype=torch.int32, device=dev)
        self.leaf_off = torch.zeros((1 << depth) + 1, dtype=torch.int32, device=dev)
        self.ws_tree_bytes = L.sb_workspace_bytes(L.SB_CALL_GROW_TREE, n=n, m=m, n_bins=n_bins, k=k, depth=depth)
        self.ws_tree = workspace(self.ws_tree_bytes, dev)
        self._ws_sketch = None
        self.norm2 = None
        self._ws_leaf = None
        self.V = None

    # ------------------------------------------------------------ sketch
    def sketch(self, kind, G_T, h, u=None, Pi=None, stream=None, norm2_in=None):
        """G_T: (d, n) float32 device tensor (column-major G); h: (n,) float32.

        norm2_in: the squared column norms of G, (d,) fp64 on the device (for
        example from sb_gradients); then G is not read for them."""
        d, n = G_T.shape
        assert n == self.n and G_T.is_contiguous() and G_T.dtype == torch.float32
        kid = L.KIND[kind]
        need = L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=self.k)
        if self._ws_sketch is None or self._ws_sketch.numel() < need:
            self._ws_sketch = workspace(need, self.device)
        if self.norm2 is None or self.norm2.numel() != d:
            self.norm2 = torch.zeros(d, dtype=torch.float64, device=self.device)
        if norm2_in is None:
            L.sb_sketch(kid, G_T, n, d, n, h, self.k, u, Pi, self.GH, self.ld_gh, self.cols, self.scales, self.norm2,
                        self.qexp, self._ws_sketch, self._ws_sketch.numel(), stream)
        else:
            L.sb_sketch_given_norms(kid, G_T, n, d, n, h, self.k, u, Pi, self.GH, self.ld_gh, self.cols, self.scales,
                                    norm2_in, self.qexp, self._ws_sketch, self._ws_sketch.numel(), stream)

    # ------------------------------------------------------------ tree
    def grow(self, stream=None):
        n = self.n
        L.sb_grow_tree(self.bins4, n, self.bins_cm, n, self.rec, self.ld_rec, n, self.m, self.n_bins, self.GH,
                       self.ld_gh, self.k, self.qexp, self.depth, self.lam, self.mcw, self.tree_feature,
                       self.tree_bin, self.tree_score, self.row_idx, self.leaf_off, self.ws_tree,
                       self.ws_tree_bytes, stream)

    def step(self, kind, G_T, h, u=None, Pi=None, stream=None):
        self.sketch(kind, G_T, h, u, Pi, stream)
        self.grow(stream)

    def grow_levelwise(self, before_histograms=None, stream=None):
        """The same tree as grow(), through the per-step calls, level by level:
        sb_build_histograms (the built nodes), sb_subtract_histograms (their
        siblings), sb_score_splits and sb_partition_rows.  before_histograms(l),
        if given, runs before level l's histogram call (bench.py streams a
        large buffer there to take the level's data out of the caches)."""
        n, m, B, k, c, D = self.n, self.m, self.n_bins, self.k, self.c, self.depth
        dev = self.device
        maxn = 1 << (D - 1)
        if getattr(self, "_lw", None) is None:
            cells = maxn * m * c * B
            self._lw = {
                "H": [torch.empty(cells, dtype=torch.float64, device=dev) for _ in range(2)],
                "rows": [torch.empty(n, dtype=torch.int32, device=dev) for _ in range(2)],
                "off": [torch.empty((1 << l) + 1, dtype=torch.int32, device=dev) for l in range(D + 1)],
                "build": [torch.empty(max(1, (1 << l) // 2), dtype=torch.int32, device=dev) for l in range(D + 1)],
                "ws_h": workspace(L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=n, m=m, n_bins=B, k=k,
                                                       n_nodes=maxn), dev),
                "ws_s": workspace(L.sb_workspace_bytes(L.SB_CALL_SCORE_SPLITS, m=m, n_nodes=2 * maxn), dev),
                "ws_p": workspace(L.sb_workspace_bytes(L.SB_CALL_PARTITION_ROWS, n=n, n_nodes=2 * maxn), dev),
            }
            self._lw["off"][0].copy_(torch.tensor([0, n], dtype=torch.int32))
        w = self._lw
        rows_in = None
        for l in range(D):
            nn = 1 << l
            H, Hp = w["H"][l & 1], w["H"][(l - 1) & 1]
            if before_histograms is not None:
                before_histograms(l)
            if l == 0:
                L.sb_build_histograms(self.bins4, n, None, 0, n, m, B, self.GH, self.ld_gh, k, self.qexp, None,
                                      w["off"][0], 1, None, 1, H, w["ws_h"], w["ws_h"].numel(), stream)
            else:
                L.sb_build_histograms(None, 0, self.rec, self.ld_rec, n, m, B, self.GH, self.ld_gh, k, self.qexp,
                                      rows_in, w["off"][l], nn, w["build"][l], nn // 2, H, w["ws_h"],
                                      w["ws_h"].numel(), stream)
                L.sb_subtract_histograms(Hp, H, nn // 2, m, B, k, w["build"][l], stream)
            base = nn - 1
            tf, tb, ts = self.tree_feature[base:base + nn], self.tree_bin[base:base + nn], self.tree_score[base:base + nn]
            L.sb_score_splits(H, nn, m, B, k, self.lam, self.mcw, tf, tb, ts, w["ws_s"], w["ws_s"].numel(), stream)
            last = l == D - 1
            rows_out = self.row_idx if last else w["rows"][l & 1]
            off_out = self.leaf_off if last else w["off"][l + 1]
            L.sb_partition_rows(self.bins_cm, n, m, n, rows_in, w["off"][l], nn, tf, tb, rows_out, off_out,
                                w["build"][l + 1], w["ws_p"], w["ws_p"].numel(), stream)
            rows_in = rows_out

    # ------------------------------------------------------------ leaf values
    def leaf_values(self, G_T, hess_T=None, h=None, stream=None):
        """Leaf values of the last grown tree from the full G (eq. 3): self.V, (2^depth, d) fp64.

        hess_T: (d, n) per-element hessians, or h: (n,) per-row hessians, or
        neither (h = 1)."""
        d, n = G_T.shape
        assert n == self.n and G_T.is_contiguous() and G_T.dtype == torch.float32
        n_leaves = 1 << self.depth
        need = L.sb_workspace_bytes(L.SB_CALL_LEAF_VALUES, n=n, d=d, n_nodes=n_leaves)
        if self._ws_leaf is None or self._ws_leaf.numel() < need:
            self._ws_leaf = workspace(need, self.device)
        if self.V is None or self.V.shape != (n_leaves, d):
            self.V = torch.zeros((n_leaves, d), dtype=torch.float64, device=self.device)
        L.sb_leaf_values(G_T, n, d, n, hess_T, n, h, self.row_idx, self.leaf_off, n_leaves, self.lam, self.V, d,
                         self._ws_leaf, self._ws_leaf.numel(), stream)
        return self.V

    def leaf_values_from_loss(self, loss, G_T, labels=None, Y=None, stream=None):
        """Leaf values with the cross-entropy hessians formed from G and the targets (eq. 3)."""
        d, n = G_T.shape
        n_leaves = 1 << self.depth
        need = L.sb_workspace_bytes(L.SB_CALL_LEAF_VALUES, n=n, d=d, n_nodes=n_leaves)
        if self._ws_leaf is None or self._ws_leaf.numel() < need:
            self._ws_leaf = workspace(need, self.device)
        if self.V is None or self.V.shape != (n_leaves, d):
            self.V = torch.zeros((n_leaves, d), dtype=torch.float64, device=self.device)
        L.sb_leaf_values_from_loss(L.LOSS[loss], G_T, n, d, n, labels, Y, n, self.row_idx, self.leaf_off, n_leaves,
                                   self.lam, self.V, d, self._ws_leaf, self._ws_leaf.numel(), stream)
        return self.V

    # ------------------------------------------------------------ readback
    def gh(self):
        """The sketch as an (n, k+1) float32 host array."""
        return np.ascontiguousarray(self.GH[:, :self.c].cpu().numpy())

    def gh_padding(self):
        """The padding floats of the sketch rows (written as 0)."""
        return self.GH[:, self.c:].cpu().numpy()

    def tree(self):
        """Host copies of the tree arrays, split per level."""
        f = self.tree_feature.cpu().numpy()
        b = self.tree_bin.cpu().numpy()
        s = self.tree_score.cpu().numpy()
        out = {"feature": [], "bin": [], "score": []}
        for l in range(self.depth):
            lo, hi = (1 << l) - 1, (1 << (l + 1)) - 1
            out["feature"].append(f[lo:hi])
            out["bin"].append(b[lo:hi])
            out["score"].append(s[lo:hi])
        out["row_idx"] = self.row_idx.cpu().numpy()
        out["leaf_off"] = self.leaf_off.cpu().numpy()
        return out


class Booster:
    """The boosting loop on the device (Section 2), one tree per ``step()``:

    1. derivatives of the loss at the current scores F (eq. 2), with the
       column norms of G, in one pass (``sb_gradients``);
    2. the sketch from those norms (``sb_sketch_given_norms``), with the
       split-search weight h = 1 for softmax (the count weight of S_G) and the
       row mean of the hessians for sigmoid;
    3. the tree (``sb_grow_tree``);
    4. leaf values from the full G and the per-element hessians (eq. 3),
       which ``sb_leaf_values_from_loss`` forms from G and the targets
       instead of storing them;
    5. F += lr * f_t.  The update is held until the next step, whose first
       call applies it and takes the derivatives at the new scores in one pass
       (``sb_update_and_gradients``); reading ``F`` (or ``flush()``) applies a
       held update on its own (``sb_update_predictions``).

    F, G and the hessians are (d, n) float32 device tensors (column-major).
    """

    def __init__(self, bins, n_bins, d, loss, kind, k, depth, lam=1.0, lr=0.01, min_child_weight=0.0,
                 device="cuda", F0=None):
        self.ss = SplitSearch(bins, n_bins, k, depth, lam, min_child_weight, device=device)
        dev, n = self.ss.device, self.ss.n
        self.n, self.d, self.loss, self.kind, self.lr = n, d, loss, kind, float(lr)
        self._F = torch.zeros((d, n), dtype=torch.float32, device=dev) if F0 is None else F0.clone()
        self.G = torch.empty((d, n), dtype=torch.float32, device=dev)
        self.h_row = torch.empty(n, dtype=torch.float32, device=dev)
        self.ones = torch.ones(n, dtype=torch.float32, device=dev)
        self.norm2 = torch.zeros(d, dtype=torch.float64, device=dev)
        self.ws_grad = workspace(L.sb_workspace_bytes(L.SB_CALL_GRADIENTS, n=n, d=d), dev)
        self.ws_upd = workspace(L.sb_workspace_bytes(L.SB_CALL_UPDATE_PREDICTIONS, n=n), dev)
        self.ws_upd_grad = workspace(L.sb_workspace_bytes(L.SB_CALL_UPDATE_AND_GRADIENTS, n=n, d=d), dev)
        self.labels = None
        self.Y = None
        self.pending = None  # leaf values of the last tree, not yet added to F

    @property
    def F(self):
        """The scores, with every grown tree added."""
        self.flush()
        return self._F

    def flush(self, stream=None):
        """Add a held update (the last tree's leaf values) to F."""
        if self.pending is not None:
            V = self.pending
            L.sb_update_predictions(self._F, self.n, self.d, self.n, self.ss.row_idx, self.ss.leaf_off, V.shape[0], V,
                                    self.d, self.lr, self.ws_upd, self.ws_upd.numel(), stream)
            self.pending = None

    def set_target(self, target):
        """Labels (n,) int32 for softmax, or a (d, n) uint8 0/1 matrix for sigmoid (device tensors)."""
        if self.loss == "softmax":
            self.labels = target
        else:
            self.Y = target

    def gradients(self, stream=None):
        """Derivatives at the current scores (a held update is applied first, in the same pass)."""
        n, d = self.n, self.d
        h_row = self.h_row if self.loss == "sigmoid" else None
        if self.pending is not None:
            V = self.pending
            L.sb_update_and_gradients(L.LOSS[self.loss], self._F, n, d, n, self.ss.row_idx, self.ss.leaf_off,
                                      V.shape[0], V, d, self.lr, self.labels, self.Y, n, self.G, n, None, 0, h_row,
                                      self.norm2, self.ws_upd_grad, self.ws_upd_grad.numel(), stream)
            self.pending = None
        else:
            L.sb_gradients(L.LOSS[self.loss], self._F, n, d, n, self.labels, self.Y, n, self.G, n, None, 0, h_row,
                           self.norm2, self.ws_grad, self.ws_grad.numel(), stream)

    def step(self, u=None, Pi=None, stream=None):
        self.gradients(stream)
        h = self.ones if self.loss == "softmax" else self.h_row
        self.ss.sketch(self.kind, self.G, h, u=u, Pi=Pi, stream=stream, norm2_in=self.norm2)
        self.ss.grow(stream)
        # the tree's leaf segments stay in ss.row_idx / ss.leaf_off until the next grow
        self.pending = self.ss.leaf_values_from_loss(self.loss, self.G, self.labels, self.Y, stream=stream)
