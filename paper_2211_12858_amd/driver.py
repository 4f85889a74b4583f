"""Device-side driver: torch allocates the buffers, libsketchboost computes.

``SplitSearch`` holds one binned dataset resident in HBM in the two layouts
the kernels read:

* row records for the histogram kernel: row i occupies ``rec_stride`` bytes,
  its m bin bytes first and, when ``interleave`` is set, its k+1 sketch
  floats after them (at an 8-byte aligned offset).  With 100 features and
  k = 5 each row is exactly one 128-byte cache line, so gathering the rows
  of a node fetches nothing it does not use.  Otherwise the sketch lives in
  its own compact (n, k+1) array;
* a column-major copy (feature-major, ``bins_cm[f, i]``) for the partition,
  which then reads one contiguous run of one feature column per node.

``step()`` runs one tree: sketch (once per tree) and the depth-wise level
loop, entirely on the device.  No computation happens in Python.
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


class SplitSearch:
    def __init__(self, bins, n_bins, k, depth, lam=1.0, min_child_weight=0.0, device="cuda", interleave=True):
        bins = np.ascontiguousarray(bins, dtype=np.uint8)
        self.n, self.m = bins.shape
        self.n_bins, self.k, self.c, self.depth = n_bins, k, k + 1, depth
        self.lam, self.mcw = float(lam), float(min_child_weight)
        self.device = torch.device(device)
        n, m, c = self.n, self.m, self.c
        self.ld_bins = _round_up(m, 4)
        if interleave:
            self.gh_offset = _round_up(self.ld_bins, 8)
            self.rec_stride = _round_up(self.gh_offset + 4 * c, 128)
        else:
            self.gh_offset = None
            self.rec_stride = self.ld_bins
        rec = np.zeros((n, self.rec_stride), dtype=np.uint8)
        rec[:, :m] = bins
        self.rec = torch.from_numpy(rec).to(self.device)
        self.bins_cm = torch.from_numpy(np.ascontiguousarray(bins.T)).to(self.device)
        if interleave:
            self.GH = None
            self.gh_ptr = self.rec.data_ptr() + self.gh_offset
            self.ld_gh = self.rec_stride // 4
        else:
            self.GH = torch.zeros((n, c), dtype=torch.float32, device=self.device)
            self.gh_ptr = self.GH.data_ptr()
            self.ld_gh = c
        dev = self.device
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

    # ------------------------------------------------------------ sketch
    def sketch(self, kind, G_T, h, u=None, Pi=None, stream=None):
        """G_T: (d, n) float32 device tensor (column-major G); h: (n,) float32."""
        d, n = G_T.shape
        assert n == self.n and G_T.is_contiguous() and G_T.dtype == torch.float32
        kid = L.KIND[kind]
        need = L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=self.k)
        if self._ws_sketch is None or self._ws_sketch.numel() < need:
            self._ws_sketch = workspace(need, self.device)
        if self.norm2 is None or self.norm2.numel() != d:
            self.norm2 = torch.zeros(d, dtype=torch.float64, device=self.device)
        L.sb_sketch(kid, G_T, n, d, n, h, self.k, u, Pi, self.gh_ptr, self.ld_gh, self.cols, self.scales,
                    self.norm2, self.qexp, self._ws_sketch, self._ws_sketch.numel(), stream)

    # ------------------------------------------------------------ tree
    def grow(self, stream=None):
        L.sb_grow_tree(self.rec, self.rec_stride, self.bins_cm, self.n, self.n, self.m, self.n_bins, self.gh_ptr,
                       self.ld_gh, self.k, self.qexp, self.depth, self.lam, self.mcw, self.tree_feature,
                       self.tree_bin, self.tree_score, self.row_idx, self.leaf_off, self.ws_tree,
                       self.ws_tree_bytes, stream)

    def step(self, kind, G_T, h, u=None, Pi=None, stream=None):
        self.sketch(kind, G_T, h, u, Pi, stream)
        self.grow(stream)

    # ------------------------------------------------------------ readback
    def gh(self):
        """The sketch records as an (n, k+1) float32 host array."""
        if self.GH is not None:
            return self.GH.cpu().numpy()
        raw = self.rec[:, self.gh_offset:self.gh_offset + 4 * self.c].contiguous()
        return raw.view(torch.float32).cpu().numpy().reshape(self.n, self.c)

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
