"""Helpers for the GPU parity tests: upload seeded inputs, call the C ABI, read back.

Expected values always come from ``oracle`` on the same host inputs; nothing
here computes the method.
"""
import math

import numpy as np
import torch

from paper_2211_12858_amd import _lib as L
from paper_2211_12858_amd.driver import workspace

DEV = torch.device("cuda:0")
TOL = 1e-4  # relative tolerance stated for histograms and scores


def up(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def sync():
    torch.cuda.synchronize()


def quad_major(bins):
    """Host copy of the quad-major layout: word q of row i holds features 4q..4q+3."""
    n, m = bins.shape
    nq = (m + 3) // 4
    pad = np.zeros((n, 4 * nq), dtype=np.uint8)
    pad[:, :m] = bins
    return np.ascontiguousarray(pad.view("<u4").reshape(n, nq).T).view(np.int32)


def run_sketch(kind, G_T, h, k, u=None, Pi=None, ld_gh=None):
    """Returns (GH as (n, k+1), cols, scales, norm2, qexp, the padding floats of the rows)."""
    d, n = G_T.shape
    ld_gh = (k + 1 + 7) // 8 * 8 if ld_gh is None else ld_gh
    Gd, hd = up(G_T), up(h)
    GH = torch.full((n, ld_gh), float("nan"), dtype=torch.float32, device=DEV)
    cols = torch.full((k,), -7, dtype=torch.int32, device=DEV)
    scales = torch.zeros(k, dtype=torch.float32, device=DEV)
    norm2 = torch.zeros(d, dtype=torch.float64, device=DEV)
    qexp = torch.zeros(k + 1, dtype=torch.int32, device=DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=n, d=d, k=k), DEV)
    ud = up(u, torch.float64) if u is not None else None
    Pid = up(Pi, torch.float32) if Pi is not None else None
    L.sb_sketch(L.KIND[kind], Gd, n, d, n, hd, k, ud, Pid, GH, ld_gh, cols, scales, norm2, qexp, ws, ws.numel())
    sync()
    g = GH.cpu().numpy()
    return (np.ascontiguousarray(g[:, :k + 1]), cols.cpu().numpy(), scales.cpu().numpy(), norm2.cpu().numpy(),
            qexp.cpu().numpy(), g[:, k + 1:])


def qexp_rule(GH):
    """Exponents by the documented rule, from a host GH (not from the device)."""
    out = []
    for t in range(GH.shape[1]):
        mx = float(np.max(np.abs(GH[:, t].astype(np.float64)))) if GH.shape[0] else 0.0
        out.append(17 - math.frexp(mx)[1] + 1 if mx > 0 else 0)  # 17 - floor(log2 mx)
    return np.array(out, dtype=np.int32)


def run_hist(bins, GH, qexp, n_bins, row_idx, node_off, build_list=None, H=None, ld_pad=0, ld_rec=None, ld_gh=None):
    """Histograms through the C ABI (device layout [node][feature][channel][bin]).

    GH is an (n, k+1) host array, uploaded row-major with ld_gh floats per
    row (default: k+1 rounded up to 8).  Without row_idx the bins go up
    quad-major (leading dimension n + ld_pad); with row_idx as row records of
    ld_rec bytes (default: m rounded up to 16).
    """
    n, m = bins.shape
    c = GH.shape[1]
    k = c - 1
    n_nodes = len(node_off) - 1
    n_build = n_nodes if build_list is None else len(build_list)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=n, m=m, n_bins=n_bins, k=k,
                                        n_nodes=max(n_nodes, n_build)), DEV)
    if H is None:
        H = torch.full((n_nodes, m, c, n_bins), float("nan"), dtype=torch.float64, device=DEV)
    ld_gh = (c + 7) // 8 * 8 if ld_gh is None else ld_gh
    gh = np.zeros((n, ld_gh), dtype=np.float32)
    gh[:, :c] = GH
    b4 = rec = None
    ld = n + ld_pad
    if row_idx is None:
        qm = quad_major(bins)
        b4 = np.zeros((qm.shape[0], ld), dtype=np.int32)
        b4[:, :n] = qm
        b4 = up(b4)
    else:
        if ld_rec is None:
            ld_rec = (m + 15) // 16 * 16
        rec = up(make_records(bins, ld_rec))
    L.sb_build_histograms(b4, ld, rec, ld_rec or 0, n, m, n_bins, up(gh), ld_gh, k, up(qexp, torch.int32),
                          None if row_idx is None else up(row_idx, torch.int32), up(node_off, torch.int32), n_nodes,
                          None if build_list is None else up(build_list, torch.int32), n_build, H, ws, ws.numel())
    sync()
    return H


def host_layout(H):
    """Device histograms [node][feature][channel][bin] as [node][feature][bin][channel] (the oracle's layout)."""
    return np.ascontiguousarray(np.swapaxes(np.asarray(H), -1, -2))


def hist_tolerance_ok(Hg, Ho, counts, qexp, mass, chan_max):
    """Check a device histogram against the oracle's.

    Two bars: (1) the fixed-point bound, |Hg - Ho| <= count * 2^-(qexp+1),
    exact arithmetic plus fp64 rounding of the oracle's own sum; (2) the
    stated 1e-4 relative bar, relative to the larger of |Ho| and the cell's
    absolute mass (sums of mixed-sign gradients cancel), with an absolute
    floor of 1e-4 of one maximal row of that channel (chan_max).
    """
    half_q = np.ldexp(1.0, -(qexp.astype(np.int64) + 1))
    bound1 = counts[..., None] * half_q + 1e-12 * mass
    err = np.abs(Hg - Ho)
    ok1 = err <= bound1
    scale = np.maximum(np.maximum(np.abs(Ho), mass), chan_max)
    ok2 = err <= TOL * scale
    return bool(ok1.all()), bool(ok2.all()), float((err / scale).max())


def run_score(H_np, n_bins, k, lam=1.0, mcw=0.0):
    """H_np in the oracle's layout [node][feature][bin][channel]."""
    n_nodes, m = H_np.shape[:2]
    Hd = up(host_layout(H_np), torch.float64)
    bf = torch.zeros(n_nodes, dtype=torch.int32, device=DEV)
    bb = torch.zeros(n_nodes, dtype=torch.int32, device=DEV)
    bs = torch.zeros(n_nodes, dtype=torch.float64, device=DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_SCORE_SPLITS, m=m, n_nodes=n_nodes), DEV)
    L.sb_score_splits(Hd, n_nodes, m, n_bins, k, lam, mcw, bf, bb, bs, ws, ws.numel())
    sync()
    return bf.cpu().numpy(), bb.cpu().numpy(), bs.cpu().numpy()


def run_partition(bins, row_in, node_off, bf, bb):
    n, m = bins.shape
    n_nodes = len(node_off) - 1
    bins_cm = up(np.ascontiguousarray(bins.T))
    row_out = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    off_out = torch.full((2 * n_nodes + 1,), -1, dtype=torch.int32, device=DEV)
    bl_out = torch.full((n_nodes,), -1, dtype=torch.int32, device=DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_PARTITION_ROWS, n=n, n_nodes=n_nodes), DEV)
    L.sb_partition_rows(bins_cm, n, m, n, None if row_in is None else up(row_in, torch.int32),
                        up(node_off, torch.int32), n_nodes, up(bf, torch.int32), up(bb, torch.int32), row_out, off_out,
                        bl_out, ws, ws.numel())
    sync()
    return row_out.cpu().numpy(), off_out.cpu().numpy(), bl_out.cpu().numpy()


def make_records(bins, ld_rec):
    """Host row records: the m bins of row i in bytes 0..m-1 of record i."""
    n, m = bins.shape
    rec = np.zeros((n, ld_rec), dtype=np.uint8)
    rec[:, :m] = bins
    return rec


def run_leaf(G_T, row_idx, leaf_off, lam, hess_T=None, h=None, ld_v=None, device_G=None):
    """sb_leaf_values on host inputs (G_T, hess_T: (d, n) column-major).  Returns V (n_leaves, d)."""
    d, n = G_T.shape if device_G is None else device_G.shape
    n_leaves = len(leaf_off) - 1
    ld_v = d if ld_v is None else ld_v
    Gd = up(G_T) if device_G is None else device_G
    Hd = up(hess_T) if hess_T is not None else None
    hd = up(h) if h is not None else None
    V = torch.full((n_leaves, ld_v), float("nan"), dtype=torch.float64, device=DEV)
    ws = workspace(L.sb_workspace_bytes(L.SB_CALL_LEAF_VALUES, n=n, d=d, n_nodes=n_leaves), DEV)
    L.sb_leaf_values(Gd, n, d, n, Hd, n, hd, up(np.asarray(row_idx, dtype=np.int32)),
                     up(np.asarray(leaf_off, dtype=np.int32)), n_leaves, lam, V, ld_v, ws, ws.numel())
    sync()
    return V.cpu().numpy()


LEAF_QUANTUM = 2.0 ** -41  # per-element error bound of the leaf sums, relative to the column's largest magnitude


def leaf_value_error_ok(V, V_o, G, rows_of, lam, hess=None, h=None, col_max=None, hess_err=0.0):
    """|V - V_o| within the bound that the fixed-point accumulation and fp64 sums allow.

    The numerator and denominator sums carry at most n_L * 2^-41 * M (M: the
    column's largest magnitude over all rows) plus 1e-13 of the leaf's absolute
    mass; the quotient adds both relative errors and one rounding.
    col_max: the columns' largest magnitudes over all n rows, when G holds only
    some of them.  hess_err: a per-element error of the hessians themselves
    (formed on the device rather than read).  Returns (ok, worst ratio of
    error to bound)."""
    G = np.asarray(G, dtype=np.float64)
    Mg = np.abs(G).max(axis=0) if col_max is None else np.asarray(col_max, dtype=np.float64)
    worst = 0.0
    for Lf, rows in enumerate(rows_of):
        nL = rows.shape[0]
        A = np.abs(G[rows]).sum(axis=0)
        eg = nL * LEAF_QUANTUM * Mg + 1e-13 * A
        if hess is not None:
            Hh = np.asarray(hess, dtype=np.float64)
            hs = Hh[rows].sum(axis=0)
            eh = nL * LEAF_QUANTUM * np.abs(Hh).max(axis=0) + 1e-13 * hs + nL * hess_err
        elif h is not None:
            hh = np.asarray(h, dtype=np.float64)
            hs = np.full(G.shape[1], hh[rows].sum())
            eh = nL * LEAF_QUANTUM * np.abs(hh).max() + 1e-13 * hs
        else:
            hs = np.full(G.shape[1], float(nL))
            eh = np.zeros(G.shape[1])
        den = hs + lam
        bound = eg / den + np.abs(V_o[Lf]) * eh / den + 4e-16 * np.abs(V_o[Lf]) + 1e-300
        ratio = np.abs(V[Lf] - V_o[Lf]) / bound
        worst = max(worst, float(ratio.max()))
    return worst <= 1.0, worst
