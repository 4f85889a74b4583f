"""C-ABI contract checks that need no GPU.

The library must load, export every function include/sb.h declares, and
reject bad arguments on the host with the documented status before any
device work (these calls never reach a kernel launch).
"""
import os
import re
import subprocess

import pytest

from paper_2211_12858_amd import build as sb_build

HDR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "sb.h")
FAKE = 0x100000  # non-NULL address that is never dereferenced (validation fails first)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sb_build.LIB):
        sb_build.build()
    from paper_2211_12858_amd import _lib
    _lib.load()
    return _lib


def header_functions():
    text = open(HDR).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**\s*(sb_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    fns = header_functions()
    for name in ("sb_sketch", "sb_build_histograms", "sb_subtract_histograms", "sb_score_splits",
                 "sb_partition_rows", "sb_layout_bins", "sb_grow_tree", "sb_leaf_values", "sb_gradients",
                 "sb_update_predictions", "sb_update_and_gradients", "sb_sketch_given_norms",
                 "sb_sketch_sparse_projection", "sb_last_error",
                 "sb_abi_version", "sb_workspace_bytes"):
        assert name in fns


def test_every_declared_symbol_is_exported(L):
    fns = header_functions()
    out = subprocess.run(["nm", "-D", "--defined-only", sb_build.LIB], capture_output=True, text=True, check=True).stdout
    exported = set(ln.split()[-1] for ln in out.splitlines() if ln.strip())
    missing = [f for f in fns if f not in exported]
    assert not missing, missing
    assert sorted(L.SYMBOLS) == fns


def test_version_and_error_text(L):
    assert L.sb_abi_version() == 4
    assert isinstance(L.sb_last_error(), str)


def test_workspace_bytes(L):
    assert L.sb_workspace_bytes(L.SB_CALL_SKETCH, n=1000, d=20, k=5) > 0
    assert L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=1000, m=100, n_bins=256, k=5, n_nodes=16) > 0
    assert L.sb_workspace_bytes(L.SB_CALL_SCORE_SPLITS, m=100, n_nodes=32) >= 32 * 100 * 12
    assert L.sb_workspace_bytes(L.SB_CALL_PARTITION_ROWS, n=10_000, n_nodes=8) >= 10_000 // 8  # one flag bit per row
    assert L.sb_workspace_bytes(L.SB_CALL_GROW_TREE, n=10_000, m=10, n_bins=256, k=5, depth=3) > 0
    with pytest.raises(L.SBError):
        L.sb_workspace_bytes(L.SB_CALL_GROW_TREE, n=10, m=10, n_bins=256, k=5, depth=13)
    assert L.sb_workspace_bytes(L.SB_CALL_LEAF_VALUES, n=10_000, d=100, n_nodes=64) >= 10_000 * 2
    with pytest.raises(L.SBError):
        L.sb_workspace_bytes(L.SB_CALL_LEAF_VALUES, n=10_000, d=100, n_nodes=4097)
    with pytest.raises(L.SBError):
        L.sb_workspace_bytes(99)
    with pytest.raises(L.SBError):  # 101 channels: more than the histogram kernels take
        L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=10, m=8, n_bins=256, k=100, n_nodes=1)


# Sizes from the valid range to the extremes of their C types, one argument
# at a time and all together: every answer is a size or -1 with an error
# text.  Run under UBSan (test_abi_sanitize.py) this also checks that no size
# arithmetic overflows.
EXTREMES = {
    "n": [-1, 0, 1, 2**31 - 1, 2**31, 2**40, 2**62, 2**63 - 1],
    "m": [-1, 0, 1, 2**16, 2**31 - 1, -2**31],
    "n_bins": [-1, 0, 1, 2, 256, 257, 2**31 - 1],
    "d": [-1, 0, 1, 2**20, 2**31 - 1],
    "k": [-1, 0, 1, 23, 24, 255, 2**31 - 1],
    "n_nodes": [-1, 0, 1, 4096, 4097, 2**31 - 1],
    "depth": [-1, 0, 1, 12, 13, 2**31 - 1],
}


def test_workspace_bytes_at_extreme_sizes(L):
    lib = L.load()
    base = dict(n=1000, m=100, n_bins=256, d=100, k=5, n_nodes=16, depth=6)
    order = ["n", "m", "n_bins", "d", "k", "n_nodes", "depth"]
    cases = []
    for name, values in EXTREMES.items():
        for v in values:
            cases.append(dict(base, **{name: v}))
    cases.append({name: values[-1] for name, values in EXTREMES.items()})
    cases.append({name: values[0] for name, values in EXTREMES.items()})
    for call in range(-1, 10):
        for kw in cases:
            got = lib.sb_workspace_bytes(call, *[kw[o] for o in order])
            assert got == -1 or 0 <= got < 2**62, (call, kw, got)
            if got == -1:
                assert L.sb_last_error(), (call, kw)


# The histogram kernels add at most 24 channels (k <= 23).  Every wider
# sketch is refused on the host, whatever the bin count: the sizes query
# returns -1 and the calls return SB_E_UNSUPPORTED before any device work.
@pytest.mark.parametrize("k,n_bins", [(24, 256), (25, 256), (26, 256), (27, 256), (28, 256), (29, 256),
                                      (40, 64), (100, 64), (24, 2)])
def test_histogram_calls_refuse_more_than_24_channels(L, k, n_bins):
    for call, kw in ((L.SB_CALL_BUILD_HISTOGRAMS, dict(n_nodes=1)), (L.SB_CALL_GROW_TREE, dict(depth=3))):
        with pytest.raises(L.SBError):
            L.sb_workspace_bytes(call, n=1000, m=10, n_bins=n_bins, k=k, **kw)
    ld_gh = (k + 1 + 7) // 8 * 8
    assert _code(L.sb_build_histograms, *hist_args(k=k, n_bins=n_bins, ld_gh=ld_gh)) == 3
    assert "24 channels" in L.sb_last_error()
    assert _code(L.sb_grow_tree, *grow_args(k=k, n_bins=n_bins, ld_gh=ld_gh)) == 3
    assert "24 channels" in L.sb_last_error()


@pytest.mark.parametrize("k,n_bins", [(23, 256), (23, 64), (20, 256), (5, 256), (1, 2)])
def test_histogram_calls_accept_up_to_24_channels(L, k, n_bins):
    assert L.sb_workspace_bytes(L.SB_CALL_BUILD_HISTOGRAMS, n=1000, m=10, n_bins=n_bins, k=k, n_nodes=1) > 0
    assert L.sb_workspace_bytes(L.SB_CALL_GROW_TREE, n=1000, m=10, n_bins=n_bins, k=k, depth=3) > 0


def _code(fn, *args):
    from paper_2211_12858_amd import _lib
    with pytest.raises(_lib.SBError) as e:
        fn(*args)
    return e.value.code


F = FAKE


def sketch_args(**kw):
    a = dict(kind=0, G=F, n=100, d=10, ld_g=100, h=F, k=3, u=F, Pi=F, GH=F, ld_gh=8, cols=F, scales=F, norm2=F,
             qexp=F, ws=F, ws_bytes=1 << 30, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(kind=7), 3),
    (dict(G=None), 1),
    (dict(n=0), 1),
    (dict(k=0), 1),
    (dict(k=11, ld_gh=12), 1),       # top outputs needs k <= d
    (dict(ld_g=99), 2),
    (dict(ld_gh=3), 2),              # row-major GH needs ld_gh >= k + 1
    (dict(GH=F + 4), 2),             # GH rows need a 16-byte aligned base
    (dict(kind=1, u=None), 1),
    (dict(kind=2, Pi=None), 1),
    (dict(kind=3, k=4), 1),          # identity needs k == d
    (dict(ws_bytes=16), 1),
    (dict(ws=F + 8), 2),             # misaligned workspace
    (dict(ws=None), 1),
])
def test_sketch_rejects(L, kw, code):
    assert _code(L.sb_sketch, *sketch_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_sketch")


def hist_args(**kw):
    a = dict(bins4=F, ld4=1000, rec=None, ld_rec=0, n=1000, m=10, n_bins=256, GH=F, ld_gh=8, k=5, qexp=F,
             row_idx=None, node_off=F, n_nodes=2, build_list=F, n_build=1, H=F, ws=F, ws_bytes=1 << 30, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(bins4=None), 1),
    (dict(H=None), 1),
    (dict(n=0), 1),
    (dict(m=0), 1),
    (dict(n_bins=1), 1),
    (dict(n_bins=257), 1),
    (dict(k=0), 1),
    (dict(ld4=999), 2),              # < n
    (dict(bins4=F + 2), 2),          # misaligned base
    (dict(ld_gh=5), 2),              # fewer floats per row than channels
    (dict(GH=None), 1),
    (dict(row_idx=F), 1),            # rows through row_idx need the records
    (dict(row_idx=F, rec=F, ld_rec=8), 2),     # records shorter than m
    (dict(row_idx=F, rec=F, ld_rec=40), 2),    # stride not a multiple of 16
    (dict(n_nodes=0), 1),
    (dict(n_build=3), 1),            # more than n_nodes
    (dict(k=100, ld_gh=104), 3),     # more than 24 channels
    (dict(k=24, ld_gh=32), 3),
    (dict(ws_bytes=100), 1),
])
def test_build_histograms_rejects(L, kw, code):
    assert _code(L.sb_build_histograms, *hist_args(**kw)) == code


def test_subtract_rejects(L):
    assert _code(L.sb_subtract_histograms, F, F, 0, 10, 256, 5, F, 0) == 1
    assert _code(L.sb_subtract_histograms, None, F, 1, 10, 256, 5, F, 0) == 1
    assert _code(L.sb_subtract_histograms, F, F, 1, 10, 300, 5, F, 0) == 1


def score_args(**kw):
    a = dict(H=F, n_nodes=4, m=10, n_bins=256, k=5, lam=1.0, mcw=0.0, bf=F, bb=F, bs=F, ws=F, ws_bytes=1 << 30,
             stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(H=None), 1),
    (dict(bs=None), 1),
    (dict(n_nodes=0), 1),
    (dict(lam=0.0), 1),
    (dict(lam=float("nan")), 1),
    (dict(mcw=-1.0), 1),
    (dict(ws_bytes=8), 1),
])
def test_score_rejects(L, kw, code):
    assert _code(L.sb_score_splits, *score_args(**kw)) == code


def part_args(**kw):
    a = dict(bins_cm=F, n=1000, m=10, ld_cm=1000, row_in=F, off_in=F, n_nodes=2, bf=F, bb=F, row_out=F + 100000,
             off_out=F, build_out=F, ws=F, ws_bytes=1 << 30, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(bins_cm=None), 1),
    (dict(row_out=None), 1),
    (dict(n=0), 1),
    (dict(ld_cm=999), 2),
    (dict(n_nodes=0), 1),
    (dict(row_out=F + 100), 2),      # overlaps row_in
    (dict(ws_bytes=10), 1),
])
def test_partition_rejects(L, kw, code):
    assert _code(L.sb_partition_rows, *part_args(**kw)) == code


def test_partition_noalloc_rejects(L):
    """The allocation-free partition checks its arguments like sb_partition_rows and refuses sizes
    beyond its static scratch before any device work."""
    args = dict(bins_cm=F, n=1000, m=10, ld_cm=1000, row_idx_in=None, node_off_in=F, n_nodes=4, best_feature=F,
                best_bin=F, row_idx_out=F, node_off_out=F, build_list_out=F, stream=0)

    def call(**kw):
        a = dict(args)
        a.update(kw)
        return _code(L.sb_partition_rows_noalloc, *a.values())

    assert call(bins_cm=None) == 1
    assert call(n=0) == 1
    assert call(ld_cm=999) == 2
    assert call(n_nodes=0) == 1
    assert call(row_idx_in=F, row_idx_out=F + 100) == 2          # overlapping row buffers
    n_big = (1 << 31) - 1                                          # needs ~280 MB of scratch
    assert call(n=n_big, ld_cm=n_big) == 3
    assert "static scratch" in L.sb_last_error()
    assert L.sb_workspace_bytes(L.SB_CALL_PARTITION_ROWS, n=50_000_000, n_nodes=64) <= 8 << 20
    assert L.sb_workspace_bytes(L.SB_CALL_PARTITION_ROWS, n=70_000_000, n_nodes=64) > 8 << 20


def layout_args(**kw):
    a = dict(bins=F, n=1000, m=10, ld_bins=10, bins4=F, ld4=1000, bins_cm=None, ld_cm=0, rec=None, ld_rec=0,
             stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(bins=None), 1),
    (dict(n=0), 1),
    (dict(ld_bins=9), 2),
    (dict(ld4=999), 2),
    (dict(bins_cm=F, ld_cm=10), 2),
    (dict(rec=F, ld_rec=24), 2),
    (dict(rec=F, ld_rec=8), 2),
])
def test_layout_rejects(L, kw, code):
    assert _code(L.sb_layout_bins, *layout_args(**kw)) == code


def grow_args(**kw):
    a = dict(bins4=F, ld4=1000, bins_cm=F, ld_cm=1000, rec=F, ld_rec=16, n=1000, m=10, n_bins=256, GH=F,
             ld_gh=8, k=5, qexp=F, depth=3, lam=1.0, mcw=0.0, tf=F, tb=F, ts=F, rows=F, leaf=F, ws=F,
             ws_bytes=1 << 34, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(bins4=None), 1),
    (dict(rec=None), 1),
    (dict(depth=0), 1),
    (dict(depth=13), 1),
    (dict(ld_cm=10), 2),
    (dict(ld4=999), 2),
    (dict(ld_gh=5), 2),
    (dict(ld_rec=8), 2),
    (dict(ld_rec=24), 2),
    (dict(lam=-1.0), 1),
    (dict(ws_bytes=1000), 1),
])
def test_grow_tree_rejects(L, kw, code):
    assert _code(L.sb_grow_tree, *grow_args(**kw)) == code


def leaf_args(**kw):
    a = dict(G=F, n=1000, d=10, ld_g=1000, hess=None, ld_hess=0, h=None, row_idx=F, leaf_off=F, n_leaves=64,
             lam=1.0, V=F, ld_v=10, ws=F, ws_bytes=1 << 30, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(G=None), 1),
    (dict(V=None), 1),
    (dict(row_idx=None), 1),
    (dict(n=0), 1),
    (dict(d=0), 1),
    (dict(n_leaves=0), 1),
    (dict(n_leaves=4097), 1),
    (dict(ld_g=999), 2),
    (dict(hess=F, ld_hess=999), 2),
    (dict(ld_v=9), 2),
    (dict(lam=0.0), 1),
    (dict(lam=float("inf")), 1),
    (dict(ws_bytes=100), 1),
    (dict(ws=F + 8), 2),
])
def test_leaf_values_rejects(L, kw, code):
    assert _code(L.sb_leaf_values, *leaf_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_leaf_values")


@pytest.mark.parametrize("kw,code", [(dict(kind=7), 3), (dict(norm2=None), 1), (dict(ld_gh=3), 2)])
def test_sketch_given_norms_rejects(L, kw, code):
    assert _code(L.sb_sketch_given_norms, *sketch_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_sketch_given_norms")


def sparse_args(**kw):
    a = dict(G=F, n=100, d=10, ld_g=100, h=F, k=5, s=1, pi_col=F, pi_val=F, GH=F, ld_gh=8, qexp=F, ws=F,
             ws_bytes=1 << 30, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(G=None), 1),
    (dict(pi_col=None), 1),
    (dict(k=0), 1),
    (dict(s=3), 3),
    (dict(ld_g=99), 2),
    (dict(ld_gh=5), 2),
    (dict(ws_bytes=16), 1),
])
def test_sketch_sparse_rejects(L, kw, code):
    assert _code(L.sb_sketch_sparse_projection, *sparse_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_sketch_sparse_projection")


def grad_args(**kw):
    a = dict(loss=0, F=F, n=1000, d=10, ld_f=1000, labels=F, Y=None, ld_y=0, G=F + 10 ** 6, ld_g=1000, hess=None,
             ld_hess=0, h_row=None, norm2=None, ws=None, ws_bytes=0, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(loss=2), 3),
    (dict(F=None), 1),
    (dict(labels=None), 1),
    (dict(loss=1, labels=None), 1),          # sigmoid needs Y
    (dict(loss=1, Y=F, ld_y=10), 2),
    (dict(n=0), 1),
    (dict(d=0), 1),
    (dict(ld_f=999), 2),
    (dict(ld_g=999), 2),
    (dict(hess=F, ld_hess=5), 2),
    (dict(G=F + 400), 2),                    # G overlaps F
    (dict(norm2=F), 1),                      # norms need a workspace
])
def test_gradients_rejects(L, kw, code):
    assert _code(L.sb_gradients, *grad_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_gradients")


def upd_args(**kw):
    a = dict(F=F, n=1000, d=10, ld_f=1000, row_idx=F, leaf_off=F, n_leaves=64, V=F, ld_v=10, lr=0.1, ws=F,
             ws_bytes=1 << 20, stream=0)
    a.update(kw)
    return list(a.values())


@pytest.mark.parametrize("kw,code", [
    (dict(F=None), 1),
    (dict(V=None), 1),
    (dict(n=0), 1),
    (dict(n_leaves=5000), 1),
    (dict(ld_f=10), 2),
    (dict(ld_v=9), 2),
    (dict(lr=float("nan")), 1),
    (dict(ws_bytes=16), 1),
])
def test_update_rejects(L, kw, code):
    assert _code(L.sb_update_predictions, *upd_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_update_predictions")


def upd_grad_args(**kw):
    a = dict(loss=0, F=F, n=1000, d=10, ld_f=1000, row_idx=F, leaf_off=F, n_leaves=64, V=F, ld_v=10, lr=0.1,
             labels=F, Y=None, ld_y=0, G=F + 10 ** 6, ld_g=1000, hess=None, ld_hess=0, h_row=None, norm2=None, ws=F,
             ws_bytes=1 << 20, stream=0)
    a.update(kw)
    return list(a.values())


# The fused call refuses what either of its two steps refuses, with its own name.
@pytest.mark.parametrize("kw,code", [
    (dict(loss=2), 3),
    (dict(F=None), 1),
    (dict(V=None), 1),
    (dict(labels=None), 1),
    (dict(n=0), 1),
    (dict(d=0), 1),
    (dict(n_leaves=5000), 1),
    (dict(ld_f=999), 2),
    (dict(ld_g=999), 2),
    (dict(ld_v=9), 2),
    (dict(lr=float("inf")), 1),
    (dict(G=F + 400), 2),
    (dict(ws_bytes=16), 1),
])
def test_update_and_gradients_rejects(L, kw, code):
    assert _code(L.sb_update_and_gradients, *upd_grad_args(**kw)) == code
    assert L.sb_last_error().startswith("sb_update_and_gradients")


def test_error_text_is_per_thread(L):
    import threading
    _code(L.sb_grow_tree, *grow_args(depth=0))
    seen = {}

    def other():
        seen["msg"] = L.sb_last_error()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["msg"] == ""
    assert "depth" in L.sb_last_error()
