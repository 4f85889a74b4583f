"""Thin ctypes binding of libsketchboost.so, one Python function per C entry point.

Argument marshalling only: every array argument may be a torch tensor (its
device pointer is passed), a raw integer address, or None (NULL).  A non-zero
status raises :class:`SBError` carrying the library's error text.  The
functions enqueue work on ``stream`` (a torch.cuda.Stream, a raw hipStream_t
integer, or None for torch's current stream) and return immediately.

Importing this module never falls back to anything: the library must be
built (``python -m paper_2211_12858_amd.build``).
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# SKETCHBOOST_LIB names another build of the same library (the host-side
# sanitizer build of the ABI tests); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("SKETCHBOOST_LIB") or os.path.join(HERE, "libsketchboost.so")

SB_OK, SB_E_ARG, SB_E_SHAPE, SB_E_UNSUPPORTED, SB_E_DEVICE = 0, 1, 2, 3, 4
SB_SKETCH_TOP_OUTPUTS, SB_SKETCH_RANDOM_SAMPLING, SB_SKETCH_RANDOM_PROJECTION, SB_SKETCH_IDENTITY = 0, 1, 2, 3
(SB_CALL_SKETCH, SB_CALL_BUILD_HISTOGRAMS, SB_CALL_SCORE_SPLITS, SB_CALL_PARTITION_ROWS, SB_CALL_GROW_TREE,
 SB_CALL_HIST_EXPONENTS, SB_CALL_LEAF_VALUES, SB_CALL_GRADIENTS, SB_CALL_UPDATE_PREDICTIONS,
 SB_CALL_UPDATE_AND_GRADIENTS) = range(10)
SB_LOSS_SOFTMAX_CE, SB_LOSS_SIGMOID_BCE = 0, 1
LOSS = {"softmax": SB_LOSS_SOFTMAX_CE, "sigmoid": SB_LOSS_SIGMOID_BCE}

KIND = {
    "top_outputs": SB_SKETCH_TOP_OUTPUTS,
    "random_sampling": SB_SKETCH_RANDOM_SAMPLING,
    "random_projection": SB_SKETCH_RANDOM_PROJECTION,
    "identity": SB_SKETCH_IDENTITY,
}

# Exported C symbols (kept in step with include/sb.h).
SYMBOLS = (
    "sb_last_error",
    "sb_abi_version",
    "sb_workspace_bytes",
    "sb_layout_bins",
    "sb_sketch",
    "sb_sketch_given_norms",
    "sb_sketch_sparse_projection",
    "sb_hist_exponents",
    "sb_build_histograms",
    "sb_subtract_histograms",
    "sb_score_splits",
    "sb_partition_rows",
    "sb_partition_rows_noalloc",
    "sb_grow_tree",
    "sb_leaf_values",
    "sb_leaf_values_from_loss",
    "sb_gradients",
    "sb_update_predictions",
    "sb_update_and_gradients",
    "sb_profile_begin",
    "sb_profile_end",
)


class SBError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("libsketchboost status %d: %s" % (code, msg))
        self.code = code


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_U64 = ctypes.c_uint64
_F64 = ctypes.c_double

_PROTOS = {
    "sb_last_error": (ctypes.c_char_p, []),
    "sb_abi_version": (_I32, []),
    "sb_workspace_bytes": (_I64, [_I32, _I64, _I32, _I32, _I32, _I32, _I32, _I32]),
    "sb_layout_bins": (_I32, [_P, _I64, _I32, _I64, _P, _I64, _P, _I64, _P, _I64, _P]),
    "sb_sketch": (_I32, [_I32, _P, _I64, _I32, _I64, _P, _I32, _P, _P, _P, _I64, _P, _P, _P, _P, _P, _I64, _P]),
    "sb_hist_exponents": (_I32, [_P, _I64, _I64, _I32, _P, _P, _I64, _P]),
    "sb_build_histograms": (_I32, [_P, _I64, _P, _I64, _I64, _I32, _I32, _P, _I64, _I32, _P, _P, _P, _I32, _P,
                                   _I32, _P, _P, _I64, _P]),
    "sb_subtract_histograms": (_I32, [_P, _P, _I32, _I32, _I32, _I32, _P, _P]),
    "sb_score_splits": (_I32, [_P, _I32, _I32, _I32, _I32, _F64, _F64, _P, _P, _P, _P, _I64, _P]),
    "sb_partition_rows": (_I32, [_P, _I64, _I32, _I64, _P, _P, _I32, _P, _P, _P, _P, _P, _P, _I64, _P]),
    "sb_partition_rows_noalloc": (_I32, [_P, _I64, _I32, _I64, _P, _P, _I32, _P, _P, _P, _P, _P, _P]),
    "sb_grow_tree": (_I32, [_P, _I64, _P, _I64, _P, _I64, _I64, _I32, _I32, _P, _I64, _I32, _P, _I32, _F64, _F64,
                            _P, _P, _P, _P, _P, _P, _I64, _P]),
}

_PROTOS["sb_leaf_values"] = (_I32, [_P, _I64, _I32, _I64, _P, _I64, _P, _P, _P, _I32, _F64, _P, _I64, _P, _I64,
                                     _P])
_PROTOS["sb_sketch_given_norms"] = _PROTOS["sb_sketch"]
_PROTOS["sb_sketch_sparse_projection"] = (_I32, [_P, _I64, _I32, _I64, _P, _I32, _I32, _P, _P, _P, _I64, _P, _P, _I64,
                                                 _P])
_PROTOS["sb_gradients"] = (_I32, [_I32, _P, _I64, _I32, _I64, _P, _P, _I64, _P, _I64, _P, _I64, _P, _P, _P, _I64, _P])
_PROTOS["sb_leaf_values_from_loss"] = (_I32, [_I32, _P, _I64, _I32, _I64, _P, _P, _I64, _P, _P, _I32, _F64, _P,
                                               _I64, _P, _I64, _P])
_PROTOS["sb_update_predictions"] = (_I32, [_P, _I64, _I32, _I64, _P, _P, _I32, _P, _I64, _F64, _P, _I64, _P])
_PROTOS["sb_update_and_gradients"] = (_I32, [_I32, _P, _I64, _I32, _I64, _P, _P, _I32, _P, _I64, _F64, _P, _P, _I64,
                                             _P, _I64, _P, _I64, _P, _P, _P, _I64, _P])
_PROTOS["sb_profile_begin"] = (_I32, [])
_PROTOS["sb_profile_end"] = (_I32, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)])

_lib = None


def load():
    """Load the shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libsketchboost.so is not built: run `python -m paper_2211_12858_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _PROTOS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(rc):
    if rc != SB_OK:
        raise SBError(rc, sb_last_error())
    return rc


def sb_last_error():
    return load().sb_last_error().decode()


def sb_abi_version():
    return load().sb_abi_version()


def sb_workspace_bytes(call, n=0, m=0, n_bins=0, d=0, k=0, n_nodes=0, depth=0):
    v = load().sb_workspace_bytes(call, n, m, n_bins, d, k, n_nodes, depth)
    if v < 0:
        raise SBError(SB_E_ARG, sb_last_error())
    return v


def sb_layout_bins(bins, n, m, ld_bins, bins4, ld4, bins_cm, ld_cm, rec, ld_rec, stream=None):
    return _check(load().sb_layout_bins(_ptr(bins), n, m, ld_bins, _ptr(bins4), ld4, _ptr(bins_cm), ld_cm, _ptr(rec),
                                        ld_rec, _stream(stream)))


def sb_sketch(kind, G, n, d, ld_g, h, k, u, Pi, GH, ld_gh, cols, scales, norm2, qexp, ws, ws_bytes, stream=None):
    return _check(load().sb_sketch(kind, _ptr(G), n, d, ld_g, _ptr(h), k, _ptr(u), _ptr(Pi), _ptr(GH), ld_gh,
                                   _ptr(cols), _ptr(scales), _ptr(norm2), _ptr(qexp), _ptr(ws), ws_bytes,
                                   _stream(stream)))


def sb_sketch_given_norms(kind, G, n, d, ld_g, h, k, u, Pi, GH, ld_gh, cols, scales, norm2, qexp, ws, ws_bytes,
                          stream=None):
    return _check(load().sb_sketch_given_norms(kind, _ptr(G), n, d, ld_g, _ptr(h), k, _ptr(u), _ptr(Pi), _ptr(GH),
                                               ld_gh, _ptr(cols), _ptr(scales), _ptr(norm2), _ptr(qexp), _ptr(ws),
                                               ws_bytes, _stream(stream)))


def sb_sketch_sparse_projection(G, n, d, ld_g, h, k, s, pi_col, pi_val, GH, ld_gh, qexp, ws, ws_bytes, stream=None):
    return _check(load().sb_sketch_sparse_projection(_ptr(G), n, d, ld_g, _ptr(h), k, s, _ptr(pi_col), _ptr(pi_val),
                                                     _ptr(GH), ld_gh, _ptr(qexp), _ptr(ws), ws_bytes,
                                                     _stream(stream)))


def sb_hist_exponents(GH, n, ld_gh, k, qexp, ws, ws_bytes, stream=None):
    return _check(load().sb_hist_exponents(_ptr(GH), n, ld_gh, k, _ptr(qexp), _ptr(ws), ws_bytes, _stream(stream)))


def sb_build_histograms(bins4, ld4, rec, ld_rec, n, m, n_bins, GH, ld_gh, k, qexp, row_idx, node_off, n_nodes,
                        build_list, n_build, H, ws, ws_bytes, stream=None):
    return _check(load().sb_build_histograms(_ptr(bins4), ld4, _ptr(rec), ld_rec, n, m, n_bins, _ptr(GH), ld_gh, k,
                                             _ptr(qexp), _ptr(row_idx), _ptr(node_off), n_nodes, _ptr(build_list),
                                             n_build, _ptr(H), _ptr(ws), ws_bytes, _stream(stream)))


def sb_subtract_histograms(H_parent, H_child, n_parents, m, n_bins, k, build_list, stream=None):
    return _check(load().sb_subtract_histograms(_ptr(H_parent), _ptr(H_child), n_parents, m, n_bins, k,
                                                _ptr(build_list), _stream(stream)))


def sb_score_splits(H, n_nodes, m, n_bins, k, lam, min_child_weight, best_feature, best_bin, best_score, ws,
                    ws_bytes, stream=None):
    return _check(load().sb_score_splits(_ptr(H), n_nodes, m, n_bins, k, lam, min_child_weight, _ptr(best_feature),
                                         _ptr(best_bin), _ptr(best_score), _ptr(ws), ws_bytes, _stream(stream)))


def sb_partition_rows(bins_cm, n, m, ld_cm, row_idx_in, node_off_in, n_nodes, best_feature, best_bin, row_idx_out,
                      node_off_out, build_list_out, ws, ws_bytes, stream=None):
    return _check(load().sb_partition_rows(_ptr(bins_cm), n, m, ld_cm, _ptr(row_idx_in), _ptr(node_off_in), n_nodes,
                                           _ptr(best_feature), _ptr(best_bin), _ptr(row_idx_out),
                                           _ptr(node_off_out), _ptr(build_list_out), _ptr(ws), ws_bytes,
                                           _stream(stream)))


def sb_partition_rows_noalloc(bins_cm, n, m, ld_cm, row_idx_in, node_off_in, n_nodes, best_feature, best_bin,
                              row_idx_out, node_off_out, build_list_out, stream=None):
    return _check(load().sb_partition_rows_noalloc(_ptr(bins_cm), n, m, ld_cm, _ptr(row_idx_in), _ptr(node_off_in),
                                                   n_nodes, _ptr(best_feature), _ptr(best_bin), _ptr(row_idx_out),
                                                   _ptr(node_off_out), _ptr(build_list_out), _stream(stream)))


def sb_grow_tree(bins4, ld4, bins_cm, ld_cm, rec, ld_rec, n, m, n_bins, GH, ld_gh, k, qexp, depth, lam,
                 min_child_weight, tree_feature, tree_bin, tree_score, row_idx_out, leaf_off_out, ws, ws_bytes,
                 stream=None):
    return _check(load().sb_grow_tree(_ptr(bins4), ld4, _ptr(bins_cm), ld_cm, _ptr(rec), ld_rec, n, m, n_bins,
                                      _ptr(GH), ld_gh, k, _ptr(qexp), depth, lam, min_child_weight,
                                      _ptr(tree_feature), _ptr(tree_bin), _ptr(tree_score), _ptr(row_idx_out),
                                      _ptr(leaf_off_out), _ptr(ws), ws_bytes, _stream(stream)))


def sb_leaf_values(G, n, d, ld_g, hess, ld_hess, h, row_idx, leaf_off, n_leaves, lam, V, ld_v, ws, ws_bytes,
                   stream=None):
    return _check(load().sb_leaf_values(_ptr(G), n, d, ld_g, _ptr(hess), ld_hess, _ptr(h), _ptr(row_idx),
                                        _ptr(leaf_off), n_leaves, lam, _ptr(V), ld_v, _ptr(ws), ws_bytes,
                                        _stream(stream)))


def sb_gradients(loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess, h_row, norm2, ws, ws_bytes,
                 stream=None):
    return _check(load().sb_gradients(loss, _ptr(F), n, d, ld_f, _ptr(labels), _ptr(Y), ld_y, _ptr(G), ld_g,
                                      _ptr(hess), ld_hess, _ptr(h_row), _ptr(norm2), _ptr(ws), ws_bytes,
                                      _stream(stream)))


def sb_leaf_values_from_loss(loss, G, n, d, ld_g, labels, Y, ld_y, row_idx, leaf_off, n_leaves, lam, V, ld_v, ws,
                             ws_bytes, stream=None):
    return _check(load().sb_leaf_values_from_loss(loss, _ptr(G), n, d, ld_g, _ptr(labels), _ptr(Y), ld_y, _ptr(row_idx),
                                                  _ptr(leaf_off), n_leaves, lam, _ptr(V), ld_v, _ptr(ws), ws_bytes,
                                                  _stream(stream)))


def sb_update_predictions(F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr, ws, ws_bytes, stream=None):
    return _check(load().sb_update_predictions(_ptr(F), n, d, ld_f, _ptr(row_idx), _ptr(leaf_off), n_leaves, _ptr(V),
                                               ld_v, lr, _ptr(ws), ws_bytes, _stream(stream)))


def sb_update_and_gradients(loss, F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr, labels, Y, ld_y, G, ld_g,
                            hess, ld_hess, h_row, norm2, ws, ws_bytes, stream=None):
    return _check(load().sb_update_and_gradients(loss, _ptr(F), n, d, ld_f, _ptr(row_idx), _ptr(leaf_off), n_leaves,
                                                 _ptr(V), ld_v, lr, _ptr(labels), _ptr(Y), ld_y, _ptr(G), ld_g,
                                                 _ptr(hess), ld_hess, _ptr(h_row), _ptr(norm2), _ptr(ws), ws_bytes,
                                                 _stream(stream)))


def sb_profile_begin():
    return _check(load().sb_profile_begin())


def sb_profile_end():
    """Returns (summed histogram-kernel milliseconds, number of launches)."""
    ms = ctypes.c_double(0.0)
    cnt = ctypes.c_int64(0)
    _check(load().sb_profile_end(ctypes.byref(ms), ctypes.byref(cnt)))
    return ms.value, cnt.value
