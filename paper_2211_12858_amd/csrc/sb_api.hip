// C ABI entry points: argument checks on the host, workspace sizing, launches,
// and the device-resident level loop of sb_grow_tree.
#include <cmath>
#include <cstring>
#include <string>
#include <utility>
#include <vector>

#include "sb_common.h"

namespace sb {

namespace {
thread_local std::string g_error;
struct Profile {
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> hist;
};
thread_local Profile g_prof;
}  // namespace

bool profile_on() { return g_prof.on; }
void profile_record(hipEvent_t start, hipEvent_t stop) { g_prof.hist.emplace_back(start, stop); }

void set_error(const std::string& msg) { g_error = msg; }

int32_t fail(int32_t code, const std::string& msg) {
  g_error = msg;
  return code;
}

int32_t check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SB_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
  return SB_OK;
}

namespace {

constexpr int64_t MAX_ROWS = (int64_t(1) << 31) - 1;
constexpr int MAX_DEPTH = 12;
constexpr int32_t MAX_LEAVES = 1 << MAX_DEPTH;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int32_t need_ws(void* ws, int64_t have, int64_t need, const char* call) {
  if (need < 0) return fail(SB_E_UNSUPPORTED, std::string(call) + ": sizes outside the supported range");
  if (need > 0 && ws == nullptr) return fail(SB_E_ARG, std::string(call) + ": workspace is NULL");
  if (have < need)
    return fail(SB_E_ARG, std::string(call) + ": workspace too small: need " + std::to_string(need) + " bytes, got " +
                              std::to_string(have));
  if (ws && !aligned(ws, 256)) return fail(SB_E_SHAPE, std::string(call) + ": workspace must be 256-byte aligned");
  return SB_OK;
}

int32_t check_hist_shape(const char* call, int64_t n, int32_t m, int32_t n_bins, int32_t k) {
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, std::string(call) + ": n must be in [1, 2^31)");
  if (m < 1 || m > 65535) return fail(SB_E_ARG, std::string(call) + ": m must be in [1, 65535]");
  if (n_bins < 2 || n_bins > 256) return fail(SB_E_ARG, std::string(call) + ": n_bins must be in [2, 256]");
  if (k < 1 || k > 255) return fail(SB_E_ARG, std::string(call) + ": k must be in [1, 255]");
  return SB_OK;
}

struct GrowLayout {
  int64_t H0, H1, rows_tmp, offs, blists, pre, feat_s, feat_b, qrow, call, total;
};

GrowLayout grow_ws_layout(int64_t n, int32_t m, int32_t n_bins, int32_t k, int32_t depth) {
  GrowLayout L{};
  const int64_t maxn = int64_t(1) << (depth - 1);
  const int64_t hbytes = align256(maxn * m * n_bins * (int64_t)(k + 1) * 8);
  const int64_t hw = hist_ws_bytes(n, m, n_bins, k, (int32_t)maxn, false);
  if (hw < 0) {
    L.total = -1;
    return L;
  }
  int64_t call = hw;
  const int64_t sw = score_ws_bytes((int32_t)maxn, m);
  const int64_t pw = partition_ws_bytes(n, (int32_t)maxn);
  if (sw > call) call = sw;
  if (pw > call) call = pw;
  const int64_t level_offs = align256(((int64_t(1) << depth) + depth) * 4);
  int64_t p = 0;
  L.H0 = p;
  p += hbytes;
  L.H1 = p;
  p += hbytes;
  L.rows_tmp = p;
  p += align256(n * 4);
  L.offs = p;
  p += level_offs;
  L.blists = p;
  p += align256((int64_t(1) << depth) * 4);
  L.pre = p;
  p += align256((maxn + 1) * 8);
  L.feat_s = p;
  p += align256(maxn * m * 8);
  L.feat_b = p;
  p += align256(maxn * m * 4);
  // quantised sketch rows of the rotated histogram kernel, written at the
  // root and read by every level
  L.qrow = p;
  p += align256(n * 16 * hist_plan(m, n_bins, k, 1).cg);
  L.call = p;
  p += call;
  L.total = p;
  return L;
}

int32_t check_rec(const char* call, const void* rec, int64_t ld_rec, int32_t m) {
  if (!aligned(rec, 16) || ld_rec % 16 != 0 || ld_rec < m)
    return fail(SB_E_SHAPE, std::string(call) + ": row records need a 16-byte aligned base, ld_rec % 16 == 0 and "
                                                "ld_rec >= m");
  return SB_OK;
}

int32_t check_gh(const char* call, const void* GH, int64_t ld_gh, int32_t k) {
  if (!aligned(GH, 16) || ld_gh < k + 1)
    return fail(SB_E_SHAPE, std::string(call) + ": GH needs a 16-byte aligned base and ld_gh >= k + 1 (row-major)");
  return SB_OK;
}

}  // namespace
}  // namespace sb

using namespace sb;

extern "C" {

const char* sb_last_error(void) { return g_error.c_str(); }

int32_t sb_abi_version(void) { return SB_ABI_VERSION; }

int32_t sb_profile_begin(void) {
  for (auto& pr : g_prof.hist) {
    (void)hipEventDestroy(pr.first);
    (void)hipEventDestroy(pr.second);
  }
  g_prof.hist.clear();
  g_prof.on = true;
  return SB_OK;
}

int32_t sb_profile_end(double* hist_kernel_ms, int64_t* hist_launches) {
  g_prof.on = false;
  double total = 0.0;
  int32_t rc = SB_OK;
  if (!g_prof.hist.empty() && hipEventSynchronize(g_prof.hist.back().second) != hipSuccess)
    rc = fail(SB_E_DEVICE, "sb_profile_end: event synchronisation failed");
  for (auto& pr : g_prof.hist) {
    float ms = 0.0f;
    if (rc == SB_OK && hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess)
      rc = fail(SB_E_DEVICE, "sb_profile_end: hipEventElapsedTime failed");
    total += ms;
    (void)hipEventDestroy(pr.first);
    (void)hipEventDestroy(pr.second);
  }
  const int64_t count = (int64_t)g_prof.hist.size();
  g_prof.hist.clear();
  if (hist_kernel_ms) *hist_kernel_ms = total;
  if (hist_launches) *hist_launches = count;
  return rc;
}

int64_t sb_workspace_bytes(int32_t call, int64_t n, int32_t m, int32_t n_bins, int32_t d, int32_t k,
                           int32_t n_nodes, int32_t depth) {
  switch (call) {
    case SB_CALL_SKETCH:
      if (n < 1 || n > MAX_ROWS || d < 1 || d > 65535 || k < 1 || k > 255) break;
      return sketch_ws_bytes(0, n, d, k);
    case SB_CALL_HIST_EXPONENTS:
      if (k < 1 || k > 255) break;
      return hist_exponents_ws_bytes(k);
    case SB_CALL_BUILD_HISTOGRAMS: {
      if (n < 1 || n > MAX_ROWS || m < 1 || m > 65535 || n_bins < 2 || n_bins > 256 || k < 1 || k > 255 ||
          n_nodes < 1 || n_nodes > (1 << 20))
        break;
      const int64_t b = hist_ws_bytes(n, m, n_bins, k, n_nodes, true);
      if (b < 0) break;
      return b;
    }
    case SB_CALL_SCORE_SPLITS:
      if (m < 1 || m > 65535 || n_nodes < 1 || n_nodes > 65535) break;
      return score_ws_bytes(n_nodes, m);
    case SB_CALL_PARTITION_ROWS:
      if (n < 1 || n > MAX_ROWS || n_nodes < 1 || n_nodes > (1 << 20)) break;
      return partition_ws_bytes(n, n_nodes);
    case SB_CALL_GROW_TREE: {
      if (n < 1 || n > MAX_ROWS || m < 1 || m > 65535 || n_bins < 2 || n_bins > 256 || k < 1 || k > 255 ||
          depth < 1 || depth > MAX_DEPTH)
        break;
      const int64_t b = grow_ws_layout(n, m, n_bins, k, depth).total;
      if (b < 0) break;
      return b;
    }
    case SB_CALL_GRADIENTS:
      if (n < 1 || n > MAX_ROWS || d < 1 || d > 65535) break;
      return grad_ws_bytes(n, d);
    case SB_CALL_UPDATE_PREDICTIONS:
      if (n < 1 || n > MAX_ROWS) break;
      return update_ws_bytes(n);
    case SB_CALL_UPDATE_AND_GRADIENTS:
      if (n < 1 || n > MAX_ROWS || d < 1 || d > 65535) break;
      return update_gradients_ws_bytes(n, d);
    case SB_CALL_LEAF_VALUES:
      if (n < 1 || n > MAX_ROWS || d < 1 || d > 65535 || n_nodes < 1 || n_nodes > MAX_LEAVES) break;
      return leaf_ws_bytes(n, d, n_nodes);
    default:
      set_error("sb_workspace_bytes: unknown call id");
      return -1;
  }
  set_error("sb_workspace_bytes: sizes outside the supported range");
  return -1;
}

int32_t sb_layout_bins(const uint8_t* bins, int64_t n, int32_t m, int64_t ld_bins, uint32_t* bins4, int64_t ld4,
                       uint8_t* bins_cm, int64_t ld_cm, uint8_t* rec, int64_t ld_rec, void* stream) {
  if (!bins) return fail(SB_E_ARG, "sb_layout_bins: bins must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, "sb_layout_bins: n must be in [1, 2^31)");
  if (m < 1 || m > 65535) return fail(SB_E_ARG, "sb_layout_bins: m must be in [1, 65535]");
  if (ld_bins < m) return fail(SB_E_SHAPE, "sb_layout_bins: ld_bins must be >= m");
  if (bins4 && (ld4 < n || !aligned(bins4, 4)))
    return fail(SB_E_SHAPE, "sb_layout_bins: bins4 needs ld4 >= n and a 4-byte aligned base");
  if (bins_cm && ld_cm < n) return fail(SB_E_SHAPE, "sb_layout_bins: ld_cm must be >= n");
  if (rec && (ld_rec < m || ld_rec % 16 != 0 || !aligned(rec, 16)))
    return fail(SB_E_SHAPE, "sb_layout_bins: rec needs ld_rec >= m, ld_rec % 16 == 0 and a 16-byte aligned base");
  return launch_layout(bins, n, m, ld_bins, bins4, ld4, bins_cm, ld_cm, rec, ld_rec,
                       static_cast<hipStream_t>(stream));
}

}  // extern "C"

namespace {

int32_t check_sketch(const char* call, int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g,
                     const float* h, int32_t k, const double* u, const float* Pi, float* GH, int64_t ld_gh,
                     int32_t* cols, float* scales, const double* norm2, int32_t* qexp, void* ws, int64_t ws_bytes) {
  const std::string c(call);
  if (kind < SB_SKETCH_TOP_OUTPUTS || kind > SB_SKETCH_IDENTITY)
    return fail(SB_E_UNSUPPORTED, c + ": unknown sketch kind " + std::to_string(kind));
  if (!G || !h || !GH || !qexp) return fail(SB_E_ARG, c + ": G, h, GH and qexp must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, c + ": n must be in [1, 2^31)");
  if (d < 1 || d > 65535) return fail(SB_E_ARG, c + ": d must be in [1, 65535]");
  if (k < 1 || k > 255) return fail(SB_E_ARG, c + ": k must be in [1, 255]");
  if (ld_g < n) return fail(SB_E_SHAPE, c + ": ld_g must be >= n");
  {
    const int32_t rr = check_gh(call, GH, ld_gh, k);
    if (rr) return rr;
  }
  switch (kind) {
    case SB_SKETCH_TOP_OUTPUTS:
      if (k > d) return fail(SB_E_ARG, c + ": top outputs needs k <= d");
      if (!cols || !scales || !norm2) return fail(SB_E_ARG, c + ": cols, scales and norm2 must not be NULL");
      break;
    case SB_SKETCH_RANDOM_SAMPLING:
      if (!u) return fail(SB_E_ARG, c + ": random sampling needs k uniforms u");
      if (!cols || !scales || !norm2) return fail(SB_E_ARG, c + ": cols, scales and norm2 must not be NULL");
      break;
    case SB_SKETCH_RANDOM_PROJECTION:
      if (!Pi) return fail(SB_E_ARG, c + ": random projection needs Pi");
      break;
    case SB_SKETCH_IDENTITY:
      if (k != d) return fail(SB_E_ARG, c + ": identity sketch needs k == d");
      if (!cols || !scales) return fail(SB_E_ARG, c + ": cols and scales must not be NULL");
      break;
  }
  return need_ws(ws, ws_bytes, sketch_ws_bytes(kind, n, d, k), call);
}

}  // namespace

extern "C" {

int32_t sb_sketch(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                  const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols, float* scales,
                  double* norm2, int32_t* qexp, void* ws, int64_t ws_bytes, void* stream) {
  const int32_t rc = check_sketch("sb_sketch", kind, G, n, d, ld_g, h, k, u, Pi, GH, ld_gh, cols, scales, norm2, qexp,
                                  ws, ws_bytes);
  if (rc) return rc;
  return launch_sketch(kind, G, n, d, ld_g, h, k, u, Pi, GH, ld_gh, cols, scales, norm2, qexp, ws,
                       static_cast<hipStream_t>(stream));
}

int32_t sb_sketch_given_norms(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h,
                              int32_t k, const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols,
                              float* scales, const double* norm2, int32_t* qexp, void* ws, int64_t ws_bytes,
                              void* stream) {
  const int32_t rc = check_sketch("sb_sketch_given_norms", kind, G, n, d, ld_g, h, k, u, Pi, GH, ld_gh, cols, scales,
                                  norm2, qexp, ws, ws_bytes);
  if (rc) return rc;
  return launch_sketch(kind, G, n, d, ld_g, h, k, u, Pi, GH, ld_gh, cols, scales, nullptr, qexp, ws,
                       static_cast<hipStream_t>(stream), norm2);
}

int32_t sb_sketch_sparse_projection(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                                    int32_t s, const int32_t* pi_col, const float* pi_val, float* GH, int64_t ld_gh,
                                    int32_t* qexp, void* ws, int64_t ws_bytes, void* stream) {
  const char* call = "sb_sketch_sparse_projection";
  if (!G || !h || !pi_col || !pi_val || !GH || !qexp)
    return fail(SB_E_ARG, "sb_sketch_sparse_projection: G, h, pi_col, pi_val, GH and qexp must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, "sb_sketch_sparse_projection: n must be in [1, 2^31)");
  if (d < 1 || d > 65535) return fail(SB_E_ARG, "sb_sketch_sparse_projection: d must be in [1, 65535]");
  if (k < 1 || k > 255) return fail(SB_E_ARG, "sb_sketch_sparse_projection: k must be in [1, 255]");
  if (s != 1 && s != 2 && s != 4 && s != 8)
    return fail(SB_E_UNSUPPORTED, "sb_sketch_sparse_projection: s must be 1, 2, 4 or 8 (pad rows with column -1)");
  if (ld_g < n) return fail(SB_E_SHAPE, "sb_sketch_sparse_projection: ld_g must be >= n");
  int32_t rc = check_gh(call, GH, ld_gh, k);
  if (rc) return rc;
  rc = need_ws(ws, ws_bytes, sketch_ws_bytes(SB_SKETCH_RANDOM_PROJECTION, n, d, k), call);
  if (rc) return rc;
  return launch_sketch_sparse(G, n, d, ld_g, h, k, s, pi_col, pi_val, GH, ld_gh, qexp, ws,
                              static_cast<hipStream_t>(stream));
}

int32_t sb_hist_exponents(const float* GH, int64_t n, int64_t ld_gh, int32_t k, int32_t* qexp, void* ws,
                          int64_t ws_bytes, void* stream) {
  if (!GH || !qexp) return fail(SB_E_ARG, "sb_hist_exponents: GH and qexp must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, "sb_hist_exponents: n must be in [1, 2^31)");
  if (k < 1 || k > 255) return fail(SB_E_ARG, "sb_hist_exponents: k must be in [1, 255]");
  if (ld_gh < k + 1) return fail(SB_E_SHAPE, "sb_hist_exponents: ld_gh must be >= k + 1 (GH is row-major)");
  int32_t rc = need_ws(ws, ws_bytes, hist_exponents_ws_bytes(k), "sb_hist_exponents");
  if (rc) return rc;
  return launch_hist_exponents(GH, n, ld_gh, k, qexp, ws, static_cast<hipStream_t>(stream));
}

int32_t sb_build_histograms(const uint32_t* bins4, int64_t ld4, const uint8_t* rec, int64_t ld_rec, int64_t n,
                            int32_t m, int32_t n_bins, const float* GH, int64_t ld_gh, int32_t k,
                            const int32_t* qexp, const int32_t* row_idx, const int32_t* node_off, int32_t n_nodes,
                            const int32_t* build_list, int32_t n_build, double* H, void* ws, int64_t ws_bytes,
                            void* stream) {
  const char* call = "sb_build_histograms";
  if (!GH || !qexp || !node_off || !H)
    return fail(SB_E_ARG, "sb_build_histograms: GH, qexp, node_off and H must not be NULL");
  int32_t rc = check_hist_shape(call, n, m, n_bins, k);
  if (rc) return rc;
  rc = check_gh(call, GH, ld_gh, k);
  if (rc) return rc;
  if (row_idx) {
    if (!rec) return fail(SB_E_ARG, "sb_build_histograms: rows through row_idx are read from rec, which is NULL");
    rc = check_rec(call, rec, ld_rec, m);
    if (rc) return rc;
  } else {
    if (!bins4) return fail(SB_E_ARG, "sb_build_histograms: without row_idx, bins4 must not be NULL");
    if (ld4 < n || !aligned(bins4, 4))
      return fail(SB_E_SHAPE, "sb_build_histograms: bins4 needs ld4 >= n and a 4-byte aligned base");
  }
  if (n_nodes < 1 || n_nodes > (1 << 20)) return fail(SB_E_ARG, "sb_build_histograms: n_nodes must be in [1, 2^20]");
  if (build_list == nullptr) n_build = n_nodes;
  if (n_build < 1 || n_build > n_nodes || n_build > 65535)
    return fail(SB_E_ARG, "sb_build_histograms: n_build must be in [1, min(n_nodes, 65535)]");
  if (hist_plan(m, n_bins, k, n_build).nq == 0)
    return fail(SB_E_UNSUPPORTED, "sb_build_histograms: at most 24 channels (k <= 23)");
  rc = need_ws(ws, ws_bytes, hist_ws_bytes(n, m, n_bins, k, n_build, true), call);
  if (rc) return rc;
  return launch_build_histograms(bins4, ld4, rec, ld_rec, n, m, n_bins, GH, ld_gh, k, qexp, row_idx, node_off, n_nodes,
                                 build_list, n_build, H, ws, static_cast<hipStream_t>(stream));
}

int32_t sb_subtract_histograms(const double* H_parent, double* H_child, int32_t n_parents, int32_t m,
                               int32_t n_bins, int32_t k, const int32_t* build_list, void* stream) {
  if (!H_parent || !H_child || !build_list)
    return fail(SB_E_ARG, "sb_subtract_histograms: H_parent, H_child and build_list must not be NULL");
  int32_t rc = check_hist_shape("sb_subtract_histograms", 1, m, n_bins, k);
  if (rc) return rc;
  if (n_parents < 1 || n_parents > 65535)
    return fail(SB_E_ARG, "sb_subtract_histograms: n_parents must be in [1, 65535]");
  return launch_subtract(H_parent, H_child, n_parents, (int64_t)m * n_bins * (k + 1), build_list,
                         static_cast<hipStream_t>(stream));
}

int32_t sb_score_splits(const double* H, int32_t n_nodes, int32_t m, int32_t n_bins, int32_t k, double lambda,
                        double min_child_weight, int32_t* best_feature, int32_t* best_bin, double* best_score,
                        void* ws, int64_t ws_bytes, void* stream) {
  if (!H || !best_feature || !best_bin || !best_score)
    return fail(SB_E_ARG, "sb_score_splits: H and the outputs must not be NULL");
  int32_t rc = check_hist_shape("sb_score_splits", 1, m, n_bins, k);
  if (rc) return rc;
  if (n_nodes < 1 || n_nodes > 65535) return fail(SB_E_ARG, "sb_score_splits: n_nodes must be in [1, 65535]");
  if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail(SB_E_ARG, "sb_score_splits: lambda must be > 0");
  if (!(min_child_weight >= 0.0) || !std::isfinite(min_child_weight))
    return fail(SB_E_ARG, "sb_score_splits: min_child_weight must be >= 0");
  rc = need_ws(ws, ws_bytes, score_ws_bytes(n_nodes, m), "sb_score_splits");
  if (rc) return rc;
  return launch_score(H, n_nodes, m, n_bins, k, lambda, min_child_weight, best_feature, best_bin, best_score, ws,
                      static_cast<hipStream_t>(stream));
}

}  // extern "C"

namespace {

int32_t check_partition(const char* call, const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm,
                        const int32_t* row_idx_in, const int32_t* node_off_in, int32_t n_nodes,
                        const int32_t* best_feature, const int32_t* best_bin, int32_t* row_idx_out,
                        int32_t* node_off_out, int32_t* build_list_out) {
  const std::string c(call);
  if (!bins_cm || !node_off_in || !best_feature || !best_bin || !row_idx_out || !node_off_out || !build_list_out)
    return fail(SB_E_ARG, c + ": bins_cm, node_off_in, the splits and the outputs must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, c + ": n must be in [1, 2^31)");
  if (m < 1) return fail(SB_E_ARG, c + ": m must be >= 1");
  if (ld_cm < n) return fail(SB_E_SHAPE, c + ": ld_cm must be >= n");
  if (n_nodes < 1 || n_nodes > (1 << 20)) return fail(SB_E_ARG, c + ": n_nodes must be in [1, 2^20]");
  if (row_idx_in) {
    const char* a0 = reinterpret_cast<const char*>(row_idx_in);
    const char* b0 = reinterpret_cast<const char*>(row_idx_out);
    if (a0 < b0 + n * 4 && b0 < a0 + n * 4) return fail(SB_E_SHAPE, c + ": row_idx_in and row_idx_out overlap");
  }
  return SB_OK;
}

int32_t check_gradients(const char* call, int32_t loss, const float* F, int64_t n, int32_t d, int64_t ld_f,
                        const int32_t* labels, const uint8_t* Y, int64_t ld_y, const float* G, int64_t ld_g,
                        const float* hess, int64_t ld_hess) {
  const std::string c(call);
  if (loss != SB_LOSS_SOFTMAX_CE && loss != SB_LOSS_SIGMOID_BCE)
    return fail(SB_E_UNSUPPORTED, c + ": unknown loss " + std::to_string(loss));
  if (!F || !G) return fail(SB_E_ARG, c + ": F and G must not be NULL");
  if (loss == SB_LOSS_SOFTMAX_CE && !labels) return fail(SB_E_ARG, c + ": softmax needs labels");
  if (loss == SB_LOSS_SIGMOID_BCE && !Y) return fail(SB_E_ARG, c + ": sigmoid needs the targets Y");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, c + ": n must be in [1, 2^31)");
  if (d < 1 || d > 65535) return fail(SB_E_ARG, c + ": d must be in [1, 65535]");
  if (ld_f < n || ld_g < n) return fail(SB_E_SHAPE, c + ": ld_f and ld_g must be >= n");
  if (hess && ld_hess < n) return fail(SB_E_SHAPE, c + ": ld_hess must be >= n");
  if (loss == SB_LOSS_SIGMOID_BCE && ld_y < n) return fail(SB_E_SHAPE, c + ": ld_y must be >= n");
  const char* f0 = reinterpret_cast<const char*>(F);
  const char* g0 = reinterpret_cast<const char*>(G);
  const int64_t fb = ((int64_t)(d - 1) * ld_f + n) * 4, gb = ((int64_t)(d - 1) * ld_g + n) * 4;
  if (f0 < g0 + gb && g0 < f0 + fb) return fail(SB_E_SHAPE, c + ": F and G overlap");
  return SB_OK;
}

int32_t check_update(const char* call, const float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                     const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr) {
  const std::string c(call);
  if (!F || !row_idx || !leaf_off || !V) return fail(SB_E_ARG, c + ": F, row_idx, leaf_off and V must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, c + ": n must be in [1, 2^31)");
  if (d < 1 || d > 65535) return fail(SB_E_ARG, c + ": d must be in [1, 65535]");
  if (n_leaves < 1 || n_leaves > MAX_LEAVES) return fail(SB_E_ARG, c + ": n_leaves must be in [1, 4096]");
  if (ld_f < n) return fail(SB_E_SHAPE, c + ": ld_f must be >= n");
  if (ld_v < d) return fail(SB_E_SHAPE, c + ": ld_v must be >= d");
  if (!std::isfinite(lr)) return fail(SB_E_ARG, c + ": lr must be finite");
  return SB_OK;
}

}  // namespace

extern "C" {

int32_t sb_partition_rows(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm,
                          const int32_t* row_idx_in, const int32_t* node_off_in, int32_t n_nodes,
                          const int32_t* best_feature, const int32_t* best_bin, int32_t* row_idx_out,
                          int32_t* node_off_out, int32_t* build_list_out, void* ws, int64_t ws_bytes,
                          void* stream) {
  int32_t rc = check_partition("sb_partition_rows", bins_cm, n, m, ld_cm, row_idx_in, node_off_in, n_nodes,
                               best_feature, best_bin, row_idx_out, node_off_out, build_list_out);
  if (rc) return rc;
  rc = need_ws(ws, ws_bytes, partition_ws_bytes(n, n_nodes), "sb_partition_rows");
  if (rc) return rc;
  return launch_partition(bins_cm, n, m, ld_cm, row_idx_in, node_off_in, n_nodes, best_feature, best_bin,
                          row_idx_out, node_off_out, build_list_out, ws, static_cast<hipStream_t>(stream));
}

int32_t sb_partition_rows_noalloc(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm,
                                  const int32_t* row_idx_in, const int32_t* node_off_in, int32_t n_nodes,
                                  const int32_t* best_feature, const int32_t* best_bin, int32_t* row_idx_out,
                                  int32_t* node_off_out, int32_t* build_list_out, void* stream) {
  const char* call = "sb_partition_rows_noalloc";
  int32_t rc = check_partition(call, bins_cm, n, m, ld_cm, row_idx_in, node_off_in, n_nodes, best_feature,
                               best_bin, row_idx_out, node_off_out, build_list_out);
  if (rc) return rc;
  const int64_t need = partition_ws_bytes(n, n_nodes);
  if (need > PARTITION_SCRATCH_BYTES)
    return fail(SB_E_UNSUPPORTED, std::string(call) + ": needs " + std::to_string(need) +
                                      " bytes of scratch; the static scratch holds " +
                                      std::to_string(PARTITION_SCRATCH_BYTES) + " (about 60 million rows)");
  void* ws = nullptr;
  rc = partition_scratch(&ws);
  if (rc) return rc;
  return launch_partition(bins_cm, n, m, ld_cm, row_idx_in, node_off_in, n_nodes, best_feature, best_bin,
                          row_idx_out, node_off_out, build_list_out, ws, static_cast<hipStream_t>(stream));
}

int32_t sb_grow_tree(const uint32_t* bins4, int64_t ld4, const uint8_t* bins_cm, int64_t ld_cm, const uint8_t* rec,
                     int64_t ld_rec, int64_t n, int32_t m, int32_t n_bins, const float* GH, int64_t ld_gh,
                     int32_t k, const int32_t* qexp, int32_t depth, double lambda,
                     double min_child_weight, int32_t* tree_feature, int32_t* tree_bin, double* tree_score,
                     int32_t* row_idx_out, int32_t* leaf_off_out, void* ws, int64_t ws_bytes, void* stream) {
  const char* call = "sb_grow_tree";
  if (!bins4 || !bins_cm || !rec || !GH || !qexp || !tree_feature || !tree_bin || !tree_score || !row_idx_out ||
      !leaf_off_out)
    return fail(SB_E_ARG, "sb_grow_tree: inputs and outputs must not be NULL");
  int32_t rc = check_hist_shape(call, n, m, n_bins, k);
  if (rc) return rc;
  if (depth < 1 || depth > MAX_DEPTH) return fail(SB_E_ARG, "sb_grow_tree: depth must be in [1, 12]");
  if (ld4 < n || !aligned(bins4, 4))
    return fail(SB_E_SHAPE, "sb_grow_tree: bins4 needs ld4 >= n and a 4-byte aligned base");
  if (ld_cm < n) return fail(SB_E_SHAPE, "sb_grow_tree: ld_cm must be >= n");
  rc = check_rec(call, rec, ld_rec, m);
  if (rc) return rc;
  rc = check_gh(call, GH, ld_gh, k);
  if (rc) return rc;
  if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail(SB_E_ARG, "sb_grow_tree: lambda must be > 0");
  if (!(min_child_weight >= 0.0) || !std::isfinite(min_child_weight))
    return fail(SB_E_ARG, "sb_grow_tree: min_child_weight must be >= 0");
  if (hist_plan(m, n_bins, k, 1).nq == 0) return fail(SB_E_UNSUPPORTED, "sb_grow_tree: at most 24 channels (k <= 23)");
  const GrowLayout G = grow_ws_layout(n, m, n_bins, k, depth);
  rc = need_ws(ws, ws_bytes, G.total, call);
  if (rc) return rc;

  hipStream_t st = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  double* Hbuf[2] = {reinterpret_cast<double*>(w + G.H0), reinterpret_cast<double*>(w + G.H1)};
  int32_t* rows_tmp = reinterpret_cast<int32_t*>(w + G.rows_tmp);
  int32_t* offs = reinterpret_cast<int32_t*>(w + G.offs);
  int32_t* blists = reinterpret_cast<int32_t*>(w + G.blists);
  int64_t* pre = reinterpret_cast<int64_t*>(w + G.pre);
  double* feat_s = reinterpret_cast<double*>(w + G.feat_s);
  int32_t* feat_b = reinterpret_cast<int32_t*>(w + G.feat_b);
  uint32_t* qrow = reinterpret_cast<uint32_t*>(w + G.qrow);
  // every level ends with the fused kernel (histogram reduction, subtraction
  // and per-feature scoring), which takes every sketch the histogram kernel
  // takes
  static_assert(FUSED_SCORE_MAX_C >= ROT_MAX_C, "the fused level end covers every histogram shape");
  void* cws = w + G.call;

  // level l node offsets start at offs + (2^l - 1) + l (2^l + 1 entries), its
  // build list at blists + 2^(l-1) - 1
  auto level_off = [&](int l) { return offs + ((int64_t(1) << l) - 1) + l; };
  auto level_build = [&](int l) { return blists + ((int64_t(1) << (l - 1)) - 1); };
  auto level_rows = [&](int l) -> int32_t* {  // rows of level l >= 1; level depth lands in row_idx_out
    return ((depth - l) % 2 == 0) ? row_idx_out : rows_tmp;
  };

  // the root's offsets and prefix {0, n} are written by the kernel that
  // quantises the sketch rows
  for (int l = 0; l < depth; ++l) {
    const int32_t nn = 1 << l;
    double* Hcur = Hbuf[l & 1];
    const int32_t* row_in = l == 0 ? nullptr : level_rows(l);
    const int32_t* off_l = level_off(l);
    // the prefix of the built nodes' sizes comes from the previous level's
    // partition (from the sketch-row quantiser at the root), and the reduce writes the
    // siblings by subtraction from the previous level
    const int64_t base = (int64_t(1) << l) - 1;
    if (l == 0) {
      rc = launch_build_histograms(bins4, ld4, rec, ld_rec, n, m, n_bins, GH, ld_gh, k, qexp, nullptr, off_l, 1,
                                   nullptr, 1, Hcur, cws, st, pre, nullptr, feat_s, feat_b, lambda,
                                   min_child_weight, qrow, false, depth > 1, const_cast<int32_t*>(off_l));
    } else {
      rc = launch_build_histograms(bins4, ld4, rec, ld_rec, n, m, n_bins, GH, ld_gh, k, qexp, row_in, off_l, nn,
                                   level_build(l), nn / 2, Hcur, cws, st, pre, Hbuf[(l - 1) & 1],
                                   feat_s, feat_b, lambda, min_child_weight, qrow, true,
                                   l < depth - 1);
    }
    if (rc) return rc;
    // node splits: picked by the partition from the fused level end's
    // per-feature results where it can, else by the node argmax kernel first
    const bool pick = partition_picks_splits(n, nn);
    if (!pick) {
      rc = launch_score_node(feat_s, feat_b, nn, m, tree_feature + base, tree_bin + base, tree_score + base, st);
      if (rc) return rc;
    }
    const bool last = l == depth - 1;
    rc = launch_partition(bins_cm, n, m, ld_cm, row_in, off_l, nn, tree_feature + base, tree_bin + base,
                          level_rows(l + 1), last ? leaf_off_out : level_off(l + 1), level_build(l + 1), cws, st,
                          last ? nullptr : pre, pick ? feat_s : nullptr, pick ? feat_b : nullptr,
                          pick ? tree_score + base : nullptr);
    if (rc) return rc;
  }
  return check_launch(call);
}

int32_t sb_leaf_values(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* hess, int64_t ld_hess,
                       const float* h, const int32_t* row_idx, const int32_t* leaf_off, int32_t n_leaves,
                       double lambda, double* V, int64_t ld_v, void* ws, int64_t ws_bytes, void* stream) {
  if (!G || !row_idx || !leaf_off || !V)
    return fail(SB_E_ARG, "sb_leaf_values: G, row_idx, leaf_off and V must not be NULL");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, "sb_leaf_values: n must be in [1, 2^31)");
  if (d < 1 || d > 65535) return fail(SB_E_ARG, "sb_leaf_values: d must be in [1, 65535]");
  if (n_leaves < 1 || n_leaves > MAX_LEAVES) return fail(SB_E_ARG, "sb_leaf_values: n_leaves must be in [1, 4096]");
  if (ld_g < n) return fail(SB_E_SHAPE, "sb_leaf_values: ld_g must be >= n");
  if (hess && ld_hess < n) return fail(SB_E_SHAPE, "sb_leaf_values: ld_hess must be >= n");
  if (ld_v < d) return fail(SB_E_SHAPE, "sb_leaf_values: ld_v must be >= d");
  if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail(SB_E_ARG, "sb_leaf_values: lambda must be > 0");
  const int32_t rc = need_ws(ws, ws_bytes, leaf_ws_bytes(n, d, n_leaves), "sb_leaf_values");
  if (rc) return rc;
  return launch_leaf_values(G, n, d, ld_g, hess, ld_hess, h, row_idx, leaf_off, n_leaves, lambda, V, ld_v, ws,
                            static_cast<hipStream_t>(stream));
}

int32_t sb_gradients(int32_t loss, const float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* labels,
                     const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g, float* hess, int64_t ld_hess,
                     float* h_row, double* norm2, void* ws, int64_t ws_bytes, void* stream) {
  int32_t rc = check_gradients("sb_gradients", loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess);
  if (rc) return rc;
  rc = need_ws(ws, ws_bytes, norm2 ? grad_ws_bytes(n, d) : 0, "sb_gradients");
  if (rc) return rc;
  return launch_gradients(loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess, h_row, norm2, ws,
                          static_cast<hipStream_t>(stream));
}

int32_t sb_leaf_values_from_loss(int32_t loss, const float* G, int64_t n, int32_t d, int64_t ld_g,
                                 const int32_t* labels, const uint8_t* Y, int64_t ld_y, const int32_t* row_idx,
                                 const int32_t* leaf_off, int32_t n_leaves, double lambda, double* V, int64_t ld_v,
                                 void* ws, int64_t ws_bytes, void* stream) {
  const char* call = "sb_leaf_values_from_loss";
  if (loss != SB_LOSS_SOFTMAX_CE && loss != SB_LOSS_SIGMOID_BCE)
    return fail(SB_E_UNSUPPORTED, "sb_leaf_values_from_loss: unknown loss " + std::to_string(loss));
  if (!G || !row_idx || !leaf_off || !V)
    return fail(SB_E_ARG, "sb_leaf_values_from_loss: G, row_idx, leaf_off and V must not be NULL");
  if (loss == SB_LOSS_SOFTMAX_CE && !labels) return fail(SB_E_ARG, "sb_leaf_values_from_loss: softmax needs labels");
  if (loss == SB_LOSS_SIGMOID_BCE && !Y) return fail(SB_E_ARG, "sb_leaf_values_from_loss: sigmoid needs Y");
  if (n < 1 || n > MAX_ROWS) return fail(SB_E_ARG, "sb_leaf_values_from_loss: n must be in [1, 2^31)");
  if (d < 1 || d > 65535) return fail(SB_E_ARG, "sb_leaf_values_from_loss: d must be in [1, 65535]");
  if (n_leaves < 1 || n_leaves > MAX_LEAVES)
    return fail(SB_E_ARG, "sb_leaf_values_from_loss: n_leaves must be in [1, 4096]");
  if (ld_g < n) return fail(SB_E_SHAPE, "sb_leaf_values_from_loss: ld_g must be >= n");
  if (loss == SB_LOSS_SIGMOID_BCE && ld_y < n) return fail(SB_E_SHAPE, "sb_leaf_values_from_loss: ld_y must be >= n");
  if (ld_v < d) return fail(SB_E_SHAPE, "sb_leaf_values_from_loss: ld_v must be >= d");
  if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail(SB_E_ARG, "sb_leaf_values_from_loss: lambda must be > 0");
  const int32_t rc = need_ws(ws, ws_bytes, leaf_ws_bytes(n, d, n_leaves), call);
  if (rc) return rc;
  return launch_leaf_values_from_loss(loss, G, n, d, ld_g, labels, Y, ld_y, row_idx, leaf_off, n_leaves, lambda, V,
                                      ld_v, ws, static_cast<hipStream_t>(stream));
}

int32_t sb_update_predictions(float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                              const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr,
                              void* ws, int64_t ws_bytes, void* stream) {
  int32_t rc = check_update("sb_update_predictions", F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr);
  if (rc) return rc;
  rc = need_ws(ws, ws_bytes, update_ws_bytes(n), "sb_update_predictions");
  if (rc) return rc;
  return launch_update(F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr, ws, static_cast<hipStream_t>(stream));
}

int32_t sb_update_and_gradients(int32_t loss, float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                                const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr,
                                const int32_t* labels, const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g,
                                float* hess, int64_t ld_hess, float* h_row, double* norm2, void* ws,
                                int64_t ws_bytes, void* stream) {
  const char* call = "sb_update_and_gradients";
  int32_t rc = check_update(call, F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr);
  if (rc) return rc;
  rc = check_gradients(call, loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess);
  if (rc) return rc;
  rc = need_ws(ws, ws_bytes, update_gradients_ws_bytes(n, d), call);
  if (rc) return rc;
  return launch_update_gradients(loss, F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr, labels, Y, ld_y, G,
                                 ld_g, hess, ld_hess, h_row, norm2, ws, static_cast<hipStream_t>(stream));
}

}  // extern "C"
