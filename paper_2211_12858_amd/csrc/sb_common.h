// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/sb.h"
#include "sb_hist_plan.h"

namespace sb {

// A load of data that is streamed once: it does not allocate in the caches.
__device__ inline float ld_stream(const float* p) { return __builtin_nontemporal_load(p); }

// Sum of x[p] over p = lane, lane + 64, ... < count, added in that order
// from 0.0 (a fixed order: the result depends only on the values); eight
// loads are issued before their adds, so the chain waits once per eight
// values rather than once per value.
__device__ inline double lane_strided_sum(const double* x, int count, int lane) {
  double s = 0.0;
  int p = lane;
  for (; p + 7 * 64 < count; p += 8 * 64) {
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = x[p + u * 64];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; p < count; p += 64) s += x[p];
  return s;
}

// A 32-bit value moved across lanes by a DPP control (row shift or row
// broadcast); lanes the control does not write get `old`.
template <int CTRL, int ROW_MASK>
__device__ inline int32_t dpp_i32(int32_t old, int32_t x) {
  return __builtin_amdgcn_update_dpp(old, x, CTRL, ROW_MASK, 0xf, false);
}

// Inclusive prefix sum over the 64 lanes of a wave (all lanes active), in
// registers: shifts by 1, 2, 4 and 8 lanes inside each row of 16, then the
// last lane of rows 0 and 2 into rows 1 and 3 (row_bcast:15) and lane 31
// into rows 2 and 3 (row_bcast:31); lanes a step does not write add 0.
__device__ inline int32_t wave_incl_scan_i32(int32_t x) {
  x += dpp_i32<0x111, 0xf>(0, x);
  x += dpp_i32<0x112, 0xf>(0, x);
  x += dpp_i32<0x114, 0xf>(0, x);
  x += dpp_i32<0x118, 0xf>(0, x);
  x += dpp_i32<0x142, 0xa>(0, x);
  x += dpp_i32<0x143, 0xc>(0, x);
  return x;
}

// Sum over each row of 16 lanes (all lanes active), in the row's last lane.
__device__ inline int32_t row16_sum_i32(int32_t x) {
  x += dpp_i32<0x111, 0xf>(0, x);
  x += dpp_i32<0x112, 0xf>(0, x);
  x += dpp_i32<0x114, 0xf>(0, x);
  x += dpp_i32<0x118, 0xf>(0, x);
  return x;
}

// One step of the wave argmax below: the candidate of the lane the DPP
// control names, where there is one ((-inf, -1), no candidate, elsewhere).
template <int CTRL, int ROW_MASK>
__device__ inline void best_step(double& s, int& f, int& b) {
  const int lo = dpp_i32<CTRL, ROW_MASK>(__double2loint(-INFINITY), __double2loint(s));
  const int hi = dpp_i32<CTRL, ROW_MASK>(__double2hiint(-INFINITY), __double2hiint(s));
  const int of = dpp_i32<CTRL, ROW_MASK>(-1, f);
  const int ob = dpp_i32<CTRL, ROW_MASK>(-1, b);
  const double os = __hiloint2double(hi, lo);
  if (of >= 0 && (f < 0 || os > s || (os == s && of < f))) {
    s = os;
    f = of;
    b = ob;
  }
}

// One step of a wave maximum of (score, index) pairs, larger score first,
// then the smaller index (index < 0: no candidate): the pair of the lane the
// DPP control names, where there is one ((-inf, -1) elsewhere).
template <int CTRL, int ROW_MASK>
__device__ inline void best_step_si(double& s, int& i) {
  const int lo = dpp_i32<CTRL, ROW_MASK>(__double2loint(-INFINITY), __double2loint(s));
  const int hi = dpp_i32<CTRL, ROW_MASK>(__double2hiint(-INFINITY), __double2hiint(s));
  const int oi = dpp_i32<CTRL, ROW_MASK>(-1, i);
  const double os = __hiloint2double(hi, lo);
  if (oi >= 0 && (i < 0 || os > s || (os == s && oi < i))) {
    s = os;
    i = oi;
  }
}

// The best (score, index) pair of a wave (all lanes active), in lane 63.
__device__ inline void wave_best_si(double& s, int& i) {
  best_step_si<0x111, 0xf>(s, i);
  best_step_si<0x112, 0xf>(s, i);
  best_step_si<0x114, 0xf>(s, i);
  best_step_si<0x118, 0xf>(s, i);
  best_step_si<0x142, 0xa>(s, i);
  best_step_si<0x143, 0xc>(s, i);
}

// Best feature of one node from its per-feature results (score s_f, bin b_f;
// b_f < 0: no valid threshold), by one wave (all lanes active): larger score
// first, then the smaller feature.  This is a maximum under a total order,
// so the result does not depend on the reduction order; the lanes' bests
// meet in registers (DPP row shifts and broadcasts, ending in lane 63) and
// every lane gets the result.  Outputs (-1, -1, -inf) when no feature has a
// valid threshold.
__device__ inline void wave_best_feature(const double* fs, const int32_t* fb, int m, int32_t* out_f, int32_t* out_b,
                                         double* out_s) {
  const int lane = threadIdx.x & 63;
  double best_s = -INFINITY;
  int best_f = -1, best_bin = -1;
  for (int f = lane; f < m; f += 64) {
    const int b = fb[f];
    const double s = fs[f];
    if (b >= 0 && (best_f < 0 || s > best_s || (s == best_s && f < best_f))) {
      best_s = s;
      best_f = f;
      best_bin = b;
    }
  }
  best_step<0x111, 0xf>(best_s, best_f, best_bin);
  best_step<0x112, 0xf>(best_s, best_f, best_bin);
  best_step<0x114, 0xf>(best_s, best_f, best_bin);
  best_step<0x118, 0xf>(best_s, best_f, best_bin);
  best_step<0x142, 0xa>(best_s, best_f, best_bin);
  best_step<0x143, 0xc>(best_s, best_f, best_bin);
  best_f = __builtin_amdgcn_readlane(best_f, 63);
  best_bin = __builtin_amdgcn_readlane(best_bin, 63);
  best_s = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(best_s), 63),
                            __builtin_amdgcn_readlane(__double2loint(best_s), 63));
  *out_f = best_f;
  *out_b = best_f >= 0 ? best_bin : -1;
  *out_s = best_f >= 0 ? best_s : -INFINITY;
}

// ---------------------------------------------------------------- errors
void set_error(const std::string& msg);
int32_t fail(int32_t code, const std::string& msg);
int32_t check_launch(const char* what);

// ---------------------------------------------------------------- launches (stream-ordered)
int32_t launch_layout(const uint8_t* bins, int64_t n, int32_t m, int64_t ld_bins, uint32_t* bins4, int64_t ld4,
                      uint8_t* bins_cm, int64_t ld_cm, uint8_t* rec, int64_t ld_rec, hipStream_t st);

// norm2_in: the squared column norms as an input (G is not read for them), or NULL.
int32_t launch_sketch(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                      const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols, float* scales,
                      double* norm2, int32_t* qexp, void* ws, hipStream_t st, const double* norm2_in = nullptr);
int64_t sketch_ws_bytes(int32_t kind, int64_t n, int32_t d, int32_t k);
int32_t launch_sketch_sparse(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k, int32_t s,
                             const int32_t* pi_col, const float* pi_val, float* GH, int64_t ld_gh, int32_t* qexp,
                             void* ws, hipStream_t st);
int64_t hist_exponents_ws_bytes(int32_t k);
int32_t launch_hist_exponents(const float* GH, int64_t n, int64_t ld_gh, int32_t k, int32_t* qexp, void* ws,
                              hipStream_t st);

int32_t launch_build_histograms(const uint32_t* bins4, int64_t ld4, const uint8_t* rec, int64_t ld_rec, int64_t n,
                                int32_t m, int32_t n_bins, const float* GH, int64_t ld_gh, int32_t k,
                                const int32_t* qexp,
                                const int32_t* row_idx, const int32_t* node_off, int32_t n_nodes,
                                const int32_t* build_list, int32_t n_build, double* H, void* ws, hipStream_t st,
                                const int64_t* pre_given = nullptr, const double* H_parent = nullptr,
                                double* feat_s = nullptr, int32_t* feat_b = nullptr, double lam = 0.0,
                                double mcw = 0.0, uint32_t* qrow = nullptr, bool qrow_ready = false,
                                bool store_h = true, int32_t* root_off = nullptr);
// The fused level end (reduction, subtraction and per-feature scoring in one
// kernel) holds a bin's channel sums of both nodes in registers: channels up
// to this many (every sketch the histogram kernel takes).
constexpr int FUSED_SCORE_MAX_C = 24;
int32_t launch_subtract(const double* Hp, double* Hc, int32_t n_parents, int64_t cells_per_node,
                        const int32_t* build_list, hipStream_t st);

int64_t score_ws_bytes(int32_t n_nodes, int32_t m);
int32_t launch_score(const double* H, int32_t n_nodes, int32_t m, int32_t n_bins, int32_t k, double lambda,
                     double mcw, int32_t* best_f, int32_t* best_b, double* best_s, void* ws, hipStream_t st);
int32_t launch_score_node(const double* feat_s, const int32_t* feat_b, int32_t n_nodes, int32_t m, int32_t* best_f,
                          int32_t* best_b, double* best_s, hipStream_t st);

int64_t partition_ws_bytes(int64_t n, int32_t n_nodes);
// The static scratch of the allocation-free partition (8 MiB per device) and
// its device address on the current device (looked up once per device).
constexpr int64_t PARTITION_SCRATCH_BYTES = int64_t(8) << 20;
int32_t partition_scratch(void** out);
// Splits come either as best_f/best_b (one per node, inputs), or, in the
// level loop, as the fused level end's per-(node, feature) results
// feat_s/feat_b: the partition then picks every node's best feature itself
// and writes it to best_f/best_b/best_s (the tree's node results).  The
// latter needs partition_picks_splits(n, n_nodes).
bool partition_picks_splits(int64_t n, int32_t n_nodes);
int32_t launch_partition(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm, const int32_t* row_in,
                         const int32_t* off_in, int32_t n_nodes, const int32_t* best_f, const int32_t* best_b,
                         int32_t* row_out, int32_t* off_out, int32_t* build_out, void* ws, hipStream_t st,
                         int64_t* next_pre = nullptr, const double* feat_s = nullptr, const int32_t* feat_b = nullptr,
                         double* best_s = nullptr);

int64_t leaf_ws_bytes(int64_t n, int32_t d, int32_t n_leaves);
int32_t launch_leaf_values(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* hess, int64_t ld_hess,
                           const float* h, const int32_t* row_idx, const int32_t* leaf_off, int32_t n_leaves,
                           double lambda, double* V, int64_t ld_v, void* ws, hipStream_t st);

int32_t launch_leaf_values_from_loss(int32_t loss, const float* G, int64_t n, int32_t d, int64_t ld_g,
                                     const int32_t* labels, const uint8_t* Y, int64_t ld_y, const int32_t* row_idx,
                                     const int32_t* leaf_off, int32_t n_leaves, double lambda, double* V, int64_t ld_v,
                                     void* ws, hipStream_t st);
int64_t grad_ws_bytes(int64_t n, int32_t d);
int32_t launch_gradients(int32_t loss, const float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* labels,
                         const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g, float* hess, int64_t ld_hess,
                         float* h_row, double* norm2, void* ws, hipStream_t st);
int64_t update_ws_bytes(int64_t n);
int32_t launch_update(float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx, const int32_t* leaf_off,
                      int32_t n_leaves, const double* V, int64_t ld_v, double lr, void* ws, hipStream_t st);
int64_t update_gradients_ws_bytes(int64_t n, int32_t d);
int32_t launch_update_gradients(int32_t loss, float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                                const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr,
                                const int32_t* labels, const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g,
                                float* hess, int64_t ld_hess, float* h_row, double* norm2, void* ws, hipStream_t st);

// ---------------------------------------------------------------- profiling
// Event pairs around histogram-kernel launches while profiling is on (per thread).
bool profile_on();
void profile_record(hipEvent_t start, hipEvent_t stop);

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

}  // namespace sb
