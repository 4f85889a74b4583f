// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/sb.h"

namespace sb {

// ---------------------------------------------------------------- errors
void set_error(const std::string& msg);
int32_t fail(int32_t code, const std::string& msg);
int32_t check_launch(const char* what);

// ---------------------------------------------------------------- fixed point
// Quantised magnitudes are <= 2^QBITS (qexp = QBITS-1 - floor(log2(max|v|))),
// so each value carries an error of at most 2^-(QBITS+1) of its channel's
// maximum magnitude.
constexpr int QBITS = 18;
// Each channel's LDS sum is a 32-bit running sum read back into int64 every
// window of WINDOW_ROWS rows (4 steps of the 768-thread workgroup).  A cell
// gets at most one value per row, and the change between two reads spans at
// most two windows, so 2 * WINDOW_ROWS * 2^QBITS must stay below 2^31.
constexpr int WINDOW_ROWS = 3072;
static_assert(2ll * WINDOW_ROWS * (1ll << QBITS) < (1ll << 31), "fixed-point window overflow");

// ---------------------------------------------------------------- histogram plan
// One histogram workgroup: 768 threads (12 waves, 3 per SIMD, so up to 168
// VGPRs per lane) and up to 40 channel cells per thread (20 64-bit LDS cells
// of two channels each: 120 KB of the 160 KB LDS).  Each thread keeps the
// int64 totals of its 40 channel cells in 80 VGPRs next to the prefetched
// row data of the step loop; with 4 waves per SIMD (128 VGPRs) they would
// spill to scratch.
constexpr int HIST_THREADS = 768;
constexpr int HIST_MAX_CELLS_PER_THREAD = 40;
constexpr int HIST_LDS_BYTES = HIST_MAX_CELLS_PER_THREAD * HIST_THREADS * 4;
// MI355X: 8 XCDs of 32 CUs; workgroup b is dispatched to XCD b % 8.
constexpr int HIST_CUS_PER_XCD = 32;
// A lane holds the bin words of up to 16 quads (64 features) of its row.
constexpr int HIST_MAX_QUADS = 16;

struct HistPlan {
  int c;          // channels k+1
  int pairs;      // 64-bit LDS cells per (feature, bin): ceil(c/2)
  int nq;         // 4-feature quads per slice
  int f;          // features per slice (4*nq)
  int slices;     // feature slices
  int rows_wave;  // rows one wave handles per step (64 / nq)
  int cells;      // 2 * pairs * f * n_bins channel cells per workgroup
  int q;          // row groups per slice
  int q_pad;      // q rounded up to a multiple of 8 (XCD-aware mapping)
  int64_t slots;  // partial slots per slice: q + n_build
};
HistPlan hist_plan(int32_t m, int32_t n_bins, int32_t k, int32_t n_build);
int64_t hist_ws_bytes(int32_t m, int32_t n_bins, int32_t k, int32_t n_build);

// ---------------------------------------------------------------- launches (stream-ordered)
int32_t launch_layout(const uint8_t* bins, int64_t n, int32_t m, int64_t ld_bins, uint32_t* bins4, int64_t ld4,
                      uint8_t* bins_cm, int64_t ld_cm, uint8_t* rec, int64_t ld_rec, hipStream_t st);

int32_t launch_sketch(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                      const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols, float* scales,
                      double* norm2, int32_t* qexp, void* ws, hipStream_t st);
int64_t sketch_ws_bytes(int32_t kind, int64_t n, int32_t d, int32_t k);
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
                                double mcw = 0.0);
// The fused level end (reduction, subtraction and per-feature scoring in one
// kernel) stages both nodes' values of one feature in LDS: channels up to
// this many (64 KB at 256 bins).
constexpr int FUSED_SCORE_MAX_C = 16;
int32_t launch_subtract(const double* Hp, double* Hc, int32_t n_parents, int64_t cells_per_node,
                        const int32_t* build_list, hipStream_t st);

int64_t score_ws_bytes(int32_t n_nodes, int32_t m);
int32_t launch_score(const double* H, int32_t n_nodes, int32_t m, int32_t n_bins, int32_t k, double lambda,
                     double mcw, int32_t* best_f, int32_t* best_b, double* best_s, void* ws, hipStream_t st);
int32_t launch_score_node(const double* feat_s, const int32_t* feat_b, int32_t n_nodes, int32_t m, int32_t* best_f,
                          int32_t* best_b, double* best_s, hipStream_t st);

int64_t partition_ws_bytes(int64_t n, int32_t n_nodes);
int32_t launch_partition(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm, const int32_t* row_in,
                         const int32_t* off_in, int32_t n_nodes, const int32_t* best_f, const int32_t* best_b,
                         int32_t* row_out, int32_t* off_out, int32_t* build_out, void* ws, hipStream_t st,
                         int64_t* next_pre = nullptr);

// ---------------------------------------------------------------- profiling
// Event pairs around histogram-kernel launches while profiling is on (per thread).
bool profile_on();
void profile_record(hipEvent_t start, hipEvent_t stop);

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

}  // namespace sb
