// Constants and work plan of the histogram kernel (fixed point, workgroup
// shape, LDS budget, feature slicing).
#pragma once

#include <cstdint>

namespace sb {

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
// The rotated kernel reads each row's quantised values, not its fp32 sketch:
// up to 6 channels as QFIELD_BITS-bit two's-complement fields of one 16-byte
// word (channels 0-2 in bits 0-62 of the low 64 bits, 3-5 in the high 64
// bits), written once per sketch, so that a row's values are one 16-byte load.
constexpr int QFIELD_BITS = 21;
constexpr int QROW_MAX_C = 6;
// More channels take several such words per row, one per channel group of
// six; each group gets workgroups of its own (up to ROT_MAX_C channels).
constexpr int ROT_MAX_C = 24;
static_assert(QBITS + 2 <= QFIELD_BITS, "a quantised value of magnitude <= 2^QBITS and its sign must fit a field");

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

// Rotated-feature workgroups (up to 3 channel pairs, c <= 6): a slice of 16
// features, LDS cells [bin][pair][feature] for 256 bins (12288 64-bit cells,
// 96 KB), ROT_CPT cells per thread.
#ifndef SB_HIST_ROT_THREADS
#define SB_HIST_ROT_THREADS 768
#endif
constexpr int ROT_THREADS = SB_HIST_ROT_THREADS;
constexpr int ROT_F = 16;
constexpr int ROT_PMAX = 3;
constexpr int ROT_CELLS = 256 * ROT_PMAX * ROT_F;
constexpr int ROT_CPT = ROT_CELLS / ROT_THREADS;
static_assert(ROT_CPT * ROT_THREADS == ROT_CELLS, "rotated cells must split evenly over the threads");
static_assert(WINDOW_ROWS % ROT_THREADS == 0, "a fixed-point window must be a whole number of steps");

struct HistPlan {
  bool rot;       // rotated-feature kernel (c <= 6), else the row-per-lane kernel
  int c;          // channels k+1
  int pairs;      // 64-bit LDS cells per (feature, bin): ceil(c/2)
  int nq;         // 4-feature quads per slice
  int f;          // features per slice (4*nq)
  int slices;     // feature slices
  int rows_wave;  // rows one wave handles per step (64 / nq)
  int cells;      // 2 * pairs * f * n_bins channel cells per workgroup
  int q;          // row groups per (full) slice
  int q_pad;      // q rounded up to a multiple of 8 (XCD-aware mapping)
  int64_t slots;  // partial slots per slice: max(q, q_thin) + n_build
  // Rotated kernel: the first slices_full slices hold 16 features each; when
  // m is not a multiple of 16 the rest go to one thin slice of f_thin
  // features (a power of two below 16), whose workgroups keep 16 / f_thin
  // copies of each cell so that its adds stay conflict-free while a row
  // costs f_thin steps instead of 16.  Per XCD: a_full row groups of every
  // full slice and b_thin row groups of the thin slice (q = 8 a_full,
  // q_thin = 8 b_thin), chosen to even out the work of its 32 CUs.  Only for
  // rows read straight from the data (the root): rows gathered through row
  // indices are cheaper to read when the slices of a row group share an XCD,
  // so there the last slice is a padded slice of 16 like the others.
  int slices_full, f_thin, a_full, b_thin, q_thin;
  // Rotated kernel with c > 6 channels: cg = ceil(c / 6) channel groups of
  // at most three pairs; every (slice, channel group) of a row group is one
  // workgroup, and all groups of a slice write the same partial slots.
  int cg;
  int grid;       // histogram workgroups
};
HistPlan hist_plan(int32_t m, int32_t n_bins, int32_t k, int32_t n_build, bool thin_ok = false);
// Workspace of one histogram launch; quant_rows adds the n quantised sketch
// rows of the rotated kernel (16 bytes each).
int64_t hist_ws_bytes(int64_t n, int32_t m, int32_t n_bins, int32_t k, int32_t n_build, bool quant_rows);

}  // namespace sb
