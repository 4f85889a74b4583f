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
// MI355X: 8 XCDs of 32 CUs; workgroup b is dispatched to XCD b % 8.
constexpr int HIST_CUS_PER_XCD = 32;

// One histogram workgroup: 768 threads (12 waves, 3 per SIMD) and the cells
// of a slice of 16 features for up to 3 channel pairs (c <= 6), laid out
// [bin][pair][feature] for 256 bins (12288 64-bit cells, 96 KB of the
// 160 KB LDS), ROT_CPT cells per thread.
constexpr int ROT_THREADS = 768;
constexpr int ROT_F = 16;
constexpr int ROT_PMAX = 3;
constexpr int ROT_CELLS = 256 * ROT_PMAX * ROT_F;
constexpr int ROT_CPT = ROT_CELLS / ROT_THREADS;
static_assert(ROT_CPT * ROT_THREADS == ROT_CELLS, "rotated cells must split evenly over the threads");
static_assert(WINDOW_ROWS % ROT_THREADS == 0, "a fixed-point window must be a whole number of steps");

struct HistPlan {
  int c;          // channels k+1
  int pairs;      // channel pairs: ceil(c/2)
  int nq;         // 4-feature quads per slice (0: the shape is not supported)
  int f;          // features per slice (16)
  int slices;     // feature slices
  int cells;      // 2 * pairs * f * n_bins channel cells of a partial
  int q;          // row groups per full slice
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
// Plan of one histogram launch; nq == 0 when c > ROT_MAX_C or n_bins > 256.
HistPlan hist_plan(int32_t m, int32_t n_bins, int32_t k, int32_t n_build, bool thin_ok = false);
// Workspace of one histogram launch (-1 when unsupported); quant_rows adds
// the n quantised sketch rows (16 * cg bytes each).
int64_t hist_ws_bytes(int64_t n, int32_t m, int32_t n_bins, int32_t k, int32_t n_build, bool quant_rows);

}  // namespace sb
