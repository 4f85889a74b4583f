// Leaf values from the full gradient matrix (Section 2, "Finding the leaf
// values": with diagonal Hessians the value of leaf R is, output by output,
// v_j = -sum_{i in R} g_ij / (sum_{i in R} h_ij + lambda), eq. 3.  Section 3:
// the sketch serves only the search for the structure; leaf values use all d
// outputs of G).
//
// A leaf's rows are scattered over the rows of G, and G is column-major, so
// gathering a leaf's rows would fetch a whole 32-byte sector for every 4-byte
// value.  The path streams G once, in row order, instead:
//   k_leaf_ids    writes every row's leaf id from the leaf segments;
//   k_leaf_accum  one block per (chunk of J channels, split of the rows).  The
//                 lanes take consecutive rows of a column (256-byte loads per
//                 wave) and add every value into an LDS cell (leaf, channel);
//   k_leaf_final  sums the splits' partials per (leaf, output) in a fixed
//                 order and divides.
// Channels are the d gradient columns followed by the hessian columns (d of
// them per element, or one per-row weight, or none: then the denominator is
// the leaf's row count).  For the cross-entropies the per-element hessians
// follow from G and the targets (p = g + target, h = p (1 - p)), so they
// can be formed while loading G instead of being stored and read.
//
// Exact, order-free accumulation.  Per tile of T = 2048 rows and per
// channel, the block takes M = max |v| over the tile, with M < 2^E, and maps
// each v to the integer rint(v * 2^(ql - E)), of magnitude <= 2^ql (ql = 41).  T * 2^ql <= 2^52, so any sum of one
// tile's integers is an integer below 2^53: the 64-bit LDS integer atomics
// reach the same sum in any order, and that sum times 2^(E - ql) is an exact
// fp64 value.  One thread
// per cell adds it to the cell's fp64 accumulator, tile after tile, so the
// rounding order is fixed and the result does not depend on timing.  Each
// element is off by at most 2^(E - ql - 1) <= M * 2^-ql.
#include <cmath>

#include "sb_common.h"
#include "sb_leaf_ids.h"

namespace sb {
namespace {

constexpr int LEAF_THREADS = 256;
// Rows per thread per tile: 8 (2048-row tiles), with plain channels and
// with the derived hessians alike (4 rows per thread, 1024-row tiles, took
// 368 against 290 us on 2M x 100: twice the per-tile maxima and cell
// flushes per row).
constexpr int LEAF_SPT = 8;
constexpr int LEAF_SPT_DERIVED = 8;
// Quantum exponent for a tile of 256 * SPT rows: tile * 2^ql <= 2^52.
constexpr int leaf_ql(int spt) { return spt == 8 ? 41 : (spt == 4 ? 42 : 40); }
static_assert((int64_t)(LEAF_THREADS * 8) << leaf_ql(8) <= (int64_t(1) << 52), "tile sums must stay exact in fp64");
static_assert((int64_t)(LEAF_THREADS * 4) << leaf_ql(4) <= (int64_t(1) << 52), "tile sums must stay exact in fp64");
constexpr int64_t LEAF_LDS_MAX = 64 * 1024;             // integer + fp64 cells of one block
constexpr int LEAF_TARGET_BLOCKS = 4096;                // 16 per CU
// channels per block (fewer for many leaves, so that the cells fit LEAF_LDS_MAX)
constexpr int LEAF_JMAX = 4;
// with derived hessians a block holds 4 outputs (8 channels), so the
// per-row leaf ids and labels are read once per 4 outputs
constexpr int LEAF_JMAX_DERIVED = 8;
// copies of each integer cell, lane l adding to copy l mod copies
constexpr int LEAF_MAX_COPIES = 4;

struct LeafArgs {
  const float* G;
  int64_t ld_g;
  int32_t d;
  const float* hess;  // per-element hessians (column-major) or NULL
  int64_t ld_h;
  const float* h;     // per-row hessian or NULL
  // hessians formed from G and the targets: 0 no, 1 softmax (labels), 2
  // sigmoid (Y).  Channels are then interleaved: 2o is g of output o, 2o+1
  // its hessian, so one block reads each column of G once.
  int32_t derive;
  const uint16_t* labels;  // narrowed to 16 bits
  const uint8_t* Y;
  int64_t ld_y;
  const void* leaf_of;  // uint8 ids for up to 256 leaves, else uint16
  int64_t n;
  int32_t n_leaves;
  int32_t nch;
  int32_t n_tiles;
  int32_t tiles_per_split;
  int32_t copies_shift;  // 2^copies_shift copies of every integer cell
  double* part;       // [leaf][nch][split]
};

__device__ inline const float* chan_ptr(const LeafArgs& a, int c) {
  if (a.derive) return a.G + (int64_t)(c >> 1) * a.ld_g;  // odd channels are transformed after the load
  if (c < a.d) return a.G + (int64_t)c * a.ld_g;
  if (a.hess) return a.hess + (int64_t)(c - a.d) * a.ld_h;
  return a.h;
}

// 2^e as a double, for |e| <= 1022.
__device__ inline double pow2(int e) { return __longlong_as_double((long long)(1023 + e) << 52); }

// rint(y) as an int64 for |y| < 2^51: adding 1.5 * 2^52 leaves the integer
// nearest to y (ties to even) in the low mantissa bits, and the fused
// multiply-add rounds the exact product v * scale only once.
__device__ inline long long rint_to_ll(float v, double scale) {
  const double t = fma((double)v, scale, 6755399441055744.0);
  return __double_as_longlong(t) - 0x4338000000000000ll;
}

template <int J, int SPT>
struct LeafTile {
  float v[SPT][J];
  int lf[SPT];
};

// DER: how the odd channels are made (0: loaded as they are; 1 softmax, 2
// sigmoid: the hessian of the even channel's output, formed after the load).
// With DER the two channels of an output come from one column of G, loaded
// once.
template <int J, int SPT, typename LT, int DER>
__device__ inline void leaf_load(const LeafArgs& a, const float* const (&col)[J], int c0, int t, int top,
                                 LeafTile<J, SPT>& x) {
  // Rows past the end load row n-1 and get a negative leaf id, which drops
  // them from the adds (they may still raise the tile maximum, which only has
  // to bound the tile's values).  No value depends on a condition, so the
  // compiler issues every load of the tile back to back instead of waiting
  // for each one inside its own branch.
  const LT* ids = static_cast<const LT*>(a.leaf_of);
  const int64_t r0 = (int64_t)t * (LEAF_THREADS * SPT);
#pragma unroll
  for (int s = 0; s < SPT; ++s) {
    const int64_t row = r0 + threadIdx.x + LEAF_THREADS * s;
    const int64_t rc = row < a.n ? row : a.n - 1;
    const int l = (int)ids[rc];
    x.lf[s] = (l > top ? top : l) - (row < a.n ? 0 : 0x10000);
#pragma unroll
    for (int j = 0; j < J; ++j) x.v[s][j] = (DER && J >= 2 && (j & 1)) ? x.v[s][j - 1] : col[j][rc];
  }
  if constexpr (DER != 0) {
    // odd channel 2o+1: the hessian of output o from g = G[i, o]:
    // softmax p = g + [o == label], sigmoid s = g + Y[i, o]; h = p (1 - p).
    // Applied after every load of the tile is issued.
    float tg[SPT][J];
#pragma unroll
    for (int s = 0; s < SPT; ++s) {
      const int64_t row = r0 + threadIdx.x + LEAF_THREADS * s;
      const int64_t rc = row < a.n ? row : a.n - 1;
      const int y = DER == 1 ? (int)a.labels[rc] : -1;
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int c = c0 + j, o = c >> 1;
        if (J >= 2 && !(j & 1)) {
          tg[s][j] = 0.0f;  // even channel: g itself
        } else if constexpr (DER == 1) {
          tg[s][j] = o == y ? 1.0f : 0.0f;
        } else {
          tg[s][j] = (float)a.Y[(int64_t)(o < a.d ? o : a.d - 1) * a.ld_y + rc];
        }
      }
    }
    // c0 is a multiple of J, so for J >= 2 channel c0 + j is odd when j is
    const bool c0_odd = (c0 & 1) != 0;
#pragma unroll
    for (int s = 0; s < SPT; ++s)
#pragma unroll
      for (int j = 0; j < J; ++j) {
        if (J >= 2 ? (j & 1) != 0 : c0_odd) {
          const float p = x.v[s][j] + tg[s][j];
          x.v[s][j] = p * (1.0f - p);
        }
      }
  }
}

// A float moved across lanes by a DPP control (row shift or row broadcast);
// lanes the control does not write get 0.
template <int CTRL, int ROW_MASK>
__device__ inline float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xf, false));
}

// Maximum of non-negative values over the 64 lanes of a wave, in registers
// (no LDS traffic): shifts by 1, 2, 4 and 8 lanes inside each row of 16, then
// the last lane of rows 0 and 2 into rows 1 and 3 (row_bcast:15) and lane 31
// into rows 2 and 3 (row_bcast:31).  Lanes a step does not write take 0,
// which leaves a maximum of non-negative values unchanged.  Lane 63 ends
// with the wave's maximum.
__device__ inline float wave_max_nonneg(float x) {
  x = fmaxf(x, dpp_f32<0x111, 0xf>(x));
  x = fmaxf(x, dpp_f32<0x112, 0xf>(x));
  x = fmaxf(x, dpp_f32<0x114, 0xf>(x));
  x = fmaxf(x, dpp_f32<0x118, 0xf>(x));
  x = fmaxf(x, dpp_f32<0x142, 0xa>(x));
  x = fmaxf(x, dpp_f32<0x143, 0xc>(x));
  return x;
}

// One tile: block-wide maximum per channel, quantisation, integer adds into
// the LDS cells, then the exact fp64 conversion into the accumulators.
template <int J, int SPT>
__device__ inline void leaf_tile(const LeafTile<J, SPT>& x, const bool (&live)[J], float (&wmax)[LEAF_THREADS / 64][J],
                                 double (&sconv)[J], unsigned long long* icell, double* acc, int NL, int rsh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cells = NL * J;
  const int copy = lane & ((1 << rsh) - 1);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    float mx = 0.0f;
#pragma unroll
    for (int s = 0; s < SPT; ++s) mx = fmaxf(mx, fabsf(x.v[s][j]));
    mx = wave_max_nonneg(mx);
    if (lane == 63) wmax[wave][j] = mx;
  }
  __syncthreads();
  double sc[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    float M = wmax[0][j];
#pragma unroll
    for (int w = 1; w < LEAF_THREADS / 64; ++w) M = fmaxf(M, wmax[w][j]);
    int E = 0;
    if (M > 0.0f) (void)frexpf(M, &E);  // M = f * 2^E with f in [0.5, 1): every |v| < 2^E
    sc[j] = M > 0.0f ? pow2(leaf_ql(SPT) - E) : 0.0;
    if (tid == j) sconv[j] = M > 0.0f ? pow2(E - leaf_ql(SPT)) : 0.0;
  }
#pragma unroll
  for (int s = 0; s < SPT; ++s) {
    // a row past the end adds 0 to leaf 0
    const bool in = x.lf[s] >= 0;
    const int l = in ? x.lf[s] : 0;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const long long q = rint_to_ll(x.v[s][j], sc[j]);
      if (live[j]) atomicAdd(&icell[((j * NL + l) << rsh) + copy], (unsigned long long)(in ? q : 0ll));
    }
  }
  __syncthreads();
  // The next tile's adds (and its writes of wmax and sconv) start only after
  // its first barrier, which every thread reaches after finishing this loop.
  for (int cell = tid; cell < cells; cell += LEAF_THREADS) {
    unsigned long long* cp = icell + ((int64_t)cell << rsh);
    long long q = 0;
    for (int r = 0; r < (1 << rsh); ++r) q += (long long)cp[r];  // exact: the copies split one tile's sum
    if (q != 0) acc[cell] += (double)q * sconv[cell / NL];
    for (int r = 0; r < (1 << rsh); ++r) cp[r] = 0ull;
  }
}

template <int J, int SPT, typename LT, int DER>
__global__ void __launch_bounds__(LEAF_THREADS) k_leaf_accum(LeafArgs a) {
  // Cells are channel-major ([J][n_leaves]): the lanes of one add instruction
  // share the channel, so their addresses differ by leaf and spread over the
  // LDS banks.  Each integer cell has 2^rsh copies side by side, lane l adding
  // to copy l mod 2^rsh: lanes whose rows share a leaf (most lanes when few
  // leaves are large) then mostly hit different addresses.
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ float wmax[LEAF_THREADS / 64][J];
  __shared__ double sconv[J];
  const int NL = a.n_leaves;
  const int cells = NL * J;
  const int rsh = a.copies_shift;
  unsigned long long* icell = reinterpret_cast<unsigned long long*>(smem);
  double* acc = reinterpret_cast<double*>(smem + ((size_t)cells << rsh) * 8);
  const int tid = threadIdx.x;
  const int c0 = blockIdx.x * J;
  const int split = blockIdx.y;

  const float* col[J];
  bool live[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    live[j] = c0 + j < a.nch;
    col[j] = chan_ptr(a, live[j] ? c0 + j : c0);  // a channel past the last one reads the chunk's first
  }
  for (int cell = tid; cell < (cells << rsh); cell += LEAF_THREADS) icell[cell] = 0ull;
  for (int cell = tid; cell < cells; cell += LEAF_THREADS) acc[cell] = 0.0;
  const int t0 = split * a.tiles_per_split;
  const int t1 = min(a.n_tiles, t0 + a.tiles_per_split);
  const int top = NL - 1;
  __syncthreads();

  for (int t = t0; t < t1; ++t) {
    LeafTile<J, SPT> x;
    leaf_load<J, SPT, LT, DER>(a, col, c0, t, top, x);
    leaf_tile(x, live, wmax, sconv, icell, acc, NL, rsh);
  }
  __syncthreads();
  for (int cell = tid; cell < cells; cell += LEAF_THREADS) {
    const int j = cell / NL, L = cell - j * NL;
    if (c0 + j < a.nch) a.part[((int64_t)L * a.nch + c0 + j) * gridDim.y + split] = acc[cell];
  }
}

// One wave per (leaf, output): the lanes sum the splits' partials (stored
// split-contiguous) in a fixed lane-strided order, then a fixed butterfly
// combines the lanes.  hmode: 0 = no hessian (row counts), 1 = per-element
// hessian channels d..2d-1, 2 = one per-row hessian channel d, 3 = g and h
// interleaved (channels 2j, 2j+1).
__global__ void __launch_bounds__(256) k_leaf_final(const double* __restrict__ part, int32_t n_splits,
                                                    int32_t n_leaves, int32_t d, int32_t nch, int32_t hmode,
                                                    const int32_t* __restrict__ leaf_off, double lam,
                                                    double* __restrict__ V, int64_t ld_v) {
  const int lane = threadIdx.x & 63;
  const int64_t out = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (out >= (int64_t)n_leaves * d) return;
  const int L = (int)(out / d), j = (int)(out % d);
  const double* pg = part + ((int64_t)L * nch + (hmode == 3 ? 2 * j : j)) * n_splits;
  const double* ph = hmode == 3   ? part + ((int64_t)L * nch + 2 * j + 1) * n_splits
                     : hmode == 1 ? part + ((int64_t)L * nch + d + j) * n_splits
                                  : part + ((int64_t)L * nch + d) * n_splits;
  const double gs0 = lane_strided_sum(pg, n_splits, lane);
  const double hs0 = hmode != 0 ? lane_strided_sum(ph, n_splits, lane) : 0.0;
  double gs = gs0, hs = hs0;
  for (int off = 32; off > 0; off >>= 1) {
    gs += __shfl_xor(gs, off, 64);
    hs += __shfl_xor(hs, off, 64);
  }
  if (lane != 0) return;
  if (hmode == 0) hs = (double)((int64_t)leaf_off[L + 1] - (int64_t)leaf_off[L]);
  V[(int64_t)L * ld_v + j] = -gs / (hs + lam);
}

// Labels as 16-bit values (labels outside [0, d) become d, which matches no output).
__global__ void __launch_bounds__(256) k_narrow_labels(const int32_t* __restrict__ labels, int64_t n, int32_t d,
                                                        uint16_t* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int32_t y = labels[i];
    out[i] = (uint16_t)((y >= 0 && y < d) ? y : d);
  }
}

struct LeafPlan {
  int J, spt, nch, n_chunks, n_tiles, tps, splits, rsh;
  int64_t lds;
};

LeafPlan leaf_plan(int64_t n, int32_t nch, int32_t n_leaves, int jmax = LEAF_JMAX, int spt = LEAF_SPT) {
  LeafPlan p{};
  p.spt = spt;
  p.J = jmax;
  while (p.J > 1 && (int64_t)n_leaves * p.J * 16 > LEAF_LDS_MAX) p.J >>= 1;
  p.nch = nch;
  p.n_chunks = (nch + p.J - 1) / p.J;
  p.n_tiles = (int)((n + LEAF_THREADS * spt - 1) / (LEAF_THREADS * spt));
  int splits = (LEAF_TARGET_BLOCKS + p.n_chunks - 1) / p.n_chunks;
  if (splits < 1) splits = 1;
  if (splits > p.n_tiles) splits = p.n_tiles;
  p.tps = (p.n_tiles + splits - 1) / splits;
  p.splits = (p.n_tiles + p.tps - 1) / p.tps;
  // as many copies of the integer cells (up to LEAF_MAX_COPIES) as the LDS budget allows
  p.rsh = 0;
  while ((1 << (p.rsh + 1)) <= LEAF_MAX_COPIES && (int64_t)n_leaves * p.J * (8 * (2 << p.rsh) + 8) <= LEAF_LDS_MAX)
    ++p.rsh;
  p.lds = (int64_t)n_leaves * p.J * (8 * (1 << p.rsh) + 8);
  return p;
}

int64_t leaf_ws_for(int64_t n, int32_t nch, int32_t n_leaves, int jmax = LEAF_JMAX, int spt = LEAF_SPT) {
  const LeafPlan p = leaf_plan(n, nch, n_leaves, jmax, spt);
  return leaf_ids_bytes(n) + align256((int64_t)p.splits * n_leaves * nch * 8) + align256(n * 2);
}

template <int J, typename LT>
void launch_accum(const LeafPlan& p, const LeafArgs& a, hipStream_t st) {
  const dim3 g(p.n_chunks, p.splits);
  if (a.derive == 1)
    hipLaunchKernelGGL((k_leaf_accum<J, LEAF_SPT_DERIVED, LT, 1>), g, dim3(LEAF_THREADS), (size_t)p.lds, st, a);
  else if (a.derive == 2)
    hipLaunchKernelGGL((k_leaf_accum<J, LEAF_SPT_DERIVED, LT, 2>), g, dim3(LEAF_THREADS), (size_t)p.lds, st, a);
  else
    hipLaunchKernelGGL((k_leaf_accum<J, LEAF_SPT, LT, 0>), g, dim3(LEAF_THREADS), (size_t)p.lds, st, a);
}

template <typename LT>
void launch_leaf_kernels(const LeafPlan& p, LeafArgs a, const int32_t* row_idx, const int32_t* leaf_off, void* ids,
                         hipStream_t st) {
  launch_leaf_ids(row_idx, leaf_off, a.n_leaves, a.n, ids, st);
  a.leaf_of = ids;
  switch (p.J) {
    case 8: launch_accum<8, LT>(p, a, st); break;
    case 4: launch_accum<4, LT>(p, a, st); break;
    case 2: launch_accum<2, LT>(p, a, st); break;
    default: launch_accum<1, LT>(p, a, st); break;
  }
}

}  // namespace

int64_t leaf_ws_bytes(int64_t n, int32_t d, int32_t n_leaves) {
  // the largest of the three hessian forms
  int64_t b = leaf_ws_for(n, d, n_leaves);
  const int64_t b1 = leaf_ws_for(n, d + 1, n_leaves);
  const int64_t b2 = leaf_ws_for(n, 2 * d, n_leaves);
  const int64_t b3 = leaf_ws_for(n, 2 * d, n_leaves, LEAF_JMAX_DERIVED, LEAF_SPT_DERIVED);
  if (b1 > b) b = b1;
  if (b2 > b) b = b2;
  if (b3 > b) b = b3;
  return b;
}

int32_t launch_leaf_values(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* hess, int64_t ld_hess,
                           const float* h, const int32_t* row_idx, const int32_t* leaf_off, int32_t n_leaves,
                           double lambda, double* V, int64_t ld_v, void* ws, hipStream_t st) {
  const int hmode = hess ? 1 : (h ? 2 : 0);
  const int32_t nch = d + (hmode == 1 ? d : (hmode == 2 ? 1 : 0));
  const LeafPlan p = leaf_plan(n, nch, n_leaves);
  char* w = static_cast<char*>(ws);
  double* part = reinterpret_cast<double*>(w + leaf_ids_bytes(n));
  const LeafArgs a{G,       ld_g,    d, hess,     ld_hess,   h,         0,     nullptr, nullptr, 0,
                   nullptr, n,       n_leaves, nch, p.n_tiles, p.tps, p.rsh, part};
  if (n_leaves <= 256)
    launch_leaf_kernels<uint8_t>(p, a, row_idx, leaf_off, w, st);
  else
    launch_leaf_kernels<uint16_t>(p, a, row_idx, leaf_off, w, st);
  const int64_t outs = (int64_t)n_leaves * d;
  hipLaunchKernelGGL(k_leaf_final, dim3((unsigned)((outs + 3) / 4)), dim3(256), 0, st, part, p.splits, n_leaves, d,
                     nch, hmode, leaf_off, lambda, V, ld_v);
  return check_launch("sb_leaf_values");
}

int32_t launch_leaf_values_from_loss(int32_t loss, const float* G, int64_t n, int32_t d, int64_t ld_g,
                                     const int32_t* labels, const uint8_t* Y, int64_t ld_y, const int32_t* row_idx,
                                     const int32_t* leaf_off, int32_t n_leaves, double lambda, double* V, int64_t ld_v,
                                     void* ws, hipStream_t st) {
  const int32_t nch = 2 * d;
  const LeafPlan p = leaf_plan(n, nch, n_leaves, LEAF_JMAX_DERIVED, LEAF_SPT_DERIVED);
  char* w = static_cast<char*>(ws);
  double* part = reinterpret_cast<double*>(w + leaf_ids_bytes(n));
  uint16_t* lab16 = reinterpret_cast<uint16_t*>(w + leaf_ids_bytes(n) + align256((int64_t)p.splits * n_leaves * nch * 8));
  if (loss == SB_LOSS_SOFTMAX_CE) {
    const int64_t b = (n + 255) / 256;
    hipLaunchKernelGGL(k_narrow_labels, dim3((unsigned)(b < 2048 ? b : 2048)), dim3(256), 0, st, labels, n, d, lab16);
  }
  const LeafArgs a{G, ld_g, d, nullptr, 0, nullptr, loss == SB_LOSS_SOFTMAX_CE ? 1 : 2, lab16, Y, ld_y, nullptr,
                   n, n_leaves, nch, p.n_tiles, p.tps, p.rsh, part};
  if (n_leaves <= 256)
    launch_leaf_kernels<uint8_t>(p, a, row_idx, leaf_off, w, st);
  else
    launch_leaf_kernels<uint16_t>(p, a, row_idx, leaf_off, w, st);
  const int64_t outs = (int64_t)n_leaves * d;
  hipLaunchKernelGGL(k_leaf_final, dim3((unsigned)((outs + 3) / 4)), dim3(256), 0, st, part, p.splits, n_leaves, d,
                     nch, 3, leaf_off, lambda, V, ld_v);
  return check_launch("sb_leaf_values_from_loss");
}

}  // namespace sb
