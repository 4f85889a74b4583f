// Per-node histograms of one tree level (Section 3.4) and sibling subtraction.
//
// Design for gfx950.  The scatter-add of random bins into LDS bounds this
// kernel where rows are contiguous (the root); below it the gathered loads
// of scattered rows weigh as much.  Every choice below serves the LDS data
// path:
//  * every sketch value is quantised to an integer rint(v * 2^qexp[t]) of
//    magnitude <= 2^QBITS (written once per tree as 21-bit fields of one
//    16-byte word per row and channel group of six);
//  * channels are packed in pairs into 64-bit LDS cells holding
//    hi * 2^32 + lo as a two's-complement sum, one ds_add_u64 per pair;
//  * a slice of 16 features keeps its cells as [bin][pair][feature] and lane
//    l adds feature (i + l) mod 16 at step i, so a cell's bank pair is its
//    feature and every instruction puts four lanes on each bank pair,
//    whatever the bins (no bank conflicts);
//  * each cell is a running sum modulo 2^64.  Its owner thread reads it back
//    every window of <= WINDOW_ROWS rows, splits the change into the two
//    channel changes (each below 2^31 in magnitude, so the split is exact)
//    and adds them into int64 register totals;
//  * a workgroup owns one feature slice and a contiguous range of the rows of
//    the built nodes, taken in build-list order; it writes one partial per
//    node it touched: every channel sum as an int32 when it fits (almost
//    always: a workgroup's sum of one bin exceeds 2^31 only past 8192 rows
//    of full-scale values in that bin), else an escape value and the exact
//    int64 pair in an overflow slot of the same index;
//  * the reduce kernels sum the partials of each node (integers, so the
//    result is independent of the grid) and write the fp64 histogram.  Sums
//    of fixed-point values are exact in fp64, which makes sibling
//    subtraction exact as well.
// Rows come either as positions of contiguous data (quad-major bins: 256
// contiguous bytes per wave and word) or through row indices from the row
// records (one record line per row).
// Workgroups that share a row range but own different slices are placed on
// the same XCD (dispatch is round-robin over the 8 XCDs by block index) so
// the rows they all read stay in that XCD's L2.
#include "sb_common.h"

namespace sb {

HistPlan hist_plan(int32_t m, int32_t n_bins, int32_t k, int32_t n_build, bool thin_ok) {
  HistPlan p{};
  p.c = k + 1;
  p.pairs = (p.c + 1) / 2;
  if (p.c <= ROT_MAX_C && n_bins <= 256) {
    p.cg = (p.c + QROW_MAX_C - 1) / QROW_MAX_C;
    p.nq = ROT_F / 4;
    p.f = ROT_F;
    p.cells = 2 * p.pairs * p.f * n_bins;
    p.slices_full = m / ROT_F;
    const int r = m % ROT_F;
    p.f_thin = 0;
    if (r) {
      int ft = 1;
      while (ft < r) ft <<= 1;
      if (ft == ROT_F || !thin_ok) ++p.slices_full;  // a padded slice of 16
      else p.f_thin = ft;
    }
    p.slices = p.slices_full + (p.f_thin ? 1 : 0);
    const int S = p.slices_full, cus = HIST_CUS_PER_XCD;
    const int uf = S * p.cg, ut = p.cg;  // workgroups per full / thin row group
    if (!p.f_thin) {
      p.a_full = cus / uf > 0 ? cus / uf : 1;
      p.b_thin = 0;
    } else if (S == 0) {
      p.a_full = 0;
      p.b_thin = cus / ut > 0 ? cus / ut : 1;
    } else {
      // per-workgroup work of a full slice is ROT_F rows-steps per row of its
      // group, of the thin slice f_thin: minimise the larger of the two
      int best_a = 1;
      double best = 1e30;
      for (int aa = 1; aa * uf < cus || aa == 1; ++aa) {
        const int bb = (cus - aa * uf) / ut > 0 ? (cus - aa * uf) / ut : 1;
        const double cost = fmax((double)ROT_F / aa, (double)p.f_thin / bb);
        if (cost < best) {
          best = cost;
          best_a = aa;
        }
      }
      p.a_full = best_a;
      p.b_thin = (cus - best_a * uf) / ut > 0 ? (cus - best_a * uf) / ut : 1;
    }
    p.q = 8 * p.a_full;
    p.q_thin = 8 * p.b_thin;
    p.slots = (int64_t)(p.q > p.q_thin ? p.q : p.q_thin) + n_build;
    p.grid = 8 * (p.a_full * uf + p.b_thin * ut);
    return p;
  }
  return p;  // more than ROT_MAX_C channels or 256 bins: unsupported (nq = 0)
}

// Workspace: [pre: n_build+1 int64][partials: slices * slots * cells int32]
// [overflow: slices * slots * cells int64][quantised rows: n * 16 * cg bytes,
// with quant_rows only]
int64_t hist_ws_bytes(int64_t n, int32_t m, int32_t n_bins, int32_t k, int32_t n_build, bool quant_rows) {
  HistPlan p = hist_plan(m, n_bins, k, n_build, false);
  if (p.nq == 0) return -1;  // unsupported shape
  const HistPlan pt = hist_plan(m, n_bins, k, n_build, true);  // rows read straight from the data
  int64_t part = (int64_t)p.slices * p.slots * p.cells;
  if ((int64_t)pt.slices * pt.slots * pt.cells > part) part = (int64_t)pt.slices * pt.slots * pt.cells;
  const int64_t q = quant_rows ? align256(n * 16 * p.cg) : 0;
  return align256((int64_t)(n_build + 1) * 8) + align256(part * 4) + align256(part * 8) + q;
}

namespace {

// Escape value of an int32 partial: the cell's exact int64 sum is in the
// overflow slot of the same index.  INT32_MIN itself is escaped too.
constexpr int32_t PART_ESC = INT32_MIN;

__device__ inline bool fits_partial(int64_t v) { return v > (int64_t)INT32_MIN && v <= (int64_t)INT32_MAX; }

struct HistArgs {
  const uint32_t* bins4;
  int64_t ld4;
  const float* GH;
  int64_t ld_gh;
  const uint8_t* rec;
  int64_t ld_rec;
  const int32_t* qexp;
  const uint32_t* qrow;  // rotated kernel: quantised sketch rows, 4 * cg words per row
  const int32_t* row_idx;
  const int32_t* node_off;
  const int32_t* build_list;
  int64_t* pre;
  int32_t* part32;  // partials, one int32 per channel cell (PART_ESC: see ovf)
  int64_t* ovf;     // exact int64 partials of the escaped cells, same index
  double* H;
  const double* Hp;  // parent level, for the fused sibling subtraction (may be null)
  bool store_h;      // fused level end: write H (skipped at a tree's last level, whose H has no reader)
  int64_t n;
  int32_t m, n_bins, c, pairs, n_nodes, n_build;
  int32_t f, slices, cells, q, steps_per_window;
  int64_t slots;
  int32_t slices_full, f_thin, a_full, b_thin, q_thin, cg;  // rotated kernel plan (see HistPlan)
};

// Row groups of slice s (the thin slice has its own count).
__device__ inline int32_t groups_of(const HistArgs& a, int s) {
  return (a.f_thin && s >= a.slices_full) ? a.q_thin : a.q;
}

__device__ inline int32_t clamp_i32(int64_t v, int64_t lo, int64_t hi) {
  return (int32_t)(v < lo ? lo : (v > hi ? hi : v));
}

__device__ inline int32_t node_of(const HistArgs& a, int p) {
  const int32_t j = a.build_list ? a.build_list[p] : p;
  return j;
}

// Prefix of the built nodes' sizes (build-list order), one block.
__global__ void __launch_bounds__(1024) k_hist_plan(HistArgs a) {
  __shared__ int64_t part[1024];
  const int per = (a.n_build + 1023) / 1024;
  const int p0 = threadIdx.x * per;
  int64_t local = 0;
  for (int i = 0; i < per; ++i) {
    const int p = p0 + i;
    if (p < a.n_build) {
      const int32_t j = node_of(a, p);
      if (j >= 0 && j < a.n_nodes) {
        const int64_t s0 = clamp_i32(a.node_off[j], 0, a.n);
        const int64_t s1 = clamp_i32(a.node_off[j + 1], 0, a.n);
        local += s1 > s0 ? s1 - s0 : 0;
      }
    }
  }
  part[threadIdx.x] = local;
  __syncthreads();
  // Hillis-Steele inclusive scan of the 1024 per-thread totals
  for (int off = 1; off < 1024; off <<= 1) {
    int64_t v = threadIdx.x >= off ? part[threadIdx.x - off] : 0;
    __syncthreads();
    part[threadIdx.x] += v;
    __syncthreads();
  }
  int64_t run = threadIdx.x ? part[threadIdx.x - 1] : 0;
  for (int i = 0; i < per; ++i) {
    const int p = p0 + i;
    if (p < a.n_build) {
      a.pre[p] = run;
      const int32_t j = node_of(a, p);
      if (j >= 0 && j < a.n_nodes) {
        const int64_t s0 = clamp_i32(a.node_off[j], 0, a.n);
        const int64_t s1 = clamp_i32(a.node_off[j + 1], 0, a.n);
        run += s1 > s0 ? s1 - s0 : 0;
      }
    }
  }
  if (threadIdx.x == 1023) a.pre[a.n_build] = part[1023];
}

// Thread t owns the 64-bit cells j = t + NT * i, i < H: consecutive threads
// own consecutive cells, so the fold's 64-bit LDS reads are contiguous per
// wave.  Cell i of the thread carries its channel totals 2i (low half) and
// 2i+1 (high half).
//
// A cell holds S = Hi * 2^32 + Lo (mod 2^64), Hi and Lo the exact running
// channel sums, and the totals hold the sums as of the previous read, so
// the change D = S - (tot_hi * 2^32 + tot_lo) is dHi * 2^32 + dLo with
// |dLo|, |dHi| < 2^31: dLo is the sign-extended low word of D and dHi the
// arithmetic high word of D - dLo.
template <int H, int NT>
__device__ inline void fold_cells(const uint64_t* lds64, int64_t* tot) {
#pragma unroll
  for (int i0 = 0; i0 < H; i0 += 4) {
    asm volatile("" ::: "memory");
    uint64_t cur[4];
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) cur[ii] = (i0 + ii < H) ? lds64[threadIdx.x + NT * (i0 + ii)] : 0;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      if (i0 + ii < H) {
        const int i = 2 * (i0 + ii);
        const uint64_t last = ((uint64_t)tot[i + 1] << 32) + (uint64_t)tot[i];
        const uint64_t d = cur[ii] - last;
        const int64_t dlo = (int64_t)(int32_t)(uint32_t)d;
        const int64_t dhi = (int64_t)(d - (uint64_t)dlo) >> 32;
        tot[i] += dlo;
        tot[i + 1] += dhi;
      }
    }
  }
  asm volatile("" ::: "memory");
}

// Barrier for the window folds: waits for this wave's LDS operations only, so
// global prefetches stay in flight across it (a plain __syncthreads also
// drains them).  0xc07f is s_waitcnt lgkmcnt(0) in the gfx9 encoding.
__device__ inline void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A lane's position in a step: `raw` is the row index as loaded (not yet
// clamped, so that issuing the load never waits for it) and `on` says whether
// the position exists.
struct RowRef {
  int32_t raw;
  bool on;
};

// N consecutive words from a 4-byte aligned address, in 16- and 8-byte loads
// (the memory system accepts multi-dword loads at dword alignment).
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x2_a4 __attribute__((ext_vector_type(2), aligned(4)));
template <int N>
__device__ inline void load_run(const uint32_t* p, uint32_t* out) {
#pragma unroll
  for (int i = 0; i + 4 <= N; i += 4) {
    const u32x4_a4 v = *reinterpret_cast<const u32x4_a4*>(p + i);
    out[i] = v.x;
    out[i + 1] = v.y;
    out[i + 2] = v.z;
    out[i + 3] = v.w;
  }
  constexpr int R = N & 3;
  if constexpr (R >= 2) {
    const u32x2_a4 v = *reinterpret_cast<const u32x2_a4*>(p + (N - R));
    out[N - R] = v.x;
    out[N - R + 1] = v.y;
  }
  if constexpr (R & 1) out[N - 1] = p[N - 1];
}

// ---------------------------------------------------------------- rotated-feature order
// With one lane per row and the whole wave on one feature, a wave's 64
// 64-bit adds go to banks chosen by 64 random bins, and the collisions set
// the speed (about two thirds of the LDS cycles).  The rotated variant lets
// the feature choose the bank instead: a slice of ROT_F = 16 features keeps
// its cells as [bin][pair][feature], so one (bin, pair) row of 16 cells fills
// the 32 banks once and a cell's bank pair is its feature; at step i lane l
// adds its row's values for feature (i + l) mod 16.  Each step then puts
// exactly four lanes on every bank pair, whatever the bins.  Measured on
// MI355X with random bins: 6.5 clocks per wave instruction (19.75
// channel-adds/clk/CU), the rate of any 64-bit LDS write or atomic, against
// 13.9 clocks for the one-feature-per-wave order.  A lane rotates its row's
// 16 bin bytes once (by l mod 16), so that step i reads byte i.  Features
// past m come from padding bytes (the row records hold ld_rec >= m bytes,
// ld_rec % 16 == 0; the quad-major planes are clamped to the last one) and
// land in feature columns that the reduction never reads.

// Byte i of out = byte (i + r) mod 16 of the 16 bytes in w: whole words by
// r / 4 in two mask stages (bitfield inserts, so that the compiler keeps the
// words in registers instead of indexing a private array), then bytes by
// r mod 4 (v_alignbyte_b32 takes the 4 bytes at offset r mod 4 of the 8-byte
// pair {hi, lo}).
__device__ inline void rotate16(const uint32_t* w, int r, uint32_t* out) {
  const uint32_t m1 = 0u - (uint32_t)((r >> 2) & 1), m2 = 0u - (uint32_t)((r >> 3) & 1);
  const uint32_t sb = (uint32_t)(r & 3);
  uint32_t t[4], u[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) t[j] = (w[(j + 1) & 3] & m1) | (w[j] & ~m1);
#pragma unroll
  for (int j = 0; j < 4; ++j) u[j] = (t[(j + 2) & 3] & m2) | (t[j] & ~m2);
#pragma unroll
  for (int j = 0; j < 4; ++j) out[j] = __builtin_amdgcn_alignbyte(u[(j + 1) & 3], u[j], sb);
}

// A row of a rotated slice of FT features: the slice's bin bytes (FT of
// them, in NW words) and the row's quantised channel values (one 16-byte
// word of 21-bit fields).
template <int FT>
struct RowRot {
  static constexpr int NW = (FT + 3) / 4;
  uint32_t word[NW];
  uint32_t q[4];
};

typedef uint32_t u32x4_a16 __attribute__((ext_vector_type(4), aligned(16)));

// The lane's row for a rotated slice: its 16 bin bytes from features f0 ..
// f0+15 and its quantised values, all loads unconditional.  Row numbers are
// below 2^31, so the row arithmetic is 32-bit with one 64-bit multiply-add
// per record address.
template <int FT, bool FROM_REC>
__device__ inline void load_row_rot(const HistArgs& a, RowRef ref, int f0, const uint32_t* qbase, uint32_t qstride,
                                    RowRot<FT>& d) {
  constexpr int NW = RowRot<FT>::NW;
  const int32_t n1 = (int32_t)a.n - 1;
  int32_t row = ref.on ? ref.raw : 0;
  row = row < 0 ? 0 : (row > n1 ? n1 : row);
  const uint32_t ur = (uint32_t)row;
  {
    const u32x4_a16 v = *reinterpret_cast<const u32x4_a16*>(qbase + (uint64_t)ur * qstride);
    d.q[0] = v.x;
    d.q[1] = v.y;
    d.q[2] = v.z;
    d.q[3] = v.w;
  }
  if constexpr (FROM_REC) {
    // f0 is a multiple of 16 and ld_rec % 16 == 0: the slice's bytes are
    // 16-byte aligned (4- or 8-byte loads for a thin slice)
    load_run<NW>(reinterpret_cast<const uint32_t*>(a.rec + (uint64_t)ur * (uint32_t)a.ld_rec + f0), d.word);
  } else {
    const int last = ((a.m + 3) >> 2) - 1;
#pragma unroll
    for (int qq = 0; qq < NW; ++qq) {
      const int plane = (f0 >> 2) + qq < last ? (f0 >> 2) + qq : last;
      d.word[qq] = (a.bins4 + (int64_t)plane * a.ld4)[ur];
    }
  }
}

// Channel value t of a quantised row: the sign-extended 21-bit field t.
__device__ inline int32_t qfield(const uint32_t* q, int t) {
  const uint32_t lo = q[(t / 3) * 2], hi = q[(t / 3) * 2 + 1];
  const int f = t % 3;
  uint32_t x;
  if (f == 0) x = lo << 11;                                    // bits 0-20
  else if (f == 1) x = ((lo >> QFIELD_BITS) | (hi << 11)) << 11;  // bits 21-41
  else x = hi << 1;                                            // bits 42-62
  return (int32_t)x >> 11;
}

// Quantised sketch rows for the rotated kernel: channel t of row i becomes
// rint(GH[i, t] * 2^qexp[t]), the same fp32 operations that define the
// histogram's fixed point, packed into the 21-bit fields of one 16-byte word.
// With root_off given (a tree's first level), the first thread also writes
// the root's node offsets {0, n} and built-size prefix {0, n}.
template <int C>
__global__ void __launch_bounds__(256)
k_quant_rows(const float* __restrict__ GH, int64_t ld_gh, int64_t n, const int32_t* __restrict__ qexp,
             uint32_t* __restrict__ qrow, int32_t* root_off, int64_t* root_pre) {
  if (root_off && blockIdx.x == 0 && threadIdx.x == 0) {
    root_off[0] = 0;
    root_off[1] = (int32_t)n;
    root_pre[0] = 0;
    root_pre[1] = n;
  }
  int qe[C];
#pragma unroll
  for (int t = 0; t < C; ++t) qe[t] = __builtin_amdgcn_readfirstlane(qexp[t]);
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  uint32_t gw[C];
  load_run<C>(reinterpret_cast<const uint32_t*>(GH + i * ld_gh), gw);
  uint64_t half[2] = {0, 0};
  constexpr uint64_t M = (uint64_t(1) << QFIELD_BITS) - 1;
#pragma unroll
  for (int t = 0; t < C; ++t) {
    const int32_t v = (int32_t)rintf(ldexpf(__uint_as_float(gw[t]), qe[t]));
    half[t / 3] |= ((uint64_t)(uint32_t)v & M) << (QFIELD_BITS * (t % 3));
  }
  u32x4_a16 o;
  o.x = (uint32_t)half[0];
  o.y = (uint32_t)(half[0] >> 32);
  o.z = (uint32_t)half[1];
  o.w = (uint32_t)(half[1] >> 32);
  *reinterpret_cast<u32x4_a16*>(qrow + i * 4) = o;
}

// The same for 6 < c <= 6 CG channels: CG words per row, word g holding
// channels 6g .. 6g + 5 (zero past c).  The row's c values come in 16-byte
// loads (dword-aligned), the last partial group of four as single loads.
template <int CG>
__global__ void __launch_bounds__(256)
k_quant_rows_wide(const float* __restrict__ GH, int64_t ld_gh, int64_t n, int c, const int32_t* __restrict__ qexp,
                  uint32_t* __restrict__ qrow, int32_t* root_off, int64_t* root_pre) {
  constexpr int CM = QROW_MAX_C * CG;
  if (root_off && blockIdx.x == 0 && threadIdx.x == 0) {
    root_off[0] = 0;
    root_off[1] = (int32_t)n;
    root_pre[0] = 0;
    root_pre[1] = n;
  }
  int qe[CM];
#pragma unroll
  for (int t = 0; t < CM; ++t) qe[t] = t < c ? __builtin_amdgcn_readfirstlane(qexp[t]) : 0;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const uint32_t* p = reinterpret_cast<const uint32_t*>(GH + i * ld_gh);
  // the values come in fours, so the row buffer is a whole number of fours
  // (CM = 18 is not)
  constexpr int CW = (CM + 3) / 4 * 4;
  uint32_t w[CW];
#pragma unroll
  for (int j = 0; j < CW; j += 4) {
    if (j + 3 < c) {
      const u32x4_a4 v = *reinterpret_cast<const u32x4_a4*>(p + j);
      w[j] = v.x;
      w[j + 1] = v.y;
      w[j + 2] = v.z;
      w[j + 3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) w[j + e] = j + e < c ? p[j + e] : 0u;
    }
  }
  constexpr uint64_t M = (uint64_t(1) << QFIELD_BITS) - 1;
#pragma unroll
  for (int g = 0; g < CG; ++g) {
    uint64_t half[2] = {0, 0};
#pragma unroll
    for (int jj = 0; jj < QROW_MAX_C; ++jj) {
      const int t = QROW_MAX_C * g + jj;
      const int32_t v = t < c ? (int32_t)rintf(ldexpf(__uint_as_float(w[t]), qe[t])) : 0;
      half[jj / 3] |= ((uint64_t)(uint32_t)v & M) << (QFIELD_BITS * (jj % 3));
    }
    u32x4_a16 o;
    o.x = (uint32_t)half[0];
    o.y = (uint32_t)(half[0] >> 32);
    o.z = (uint32_t)half[1];
    o.w = (uint32_t)(half[1] >> 32);
    *reinterpret_cast<u32x4_a16*>(qrow + (i * CG + g) * 4) = o;
  }
}

typedef __attribute__((address_space(3))) unsigned long long lds_u64;

// Cell (bin, pair, slot) of a rotated slice is the 64-bit LDS word
// (bin * P + pair) * 16 + slot; offsets are 32-bit LDS byte offsets.  In a
// slice of 16 features the slot is the feature.  A thin slice of FT < 16
// features keeps R = 16 / FT copies: lane l adds into copy (l / FT) mod R,
// slot feature + FT * copy, and at step i handles feature (i + l) mod FT.
// Any 16 consecutive lanes then cover the 16 slots once, so every step puts
// four lanes on each bank pair, as in a full slice.
template <int C, int FT>
__device__ inline void add_row_rot(lds_u64* lds, const RowRot<FT>& d, uint32_t r, uint32_t slot0, uint32_t B) {
  constexpr int P = (C + 1) / 2;
  int32_t vq[2 * P];
#pragma unroll
  for (int t = 0; t < 2 * P; ++t) vq[t] = t < C ? qfield(d.q, t) : 0;
  uint64_t pk[P];
#pragma unroll
  for (int p = 0; p < P; ++p) pk[p] = ((uint64_t)(uint32_t)vq[2 * p + 1] << 32) + (uint64_t)(int64_t)vq[2 * p];
  // LDS byte address of cell (0, 0, 0); the cell addresses are formed as
  // 32-bit integers (the compiler otherwise keeps 64-bit pointer sums)
  const uint32_t base = (uint32_t)(size_t)lds;
  const int bmax = (int)((B - 1) & 0xffu);  // B <= 256: the 8-bit mask lets the products use 24-bit multiplies
  if constexpr (FT < ROT_F) {
#pragma unroll
    for (int i = 0; i < FT; ++i) {
      const uint32_t fi = (r + (uint32_t)i) & (FT - 1);  // this step's feature
      // the word is chosen by a bit mask (a select or a per-lane index into
      // d.word is turned into scratch-memory indexing by the compiler)
      const uint32_t sel = FT > 4 ? 0u - ((fi >> 2) & 1u) : 0u;
      const uint32_t w = d.word[0] ^ ((d.word[0] ^ d.word[RowRot<FT>::NW - 1]) & sel);
      int bin = (int)((w >> (8 * (fi & 3))) & 0xffu);
      bin = bin < bmax ? bin : bmax;
      const uint32_t addr = base + (uint32_t)bin * (uint32_t)(P * ROT_F * 8) + (slot0 + fi) * 8u;
#pragma unroll
      for (int p = 0; p < P; ++p)
        __hip_atomic_fetch_add((lds_u64*)(size_t)(addr + p * ROT_F * 8), (unsigned long long)pk[p], __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    return;
  }
  uint32_t rw[4];
  rotate16(d.word, (int)r, rw);
#pragma unroll
  for (int i = 0; i < ROT_F; ++i) {
    int bin = (int)((rw[i >> 2] >> (8 * (i & 3))) & 0xffu);
    bin = bin < bmax ? bin : bmax;
    const uint32_t addr = base + (uint32_t)bin * (uint32_t)(P * ROT_F * 8) + ((r + (uint32_t)i) & (ROT_F - 1)) * 8u;
#pragma unroll
    for (int p = 0; p < P; ++p)
      __hip_atomic_fetch_add((lds_u64*)(size_t)(addr + p * ROT_F * 8), (unsigned long long)pk[p], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_WORKGROUP);
  }
}

// Accumulate the lane's rows of virtual positions [v, vend) of one node
// (segment start seg0, first virtual position pstart) into the LDS cells of
// a rotated slice, folding into `tot` at every window.  HAS_IDX: rows come
// through row_idx and are read from their records (otherwise the position is
// the row of the contiguous data).  Positions are 32-bit (every position and
// row is below 2^31, so unsigned 32-bit sums of them do not wrap).  The
// row-index load of a lane is unconditional (positions past the end are
// clamped into the segment and marked off), so the load path has no
// branches.  The next step's row is loaded before the current one is added,
// so its memory latency hides behind the current step's LDS work; the
// prefetched row stays in flight across the window folds.
template <int C, int FT, bool HAS_IDX>
__device__ inline void run_segment_rot(const HistArgs& a, lds_u64* lds, int64_t* tot, uint32_t v,
                                       uint32_t vend, uint32_t pstart, uint32_t seg0, int wave, int lane, int f0,
                                       uint32_t B, int grp) {
  // this workgroup's word of each quantised row (channel group grp)
  const uint32_t* qbase = a.qrow + 4 * grp;
  const uint32_t qstride = 4u * (uint32_t)a.cg;
  constexpr uint32_t rows_step = ROT_THREADS;
  const uint32_t last_pos = seg0 + (vend - 1 - pstart);
  const uint32_t lane_off = (uint32_t)(wave * 64 + lane);
  const uint32_t r = (uint32_t)lane & (FT - 1);
  const uint32_t slot0 = FT < ROT_F ? (((uint32_t)lane / FT) & (ROT_F / FT - 1)) * FT : 0u;
  auto row_at = [&](uint32_t vs) -> RowRef {
    const uint32_t vv = vs + lane_off;
    RowRef rr;
    rr.on = vv < vend;
    uint32_t pos = seg0 + (vv - pstart);
    pos = pos < last_pos ? pos : last_pos;
    rr.raw = HAS_IDX ? a.row_idx[pos] : (int32_t)pos;
    return rr;
  };
  RowRef r0 = row_at(v);
  RowRef r1 = row_at(v + rows_step);
  RowRot<FT> d0, d1;
  load_row_rot<FT, HAS_IDX>(a, r0, f0, qbase, qstride, d0);
  int steps = 0;
#pragma unroll 1
  for (uint32_t vs = v; vs < vend; vs += rows_step) {
    const RowRef r2 = row_at(vs + 2 * rows_step);
    load_row_rot<FT, HAS_IDX>(a, r1, f0, qbase, qstride, d1);
    if (r0.on) add_row_rot<C, FT>(lds, d0, r, slot0, B);
    r0 = r1;
    d0 = d1;
    r1 = r2;
    if (++steps == a.steps_per_window) {
      steps = 0;
      lds_barrier();
      fold_cells<ROT_CPT, ROT_THREADS>((const uint64_t*)lds, tot);
    }
  }
}

// One workgroup's share of a level: the slice's cells in [bin][pair][slot]
// order, thread t owning the 64-bit cells t + ROT_THREADS * i, i < ROT_CPT.
// At the end of a node's part the totals go out through LDS, one pair at a
// time, as partials laid out [pair][feature][bin] (16-byte channel pairs).
// Slice s of FT features (16, or a thin slice's f_thin), row group q of
// qn: the rows of virtual positions [q T / qn, (q+1) T / qn).
template <int C, int FT>
__device__ __forceinline__ void hist_rot_group(const HistArgs& a, uint64_t* lds64, int s, int grp, int q, int qn) {
  constexpr int P = (C + 1) / 2;
  constexpr int R = ROT_F / FT;  // copies of each cell in the slice
  const int64_t T = a.pre[a.n_build];
  const int64_t v0 = (int64_t)q * T / qn;
  const int64_t v1 = (int64_t)(q + 1) * T / qn;
  if (v0 >= v1) return;

  int lo = 0, hi = a.n_build;  // pre[lo] <= v0 < pre[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.pre[mid] <= v0) lo = mid;
    else hi = mid;
  }
  int p = lo;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int f0 = s * ROT_F;
  const int B = a.n_bins;

  int64_t tot[2 * ROT_CPT];
#pragma unroll
  for (int jj = 0; jj < 2 * ROT_CPT; ++jj) tot[jj] = 0;
#pragma unroll
  for (int i = 0; i < ROT_CPT; ++i) lds64[tid + ROT_THREADS * i] = 0;
  __syncthreads();

  longlong2* stage = reinterpret_cast<longlong2*>(lds64);  // [slot][B + 1] channel pairs
  int64_t v = v0;
  while (v < v1) {
    const int32_t j = node_of(a, p);
    const int64_t pstart = a.pre[p];
    const int64_t vend = v1 < a.pre[p + 1] ? v1 : a.pre[p + 1];
    const int64_t seg0 = clamp_i32(a.node_off[j], 0, a.n);
    lds_u64* L = (lds_u64*)lds64;  // generic to LDS address space: 32-bit offsets
    if (a.row_idx)
      run_segment_rot<C, FT, true>(a, L, tot, (uint32_t)v, (uint32_t)vend, (uint32_t)pstart, (uint32_t)seg0, wave,
                                   lane, f0, (uint32_t)B, grp);
    else
      run_segment_rot<C, FT, false>(a, L, tot, (uint32_t)v, (uint32_t)vend, (uint32_t)pstart, (uint32_t)seg0,
                                    wave, lane, f0, (uint32_t)B, grp);
    // The node-end barriers wait for LDS operations only: the partial stores
    // take their data from registers, so nothing here waits for them.
    lds_barrier();
    fold_cells<ROT_CPT, ROT_THREADS>(lds64, tot);
    lds_barrier();  // every fold read is done: the LDS becomes the staging area
    const int64_t slot = ((int64_t)s * a.slots + q + p) * a.cells;  // channel cells
    int2* dst = reinterpret_cast<int2*>(a.part32 + slot);
    longlong2* dov = reinterpret_cast<longlong2*>(a.ovf + slot);
    // this channel group's pairs are pairs 3 grp .. 3 grp + P - 1 of the
    // slot; pairs past the last (a short final group) are not written
#pragma unroll 1
    for (int pr = 0; pr < P && ROT_PMAX * grp + pr < a.pairs; ++pr) {
#pragma unroll
      for (int i = 0; i < ROT_CPT; ++i) {
        const int j64 = tid + ROT_THREADS * i;
        const int row = j64 >> 4, bin = row / P, fl = j64 & (ROT_F - 1);
        if (row - bin * P == pr && bin < B) stage[fl * (B + 1) + bin] = make_longlong2(tot[2 * i], tot[2 * i + 1]);
      }
      lds_barrier();
      // features 0 .. FT-1 of the slice; a thin slice adds its R copies
      for (int e = tid; e < FT * B; e += ROT_THREADS) {
        const int fl = e / B, bin = e - fl * B;
        longlong2 x = stage[fl * (B + 1) + bin];
#pragma unroll
        for (int rc = 1; rc < R; ++rc) {
          const longlong2 y = stage[(fl + FT * rc) * (B + 1) + bin];
          x.x += y.x;
          x.y += y.y;
        }
        const int64_t at = (int64_t)(ROT_PMAX * grp + pr) * ROT_F * B + e;
        const bool fx = fits_partial(x.x), fy = fits_partial(x.y);
        dst[at] = make_int2(fx ? (int32_t)x.x : PART_ESC, fy ? (int32_t)x.y : PART_ESC);
        if (!(fx && fy)) dov[at] = x;
      }
      lds_barrier();
    }
#pragma unroll
    for (int i = 0; i < ROT_CPT; ++i) {
      lds64[tid + ROT_THREADS * i] = 0;
      tot[2 * i] = 0;
      tot[2 * i + 1] = 0;
    }
    lds_barrier();
    v = vend;
    ++p;
    while (p < a.n_build && a.pre[p + 1] <= v) ++p;
  }
}

// The histogram kernel.  Workgroup b runs on XCD b % 8; on each XCD the
// first a_full * slices_full * cg workgroups take the (full slice, channel
// group) pairs of a_full row groups (so the slices of a row group share the
// XCD's L2) and the next b_thin * cg the thin slice.
template <int C>
__global__ void __launch_bounds__(ROT_THREADS)
k_hist_rot(HistArgs a) {
  extern __shared__ uint64_t lds64[];
  const int b = blockIdx.x;
  const int xcd = b & 7, g = b >> 3;
  const int uf = a.slices_full * a.cg;  // workgroups per full row group: (slice, channel group)
  const int nfull = a.a_full * uf;
  if (g < nfull) {
    const int q = (g / uf) * 8 + xcd;
    const int u = g % uf;
    if (q < a.q) hist_rot_group<C, ROT_F>(a, lds64, u / a.cg, u % a.cg, q, a.q);
    return;
  }
  const int t = g - nfull;
  const int q = (t / a.cg) * 8 + xcd, grp = t % a.cg;
  if (!a.f_thin || q >= a.q_thin) return;
  const int s = a.slices_full;
  switch (a.f_thin) {
    case 1: hist_rot_group<C, 1>(a, lds64, s, grp, q, a.q_thin); break;
    case 2: hist_rot_group<C, 2>(a, lds64, s, grp, q, a.q_thin); break;
    case 4: hist_rot_group<C, 4>(a, lds64, s, grp, q, a.q_thin); break;
    default: hist_rot_group<C, 8>(a, lds64, s, grp, q, a.q_thin); break;
  }
}

__device__ inline int64_t group_of(int64_t x, int64_t T, int64_t Q) { return ((x + 1) * Q - 1) / T; }

// H[node][f][t][b] = sum of the partials of the row groups that covered the
// node.  Partial channel cell e = 2 * e64 + half, with 64-bit LDS cell e64
// laid out [channel pair][feature in slice][bin] and t = 2 * pair + half.
// With the parent level given (Hp), the built node j of pair p also yields
// its sibling: H[j ^ 1] = Hp[p] - H[j], exact in fixed point.
__global__ void __launch_bounds__(256) k_hist_reduce(HistArgs a) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int p = blockIdx.y, s = blockIdx.z;
  if (e >= a.cells) return;
  const int32_t j = node_of(a, p);
  if (j < 0 || j >= a.n_nodes) return;
  const int FB = a.f * a.n_bins;
  const int e64 = e >> 1;
  const int pair = e64 / FB;
  const int rem = e64 - pair * FB;
  const int fl = rem / a.n_bins;
  const int bin = rem - fl * a.n_bins;
  const int t = 2 * pair + (e & 1);
  const int f = s * a.f + fl;
  if (f >= a.m || t >= a.c) return;
  const int64_t T = a.pre[a.n_build];
  const int64_t lo = a.pre[p], hi = a.pre[p + 1];
  int64_t sum = 0;
  if (hi > lo) {
    const int32_t qn = groups_of(a, s);
    const int64_t qlo = group_of(lo, T, qn), qhi = group_of(hi - 1, T, qn);
    const int64_t base = ((int64_t)s * a.slots + p) * a.cells + e;
    const int32_t* src = a.part32 + base;
    const int64_t* ov = a.ovf + base;
    const bool dense = T >= qn;  // every row group holds at least one position
    auto live = [&](int64_t q) { return q <= qhi && (dense || q * T / qn < (q + 1) * T / qn); };
    // batches of eight row groups, loads unconditional (clamped to the last
    // group, dropped past it); escapes are flagged, and a thread that met one
    // sums again with the overflow slots
    bool esc = false;
    for (int64_t q = qlo; q <= qhi; q += 8) {
      int32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[(q + u <= qhi ? q + u : qhi) * a.cells];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool use = live(q + u);
        sum += use ? v[u] : 0;
        esc |= use && v[u] == PART_ESC;
      }
    }
    if (esc) {
      sum = 0;
      for (int64_t q = qlo; q <= qhi; ++q)
        if (live(q)) {
          const int32_t x = src[q * a.cells];
          sum += x == PART_ESC ? ov[q * a.cells] : (int64_t)x;
        }
    }
  }
  const int64_t cpn = (int64_t)a.m * a.c * a.n_bins;
  const int64_t idx = ((int64_t)f * a.c + t) * a.n_bins + bin;
  const double v = ldexp((double)sum, -a.qexp[t]);
  a.H[(int64_t)j * cpn + idx] = v;
  if (a.Hp && (j == 2 * p || j == 2 * p + 1)) a.H[(int64_t)(j ^ 1) * cpn + idx] = a.Hp[(int64_t)p * cpn + idx] - v;
}

__global__ void __launch_bounds__(256)
k_subtract(const double* __restrict__ Hp, double* __restrict__ Hc, int64_t cpn, const int32_t* __restrict__ build) {
  const int p = blockIdx.y;
  const int32_t c = build[p];
  if (c != 2 * p && c != 2 * p + 1) return;
  const int32_t sib = c ^ 1;
  const double* src = Hp + (int64_t)p * cpn;
  const double* built = Hc + (int64_t)c * cpn;
  double* dst = Hc + (int64_t)sib * cpn;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < cpn; i += (int64_t)gridDim.x * 256)
    dst[i] = src[i] - built[i];
}

// A double moved across lanes by a DPP control (row shift or row broadcast),
// both 32-bit halves alike; lanes the control does not write get 0.
template <int CTRL, int ROW_MASK>
__device__ inline double dpp_move(double x) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, ROW_MASK, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, ROW_MASK, 0xf, false);
  return __hiloint2double(hi, lo);
}

// Inclusive prefix sum over the 64 lanes of a wave (all lanes active), in
// registers: shifts by 1, 2, 4 and 8 lanes inside each row of 16, then the
// last lane of rows 0 and 2 is added to rows 1 and 3 (row_bcast:15) and
// lane 31 to rows 2 and 3 (row_bcast:31).
__device__ inline double wave_inclusive_scan(double x) {
  x += dpp_move<0x111, 0xf>(x);
  x += dpp_move<0x112, 0xf>(x);
  x += dpp_move<0x114, 0xf>(x);
  x += dpp_move<0x118, 0xf>(x);
  x += dpp_move<0x142, 0xa>(x);
  x += dpp_move<0x143, 0xc>(x);
  return x;
}

__device__ inline bool score_better(double sa, int ia, double sb_, int ib) {
  return sa > sb_ || (sa == sb_ && ia < ib);
}

// Fused end of a level (the level loop's path): one block per (feature f,
// built node p), one thread per bin.  The block sums feature f's int32
// partials of node p (with the int64 overflow slots where a sum escaped),
// writes the fp64 histogram of the built node j (and, with the parent level
// given, of its sibling by exact subtraction), then scores every threshold
// of f for both nodes as k_score_feature does (Section 2, eq. 4: prefix sums
// over bins, fp64, ties to the lower bin) and writes the best (score, bin)
// per (node, feature) for the node argmax (in the partition's first kernel,
// or k_score_node).
struct ScoreOut {
  double* s;
  int32_t* b;
  double lam, mcw;
};

// RQ threads per bin: each sums its share of the node's row groups, and the
// shares meet in LDS (integers, so the order does not matter).  The first
// 256 threads then carry the bin through the rest.  RQ = 4 where a node
// spans many row groups (the first levels), else 1.  The scan over bins runs
// in registers (DPP inside each wave, wave totals through LDS), so a block
// holds under 1 KB of LDS past the quarters' sums and the deep levels, with
// thousands of blocks, are limited by registers: 4 to 6 blocks per CU.
template <int PMAX, int RQ>
__global__ void __launch_bounds__(256 * RQ) k_hist_reduce_score(HistArgs a, ScoreOut so) {
  const int f = blockIdx.x, p = blockIdx.y;
  const int32_t j = node_of(a, p);
  if (j < 0 || j >= a.n_nodes || f >= a.m) return;
  const int B = a.n_bins, c = a.c, k = c - 1;
  const int s = f / a.f, fl = f - s * a.f;
  const int FB = a.f * B;
  const int bin = threadIdx.x & 255, quarter = threadIdx.x >> 8;
  const bool on = bin < B;
  const bool sib = a.Hp && (j == 2 * p || j == 2 * p + 1);
  const int64_t cpn = (int64_t)a.m * c * B;
  const int64_t T = a.pre[a.n_build];
  const int64_t lo = a.pre[p], hi = a.pre[p + 1];
  const int32_t qn = groups_of(a, s);
  const int64_t nlo = hi > lo ? group_of(lo, T, qn) : 0, nhi = hi > lo ? group_of(hi - 1, T, qn) : -1;
  // this thread's quarter of the node's row groups [nlo, nhi]
  const int64_t per = (nhi - nlo + RQ) / RQ;
  const int64_t qlo = nlo + quarter * per;
  const int64_t qhi = (qlo + per - 1 < nhi) ? qlo + per - 1 : nhi;
  const bool dense = T >= qn;  // every row group holds at least one position
  // The parent's values for the sibling, loaded first so that this read and
  // the partials' are in flight together (a block reads them once each).
  double hp[2 * PMAX];
#pragma unroll
  for (int t = 0; t < 2 * PMAX; ++t) {
    hp[t] = 0.0;
    if (sib && t < c && on && quarter == 0) hp[t] = a.Hp[(int64_t)p * cpn + ((int64_t)f * c + t) * B + bin];
  }
  // int64 channel sums of this bin over the node's row groups, from the
  // int32 partials.  Fast path: batches of BQ row groups and every channel
  // pair, loads unconditional (groups past the node's last and pairs past
  // the last repeat it; the extra values are dropped), no branch on the
  // values: escapes are only flagged.  A lane that met an escape sums its
  // bin again with the overflow slots (rare: a workgroup's sum of one bin
  // must pass 2^31).
  int64_t acc_lo[PMAX], acc_hi[PMAX];
#pragma unroll
  for (int pr = 0; pr < PMAX; ++pr) acc_lo[pr] = acc_hi[pr] = 0;
  if (on && qlo <= qhi) {
    const int64_t e64 = (int64_t)fl * B + bin;
    const int64_t base = ((int64_t)s * a.slots + p) * a.cells;
    const int2* src = reinterpret_cast<const int2*>(a.part32 + base) + e64;
    const longlong2* ov = reinterpret_cast<const longlong2*>(a.ovf + base) + e64;
    const int64_t stride = a.cells / 2;  // one row group, in channel pairs
    auto live = [&](int64_t q) { return q <= qhi && (dense || q * T / qn < (q + 1) * T / qn); };
    bool esc = false;
    if (dense) {
      constexpr int BQ = PMAX <= 4 ? 4 : 2;
      auto load = [&](int64_t q0, int2 (&v)[BQ][PMAX]) {
#pragma unroll
        for (int u = 0; u < BQ; ++u)
#pragma unroll
          for (int pr = 0; pr < PMAX; ++pr)
            v[u][pr] = src[(q0 + u <= qhi ? q0 + u : qhi) * stride + (int64_t)(pr < a.pairs ? pr : a.pairs - 1) * FB];
      };
      auto add = [&](int64_t q0, const int2 (&v)[BQ][PMAX]) {
#pragma unroll
        for (int u = 0; u < BQ; ++u)
#pragma unroll
          for (int pr = 0; pr < PMAX; ++pr) {
            const bool use = q0 + u <= qhi && pr < a.pairs;
            const int2 x = v[u][pr];
            acc_lo[pr] += use ? x.x : 0;
            acc_hi[pr] += use ? x.y : 0;
            esc |= use && (x.x == PART_ESC || x.y == PART_ESC);
          }
      };
      for (int64_t q = qlo; q <= qhi; q += BQ) {
        int2 vq[BQ][PMAX];
        load(q, vq);
        add(q, vq);
      }
    } else {
      // fewer positions than row groups (tiny levels): empty groups wrote nothing
      for (int64_t q = qlo; q <= qhi; ++q) {
        if (!live(q)) continue;
#pragma unroll
        for (int pr = 0; pr < PMAX; ++pr) {
          if (pr >= a.pairs) continue;
          const int2 x = src[q * stride + (int64_t)pr * FB];
          acc_lo[pr] += x.x;
          acc_hi[pr] += x.y;
          esc |= x.x == PART_ESC || x.y == PART_ESC;
        }
      }
    }
    if (esc) {
#pragma unroll
      for (int pr = 0; pr < PMAX; ++pr) acc_lo[pr] = acc_hi[pr] = 0;
      for (int64_t q = qlo; q <= qhi; ++q) {
        if (!live(q)) continue;
        for (int pr = 0; pr < PMAX && pr < a.pairs; ++pr) {
          const int2 x = src[q * stride + (int64_t)pr * FB];
          if (x.x == PART_ESC || x.y == PART_ESC) {
            const longlong2 o = ov[q * stride + (int64_t)pr * FB];
            acc_lo[pr] += o.x;
            acc_hi[pr] += o.y;
          } else {
            acc_lo[pr] += x.x;
            acc_hi[pr] += x.y;
          }
        }
      }
    }
  }
  // the quarters meet: quarters 1..3 leave their sums in LDS, quarter 0
  // adds them
  extern __shared__ longlong2 part[];  // [quarter - 1][pair][256]
  if (RQ > 1 && quarter > 0) {
#pragma unroll
    for (int pr = 0; pr < PMAX; ++pr) part[((quarter - 1) * PMAX + pr) * 256 + bin] = make_longlong2(acc_lo[pr], acc_hi[pr]);
  }
  if (RQ > 1) __syncthreads();
  if (RQ > 1 && quarter == 0) {
#pragma unroll
    for (int qq = 0; qq < RQ - 1; ++qq)
#pragma unroll
      for (int pr = 0; pr < PMAX; ++pr) {
        const longlong2 v = part[(qq * PMAX + pr) * 256 + bin];
        acc_lo[pr] += v.x;
        acc_hi[pr] += v.y;
      }
  }
  // fp64 histogram values of this bin, v[0] of the built node j and v[1] of
  // its sibling (by subtraction), written to H and kept in registers for the
  // scan: the bins are the block's first 256 threads, so the prefix over
  // bins is a prefix over lanes, then over the block's first waves
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nw = (B + 63) >> 6;  // waves that hold bins
  const bool scan_wave = quarter == 0 && wave < nw;
  double v[2][2 * PMAX];
#pragma unroll
  for (int t = 0; t < 2 * PMAX; ++t) {
    v[0][t] = v[1][t] = 0.0;
    if (t < c && on && quarter == 0) {
      const int64_t idx = ((int64_t)f * c + t) * B + bin;
      const double x = ldexp((double)((t & 1) ? acc_hi[t >> 1] : acc_lo[t >> 1]), -a.qexp[t]);
      if (a.store_h) a.H[(int64_t)j * cpn + idx] = x;
      v[0][t] = x;
      if (sib) {
        const double xs = hp[t] - x;
        if (a.store_h) a.H[(int64_t)(j ^ 1) * cpn + idx] = xs;
        v[1][t] = xs;
      }
    }
  }
  // Every value is a multiple of 2^-qexp below 2^53 of those units in
  // magnitude (a node's channel sum is at most 2^31 rows of 2^QBITS), so
  // fp64 sums of them are exact and any order of the scan gives the same
  // bits.  Wave totals meet in LDS as [node][channel][wave].
  __shared__ double wtot[2][2 * PMAX][4];
  __shared__ double wbest_s[2][4];
  __shared__ int32_t wbest_b[2][4];
  const int nodes = sib ? 2 : 1;
  if (scan_wave) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < 2 * PMAX; ++t)
        if (u < nodes && t < c) {
          v[u][t] = wave_inclusive_scan(v[u][t]);
          if (lane == 63) wtot[u][t][wave] = v[u][t];
        }
  } else if (quarter == 0 && lane == 0) {
    // a wave past the last bin adds nothing
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < 2 * PMAX; ++t) wtot[u][t][wave] = 0.0;
  }
  __syncthreads();
  if (scan_wave) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (u < nodes) {
        // Section 2, eq. 4 for every threshold b (left: bins <= b): gradient
        // channels t < k add L^2 and R^2, the last channel is the hessian
        double sl = 0.0, sr = 0.0, HL = 0.0, HR = 0.0;
#pragma unroll
        for (int t = 0; t < 2 * PMAX; ++t) {
          if (t < c) {
            double before = 0.0, tot = 0.0;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const double x = wtot[u][t][w];
              tot += x;
              before += w < wave ? x : 0.0;
            }
            const double L = v[u][t] + before, R = tot - L;
            if (t < k) {
              sl += L * L;
              sr += R * R;
            } else {
              HL = L;
              HR = R;
            }
          }
        }
        double best_s = -INFINITY;
        int best_b = -1;
        if (on && bin <= B - 2 && HL > so.mcw && HR > so.mcw) {
          best_s = sl / (HL + so.lam) + sr / (HR + so.lam);
          best_b = bin;
        }
        wave_best_si(best_s, best_b);  // in lane 63, the reduction in registers
        if (lane == 63) {
          wbest_s[u][wave] = best_s;
          wbest_b[u][wave] = best_b;
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x < nodes) {
    const int u = threadIdx.x;
    double best_s = -INFINITY;
    int best_b = -1;
    for (int w = 0; w < nw; ++w) {
      const double os = wbest_s[u][w];
      const int ob = wbest_b[u][w];
      if (ob >= 0 && (best_b < 0 || score_better(os, ob, best_s, best_b))) {
        best_s = os;
        best_b = ob;
      }
    }
    const int32_t nd = u ? (j ^ 1) : j;
    so.s[(int64_t)nd * a.m + f] = best_s;
    so.b[(int64_t)nd * a.m + f] = best_b;
  }
}

}  // namespace

int32_t launch_build_histograms(const uint32_t* bins4, int64_t ld4, const uint8_t* rec, int64_t ld_rec, int64_t n,
                                int32_t m, int32_t n_bins, const float* GH, int64_t ld_gh, int32_t k,
                                const int32_t* qexp,
                                const int32_t* row_idx, const int32_t* node_off, int32_t n_nodes,
                                const int32_t* build_list, int32_t n_build, double* H, void* ws, hipStream_t st,
                                const int64_t* pre_given, const double* H_parent, double* feat_s, int32_t* feat_b,
                                double lam, double mcw, uint32_t* qrow, bool qrow_ready, bool store_h,
                                int32_t* root_off) {
  const HistPlan pl = hist_plan(m, n_bins, k, n_build, row_idx == nullptr);
  if (pl.nq == 0) return fail(SB_E_UNSUPPORTED, "sb_build_histograms: at most 24 channels (k <= 23) and 256 bins");
  HistArgs a{};
  a.bins4 = bins4;
  a.ld4 = ld4;
  a.rec = rec;
  a.ld_rec = ld_rec;
  a.GH = GH;
  a.ld_gh = ld_gh;
  a.qexp = qexp;
  a.row_idx = row_idx;
  a.node_off = node_off;
  a.build_list = build_list;
  char* w = static_cast<char*>(ws);
  a.pre = pre_given ? const_cast<int64_t*>(pre_given) : reinterpret_cast<int64_t*>(w);
  {
    const HistPlan pt = hist_plan(m, n_bins, k, n_build, true);
    int64_t part = (int64_t)pl.slices * pl.slots * pl.cells;
    if ((int64_t)pt.slices * pt.slots * pt.cells > part) part = (int64_t)pt.slices * pt.slots * pt.cells;
    char* p0 = w + align256((int64_t)(n_build + 1) * 8);
    a.part32 = reinterpret_cast<int32_t*>(p0);
    a.ovf = reinterpret_cast<int64_t*>(p0 + align256(part * 4));
  }
  // the quantised rows live in the caller's buffer (kept across a tree's
  // levels) or else at the end of this call's workspace
  if (!qrow) qrow = reinterpret_cast<uint32_t*>(w + hist_ws_bytes(n, m, n_bins, k, n_build, false));
  a.qrow = qrow;
  if (!qrow_ready) {
    const unsigned qb = (unsigned)((n + 255) / 256);
    int64_t* rp = const_cast<int64_t*>(pre_given);
    switch (pl.c) {
      case 1: hipLaunchKernelGGL(k_quant_rows<1>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, qexp, qrow, root_off, rp); break;
      case 2: hipLaunchKernelGGL(k_quant_rows<2>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, qexp, qrow, root_off, rp); break;
      case 3: hipLaunchKernelGGL(k_quant_rows<3>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, qexp, qrow, root_off, rp); break;
      case 4: hipLaunchKernelGGL(k_quant_rows<4>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, qexp, qrow, root_off, rp); break;
      case 5: hipLaunchKernelGGL(k_quant_rows<5>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, qexp, qrow, root_off, rp); break;
      case 6: hipLaunchKernelGGL(k_quant_rows<6>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, qexp, qrow, root_off, rp); break;
      default:
        if (pl.cg == 2)
          hipLaunchKernelGGL(k_quant_rows_wide<2>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, pl.c, qexp, qrow, root_off, rp);
        else if (pl.cg == 3)
          hipLaunchKernelGGL(k_quant_rows_wide<3>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, pl.c, qexp, qrow, root_off, rp);
        else
          hipLaunchKernelGGL(k_quant_rows_wide<4>, dim3(qb), dim3(256), 0, st, GH, ld_gh, n, pl.c, qexp, qrow, root_off, rp);
        break;
    }
  }
  a.H = H;
  a.Hp = H_parent;
  a.store_h = store_h;
  a.n = n;
  a.m = m;
  a.n_bins = n_bins;
  a.c = pl.c;
  a.pairs = pl.pairs;
  a.n_nodes = n_nodes;
  a.n_build = n_build;
  a.f = pl.f;
  a.slices = pl.slices;
  a.cells = pl.cells;
  a.q = pl.q;
  a.slices_full = pl.slices_full;
  a.f_thin = pl.f_thin;
  a.a_full = pl.a_full;
  a.b_thin = pl.b_thin;
  a.q_thin = pl.q_thin;
  a.cg = pl.cg;
  a.steps_per_window = WINDOW_ROWS / ROT_THREADS;
  a.slots = pl.slots;

  if (!pre_given) hipLaunchKernelGGL(k_hist_plan, dim3(1), dim3(1024), 0, st, a);
  const int grid = pl.grid;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  const bool prof = profile_on() && hipEventCreate(&e0) == hipSuccess && hipEventCreate(&e1) == hipSuccess;
  if (prof) (void)hipEventRecord(e0, st);
  const size_t lds_bytes = (size_t)ROT_CELLS * 8;
  // up to six channels: one workgroup per (slice, row group); more: channel
  // groups of six (three pairs) each, one workgroup per (slice, group)
  switch (pl.c) {
    case 1: hipLaunchKernelGGL(k_hist_rot<1>, dim3(grid), dim3(ROT_THREADS), lds_bytes, st, a); break;
    case 2: hipLaunchKernelGGL(k_hist_rot<2>, dim3(grid), dim3(ROT_THREADS), lds_bytes, st, a); break;
    case 3: hipLaunchKernelGGL(k_hist_rot<3>, dim3(grid), dim3(ROT_THREADS), lds_bytes, st, a); break;
    case 4: hipLaunchKernelGGL(k_hist_rot<4>, dim3(grid), dim3(ROT_THREADS), lds_bytes, st, a); break;
    case 5: hipLaunchKernelGGL(k_hist_rot<5>, dim3(grid), dim3(ROT_THREADS), lds_bytes, st, a); break;
    default: hipLaunchKernelGGL(k_hist_rot<QROW_MAX_C>, dim3(grid), dim3(ROT_THREADS), lds_bytes, st, a); break;
  }
  if (prof) {
    (void)hipEventRecord(e1, st);
    profile_record(e0, e1);
  }
  if (feat_s) {
    ScoreOut so{feat_s, feat_b, lam, mcw};
    const dim3 g(m, n_build);
    // dynamic LDS: the partial sums of quarters 1..3 ([quarter][pair][256])
    const int pm = pl.pairs <= 3 ? 3 : pl.pairs <= 4 ? 4 : pl.pairs <= 6 ? 6 : pl.pairs <= 8 ? 8 : 12;
    // four threads per bin where a node spans about q / n_build >= 12 row
    // groups; not at 12 pairs, where the 1024-thread block would spill
    const bool wide = pl.q >= 12 * n_build && pm < 12;
    const int rq = wide ? 4 : 1;
    const size_t lds = (size_t)(rq - 1) * pm * 256 * 16;
#define SB_RS(P, R) hipLaunchKernelGGL((k_hist_reduce_score<P, R>), g, dim3(256 * R), lds, st, a, so)
    if (pm == 3) { if (wide) SB_RS(3, 4); else SB_RS(3, 1); }
    else if (pm == 4) { if (wide) SB_RS(4, 4); else SB_RS(4, 1); }
    else if (pm == 6) { if (wide) SB_RS(6, 4); else SB_RS(6, 1); }
    else if (pm == 8) { if (wide) SB_RS(8, 4); else SB_RS(8, 1); }
    else if (pl.pairs <= 12) SB_RS(12, 1);
#undef SB_RS
    else return fail(SB_E_UNSUPPORTED, "sb_grow_tree: the fused histogram scoring takes at most 24 channels");
  } else {
    dim3 rg((pl.cells + 255) / 256, n_build, pl.slices);
    hipLaunchKernelGGL(k_hist_reduce, rg, dim3(256), 0, st, a);
  }
  return check_launch("sb_build_histograms");
}

int32_t launch_subtract(const double* Hp, double* Hc, int32_t n_parents, int64_t cells_per_node,
                        const int32_t* build_list, hipStream_t st) {
  int64_t bx = (cells_per_node + 255) / 256;
  if (bx > 1024) bx = 1024;
  hipLaunchKernelGGL(k_subtract, dim3((unsigned)bx, n_parents), dim3(256), 0, st, Hp, Hc, cells_per_node,
                     build_list);
  return check_launch("sb_subtract_histograms");
}

}  // namespace sb
