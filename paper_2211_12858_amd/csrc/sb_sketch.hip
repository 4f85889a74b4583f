// Gradient sketches of Section 3 on gfx950.
//
//   k_colnorm_partial / k_colnorm_final : ||g_j||^2 in fp64, fixed reduction
//       order (Section 3.1 ranks columns by norm; Section 3.2 samples with
//       p_j proportional to it).
//   k_select   : Top Outputs ranks, Random Sampling inverse-CDF draws from
//       given uniforms, identity.
//   k_pack     : GH[i, t] = fp32(G[i, col_t] * scale_t), GH[i, k] = h_i
//       (row-major, rows written whole), plus per-block maxima of |value|
//       for the fixed-point histogram exponents.
//   k_project  : GH[i, 0:k] = (G Pi)[i, :] (Section 3.3), fp32 accumulation.
//   k_project_sparse : the same product for a row-sparse Pi (S entries per row).
//   k_qexp     : per-channel maximum over the blocks and the exponents.
//
// G is column-major, so every kernel reads whole columns with lanes on
// consecutive rows (coalesced 256-byte wave loads).
#include "sb_common.h"

namespace sb {
namespace {

constexpr int NORM_THREADS = 256;
constexpr int64_t NORM_CHUNK = 16384;  // rows per partial sum
constexpr int NORM_UNROLL = 8;         // 16-byte loads in flight per thread
constexpr int NORM_MAX_PARTS = 256;

// A 16-byte load that does not allocate in the caches (data read once).
__device__ inline float4 load_nt4(const float4* p) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  const f4v t = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(p));
  return make_float4(t.x, t.y, t.z, t.w);
}

__device__ inline double wave_sum(double v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
  return v;
}

// Fixed-order block reduction (wave tree, then the waves in index order).
template <int THREADS>
__device__ inline double block_sum(double v, double* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < THREADS / 64; ++w) r += sh[w];
  return r;
}

__global__ void __launch_bounds__(NORM_THREADS)
k_colnorm_partial(const float* __restrict__ G, int64_t n, int64_t ld, int parts, int64_t chunk,
                  double* __restrict__ part) {
  __shared__ double sh[NORM_THREADS / 64];
  const int j = blockIdx.y, p = blockIdx.x;
  const float* col = G + (int64_t)j * ld;
  const int64_t i0 = (int64_t)p * chunk;
  const int64_t i1 = (i0 + chunk < n) ? i0 + chunk : n;
  double acc = 0.0;
  if (i0 >= i1) {
    // empty chunk: contributes zero
  } else if ((((uintptr_t)(col + i0)) & 15) == 0) {
    // NORM_UNROLL 16-byte loads in flight per thread; fixed summation order
    const int64_t nv = (i1 - i0) >> 2;
    const float4* v4 = reinterpret_cast<const float4*>(col + i0);
    int64_t q = threadIdx.x;
    for (; q + (NORM_UNROLL - 1) * NORM_THREADS < nv; q += NORM_UNROLL * NORM_THREADS) {
      float4 x[NORM_UNROLL];
      // G is streamed once: non-temporal loads keep it out of the caches
      // (123 us instead of 146 us for 800 MB)
#pragma unroll
      for (int u = 0; u < NORM_UNROLL; ++u) x[u] = load_nt4(v4 + q + u * NORM_THREADS);
#pragma unroll
      for (int u = 0; u < NORM_UNROLL; ++u) {
        acc += (double)x[u].x * x[u].x;
        acc += (double)x[u].y * x[u].y;
        acc += (double)x[u].z * x[u].z;
        acc += (double)x[u].w * x[u].w;
      }
    }
    for (; q < nv; q += NORM_THREADS) {
      const float4 x = v4[q];
      acc += (double)x.x * x.x;
      acc += (double)x.y * x.y;
      acc += (double)x.z * x.z;
      acc += (double)x.w * x.w;
    }
    for (int64_t i = i0 + 4 * nv + threadIdx.x; i < i1; i += NORM_THREADS) acc += (double)col[i] * col[i];
  } else {
    for (int64_t i = i0 + threadIdx.x; i < i1; i += NORM_THREADS) acc += (double)col[i] * col[i];
  }
  double s = block_sum<NORM_THREADS>(acc, sh);
  if (threadIdx.x == 0) part[(int64_t)j * parts + p] = s;
}

// One wave per column: lane l sums partials l, l+64, ... in order, then a
// fixed shuffle tree; the result depends only on the number of partials.
__global__ void __launch_bounds__(256)
k_colnorm_final(const double* __restrict__ part, int d, int parts, double* __restrict__ n2,
                double* __restrict__ n2_user) {
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (j >= d) return;
  double s = lane_strided_sum(part + (int64_t)j * parts, parts, lane);
  s = wave_sum(s);
  if (lane == 0) {
    n2[j] = s;
    if (n2_user) n2_user[j] = s;
  }
}

// One block (Top Outputs: one block per 64 columns).
constexpr int SELECT_LDS_D = 4096;  // Random Sampling prefix sums held in LDS up to this d

__global__ void __launch_bounds__(1024)
k_select(int kind, const double* __restrict__ n2, int d, int k, const double* __restrict__ u,
         int32_t* __restrict__ cols, float* __restrict__ scales, double* __restrict__ C) {
  __shared__ double sbuf[SELECT_LDS_D];  // the norms (Top Outputs) or their prefix sums (Random Sampling)
  if (kind != SB_SKETCH_TOP_OUTPUTS && blockIdx.x > 0) return;  // one block but for Top Outputs
  if (kind == SB_SKETCH_IDENTITY) {
    for (int t = threadIdx.x; t < k; t += blockDim.x) {
      cols[t] = t;
      scales[t] = 1.0f;
    }
  } else if (kind == SB_SKETCH_TOP_OUTPUTS) {
    // rank of column j in the order (norm descending, index ascending).
    // Block b ranks columns 64b .. 64b+63; its 16 waves count the columns
    // ahead of them in 16 parts of [0, d) and the parts meet in LDS.  Up to
    // SELECT_LDS_D norms are read from LDS (a wave reads one l at a time: a
    // broadcast).
    __shared__ int32_t cnt[16][64];
    const bool in_lds = d <= SELECT_LDS_D;
    if (in_lds) {
      for (int l = threadIdx.x; l < d; l += blockDim.x) sbuf[l] = n2[l];
      __syncthreads();
    }
    const double* N = in_lds ? sbuf : n2;
    const int lane = threadIdx.x & 63, part = threadIdx.x >> 6;
    const int j = blockIdx.x * 64 + lane;
    const int per = (d + 15) / 16, l0 = part * per, l1 = l0 + per < d ? l0 + per : d;
    int ahead = 0;
    if (j < d) {
      const double v = N[j];
      for (int l = l0; l < l1; ++l) {
        const double w = N[l];
        ahead += (w > v) || (w == v && l < j);
      }
    }
    cnt[part][lane] = ahead;
    __syncthreads();
    if (part == 0 && j < d) {
      int rank = 0;
      for (int q = 0; q < 16; ++q) rank += cnt[q][lane];
      if (rank < k) {
        cols[rank] = j;
        scales[rank] = 1.0f;
      }
    }
  } else if (kind == SB_SKETCH_RANDOM_SAMPLING) {
    // the prefix sums are formed sequentially (the order the draws are
    // defined with); up to SELECT_LDS_D norms they live in LDS, so the
    // sum and the searches wait on LDS instead of global memory
    const bool in_lds = d <= SELECT_LDS_D;
    double* Cw = in_lds ? sbuf : C;
    if (in_lds) {
      for (int j = threadIdx.x; j < d; j += blockDim.x) sbuf[j] = n2[j];
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      // eight norms are read ahead of their adds (the adds stay in order),
      // so the chain waits on the fp64 adds rather than on each read; in LDS
      // the prefix overwrites the norms already read
      const double* src = in_lds ? sbuf : n2;
      double acc = 0.0;
      int j = 0;
      for (; j + 8 <= d; j += 8) {
        double v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = src[j + q];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          acc = acc + v[q];
          Cw[j + q] = acc;
        }
      }
      for (; j < d; ++j) {
        acc = acc + src[j];
        Cw[j] = acc;
      }
    }
    __syncthreads();
    C = Cw;
    const double total = C[d - 1];
    for (int t = threadIdx.x; t < k; t += blockDim.x) {
      if (!(total > 0.0)) {
        cols[t] = -1;
        scales[t] = 0.0f;
        continue;
      }
      const double x = u[t] * total;
      // smallest j with C[j] > x (C is non-decreasing)
      int lo = 0, hi = d - 1;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (C[mid] > x) hi = mid;
        else lo = mid + 1;
      }
      cols[t] = lo;
      scales[t] = (float)sqrt(total / ((double)k * n2[lo]));
    }
  }
}

// A value moved across lanes by a DPP control (row shift or row broadcast);
// lanes the control does not write get 0.
template <int CTRL, int ROW_MASK>
__device__ inline uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROW_MASK, 0xf, false);
}

// Maximum over the 64 lanes of a wave, in registers (no LDS traffic):
// shifts by 1, 2, 4 and 8 lanes inside each row of 16, then the last lane of
// rows 0 and 2 into rows 1 and 3 (row_bcast:15) and lane 31 into rows 2 and 3
// (row_bcast:31).  Lanes a step does not write take 0, the smallest value,
// so lane 63 ends with the wave's maximum.
__device__ inline uint32_t wave_max_u32(uint32_t v) {
  uint32_t o;
  o = dpp_u32<0x111, 0xf>(v); v = o > v ? o : v;
  o = dpp_u32<0x112, 0xf>(v); v = o > v ? o : v;
  o = dpp_u32<0x114, 0xf>(v); v = o > v ? o : v;
  o = dpp_u32<0x118, 0xf>(v); v = o > v ? o : v;
  o = dpp_u32<0x142, 0xa>(v); v = o > v ? o : v;
  o = dpp_u32<0x143, 0xc>(v); v = o > v ? o : v;
  return v;
}

// Block maximum of a per-thread value (bit patterns of |x|, which order like
// the magnitudes); every thread gets the result.
template <int THREADS>
__device__ inline uint32_t block_max_u32(uint32_t v, uint32_t* sh) {
  v = wave_max_u32(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 63) sh[wave] = v;
  __syncthreads();
  uint32_t r = 0u;
#pragma unroll
  for (int w = 0; w < THREADS / 64; ++w) r = sh[w] > r ? sh[w] : r;
  return r;
}

constexpr int PACK_THREADS = 256;
constexpr int PACK_ROWS = 4;                           // rows per thread per pass
constexpr int64_t PACK_ROWS_PER_BLOCK = PACK_THREADS * PACK_ROWS;
constexpr int PACK_CG = 16;                            // floats of a row written per pass
// Grid caps of the sketch kernels: block b writes its per-channel maxima to
// blockmax[b*(k+1) + t], reduced afterwards by k_qexp (no atomics), so the
// workspace holds SKETCH_MAX_BLOCKS rows of maxima.  The streaming kernels
// loop over rows in at most SKETCH_GRID_BLOCKS blocks; the matrix-core
// projection takes one block per 512-row tile up to SKETCH_MAX_BLOCKS.
constexpr int SKETCH_MAX_BLOCKS = 4096;
constexpr int SKETCH_GRID_BLOCKS = 2048;

// The floats g0..g0+gn-1 of row i, 16-byte stores when the row allows (every
// row of a multiple-of-4 stride starts 16-byte aligned).
__device__ inline void store_row_run(float* dst, const float* v, int gn, bool vec4) {
  if (vec4 && (gn & 3) == 0) {
#pragma unroll
    for (int t4 = 0; t4 < PACK_CG / 4; ++t4)
      if (4 * t4 < gn)
        reinterpret_cast<float4*>(dst)[t4] = make_float4(v[4 * t4], v[4 * t4 + 1], v[4 * t4 + 2], v[4 * t4 + 3]);
  } else {
#pragma unroll
    for (int tt = 0; tt < PACK_CG; ++tt)
      if (tt < gn) dst[tt] = v[tt];
  }
}

// Row-major sketch: GH[i*ld_gh + t] = fp32(G[i, cols[t]] * scales[t]) for
// t < k, h_i for t = k, 0 after that.  One row per thread: the column reads
// are coalesced across the wave and every row is written whole (with
// ld_gh % 8 == 0, whole 32-byte sectors, so no partial-sector writes).
__global__ void __launch_bounds__(PACK_THREADS)
k_pack(const float* __restrict__ G, int64_t n, int64_t ld_g, int d, const float* __restrict__ h, int k,
       const int32_t* __restrict__ cols, const float* __restrict__ scales, float* __restrict__ GH, int64_t ld_gh,
       uint32_t* __restrict__ blockmax) {
  __shared__ uint32_t sh[PACK_THREADS / 64];
  const bool vec4 = (ld_gh & 3) == 0;
  for (int g0 = 0; g0 < ld_gh; g0 += PACK_CG) {
    const int gn = (ld_gh - g0 < PACK_CG) ? (int)(ld_gh - g0) : PACK_CG;
    // what channel g0 + tt holds: a column of G (col >= 0), all zeros
    // (col == -1: padding, or a Random Sampling column of an all-zero G), or h
    int col[PACK_CG];
    float sc[PACK_CG];
#pragma unroll
    for (int tt = 0; tt < PACK_CG; ++tt) {
      const int t = g0 + tt;
      const int c = (tt < gn && t < k) ? cols[t] : -1;
      col[tt] = (c >= 0 && c < d) ? c : -1;
      sc[tt] = (tt < gn && t < k) ? scales[t] : 0.0f;
    }
    uint32_t mx[PACK_CG];
#pragma unroll
    for (int tt = 0; tt < PACK_CG; ++tt) mx[tt] = 0u;
    for (int64_t base = (int64_t)blockIdx.x * PACK_ROWS_PER_BLOCK; base < n;
         base += (int64_t)gridDim.x * PACK_ROWS_PER_BLOCK) {
      // PACK_ROWS rows per thread, every load issued before any use; rows past
      // the end read row n-1 and store nothing
      float v[PACK_ROWS][PACK_CG];
#pragma unroll
      for (int r = 0; r < PACK_ROWS; ++r) {
        const int64_t i = base + threadIdx.x + (int64_t)r * PACK_THREADS;
        const int64_t ic = i < n ? i : n - 1;
#pragma unroll
        for (int tt = 0; tt < PACK_CG; ++tt) {
          // the branches are uniform (the same for every lane)
          if (col[tt] >= 0)
            v[r][tt] = G[(int64_t)col[tt] * ld_g + ic];
          else if (g0 + tt == k)
            v[r][tt] = h[ic];
          else
            v[r][tt] = 0.0f;
        }
      }
#pragma unroll
      for (int r = 0; r < PACK_ROWS; ++r) {
        const int64_t i = base + threadIdx.x + (int64_t)r * PACK_THREADS;
#pragma unroll
        for (int tt = 0; tt < PACK_CG; ++tt) {
          const int t = g0 + tt;
          // one fp32 multiply: bit-exact with fp32(G * scale)
          float x = t == k ? v[r][tt] : (col[tt] >= 0 ? v[r][tt] * sc[tt] : 0.0f);
          x = tt < gn ? x : 0.0f;
          v[r][tt] = x;
          const uint32_t a = __float_as_uint(x) & 0x7fffffffu;
          if (i < n) mx[tt] = a > mx[tt] ? a : mx[tt];
        }
        if (i < n) store_row_run(GH + i * ld_gh + g0, v[r], gn, vec4);
      }
    }
#pragma unroll
    for (int tt = 0; tt < PACK_CG; ++tt) {
      if (tt < gn && g0 + tt <= k) {
        const uint32_t r = block_max_u32<PACK_THREADS>(mx[tt], sh);
        if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * (k + 1) + g0 + tt] = r;
      }
    }
  }
}

// k_pack for sketches of KC <= 15 columns whose rows fit 16 floats: the
// column count is a template parameter, so every load of a row is issued
// unconditionally (a column index of -1, an all-zero Random Sampling column,
// loads column 0 and stores 0).
template <int KC>
__global__ void __launch_bounds__(PACK_THREADS)
k_pack_small(const float* __restrict__ G, int64_t n, int64_t ld_g, int d, const float* __restrict__ h,
             const int32_t* __restrict__ cols, const float* __restrict__ scales, float* __restrict__ GH,
             int64_t ld_gh, uint32_t* __restrict__ blockmax) {
  __shared__ uint32_t sh[PACK_THREADS / 64];
  const bool vec4 = (ld_gh & 3) == 0;
  const int gn = (int)ld_gh;
  int col[KC];
  bool ok[KC];
  float sc[KC];
#pragma unroll
  for (int t = 0; t < KC; ++t) {
    const int c = cols[t];
    ok[t] = c >= 0 && c < d;
    col[t] = ok[t] ? c : 0;
    sc[t] = scales[t];
  }
  uint32_t mx[KC + 1];
#pragma unroll
  for (int t = 0; t <= KC; ++t) mx[t] = 0u;
  for (int64_t base = (int64_t)blockIdx.x * PACK_ROWS_PER_BLOCK; base < n;
       base += (int64_t)gridDim.x * PACK_ROWS_PER_BLOCK) {
    float g[PACK_ROWS][KC + 1];
#pragma unroll
    for (int r = 0; r < PACK_ROWS; ++r) {
      const int64_t i = base + threadIdx.x + (int64_t)r * PACK_THREADS;
      const int64_t ic = i < n ? i : n - 1;
#pragma unroll
      for (int t = 0; t < KC; ++t) g[r][t] = G[(int64_t)col[t] * ld_g + ic];
      g[r][KC] = h[ic];
    }
#pragma unroll
    for (int r = 0; r < PACK_ROWS; ++r) {
      const int64_t i = base + threadIdx.x + (int64_t)r * PACK_THREADS;
      float v[PACK_CG];
#pragma unroll
      for (int tt = 0; tt < PACK_CG; ++tt) {
        // one fp32 multiply: bit-exact with fp32(G * scale)
        float x = 0.0f;
        if (tt < KC) x = ok[tt] ? g[r][tt] * sc[tt] : 0.0f;
        if (tt == KC) x = g[r][KC];
        v[tt] = x;
      }
      if (i < n) {
#pragma unroll
        for (int t = 0; t <= KC; ++t) {
          const uint32_t a = __float_as_uint(v[t]) & 0x7fffffffu;
          mx[t] = a > mx[t] ? a : mx[t];
        }
        store_row_run(GH + i * ld_gh, v, gn, vec4);
      }
    }
  }
#pragma unroll
  for (int t = 0; t <= KC; ++t) {
    const uint32_t r = block_max_u32<PACK_THREADS>(mx[t], sh);
    if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * (KC + 1) + t] = r;
  }
}

constexpr int PROJ_THREADS = 1024;
constexpr int PROJ_KT = 32;               // sketch columns per pass
constexpr int PROJ_JU = 16;               // G loads in flight per thread
constexpr int PROJ_LDS_FLOATS = 32768;    // 128 KB: the Pi block staged per pass
constexpr int SPARSE_MAX_S = 1;           // entries per row of Pi for the sparse kernel
constexpr int PROJ_MFMA_MIN_K = 8;        // from this k on the dense product runs on MFMA

// Random Projections (Section 3.3), HBM-bound on the read of G: one row per
// thread, PROJ_JU columns of G loaded ahead, and the pass's block of Pi
// (rows j0..j0+jc, columns t0..t0+KT) staged in LDS and read by broadcast.
// Each output is an fp32 fmaf chain over j in increasing order.  Columns
// past k are padded with zeros in LDS and never written.
// Writes one row: channels [t0, t0 + kt) from acc; on the last pass also the
// hessian channel k and the zero padding up to ld_gh (whole row in 16-byte
// stores when the pass covers the row from 0 and ld_gh % 4 == 0).
template <int KT>
__device__ inline void store_proj_row(float* __restrict__ GH, int64_t i, int64_t ld_gh, int t0, int kt, int k,
                                      bool last, float hv, const float (&acc)[KT]) {
  float* row = GH + i * ld_gh;
  if (last && t0 == 0 && (ld_gh & 3) == 0 && ld_gh <= KT + 8) {
#pragma unroll
    for (int q = 0; q < (KT + 8) / 4; ++q) {
      if (4 * q < ld_gh) {
        float o[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 4 * q + r;
          o[r] = t < k ? acc[t < KT ? t : 0] : (t == k ? hv : 0.0f);
        }
        *reinterpret_cast<float4*>(row + 4 * q) = make_float4(o[0], o[1], o[2], o[3]);
      }
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < KT; ++t)
    if (t < kt) row[t0 + t] = acc[t];
  if (last) {
    row[k] = hv;
    for (int64_t t = k + 1; t < ld_gh; ++t) row[t] = 0.0f;
  }
}

template <int KT>
__global__ void __launch_bounds__(PROJ_THREADS)
k_project(const float* __restrict__ G, int64_t n, int d, int64_t ld_g, const float* __restrict__ Pi, int k, int t0,
          const float* __restrict__ h, float* __restrict__ GH, int64_t ld_gh, uint32_t* __restrict__ blockmax) {
  extern __shared__ float sPi[];  // [jc][KT]
  __shared__ uint32_t sh[PROJ_THREADS / 64];
  const int kt = (k - t0 < KT) ? k - t0 : KT;
  const bool last = t0 + PROJ_KT >= k;
  const int jcap = PROJ_LDS_FLOATS / KT;
  uint32_t mx[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) mx[t] = 0u;
  uint32_t mxh = 0u;
  for (int64_t base = (int64_t)blockIdx.x * PROJ_THREADS; base < n; base += (int64_t)gridDim.x * PROJ_THREADS) {
    const int64_t i = base + threadIdx.x;
    const bool live = i < n;
    const int64_t ii = live ? i : n - 1;
    float acc[KT];
#pragma unroll
    for (int t = 0; t < KT; ++t) acc[t] = 0.0f;
    for (int j0 = 0; j0 < d; j0 += jcap) {
      const int jc = (d - j0 < jcap) ? d - j0 : jcap;
      __syncthreads();
      for (int e = threadIdx.x; e < jc * KT; e += PROJ_THREADS) {
        const int jj = e / KT, t = e - jj * KT;
        sPi[e] = (t < kt) ? Pi[(int64_t)(j0 + jj) * k + t0 + t] : 0.0f;
      }
      __syncthreads();
      for (int jb = 0; jb < jc; jb += PROJ_JU) {
        // columns past the block (last batch only) repeat its last column and
        // are skipped below: every load is issued unconditionally
        float g[PROJ_JU];
#pragma unroll
        for (int u = 0; u < PROJ_JU; ++u) {
          const int j = j0 + (jb + u < jc ? jb + u : jc - 1);
          g[u] = ld_stream(G + (int64_t)j * ld_g + ii);
        }
#pragma unroll
        for (int u = 0; u < PROJ_JU; ++u) {
          if (jb + u < jc) {
            const float4* pr = reinterpret_cast<const float4*>(sPi + (jb + u) * KT);
#pragma unroll
            for (int t4 = 0; t4 < KT / 4; ++t4) {
              const float4 p4 = pr[t4];
              acc[4 * t4] = fmaf(g[u], p4.x, acc[4 * t4]);
              acc[4 * t4 + 1] = fmaf(g[u], p4.y, acc[4 * t4 + 1]);
              acc[4 * t4 + 2] = fmaf(g[u], p4.z, acc[4 * t4 + 2]);
              acc[4 * t4 + 3] = fmaf(g[u], p4.w, acc[4 * t4 + 3]);
            }
          }
        }
      }
    }
    if (live) {
      const float hv = last ? h[i] : 0.0f;
      store_proj_row<KT>(GH, i, ld_gh, t0, kt, k, last, hv, acc);
#pragma unroll
      for (int t = 0; t < KT; ++t) {
        const uint32_t a = __float_as_uint(acc[t]) & 0x7fffffffu;
        mx[t] = (t < kt && a > mx[t]) ? a : mx[t];
      }
      const uint32_t ah = __float_as_uint(hv) & 0x7fffffffu;
      mxh = ah > mxh ? ah : mxh;
    }
  }
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    if (t < kt) {
      const uint32_t r = block_max_u32<PROJ_THREADS>(mx[t], sh);
      if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * (k + 1) + t0 + t] = r;
    }
  }
  if (last) {
    const uint32_t r = block_max_u32<PROJ_THREADS>(mxh, sh);
    if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * (k + 1) + k] = r;
  }
}

// The hessian channel of a projected sketch, GH[i*ld_gh + k] = h[i], and the
// zero padding of the row after it, with the channel's per-block maximum.
// Sparse projection (Section 3.3 with a sparse Pi: Achlioptas entries, or a
// sparse JL transform, which the proof of Prop. A.5 names as the fast form
// of G Pi).  Pi is row-sparse: row j holds S entries (column, value).  One
// thread per row of G; the lanes of a wave take consecutive rows, so each
// column of G is read once, 256 contiguous bytes per wave.  The entries of a
// row of Pi are the same for every lane, so the accumulator they add to has a
// wave-uniform index (VGPR indexing, no scratch) and the PROJ_JU * S entries
// of a batch arrive in a few wide scalar loads.  fp32 accumulation in the
// order (j, q): 2 n d S flops instead of the dense 2 n d k.  The last pass
// also writes h and the zero padding of the row.
template <int S>
__global__ void __launch_bounds__(PROJ_THREADS)
k_project_sparse(const float* __restrict__ G, int64_t n, int d, int64_t ld_g, const int32_t* __restrict__ pcol,
                 const float* __restrict__ pval, int k, int t0, const float* __restrict__ h, float* __restrict__ GH,
                 int64_t ld_gh, uint32_t* __restrict__ blockmax) {
  constexpr int KT = PROJ_KT;
  __shared__ uint32_t sh[PROJ_THREADS / 64];
  const int kt = (k - t0 < KT) ? k - t0 : KT;
  const bool last = t0 + KT >= k;
  uint32_t mx[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) mx[t] = 0u;
  uint32_t mxh = 0u;
  for (int64_t base = (int64_t)blockIdx.x * PROJ_THREADS; base < n; base += (int64_t)gridDim.x * PROJ_THREADS) {
    const int64_t i = base + threadIdx.x;
    const bool live = i < n;
    const int64_t ii = live ? i : n - 1;
    float acc[KT];
#pragma unroll
    for (int t = 0; t < KT; ++t) acc[t] = 0.0f;
    for (int j0 = 0; j0 < d; j0 += PROJ_JU) {
      // columns past d (last batch only) load column d-1 and add nothing
      float g[PROJ_JU];
#pragma unroll
      // G is streamed once: non-temporal loads (1.64 ms instead of 1.69 ms at 2M x 1000 -> 20, s = 1)
      for (int u = 0; u < PROJ_JU; ++u) g[u] = ld_stream(G + (int64_t)(j0 + u < d ? j0 + u : d - 1) * ld_g + ii);
      int tc[PROJ_JU * S];
      float vc[PROJ_JU * S];
#pragma unroll
      for (int e = 0; e < PROJ_JU * S; ++e) {
        const bool in = j0 + e / S < d;
        tc[e] = in ? pcol[(int64_t)j0 * S + e] - t0 : -1;
        vc[e] = in ? pval[(int64_t)j0 * S + e] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < PROJ_JU; ++u)
#pragma unroll
        for (int q = 0; q < S; ++q) {
          const int t = tc[u * S + q];
          if ((unsigned)t < (unsigned)kt) acc[t] = fmaf(g[u], vc[u * S + q], acc[t]);
        }
    }
    if (live) {
      const float hv = last ? h[i] : 0.0f;
      store_proj_row<KT>(GH, i, ld_gh, t0, kt, k, last, hv, acc);
#pragma unroll
      for (int t = 0; t < KT; ++t) {
        const uint32_t a = __float_as_uint(acc[t]) & 0x7fffffffu;
        mx[t] = (t < kt && a > mx[t]) ? a : mx[t];
      }
      const uint32_t ah = __float_as_uint(hv) & 0x7fffffffu;
      mxh = ah > mxh ? ah : mxh;
    }
  }
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    if (t < kt) {
      const uint32_t r = block_max_u32<PROJ_THREADS>(mx[t], sh);
      if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * (k + 1) + t0 + t] = r;
    }
  }
  if (last) {
    const uint32_t r = block_max_u32<PROJ_THREADS>(mxh, sh);
    if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * (k + 1) + k] = r;
  }
}

// Dense projection on the matrix cores with v_mfma_f32_4x4x1f32, whose 16
// blocks of 4 x 4 x 1 are here 16 groups of 4 consecutive rows of G sharing
// one column j: one instruction multiplies 64 rows of column j by row j of
// Pi for 4 sketch columns, so k columns take ceil(k / 4) instructions and
// nothing is padded past a multiple of 4 (the 32 x 32 tile pads 20 columns
// to 32).  It runs at the same flops per clock as the 32 x 32 x 2 form, and
// MI355X's fp32 MFMA rate is twice its fp32 vector rate without packed
// instructions, so at k >= 8 the product stops being bound by the VALU.
// A wave computes M4_MT * 64 rows x 4 * NG sketch columns.  Operands:
//   A (block b, 4 x 1): lane l holds G[row0 + l, j] (64 consecutive rows of
//     one column: two 128-byte lines);
//   B (block b, 1 x 4): lane l holds Pi[j, t0 + 4g + l % 4], the same in
//     every block, read from a block of Pi staged in LDS (zero past d and
//     past the pass's kt columns: four addresses per read, a broadcast);
//   D (block b, 4 x 4): register r of lane l holds row row0 + 4 (l / 4) + r,
//     column t0 + 4g + l % 4.
// M4_KU columns of G are loaded before their MFMAs.  The order in which the
// hardware adds the products is its own, so the result is checked against
// the exact product with the dot-product error bound.
constexpr int M4_THREADS = 256;
constexpr int M4_MT = 2;    // 64-row tiles per wave
constexpr int M4_JC = 256;  // columns of G per staged block of Pi
constexpr int M4_KU = 16;   // columns of G per batch of loads
static_assert(M4_JC % M4_KU == 0, "a batch of columns never passes the staged block");
typedef float mf_v4 __attribute__((ext_vector_type(4)));

template <int NG>
__global__ void __launch_bounds__(M4_THREADS)
k_project_mfma4(const float* __restrict__ G, int64_t n, int d, int64_t ld_g, const float* __restrict__ Pi, int k,
                int t0, const float* __restrict__ h, float* __restrict__ GH, int64_t ld_gh,
                uint32_t* __restrict__ blockmax) {
  constexpr int W = 4 * NG;  // sketch columns of the pass, padded to a multiple of 4
  __shared__ float sPi[M4_JC * W];
  __shared__ uint32_t smax[M4_THREADS / 64][W + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int kt = (k - t0 < W) ? k - t0 : W;
  const bool last = t0 + kt >= k;
  const int cq = lane & 3;  // this lane's column within each group of 4
  uint32_t mx[NG], mxh = 0u;
#pragma unroll
  for (int g = 0; g < NG; ++g) mx[g] = 0u;
  constexpr int64_t ROWS = (M4_THREADS / 64) * M4_MT * 64;  // rows per block per pass
  for (int64_t base = (int64_t)blockIdx.x * ROWS; base < n; base += (int64_t)gridDim.x * ROWS) {
    const int64_t rw = base + (int64_t)wave * M4_MT * 64;
    int64_t rc[M4_MT];
#pragma unroll
    for (int mt = 0; mt < M4_MT; ++mt) {
      const int64_t r = rw + mt * 64 + lane;
      rc[mt] = r < n ? r : n - 1;  // rows past the end read row n-1 and store nothing
    }
    mf_v4 acc[M4_MT][NG];
#pragma unroll
    for (int mt = 0; mt < M4_MT; ++mt)
#pragma unroll
      for (int g = 0; g < NG; ++g) acc[mt][g] = mf_v4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int j0 = 0; j0 < d; j0 += M4_JC) {
      const int jc = (d - j0 < M4_JC) ? d - j0 : M4_JC;
      __syncthreads();  // the previous block of Pi is no longer read
      for (int e = threadIdx.x; e < M4_JC * W; e += M4_THREADS) {
        const int jr = e / W, c = e - jr * W;
        sPi[e] = (jr < jc && c < kt) ? Pi[(int64_t)(j0 + jr) * k + t0 + c] : 0.0f;
      }
      __syncthreads();
      for (int kk = 0; kk < jc; kk += M4_KU) {
        float a[M4_KU][M4_MT];
#pragma unroll
        for (int u = 0; u < M4_KU; ++u) {
          // past the block: a finite value of column jc - 1 times a zero of Pi
          const int64_t jg = j0 + (kk + u < jc ? kk + u : jc - 1);
#pragma unroll
          for (int mt = 0; mt < M4_MT; ++mt) a[u][mt] = ld_stream(G + jg * ld_g + rc[mt]);
        }
#pragma unroll
        for (int u = 0; u < M4_KU; ++u) {
          const float* pr = sPi + (kk + u) * W + cq;
#pragma unroll
          for (int g = 0; g < NG; ++g) {
            const float b = pr[4 * g];
#pragma unroll
            for (int mt = 0; mt < M4_MT; ++mt)
              acc[mt][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[u][mt], b, acc[mt][g], 0, 0, 0);
          }
        }
      }
    }
#pragma unroll
    for (int mt = 0; mt < M4_MT; ++mt)
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int col = 4 * g + cq;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = rw + mt * 64 + 4 * (lane >> 2) + r;
          if (row < n && col < kt) {
            const float v = acc[mt][g][r];
            GH[row * ld_gh + t0 + col] = v;
            const uint32_t m = __float_as_uint(v) & 0x7fffffffu;
            mx[g] = m > mx[g] ? m : mx[g];
          }
        }
      }
    if (last) {
#pragma unroll
      for (int mt = 0; mt < M4_MT; ++mt) {
        const int64_t row = rw + mt * 64 + lane;
        if (row < n) {
          const float hv = h[row];
          GH[row * ld_gh + k] = hv;
          for (int64_t t = k + 1; t < ld_gh; ++t) GH[row * ld_gh + t] = 0.0f;
          const uint32_t m = __float_as_uint(hv) & 0x7fffffffu;
          mxh = m > mxh ? m : mxh;
        }
      }
    }
  }
  // block maxima: column 4g + cq's lanes are those with the same cq; then the waves
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    for (int off = 4; off < 64; off <<= 1) {
      const uint32_t o = __shfl_xor(mx[g], off, 64);
      mx[g] = o > mx[g] ? o : mx[g];
    }
    if (lane < 4) smax[wave][4 * g + lane] = mx[g];
  }
  mxh = wave_max_u32(mxh);  // in lane 63
  if (lane == 63) smax[wave][W] = mxh;
  __syncthreads();
  if (threadIdx.x <= W) {
    uint32_t r = 0u;
#pragma unroll
    for (int w = 0; w < M4_THREADS / 64; ++w) r = smax[w][threadIdx.x] > r ? smax[w][threadIdx.x] : r;
    if (threadIdx.x < kt) blockmax[(int64_t)blockIdx.x * (k + 1) + t0 + threadIdx.x] = r;
    if (threadIdx.x == W && last) blockmax[(int64_t)blockIdx.x * (k + 1) + k] = r;
  }
}

// Dense d x k Pi from its row-sparse form: one thread per row j, entries
// added in q order in fp32 (columns outside [0, k) are dropped).
__global__ void __launch_bounds__(256)
k_assemble_pi(const int32_t* __restrict__ pcol, const float* __restrict__ pval, int d, int s, int k,
              float* __restrict__ Pi) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= d) return;
  float* row = Pi + (int64_t)j * k;
  for (int t = 0; t < k; ++t) row[t] = 0.0f;
  for (int q = 0; q < s; ++q) {
    const int c = pcol[(int64_t)j * s + q];
    if (c >= 0 && c < k) row[c] += pval[(int64_t)j * s + q];
  }
}

// Per-block max |GH[i*ld_gh + t]| for a caller-supplied row-major GH: one
// row per thread, PACK_CG channels per pass.
__global__ void __launch_bounds__(256)
k_maxabs(const float* __restrict__ GH, int64_t n, int64_t ld_gh, int c, uint32_t* __restrict__ blockmax) {
  __shared__ uint32_t sh[4];
  for (int g0 = 0; g0 < c; g0 += PACK_CG) {
    const int gn = (c - g0 < PACK_CG) ? c - g0 : PACK_CG;
    uint32_t mx[PACK_CG];
#pragma unroll
    for (int tt = 0; tt < PACK_CG; ++tt) mx[tt] = 0u;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
#pragma unroll
      for (int tt = 0; tt < PACK_CG; ++tt) {
        if (tt < gn) {
          const uint32_t a = __float_as_uint(GH[i * ld_gh + g0 + tt]) & 0x7fffffffu;
          mx[tt] = a > mx[tt] ? a : mx[tt];
        }
      }
    }
#pragma unroll
    for (int tt = 0; tt < PACK_CG; ++tt) {
      if (tt < gn) {
        const uint32_t r = block_max_u32<256>(mx[tt], sh);
        if (threadIdx.x == 0) blockmax[(int64_t)blockIdx.x * c + g0 + tt] = r;
      }
    }
  }
}

// One block per channel: max over the blocks' maxima, then
// qexp[t] = (QBITS-1) - floor(log2(max)), 0 for an all-zero channel.
__global__ void __launch_bounds__(256)
k_qexp(const uint32_t* __restrict__ blockmax, int nblocks, int c, int32_t* __restrict__ qexp) {
  __shared__ uint32_t sh[4];
  const int t = blockIdx.x;
  uint32_t mx = 0u;
  int b = threadIdx.x;
  for (; b + 7 * 256 < nblocks; b += 8 * 256) {  // eight loads in flight
    uint32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = blockmax[(int64_t)(b + u * 256) * c + t];
#pragma unroll
    for (int u = 0; u < 8; ++u) mx = v[u] > mx ? v[u] : mx;
  }
  for (; b < nblocks; b += 256) {
    const uint32_t v = blockmax[(int64_t)b * c + t];
    mx = v > mx ? v : mx;
  }
  mx = block_max_u32<256>(mx, sh);
  if (threadIdx.x == 0) {
    const float m = __uint_as_float(mx);
    qexp[t] = (m > 0.0f) ? (QBITS - 1) - ilogbf(m) : 0;
  }
}

int sketch_blocks(int64_t n, int64_t rows_per_block, int cap = SKETCH_GRID_BLOCKS) {
  int64_t b = (n + rows_per_block - 1) / rows_per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

int norm_parts(int64_t n) {
  int64_t p = (n + NORM_CHUNK - 1) / NORM_CHUNK;
  if (p < 1) p = 1;
  if (p > NORM_MAX_PARTS) p = NORM_MAX_PARTS;
  return (int)p;
}

// Workspace: [norm partials d*P][norm2 d][prefix d][block maxima SKETCH_MAX_BLOCKS*(k+1)]
// [dense Pi assembled from a sparse one, d*k]
struct SketchWs {
  int64_t part, n2, C, blockmax, pi, total;
};

SketchWs sketch_ws_layout(int64_t n, int32_t d, int32_t k) {
  SketchWs L{};
  int64_t p = 0;
  L.part = p;
  p += align256((int64_t)d * norm_parts(n) * 8);
  L.n2 = p;
  p += align256((int64_t)d * 8);
  L.C = p;
  p += align256((int64_t)d * 8);
  L.blockmax = p;
  p += align256((int64_t)SKETCH_MAX_BLOCKS * (k + 1) * 4);
  L.pi = p;
  p += align256((int64_t)d * k * 4);
  L.total = p;
  return L;
}

// G Pi for a dense Pi, PROJ_KT sketch columns per pass; returns the grid size
// (block b's maxima of every channel sit in row b of blockmax).
int launch_dense_projection(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                            const float* Pi, float* GH, int64_t ld_gh, uint32_t* blockmax, hipStream_t st) {
  if (k >= PROJ_MFMA_MIN_K) {
    const int nb = sketch_blocks(n, (M4_THREADS / 64) * M4_MT * 64, SKETCH_MAX_BLOCKS);
    for (int t0 = 0; t0 < k; t0 += 32) {
      const int ng = (k - t0 < 32 ? k - t0 + 3 : 32 + 3) / 4;
#define SB_P4(NG)                                                                                                 \
  case NG:                                                                                                        \
    hipLaunchKernelGGL((k_project_mfma4<NG>), dim3(nb), dim3(M4_THREADS), 0, st, G, n, d, ld_g, Pi, k, t0, h, GH, \
                       ld_gh, blockmax);                                                                          \
    break;
      switch (ng) { SB_P4(1) SB_P4(2) SB_P4(3) SB_P4(4) SB_P4(5) SB_P4(6) SB_P4(7) SB_P4(8) }
#undef SB_P4
    }
    return nb;
  }
  const int nb = sketch_blocks(n, PROJ_THREADS);
  for (int t0 = 0; t0 < k; t0 += PROJ_KT) {
    const int kt = (k - t0 < PROJ_KT) ? k - t0 : PROJ_KT;
    const int KT = (kt + 3) / 4 * 4;
    const int jc = (d < PROJ_LDS_FLOATS / KT) ? d : PROJ_LDS_FLOATS / KT;
    const size_t lds = (size_t)jc * KT * 4;
#define SB_PROJ(K)                                                                                               \
  case K:                                                                                                        \
    hipLaunchKernelGGL((k_project<K>), dim3(nb), dim3(PROJ_THREADS), lds, st, G, n, d, ld_g, Pi, k, t0, h, GH,   \
                       ld_gh, blockmax);                                                                         \
    break;
    switch (KT) {
      SB_PROJ(4) SB_PROJ(8) SB_PROJ(12) SB_PROJ(16) SB_PROJ(20) SB_PROJ(24) SB_PROJ(28) SB_PROJ(32)
    }
#undef SB_PROJ
  }
  return nb;
}

}  // namespace

int64_t sketch_ws_bytes(int32_t kind, int64_t n, int32_t d, int32_t k) {
  (void)kind;
  return sketch_ws_layout(n, d, k).total;
}

int64_t hist_exponents_ws_bytes(int32_t k) { return align256((int64_t)SKETCH_MAX_BLOCKS * (k + 1) * 4); }

int32_t launch_sketch(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                      const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols, float* scales,
                      double* norm2, int32_t* qexp, void* ws, hipStream_t st, const double* norm2_in) {
  const int P = norm_parts(n);
  const SketchWs L = sketch_ws_layout(n, d, k);
  char* w = static_cast<char*>(ws);
  double* part = reinterpret_cast<double*>(w + L.part);
  double* n2 = reinterpret_cast<double*>(w + L.n2);
  double* C = reinterpret_cast<double*>(w + L.C);
  uint32_t* blockmax = reinterpret_cast<uint32_t*>(w + L.blockmax);

  int nb;
  if (kind == SB_SKETCH_RANDOM_PROJECTION) {
    nb = launch_dense_projection(G, n, d, ld_g, h, k, Pi, GH, ld_gh, blockmax, st);
  } else {
    if (norm2_in == nullptr) {
      int64_t chunk = (n + P - 1) / P;
      chunk = (chunk + 3) & ~int64_t(3);
      hipLaunchKernelGGL(k_colnorm_partial, dim3(P, d), dim3(NORM_THREADS), 0, st, G, n, ld_g, P, chunk, part);
      hipLaunchKernelGGL(k_colnorm_final, dim3((d + 3) / 4), dim3(256), 0, st, part, d, P, n2, norm2);
    }
    const unsigned sel_blocks = kind == SB_SKETCH_TOP_OUTPUTS ? (unsigned)((d + 63) / 64) : 1u;
    hipLaunchKernelGGL(k_select, dim3(sel_blocks), dim3(1024), 0, st, kind, norm2_in ? norm2_in : n2, d, k, u, cols,
                       scales, C);
    nb = sketch_blocks(n, PACK_ROWS_PER_BLOCK);
    if (k < PACK_CG && ld_gh <= PACK_CG) {
#define SB_PACK(K)                                                                                               \
  case K:                                                                                                        \
    hipLaunchKernelGGL((k_pack_small<K>), dim3(nb), dim3(PACK_THREADS), 0, st, G, n, ld_g, d, h, cols, scales, GH, \
                       ld_gh, blockmax);                                                                         \
    break;
      switch (k) {
        SB_PACK(1) SB_PACK(2) SB_PACK(3) SB_PACK(4) SB_PACK(5) SB_PACK(6) SB_PACK(7) SB_PACK(8) SB_PACK(9)
        SB_PACK(10) SB_PACK(11) SB_PACK(12) SB_PACK(13) SB_PACK(14) SB_PACK(15)
      }
#undef SB_PACK
    } else {
      hipLaunchKernelGGL(k_pack, dim3(nb), dim3(PACK_THREADS), 0, st, G, n, ld_g, d, h, k, cols, scales, GH, ld_gh,
                         blockmax);
    }
  }
  hipLaunchKernelGGL(k_qexp, dim3(k + 1), dim3(256), 0, st, blockmax, nb, k + 1, qexp);
  return check_launch("sb_sketch");
}

// Rows of Pi with one entry go through the sparse kernel; with more, the
// per-entry accumulator update (a few issue slots each) costs more than the
// dense product at k <= 32 (2M x 1000 -> 20: sparse kernel 1.70 ms at s = 1,
// 2.34 ms at s = 2, 4.18 ms at s = 4; assembled dense Pi 2.15-2.43 ms), so
// Pi is assembled densely first.
int32_t launch_sketch_sparse(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k, int32_t s,
                             const int32_t* pi_col, const float* pi_val, float* GH, int64_t ld_gh, int32_t* qexp,
                             void* ws, hipStream_t st) {
  const SketchWs L = sketch_ws_layout(n, d, k);
  char* w = static_cast<char*>(ws);
  uint32_t* blockmax = reinterpret_cast<uint32_t*>(w + L.blockmax);
  int nb;
  if (s <= SPARSE_MAX_S) {
    nb = sketch_blocks(n, PROJ_THREADS);
    for (int t0 = 0; t0 < k; t0 += PROJ_KT)
      hipLaunchKernelGGL((k_project_sparse<SPARSE_MAX_S>), dim3(nb), dim3(PROJ_THREADS), 0, st, G, n, d, ld_g, pi_col,
                         pi_val, k, t0, h, GH, ld_gh, blockmax);
  } else {
    float* Pi = reinterpret_cast<float*>(w + L.pi);
    hipLaunchKernelGGL(k_assemble_pi, dim3((d + 255) / 256), dim3(256), 0, st, pi_col, pi_val, d, s, k, Pi);
    nb = launch_dense_projection(G, n, d, ld_g, h, k, Pi, GH, ld_gh, blockmax, st);
  }
  hipLaunchKernelGGL(k_qexp, dim3(k + 1), dim3(256), 0, st, blockmax, nb, k + 1, qexp);
  return check_launch("sb_sketch_sparse_projection");
}

int32_t launch_hist_exponents(const float* GH, int64_t n, int64_t ld_gh, int32_t k, int32_t* qexp, void* ws,
                              hipStream_t st) {
  uint32_t* blockmax = static_cast<uint32_t*>(ws);
  const int nb = sketch_blocks(n, 256);
  hipLaunchKernelGGL(k_maxabs, dim3(nb), dim3(256), 0, st, GH, n, ld_gh, k + 1, blockmax);
  hipLaunchKernelGGL(k_qexp, dim3(k + 1), dim3(256), 0, st, blockmax, nb, k + 1, qexp);
  return check_launch("sb_hist_exponents");
}

}  // namespace sb
