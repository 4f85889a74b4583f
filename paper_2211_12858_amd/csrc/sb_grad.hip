// Loss derivatives with fused column norms, and the prediction update
// (Section 2: eq. 2 gives the first and second derivatives of the loss at the
// current predictions; the model is updated by a_t = a_{t-1} + eps * f_t).
//
// k_grad: one thread per row, the rows of a block in one 256-row tile, tiles
//   grid-strided.  The lanes of a wave take consecutive rows, so every load
//   and store is one 256-byte run of a column of the column-major matrices.
//   Softmax cross-entropy: a first pass over the row's scores keeps a running
//   maximum and the sum of exp(a - max), rescaled chunk by chunk; the second
//   pass re-reads the scores and writes g = p - onehot(y), h = p (1 - p).
//   Sigmoid cross-entropy needs one pass: g = s - Y, h = s (1 - s).
//   The squared column norms of the stored G (what Top Outputs and Random
//   Sampling rank and draw by, Sections 3.1, 3.2) are summed in the same pass:
//   each 16-column chunk of g goes through LDS, 16 threads per column add 16
//   rows each in fp64, a fixed shift-and-add over their 16 lanes (DPP, in
//   registers) joins them, and one thread adds the
//   tile's sum to its slot's partial (slot = tile mod GRAD_PARTS, always the
//   same thread of the same block, in tile order).  k_grad_norm_final adds the
//   slots in a fixed order, so the norms are deterministic and the same for
//   every grid that divides the slot count (the fused update below launches
//   fewer blocks than the derivatives alone).
// k_update: F[i, j] += lr * V[leaf of i, j] in fp64, rounded once to fp32.
//   lr * V of a chunk of columns is staged in LDS; the leaf ids come from the
//   leaf segments (k_leaf_ids, shared with the leaf values).
// The update of one tree followed by the derivatives of the next (the two
// consecutive steps of the boosting loop) can run as one pass for softmax
// with d <= 104: k_grad_softmax_regs with UPD loads a row's scores, adds
// lr * V of the row's leaf (all of lr * V staged in LDS), stores the new
// scores and goes on from them, so F is read once instead of twice.  The
// arithmetic is k_update's, so the result is bit-identical to the two calls.
#include <cmath>

#include "sb_common.h"
#include "sb_leaf_ids.h"

namespace sb {
namespace {

// Sum over each row of 16 lanes, in registers (no LDS traffic): shifts by 1,
// 2, 4 and 8 lanes (lanes a shift does not write add 0), so the last lane of
// each row ends with the row's sum, always added in the same order.
template <int CTRL>
__device__ inline double dpp_row_shr(double x) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}

__device__ inline double row16_sum(double x) {
  x += dpp_row_shr<0x111>(x);
  x += dpp_row_shr<0x112>(x);
  x += dpp_row_shr<0x114>(x);
  x += dpp_row_shr<0x118>(x);
  return x;
}

constexpr int GRAD_THREADS = 256;
constexpr int GRAD_JA = 8;          // columns per load batch of the softmax first pass
constexpr int GRAD_JC = 16;         // columns per chunk of the second pass (norm staging)
// Column-norm partial slots: tile t adds into slot t % GRAD_PARTS, and the
// grid divides the slot count (or is one block per tile), so every slot
// belongs to one block and sums its tiles in tile order: the norms do not
// depend on the grid.  1536 = 2^9 * 3 has the divisors 512 and 768 (two and
// three blocks per CU of MI355X).
constexpr int GRAD_PARTS = 1536;
constexpr int UPD_THREADS = 256;
constexpr int UPD_LDS_DOUBLES = 8192;  // lr * V of one column chunk: at most 64 KB
constexpr int UPD_JC = 16;             // columns per chunk at most
constexpr int UPD_MAX_BLOCKS = 2048;

struct GradArgs {
  int loss;
  const float* F;
  int64_t n;
  int32_t d;
  int64_t ld_f;
  const int32_t* labels;
  const uint8_t* Y;
  int64_t ld_y;
  float* G;
  int64_t ld_g;
  float* hess;
  int64_t ld_h;
  float* h_row;
  double* npart;  // [d][n_parts] or NULL: sums of g^2 per column and slot
  int32_t n_tiles;
  int32_t n_parts;  // min(n_tiles, GRAD_PARTS)
  // update before the derivatives (k_grad_softmax_regs with UPD): F_upd is F
  // (updated in place), ids the leaf of every row, lv_stride the doubles per
  // leaf of lr * V in LDS
  float* F_upd;
  const uint8_t* ids;
  int32_t n_leaves;
  int32_t lv_stride;
  const double* V;
  int64_t ld_v;
  double lr;
};

// Barrier for the norm staging: waits for this wave's LDS operations only.
// A plain __syncthreads also waits for every outstanding global access,
// here the stores of G (and the hessians) of the chunk just written.
// 0xc07f is s_waitcnt lgkmcnt(0) in the gfx9 encoding.
__device__ inline void lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One tile of k_grad (the loss, whether the tile is full and whether the
// hessians are stored are template parameters, so the column loop has no
// runtime branch).  Columns past d in the last chunk load column d-1 and
// store column d-1's own values there (same address, same value), and d is
// passed in opaque to the compiler, as in grad_softmax_tile below.
template <int LOSS, bool FULL, bool HESS>
__device__ inline void grad_tile(const GradArgs& a, float (*gbuf)[GRAD_THREADS], int64_t base, int d) {
  const int tid = threadIdx.x;
  const int64_t row = base + tid;
  const bool ok = FULL || row < a.n;
  const int64_t rc = ok ? row : a.n - 1;  // rows past the end read row n-1 and store nothing
  float m = -INFINITY, s = 0.0f, inv = 0.0f;
  int y = -1;
  if constexpr (LOSS == SB_LOSS_SOFTMAX_CE) {
    y = a.labels[rc];
    for (int j0 = 0; j0 < d; j0 += GRAD_JA) {
      float x[GRAD_JA];
      // columns past d (last chunk only) repeat column d-1: a repeat of
      // the row's own score leaves the maximum unchanged, and its exp is
      // dropped from the sum below
#pragma unroll
      for (int u = 0; u < GRAD_JA; ++u) x[u] = a.F[(int64_t)(j0 + u < d ? j0 + u : d - 1) * a.ld_f + rc];
      float cm = x[0];
#pragma unroll
      for (int u = 1; u < GRAD_JA; ++u) cm = fmaxf(cm, x[u]);
      const float mn = fmaxf(m, cm);
      float add = 0.0f;
#pragma unroll
      for (int u = 0; u < GRAD_JA; ++u) add += (j0 + u < d) ? expf(x[u] - mn) : 0.0f;
      s = s * expf(m - mn) + add;
      m = mn;
    }
    inv = 1.0f / s;
  }
  float hsum = 0.0f;
  for (int j0 = 0; j0 < d; j0 += GRAD_JC) {
    float x[GRAD_JC];
#pragma unroll
    for (int u = 0; u < GRAD_JC; ++u) x[u] = a.F[(int64_t)(j0 + u < d ? j0 + u : d - 1) * a.ld_f + rc];
    uint8_t yb[GRAD_JC];
    if constexpr (LOSS == SB_LOSS_SIGMOID_BCE) {
#pragma unroll
      for (int u = 0; u < GRAD_JC; ++u) yb[u] = a.Y[(int64_t)(j0 + u < d ? j0 + u : d - 1) * a.ld_y + rc];
    }
#pragma unroll
    for (int u = 0; u < GRAD_JC; ++u) {
      const int j = j0 + u;
      const int jj = j < d ? j : d - 1;
      float g, hh;
      if constexpr (LOSS == SB_LOSS_SOFTMAX_CE) {
        const float p = expf(x[u] - m) * inv;
        g = (jj == y) ? p - 1.0f : p;
        hh = p * (1.0f - p);
      } else {
        // e = exp(-|a|) never overflows, so s keeps its relative accuracy
        // for scores far below zero (down to fp32's subnormals)
        const float e = expf(-fabsf(x[u]));
        const float sg = x[u] >= 0.0f ? 1.0f / (1.0f + e) : e / (1.0f + e);
        g = sg - (float)yb[u];
        hh = sg * (1.0f - sg);
      }
      if (ok) {
        a.G[(int64_t)jj * a.ld_g + row] = g;
        if (HESS) a.hess[(int64_t)jj * a.ld_h + row] = hh;
      }
      hsum += (j < d) ? hh : 0.0f;
      gbuf[u][tid] = ok ? g : 0.0f;
    }
    if (a.npart) {
      lds_sync();
      // 16 threads per column, 16 rows each; lanes c*16 .. c*16+15 share column c
      const int c = tid >> 4, seg = tid & 15;
      const float4* src = reinterpret_cast<const float4*>(&gbuf[c][seg * 16]);
      double acc = 0.0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = src[q];
        acc += (double)v.x * v.x;
        acc += (double)v.y * v.y;
        acc += (double)v.z * v.z;
        acc += (double)v.w * v.w;
      }
      acc = row16_sum(acc);  // in the row's last lane
      if (seg == 15 && j0 + c < d) {
        const int tile = (int)(base / GRAD_THREADS);
        double* pp = a.npart + (int64_t)(j0 + c) * a.n_parts + tile % a.n_parts;
        *pp = tile < a.n_parts ? acc : *pp + acc;  // the slot's first tile writes it
      }
      lds_sync();
    }
  }
  if (a.h_row && ok) a.h_row[row] = hsum * (1.0f / (float)d);
}

template <int LOSS>
__global__ void __launch_bounds__(GRAD_THREADS) k_grad(GradArgs a) {
  __shared__ __align__(16) float gbuf[GRAD_JC][GRAD_THREADS];
  for (int tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
    int d = a.d;
    asm volatile("" : "+s"(d));
    const int64_t base = (int64_t)tile * GRAD_THREADS;
    const bool full = base + GRAD_THREADS <= a.n;
    if (a.hess) {
      if (full) grad_tile<LOSS, true, true>(a, gbuf, base, d);
      else grad_tile<LOSS, false, true>(a, gbuf, base, d);
    } else {
      if (full) grad_tile<LOSS, true, false>(a, gbuf, base, d);
      else grad_tile<LOSS, false, false>(a, gbuf, base, d);
    }
  }
}

// Softmax cross-entropy with the row's d <= DMAX scores held in registers:
// F is read once.  Columns past d load column d-1 (the maximum is unchanged
// and the sum skips them), so every load is unconditional and all of them
// are in flight together.  The maximum is exact, the sum of exp(a - max) is
// taken in column order and its terms are kept for p = exp(a - max) / sum,
// then the second half as in k_grad (stores, the hessians and the
// column-norm staging).  The grid holds as many blocks as fit on the GPU at
// once, each looping over tiles, so no last round of blocks runs part-empty.
//
// The column count d reaches this function opaque to the compiler, and is
// made opaque again between the loads and the stores, so that the
// per-column tests j < d (uniform lane masks) and column offsets are formed
// where they are used instead of all at once and held, spilled, across a
// phase or the tile loop.  Columns past d stay on column d-1 and store
// column d-1's own values there (same address, same value), so the stores
// need no branch; a full tile stores without a row guard.
template <int DMAX, bool FULL, bool HESS, bool UPD>
__device__ inline void grad_softmax_tile(const GradArgs& a, float (*gbuf)[GRAD_THREADS], const double* lv,
                                         int64_t base, int64_t ld_f, int64_t ld_g, int64_t ld_h, int d) {
  const int tid = threadIdx.x;
  const int64_t row = base + tid;
  const bool ok = FULL || row < a.n;
  const int loc = ok ? tid : (int)(a.n - 1 - base);  // rows past the end read row n-1 and store nothing
  const int y = a.labels[base + loc];
  const float* Fb = a.F + base;
  float x[DMAX];
#pragma unroll
  for (int j = 0; j < DMAX; ++j) x[j] = Fb[(int64_t)(j < d ? j : d - 1) * ld_f + loc];
  if constexpr (UPD) {
    // the update of the previous tree, as k_update: fp64 sum, rounded once;
    // columns past d repeat column d-1 and store its own value there
    int L = a.ids[base + loc];
    L = L < a.n_leaves ? L : a.n_leaves - 1;
    const double* lvL = lv + L * a.lv_stride;
    asm volatile("" : "+s"(d));
#pragma unroll
    for (int j = 0; j < DMAX; ++j) x[j] = (float)((double)x[j] + lvL[j < d ? j : d - 1]);
    asm volatile("" : "+s"(d));
    float* Fw = a.F_upd + base;
#pragma unroll
    for (int j = 0; j < DMAX; ++j)
      if (ok) Fw[(int64_t)(j < d ? j : d - 1) * ld_f + tid] = x[j];
    asm volatile("" : "+s"(d));
  }
  float m = x[0];
#pragma unroll
  for (int j = 1; j < DMAX; ++j) m = fmaxf(m, x[j]);
  // x[j] becomes exp(x[j] - max), reused for p below
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < DMAX; ++j) {
    x[j] = expf(x[j] - m);
    s += (j < d) ? x[j] : 0.0f;
  }
  const float inv = 1.0f / s;
  float hsum = 0.0f;
  asm volatile("" : "+s"(d));
  float* Gb = a.G + base;
  float* Hb = HESS ? a.hess + base : nullptr;
#pragma unroll
  for (int j0 = 0; j0 < DMAX; j0 += GRAD_JC) {
    if (j0 >= d) break;
#pragma unroll
    for (int u = 0; u < GRAD_JC; ++u) {
      const int j = j0 + u;
      const int jj = j < d ? j : d - 1;
      const float p = x[j] * inv;
      const float hh = p * (1.0f - p);
      const float g = (jj == y) ? p - 1.0f : p;
      if (ok) {
        Gb[(int64_t)jj * ld_g + tid] = g;
        if (HESS) Hb[(int64_t)jj * ld_h + tid] = hh;
      }
      hsum += (j < d) ? hh : 0.0f;
      gbuf[u][tid] = ok ? g : 0.0f;
    }
    if (a.npart) {
      lds_sync();
      const int c = tid >> 4, seg = tid & 15;
      const float4* src = reinterpret_cast<const float4*>(&gbuf[c][seg * 16]);
      double acc = 0.0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = src[q];
        acc += (double)v.x * v.x;
        acc += (double)v.y * v.y;
        acc += (double)v.z * v.z;
        acc += (double)v.w * v.w;
      }
      acc = row16_sum(acc);  // in the row's last lane
      if (seg == 15 && j0 + c < d) {
        const int tile = (int)(base / GRAD_THREADS);
        double* pp = a.npart + (int64_t)(j0 + c) * a.n_parts + tile % a.n_parts;
        *pp = tile < a.n_parts ? acc : *pp + acc;  // the slot's first tile writes it
      }
      lds_sync();
    }
  }
  if (a.h_row && ok) a.h_row[row] = hsum * (1.0f / (float)d);
}

template <int DMAX, bool UPD>
__global__ void __launch_bounds__(GRAD_THREADS) k_grad_softmax_regs(GradArgs a) {
  __shared__ __align__(16) float gbuf[GRAD_JC][GRAD_THREADS];
  extern __shared__ double lv[];  // UPD: lr * V, [leaf][lv_stride]
  if constexpr (UPD) {
    for (int e = threadIdx.x; e < a.n_leaves * a.d; e += GRAD_THREADS) {
      const int L = e / a.d, j = e - L * a.d;
      lv[L * a.lv_stride + j] = a.lr * a.V[(int64_t)L * a.ld_v + j];
    }
    __syncthreads();
  }
  for (int tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
    const int64_t ld_f = a.ld_f, ld_g = a.ld_g, ld_h = a.ld_h;
    // d as seen by the compiler changes at every tile: the per-column tests
    // j < d are made where they are used, not hoisted out of the tile loop
    // as DMAX lane masks held (spilled) across it
    int d = a.d;
    asm volatile("" : "+s"(d));
    const int64_t base = (int64_t)tile * GRAD_THREADS;
    const bool full = base + GRAD_THREADS <= a.n;
    if (a.hess) {
      if (full) grad_softmax_tile<DMAX, true, true, UPD>(a, gbuf, lv, base, ld_f, ld_g, ld_h, d);
      else grad_softmax_tile<DMAX, false, true, UPD>(a, gbuf, lv, base, ld_f, ld_g, ld_h, d);
    } else {
      if (full) grad_softmax_tile<DMAX, true, false, UPD>(a, gbuf, lv, base, ld_f, ld_g, ld_h, d);
      else grad_softmax_tile<DMAX, false, false, UPD>(a, gbuf, lv, base, ld_f, ld_g, ld_h, d);
    }
  }
}

// One wave per column: lane l adds partials l, l+64, ... in order, then a fixed butterfly.
__global__ void __launch_bounds__(256) k_grad_norm_final(const double* __restrict__ npart, int32_t d, int32_t parts,
                                                         double* __restrict__ norm2) {
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (j >= d) return;
  double s = lane_strided_sum(npart + (int64_t)j * parts, parts, lane);
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) norm2[j] = s;
}

struct UpdArgs {
  float* F;
  int64_t n;
  int32_t d;
  int64_t ld_f;
  const void* ids;
  int32_t n_leaves;
  const double* V;
  int64_t ld_v;
  double lr;
  int32_t jc;  // columns per chunk
  int32_t n_tiles;
};

template <typename LT>
__global__ void __launch_bounds__(UPD_THREADS) k_update(UpdArgs a) {
  // lr * V of the chunk's columns, leaf-major with an odd stride (jc + 1
  // doubles) so that lanes of different leaves fall on different banks
  extern __shared__ double lv[];
  const LT* ids = static_cast<const LT*>(a.ids);
  const int top = a.n_leaves - 1;
  const int stride = a.jc + 1;
  for (int j0 = 0; j0 < a.d; j0 += a.jc) {
    const int w = (a.d - j0 < a.jc) ? a.d - j0 : a.jc;
    __syncthreads();  // the previous chunk's readers are done
    for (int e = threadIdx.x; e < a.n_leaves * a.jc; e += UPD_THREADS) {
      const int L = e / a.jc, u = e - L * a.jc;
      lv[L * stride + u] = u < w ? a.lr * a.V[(int64_t)L * a.ld_v + j0 + u] : 0.0;
    }
    __syncthreads();
    for (int tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
      const int64_t row = (int64_t)tile * UPD_THREADS + threadIdx.x;
      const bool ok = row < a.n;
      const int64_t rc = ok ? row : a.n - 1;
      int L = (int)ids[rc];
      L = L > top ? top : L;
      const double* lvL = lv + L * stride;
      // every load of the chunk first (columns past w repeat the last one),
      // then the sums and the stores
      float f[UPD_JC];
#pragma unroll
      // streamed once (non-temporal): 301 us instead of 328 us at 2M x 100
      for (int u = 0; u < UPD_JC; ++u) f[u] = ld_stream(a.F + (int64_t)(j0 + (u < w ? u : w - 1)) * a.ld_f + rc);
#pragma unroll
      for (int u = 0; u < UPD_JC; ++u)
        if (u < w && ok) a.F[(int64_t)(j0 + u) * a.ld_f + row] = (float)((double)f[u] + lvL[u]);
    }
  }
}

// Blocks of a kernel that fit on the current device at once (at least 1),
// with lds bytes of dynamic LDS per block.
template <typename K>
int resident_blocks(K kernel, int threads, size_t lds = 0) {
  int dev = 0, cus = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, lds) != hipSuccess)
    return GRAD_PARTS;
  const int r = cus * per;
  return r > 0 ? r : 1;
}

// Largest lr * V table (n_leaves x lv_stride doubles) the fused update takes.
constexpr int64_t UPDGRAD_LDS_BYTES = 64 * 1024;

// Grid of a gradient launch over `tiles` tiles, at most `cap` blocks: one
// block per tile up to GRAD_PARTS tiles, else the largest divisor of
// GRAD_PARTS within the cap, so that block b owns the slots b mod grid.
int grad_grid(int64_t tiles, int cap) {
  if (tiles <= GRAD_PARTS) return (int)tiles;
  int g = cap < GRAD_PARTS ? (cap > 1 ? cap : 1) : GRAD_PARTS;
  while (GRAD_PARTS % g) --g;
  return g;
}

// The register softmax kernel for d <= 104, with or without the update (lds:
// the update's table).  Where the rows are wide (DMAX = 104) or the update's
// table takes LDS, the grid is capped at the blocks that fit at once, each
// looping over tiles.
template <bool UPD>
void launch_softmax_regs(const GradArgs& a, size_t lds, hipStream_t st) {
  auto grid = [&](auto kernel, bool wide) {
    if (!wide && !UPD) return grad_grid(a.n_tiles, GRAD_PARTS);
    static thread_local size_t fit_lds = ~size_t(0);  // per-thread cache of the occupancy query
    static thread_local int fit = 0;
    if (fit_lds != lds) {
      fit = resident_blocks(kernel, GRAD_THREADS, lds);
      fit_lds = lds;
    }
    return grad_grid(a.n_tiles, fit);
  };
  if (a.d <= 16) {
    const int b = grid(k_grad_softmax_regs<16, UPD>, false);
    hipLaunchKernelGGL((k_grad_softmax_regs<16, UPD>), dim3(b), dim3(GRAD_THREADS), lds, st, a);
  } else if (a.d <= 32) {
    const int b = grid(k_grad_softmax_regs<32, UPD>, false);
    hipLaunchKernelGGL((k_grad_softmax_regs<32, UPD>), dim3(b), dim3(GRAD_THREADS), lds, st, a);
  } else if (a.d <= 64) {
    const int b = grid(k_grad_softmax_regs<64, UPD>, false);
    hipLaunchKernelGGL((k_grad_softmax_regs<64, UPD>), dim3(b), dim3(GRAD_THREADS), lds, st, a);
  } else {
    const int b = grid(k_grad_softmax_regs<104, UPD>, true);
    hipLaunchKernelGGL((k_grad_softmax_regs<104, UPD>), dim3(b), dim3(GRAD_THREADS), lds, st, a);
  }
}

}  // namespace

int64_t grad_ws_bytes(int64_t n, int32_t d) {
  const int64_t tiles = (n + GRAD_THREADS - 1) / GRAD_THREADS;
  return align256((int64_t)d * (tiles < GRAD_PARTS ? tiles : GRAD_PARTS) * 8);
}

int32_t launch_gradients(int32_t loss, const float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* labels,
                         const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g, float* hess, int64_t ld_hess,
                         float* h_row, double* norm2, void* ws, hipStream_t st) {
  const int64_t tiles = (n + GRAD_THREADS - 1) / GRAD_THREADS;
  const int parts = (int)(tiles < GRAD_PARTS ? tiles : GRAD_PARTS);
  double* npart = norm2 ? static_cast<double*>(ws) : nullptr;
  GradArgs a{loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess, h_row, npart, (int32_t)tiles, parts};
  const int blocks = grad_grid(tiles, GRAD_PARTS);
  if (loss == SB_LOSS_SOFTMAX_CE && d <= 104)
    launch_softmax_regs<false>(a, 0, st);
  else if (loss == SB_LOSS_SOFTMAX_CE)
    hipLaunchKernelGGL(k_grad<SB_LOSS_SOFTMAX_CE>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  else
    hipLaunchKernelGGL(k_grad<SB_LOSS_SIGMOID_BCE>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  if (norm2) hipLaunchKernelGGL(k_grad_norm_final, dim3((d + 3) / 4), dim3(256), 0, st, npart, d, parts, norm2);
  return check_launch("sb_gradients");
}

int64_t update_ws_bytes(int64_t n) { return leaf_ids_bytes(n); }

int32_t launch_update(float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx, const int32_t* leaf_off,
                      int32_t n_leaves, const double* V, int64_t ld_v, double lr, void* ws, hipStream_t st) {
  const int64_t tiles = (n + UPD_THREADS - 1) / UPD_THREADS;
  const int blocks = (int)(tiles < UPD_MAX_BLOCKS ? tiles : UPD_MAX_BLOCKS);
  int jc = UPD_LDS_DOUBLES / n_leaves - 1;  // (jc + 1) doubles per leaf
  if (jc > UPD_JC) jc = UPD_JC;
  if (jc > d) jc = d;
  launch_leaf_ids(row_idx, leaf_off, n_leaves, n, ws, st);
  const UpdArgs a{F, n, d, ld_f, ws, n_leaves, V, ld_v, lr, jc, (int32_t)tiles};
  const size_t lds = (size_t)n_leaves * (jc + 1) * 8;
  if (n_leaves <= 256)
    hipLaunchKernelGGL(k_update<uint8_t>, dim3(blocks), dim3(UPD_THREADS), lds, st, a);
  else
    hipLaunchKernelGGL(k_update<uint16_t>, dim3(blocks), dim3(UPD_THREADS), lds, st, a);
  return check_launch("sb_update_predictions");
}

// Workspace: [norm partials (grad_ws_bytes)][leaf ids (update_ws_bytes)]
int64_t update_gradients_ws_bytes(int64_t n, int32_t d) { return grad_ws_bytes(n, d) + update_ws_bytes(n); }

int32_t launch_update_gradients(int32_t loss, float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                                const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr,
                                const int32_t* labels, const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g,
                                float* hess, int64_t ld_hess, float* h_row, double* norm2, void* ws,
                                hipStream_t st) {
  char* w = static_cast<char*>(ws);
  void* ws_ids = w + grad_ws_bytes(n, d);
  const int stride = d | 1;  // odd: lanes of different leaves fall on different banks
  const int64_t table = (int64_t)n_leaves * stride * 8;
  if (!(loss == SB_LOSS_SOFTMAX_CE && d <= 104 && n_leaves <= 256 && table <= UPDGRAD_LDS_BYTES)) {
    const int32_t rc = launch_update(F, n, d, ld_f, row_idx, leaf_off, n_leaves, V, ld_v, lr, ws_ids, st);
    if (rc) return rc;
    return launch_gradients(loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess, h_row, norm2, ws, st);
  }
  launch_leaf_ids(row_idx, leaf_off, n_leaves, n, ws_ids, st);
  const int64_t tiles = (n + GRAD_THREADS - 1) / GRAD_THREADS;
  const int parts = (int)(tiles < GRAD_PARTS ? tiles : GRAD_PARTS);
  double* npart = norm2 ? reinterpret_cast<double*>(w) : nullptr;
  GradArgs a{loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess, h_row, npart, (int32_t)tiles, parts};
  a.F_upd = F;
  a.ids = static_cast<const uint8_t*>(ws_ids);
  a.n_leaves = n_leaves;
  a.lv_stride = stride;
  a.V = V;
  a.ld_v = ld_v;
  a.lr = lr;
  launch_softmax_regs<true>(a, (size_t)table, st);
  if (norm2) hipLaunchKernelGGL(k_grad_norm_final, dim3((d + 3) / 4), dim3(256), 0, st, npart, d, parts, norm2);
  return check_launch("sb_update_and_gradients");
}

}  // namespace sb
