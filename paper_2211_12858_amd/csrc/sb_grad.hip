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
//   rows each in fp64, a fixed butterfly joins them, and one thread adds the
//   tile's sum to the block's partial (a fixed order).  k_grad_norm_final adds
//   the blocks' partials in a fixed order, so the norms are deterministic.
// k_update: F[i, j] += lr * V[leaf of i, j] in fp64, rounded once to fp32.
//   lr * V of a chunk of columns is staged in LDS; the leaf ids come from the
//   leaf segments (k_leaf_ids, shared with the leaf values).
#include <cmath>

#include "sb_common.h"
#include "sb_leaf_ids.h"

namespace sb {
namespace {

constexpr int GRAD_THREADS = 256;
constexpr int GRAD_JA = 8;          // columns per load batch of the softmax first pass
constexpr int GRAD_JC = 16;         // columns per chunk of the second pass (norm staging)
constexpr int GRAD_MAX_BLOCKS = 2048;
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
  double* npart;  // [d][blocks] or NULL
  int32_t n_tiles;
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
__device__ inline void grad_tile(const GradArgs& a, float (*gbuf)[GRAD_THREADS], int64_t base, bool first, int d) {
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
      for (int off = 8; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
      if (seg == 0 && j0 + c < d) {
        double* pp = a.npart + (int64_t)(j0 + c) * gridDim.x + blockIdx.x;
        *pp = first ? acc : *pp + acc;
      }
      lds_sync();
    }
  }
  if (a.h_row && ok) a.h_row[row] = hsum * (1.0f / (float)d);
}

template <int LOSS>
__global__ void __launch_bounds__(GRAD_THREADS) k_grad(GradArgs a) {
  __shared__ __align__(16) float gbuf[GRAD_JC][GRAD_THREADS];
  bool first = true;
  for (int tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
    int d = a.d;
    asm volatile("" : "+s"(d));
    const int64_t base = (int64_t)tile * GRAD_THREADS;
    const bool full = base + GRAD_THREADS <= a.n;
    if (a.hess) {
      if (full) grad_tile<LOSS, true, true>(a, gbuf, base, first, d);
      else grad_tile<LOSS, false, true>(a, gbuf, base, first, d);
    } else {
      if (full) grad_tile<LOSS, true, false>(a, gbuf, base, first, d);
      else grad_tile<LOSS, false, false>(a, gbuf, base, first, d);
    }
    first = false;
  }
  // a block without tiles still defines its partials
  if (a.npart && first)
    for (int j = threadIdx.x; j < a.d; j += GRAD_THREADS) a.npart[(int64_t)j * gridDim.x + blockIdx.x] = 0.0;
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
template <int DMAX, bool FULL, bool HESS>
__device__ inline void grad_softmax_tile(const GradArgs& a, float (*gbuf)[GRAD_THREADS], int64_t base, bool first,
                                         int64_t ld_f, int64_t ld_g, int64_t ld_h, int d) {
  const int tid = threadIdx.x;
  const int64_t row = base + tid;
  const bool ok = FULL || row < a.n;
  const int loc = ok ? tid : (int)(a.n - 1 - base);  // rows past the end read row n-1 and store nothing
  const int y = a.labels[base + loc];
  const float* Fb = a.F + base;
  float x[DMAX];
#pragma unroll
  for (int j = 0; j < DMAX; ++j) x[j] = Fb[(int64_t)(j < d ? j : d - 1) * ld_f + loc];
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
      for (int off = 8; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
      if (seg == 0 && j0 + c < d) {
        double* pp = a.npart + (int64_t)(j0 + c) * gridDim.x + blockIdx.x;
        *pp = first ? acc : *pp + acc;
      }
      lds_sync();
    }
  }
  if (a.h_row && ok) a.h_row[row] = hsum * (1.0f / (float)d);
}

template <int DMAX>
__global__ void __launch_bounds__(GRAD_THREADS) k_grad_softmax_regs(GradArgs a) {
  __shared__ __align__(16) float gbuf[GRAD_JC][GRAD_THREADS];
  bool first = true;
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
      if (full) grad_softmax_tile<DMAX, true, true>(a, gbuf, base, first, ld_f, ld_g, ld_h, d);
      else grad_softmax_tile<DMAX, false, true>(a, gbuf, base, first, ld_f, ld_g, ld_h, d);
    } else {
      if (full) grad_softmax_tile<DMAX, true, false>(a, gbuf, base, first, ld_f, ld_g, ld_h, d);
      else grad_softmax_tile<DMAX, false, false>(a, gbuf, base, first, ld_f, ld_g, ld_h, d);
    }
    first = false;
  }
  if (a.npart && first)
    for (int j = threadIdx.x; j < a.d; j += GRAD_THREADS) a.npart[(int64_t)j * gridDim.x + blockIdx.x] = 0.0;
}

// One wave per column: lane l adds partials l, l+64, ... in order, then a fixed butterfly.
__global__ void __launch_bounds__(256) k_grad_norm_final(const double* __restrict__ npart, int32_t d, int32_t parts,
                                                         double* __restrict__ norm2) {
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (j >= d) return;
  double s = 0.0;
  for (int p = lane; p < parts; p += 64) s += npart[(int64_t)j * parts + p];
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

}  // namespace

int64_t grad_ws_bytes(int64_t n, int32_t d) {
  const int64_t tiles = (n + GRAD_THREADS - 1) / GRAD_THREADS;
  const int64_t blocks = tiles < GRAD_MAX_BLOCKS ? tiles : GRAD_MAX_BLOCKS;
  return align256((int64_t)d * blocks * 8);
}

// Blocks of a kernel that fit on the current device at once (at least 1).
template <typename K>
int resident_blocks(K kernel, int threads) {
  int dev = 0, cus = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, 0) != hipSuccess)
    return GRAD_MAX_BLOCKS;
  const int r = cus * per;
  return r > 0 ? r : 1;
}

int32_t launch_gradients(int32_t loss, const float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* labels,
                         const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g, float* hess, int64_t ld_hess,
                         float* h_row, double* norm2, void* ws, hipStream_t st) {
  const int64_t tiles = (n + GRAD_THREADS - 1) / GRAD_THREADS;
  int blocks = (int)(tiles < GRAD_MAX_BLOCKS ? tiles : GRAD_MAX_BLOCKS);
  if (loss == SB_LOSS_SOFTMAX_CE && d <= 104 && d > 64) {
    static thread_local int fit = 0;  // per-thread cache of the occupancy query
    if (!fit) fit = resident_blocks(k_grad_softmax_regs<104>, GRAD_THREADS);
    if (fit < blocks) blocks = fit;
  }
  double* npart = norm2 ? static_cast<double*>(ws) : nullptr;
  const GradArgs a{loss, F, n, d, ld_f, labels, Y, ld_y, G, ld_g, hess, ld_hess, h_row, npart, (int32_t)tiles};
  if (loss == SB_LOSS_SOFTMAX_CE && d <= 16)
    hipLaunchKernelGGL(k_grad_softmax_regs<16>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  else if (loss == SB_LOSS_SOFTMAX_CE && d <= 32)
    hipLaunchKernelGGL(k_grad_softmax_regs<32>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  else if (loss == SB_LOSS_SOFTMAX_CE && d <= 64)
    hipLaunchKernelGGL(k_grad_softmax_regs<64>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  else if (loss == SB_LOSS_SOFTMAX_CE && d <= 104)
    hipLaunchKernelGGL(k_grad_softmax_regs<104>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  else if (loss == SB_LOSS_SOFTMAX_CE)
    hipLaunchKernelGGL(k_grad<SB_LOSS_SOFTMAX_CE>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  else
    hipLaunchKernelGGL(k_grad<SB_LOSS_SIGMOID_BCE>, dim3(blocks), dim3(GRAD_THREADS), 0, st, a);
  if (norm2) hipLaunchKernelGGL(k_grad_norm_final, dim3((d + 3) / 4), dim3(256), 0, st, npart, d, blocks, norm2);
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

}  // namespace sb
