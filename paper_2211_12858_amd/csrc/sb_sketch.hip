// Gradient sketches of Section 3 on gfx950.
//
//   k_colnorm_partial / k_colnorm_final : ||g_j||^2 in fp64, fixed reduction
//       order (Section 3.1 ranks columns by norm; Section 3.2 samples with
//       p_j proportional to it).
//   k_select   : Top Outputs ranks, Random Sampling inverse-CDF draws from
//       given uniforms, identity.
//   k_pack     : GH[i, t] = fp32(G[i, col_t] * scale_t), GH[i, k] = h_i, plus
//       the per-channel max |value| for the fixed-point histogram exponents.
//   k_project  : GH[i, 0:k] = G[i, :] Pi (Section 3.3), fp32 accumulation.
//
// G is column-major, so every kernel reads whole columns with lanes on
// consecutive rows (coalesced 256-byte wave loads).
#include "sb_common.h"

namespace sb {
namespace {

constexpr int NORM_THREADS = 256;
constexpr int64_t NORM_CHUNK = 16384;  // rows per partial sum
constexpr int NORM_MAX_PARTS = 256;

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
    const int64_t nv = (i1 - i0) >> 2;
    const float4* v4 = reinterpret_cast<const float4*>(col + i0);
    for (int64_t q = threadIdx.x; q < nv; q += NORM_THREADS) {
      float4 x = v4[q];
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
  double s = 0.0;
  for (int p = lane; p < parts; p += 64) s += part[(int64_t)j * parts + p];
  s = wave_sum(s);
  if (lane == 0) {
    n2[j] = s;
    if (n2_user) n2_user[j] = s;
  }
}

// One block.  Also clears the per-channel max bits used by k_pack.
__global__ void __launch_bounds__(1024)
k_select(int kind, const double* __restrict__ n2, int d, int k, const double* __restrict__ u,
         int32_t* __restrict__ cols, float* __restrict__ scales, double* __restrict__ C,
         uint32_t* __restrict__ maxbits) {
  for (int t = threadIdx.x; t <= k; t += blockDim.x) maxbits[t] = 0u;
  if (kind == SB_SKETCH_IDENTITY) {
    for (int t = threadIdx.x; t < k; t += blockDim.x) {
      cols[t] = t;
      scales[t] = 1.0f;
    }
  } else if (kind == SB_SKETCH_TOP_OUTPUTS) {
    // rank of column j in the order (norm descending, index ascending)
    for (int j = threadIdx.x; j < d; j += blockDim.x) {
      const double v = n2[j];
      int rank = 0;
      for (int l = 0; l < d; ++l) {
        const double w = n2[l];
        rank += (w > v) || (w == v && l < j);
      }
      if (rank < k) {
        cols[rank] = j;
        scales[rank] = 1.0f;
      }
    }
  } else if (kind == SB_SKETCH_RANDOM_SAMPLING) {
    if (threadIdx.x == 0) {
      double acc = 0.0;
      for (int j = 0; j < d; ++j) {
        acc = acc + n2[j];
        C[j] = acc;
      }
    }
    __syncthreads();
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

__device__ inline uint32_t wave_max_u32(uint32_t v) {
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = __shfl_down(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

constexpr int PACK_THREADS = 256;
constexpr int PACK_ROWS_PER_THREAD = 4;

// One thread per row and channel loop; |value| maxima per channel go through
// LDS and one global atomicMax per block and channel (order-independent).
__global__ void __launch_bounds__(PACK_THREADS)
k_pack(const float* __restrict__ G, int64_t n, int64_t ld_g, int d, const float* __restrict__ h, int k,
       const int32_t* __restrict__ cols, const float* __restrict__ scales, float* __restrict__ GH, int64_t ld_gh,
       uint32_t* __restrict__ maxbits) {
  extern __shared__ uint32_t smax[];
  for (int t = threadIdx.x; t <= k; t += PACK_THREADS) smax[t] = 0u;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * PACK_THREADS * PACK_ROWS_PER_THREAD + threadIdx.x;
  for (int t = 0; t <= k; ++t) {
    const float* src;
    float sc = 1.0f;
    bool zero = false;
    if (t < k) {
      const int col = cols[t];
      zero = col < 0 || col >= d;  // -1 marks an all-zero sketch column
      src = G + (int64_t)(zero ? 0 : col) * ld_g;
      sc = scales[t];
    } else {
      src = h;
    }
    uint32_t mx = 0u;
#pragma unroll
    for (int r = 0; r < PACK_ROWS_PER_THREAD; ++r) {
      const int64_t i = base + (int64_t)r * PACK_THREADS;
      if (i < n) {
        float v = zero ? 0.0f : (t < k ? src[i] * sc : src[i]);
        GH[i * ld_gh + t] = v;
        const uint32_t a = __float_as_uint(v) & 0x7fffffffu;
        mx = a > mx ? a : mx;
      }
    }
    mx = wave_max_u32(mx);
    if ((threadIdx.x & 63) == 0) atomicMax(&smax[t], mx);
  }
  __syncthreads();
  for (int t = threadIdx.x; t <= k; t += PACK_THREADS)
    if (smax[t]) atomicMax(&maxbits[t], smax[t]);
}

constexpr int PROJ_THREADS = 256;
constexpr int PROJ_KT = 32;  // sketch columns per pass

// VALU projection: one row per thread, Pi read with uniform (scalar) loads.
__global__ void __launch_bounds__(PROJ_THREADS)
k_project(const float* __restrict__ G, int64_t n, int d, int64_t ld_g, const float* __restrict__ Pi, int k,
          const float* __restrict__ h, float* __restrict__ GH, int64_t ld_gh, uint32_t* __restrict__ maxbits) {
  extern __shared__ uint32_t smax[];
  for (int t = threadIdx.x; t <= k; t += PROJ_THREADS) smax[t] = 0u;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * PROJ_THREADS + threadIdx.x;
  const bool live = i < n;
  const int64_t ii = live ? i : 0;
  for (int t0 = 0; t0 < k; t0 += PROJ_KT) {
    float acc[PROJ_KT];
#pragma unroll
    for (int t = 0; t < PROJ_KT; ++t) acc[t] = 0.0f;
    const int kt = (k - t0 < PROJ_KT) ? k - t0 : PROJ_KT;
    for (int j = 0; j < d; ++j) {
      const float g = G[(int64_t)j * ld_g + ii];
      const float* pr = Pi + (int64_t)j * k + t0;
#pragma unroll
      for (int t = 0; t < PROJ_KT; ++t)
        if (t < kt) acc[t] = fmaf(g, pr[t], acc[t]);
    }
#pragma unroll
    for (int t = 0; t < PROJ_KT; ++t) {
      if (t < kt) {
        uint32_t a = 0u;
        if (live) {
          GH[i * ld_gh + t0 + t] = acc[t];
          a = __float_as_uint(acc[t]) & 0x7fffffffu;
        }
        a = wave_max_u32(a);
        if ((threadIdx.x & 63) == 0) atomicMax(&smax[t0 + t], a);
      }
    }
  }
  uint32_t a = 0u;
  if (live) {
    const float hv = h[i];
    GH[i * ld_gh + k] = hv;
    a = __float_as_uint(hv) & 0x7fffffffu;
  }
  a = wave_max_u32(a);
  if ((threadIdx.x & 63) == 0) atomicMax(&smax[k], a);
  __syncthreads();
  for (int t = threadIdx.x; t <= k; t += PROJ_THREADS)
    if (smax[t]) atomicMax(&maxbits[t], smax[t]);
}

__global__ void k_zero_u32(uint32_t* p, int cnt) {
  for (int i = threadIdx.x; i < cnt; i += blockDim.x) p[i] = 0u;
}

// Max |GH[:, t]| over all rows for a caller-supplied GH.
__global__ void __launch_bounds__(256)
k_maxabs(const float* __restrict__ GH, int64_t n, int64_t ld_gh, int c, uint32_t* __restrict__ maxbits) {
  extern __shared__ uint32_t smax[];
  for (int t = threadIdx.x; t < c; t += 256) smax[t] = 0u;
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int t = 0; t < c; ++t) {
    uint32_t mx = 0u;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
      const uint32_t a = __float_as_uint(GH[i * ld_gh + t]) & 0x7fffffffu;
      mx = a > mx ? a : mx;
    }
    mx = wave_max_u32(mx);
    if ((threadIdx.x & 63) == 0) atomicMax(&smax[t], mx);
  }
  __syncthreads();
  for (int t = threadIdx.x; t < c; t += 256)
    if (smax[t]) atomicMax(&maxbits[t], smax[t]);
}

// qexp[t] = (QBITS-1) - floor(log2(max)), 0 for an all-zero channel.
__global__ void k_qexp(const uint32_t* __restrict__ maxbits, int c, int32_t* __restrict__ qexp) {
  for (int t = threadIdx.x; t < c; t += blockDim.x) {
    const float mx = __uint_as_float(maxbits[t]);
    qexp[t] = (mx > 0.0f) ? (QBITS - 1) - ilogbf(mx) : 0;
  }
}

int norm_parts(int64_t n) {
  int64_t p = (n + NORM_CHUNK - 1) / NORM_CHUNK;
  if (p < 1) p = 1;
  if (p > NORM_MAX_PARTS) p = NORM_MAX_PARTS;
  return (int)p;
}

}  // namespace

// Workspace: [norm partials d*P][norm2 d][prefix d][maxbits k+1]
int64_t sketch_ws_bytes(int32_t kind, int64_t n, int32_t d, int32_t k) {
  (void)kind;
  const int P = norm_parts(n);
  return align256((int64_t)d * P * 8) + align256((int64_t)d * 8) * 2 + align256((int64_t)(k + 1) * 4);
}

int32_t launch_sketch(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                      const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols, float* scales,
                      double* norm2, int32_t* qexp, void* ws, hipStream_t st) {
  const int P = norm_parts(n);
  char* w = static_cast<char*>(ws);
  double* part = reinterpret_cast<double*>(w);
  w += align256((int64_t)d * P * 8);
  double* n2 = reinterpret_cast<double*>(w);
  w += align256((int64_t)d * 8);
  double* C = reinterpret_cast<double*>(w);
  w += align256((int64_t)d * 8);
  uint32_t* maxbits = reinterpret_cast<uint32_t*>(w);
  const size_t smax_bytes = (size_t)(k + 1) * 4;

  if (kind == SB_SKETCH_RANDOM_PROJECTION) {
    hipLaunchKernelGGL(k_zero_u32, dim3(1), dim3(256), 0, st, maxbits, k + 1);
    const int64_t blocks = (n + PROJ_THREADS - 1) / PROJ_THREADS;
    hipLaunchKernelGGL(k_project, dim3((unsigned)blocks), dim3(PROJ_THREADS), smax_bytes, st, G, n, d, ld_g, Pi, k,
                       h, GH, ld_gh, maxbits);
  } else {
    int64_t chunk = (n + P - 1) / P;
    chunk = (chunk + 3) & ~int64_t(3);
    hipLaunchKernelGGL(k_colnorm_partial, dim3(P, d), dim3(NORM_THREADS), 0, st, G, n, ld_g, P, chunk, part);
    hipLaunchKernelGGL(k_colnorm_final, dim3((d + 3) / 4), dim3(256), 0, st, part, d, P, n2, norm2);
    hipLaunchKernelGGL(k_select, dim3(1), dim3(1024), 0, st, kind, n2, d, k, u, cols, scales, C, maxbits);
    const int64_t rows_per_block = (int64_t)PACK_THREADS * PACK_ROWS_PER_THREAD;
    const int64_t blocks = (n + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL(k_pack, dim3((unsigned)blocks), dim3(PACK_THREADS), smax_bytes, st, G, n, ld_g, d, h, k, cols,
                       scales, GH, ld_gh, maxbits);
  }
  hipLaunchKernelGGL(k_qexp, dim3(1), dim3(256), 0, st, maxbits, k + 1, qexp);
  return check_launch("sb_sketch");
}

int32_t launch_hist_exponents(const float* GH, int64_t n, int64_t ld_gh, int32_t k, int32_t* qexp, void* ws,
                              hipStream_t st) {
  uint32_t* maxbits = static_cast<uint32_t*>(ws);
  hipLaunchKernelGGL(k_zero_u32, dim3(1), dim3(256), 0, st, maxbits, k + 1);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_maxabs, dim3((unsigned)blocks), dim3(256), (size_t)(k + 1) * 4, st, GH, n, ld_gh, k + 1,
                     maxbits);
  hipLaunchKernelGGL(k_qexp, dim3(1), dim3(256), 0, st, maxbits, k + 1, qexp);
  return check_launch("sb_hist_exponents");
}

}  // namespace sb
