// The three device layouts of a binned dataset, built once from a row-major
// bin matrix: quad-major words (histograms), column-major bytes (partition)
// and row records (histograms of the deeper levels).  Setup work, outside the per-tree path.
#include "sb_common.h"

namespace sb {
namespace {

constexpr int LAYOUT_THREADS = 256;
constexpr int64_t LAYOUT_MAX_BLOCKS = 65536;

__global__ void __launch_bounds__(LAYOUT_THREADS)
k_layout_quad(const uint8_t* __restrict__ bins, int64_t n, int m, int64_t ld_bins, uint32_t* __restrict__ bins4,
              int64_t ld4) {
  const int nq = (m + 3) / 4;
  const int64_t total = (int64_t)nq * n;
  for (int64_t e = (int64_t)blockIdx.x * LAYOUT_THREADS + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * LAYOUT_THREADS) {
    const int64_t q = e / n, i = e - q * n;
    uint32_t w = 0u;
    for (int u = 0; u < 4; ++u) {
      const int64_t f = 4 * q + u;
      if (f < m) w |= (uint32_t)bins[i * ld_bins + f] << (8 * u);
    }
    bins4[q * ld4 + i] = w;
  }
}

__global__ void __launch_bounds__(LAYOUT_THREADS)
k_layout_cm(const uint8_t* __restrict__ bins, int64_t n, int m, int64_t ld_bins, uint8_t* __restrict__ bins_cm,
            int64_t ld_cm) {
  const int64_t total = (int64_t)m * n;
  for (int64_t e = (int64_t)blockIdx.x * LAYOUT_THREADS + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * LAYOUT_THREADS) {
    const int64_t f = e / n, i = e - f * n;
    bins_cm[f * ld_cm + i] = bins[i * ld_bins + f];
  }
}

__global__ void __launch_bounds__(LAYOUT_THREADS)
k_layout_rec(const uint8_t* __restrict__ bins, int64_t n, int m, int64_t ld_bins, uint8_t* __restrict__ rec,
             int64_t ld_rec) {
  const int64_t total = (int64_t)m * n;
  for (int64_t e = (int64_t)blockIdx.x * LAYOUT_THREADS + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * LAYOUT_THREADS) {
    const int64_t i = e / m, f = e - i * m;
    rec[i * ld_rec + f] = bins[i * ld_bins + f];
  }
}

unsigned layout_blocks(int64_t total) {
  int64_t b = (total + LAYOUT_THREADS - 1) / LAYOUT_THREADS;
  if (b < 1) b = 1;
  if (b > LAYOUT_MAX_BLOCKS) b = LAYOUT_MAX_BLOCKS;
  return (unsigned)b;
}

}  // namespace

int32_t launch_layout(const uint8_t* bins, int64_t n, int32_t m, int64_t ld_bins, uint32_t* bins4, int64_t ld4,
                      uint8_t* bins_cm, int64_t ld_cm, uint8_t* rec, int64_t ld_rec, hipStream_t st) {
  const int64_t nq = (m + 3) / 4;
  if (bins4)
    hipLaunchKernelGGL(k_layout_quad, dim3(layout_blocks(nq * n)), dim3(LAYOUT_THREADS), 0, st, bins, n, m, ld_bins,
                       bins4, ld4);
  if (bins_cm)
    hipLaunchKernelGGL(k_layout_cm, dim3(layout_blocks((int64_t)m * n)), dim3(LAYOUT_THREADS), 0, st, bins, n, m,
                       ld_bins, bins_cm, ld_cm);
  if (rec)
    hipLaunchKernelGGL(k_layout_rec, dim3(layout_blocks((int64_t)m * n)), dim3(LAYOUT_THREADS), 0, st, bins, n, m,
                       ld_bins, rec, ld_rec);
  return check_launch("sb_layout_bins");
}

}  // namespace sb
