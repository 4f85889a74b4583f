// Leaf id of every row from the leaf segments of a grown tree: row
// row_idx[p] belongs to the last leaf L with leaf_off[L] <= p (empty leaves
// are skipped).  The offsets are searched in LDS.  Ids are 1 byte for up to
// 256 leaves, else 2.  Row indices are clamped into [0, n), so bad input
// cannot write outside the id array.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace sb {

constexpr int LEAF_IDS_MAX_LEAVES = 4096;

template <typename LT>
__global__ void __launch_bounds__(256) k_leaf_ids(const int32_t* __restrict__ row_idx,
                                                   const int32_t* __restrict__ leaf_off, int32_t n_leaves, int64_t n,
                                                   LT* __restrict__ ids) {
  __shared__ int32_t soff[LEAF_IDS_MAX_LEAVES];
  for (int L = threadIdx.x; L < n_leaves; L += blockDim.x) soff[L] = leaf_off[L];
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n; p += stride) {
    int lo = 0, hi = n_leaves - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((int64_t)soff[mid] <= p)
        lo = mid;
      else
        hi = mid - 1;
    }
    int64_t r = row_idx[p];
    r = r < 0 ? 0 : (r >= n ? n - 1 : r);
    ids[r] = (LT)lo;
  }
}

// Bytes of the id array (2 per row covers both widths).
inline int64_t leaf_ids_bytes(int64_t n) { return (n * 2 + 255) & ~int64_t(255); }

// Enqueue k_leaf_ids with 1-byte ids when n_leaves <= 256, else 2-byte ids.
inline void launch_leaf_ids(const int32_t* row_idx, const int32_t* leaf_off, int32_t n_leaves, int64_t n, void* ids,
                            hipStream_t st) {
  const int64_t b = (n + 255) / 256;
  const unsigned blocks = (unsigned)(b < 2048 ? b : 2048);
  if (n_leaves <= 256)
    hipLaunchKernelGGL(k_leaf_ids<uint8_t>, dim3(blocks), dim3(256), 0, st, row_idx, leaf_off, n_leaves, n,
                       static_cast<uint8_t*>(ids));
  else
    hipLaunchKernelGGL(k_leaf_ids<uint16_t>, dim3(blocks), dim3(256), 0, st, row_idx, leaf_off, n_leaves, n,
                       static_cast<uint16_t*>(ids));
}

}  // namespace sb
