// Stable row partition of every node of a level (the split that turns leaf R
// into R_left = {bin <= b*} and R_right, Section 2).
//
// A global exclusive prefix L[i] of the "goes left" flags over the level's
// row positions gives every row its destination: with node j owning
// positions [o_j, o_{j+1}) and Lb_j = L[o_j] (= left rows of nodes before j),
//   left  row at i -> o_j + (L[i] - Lb_j)
//   right row at i -> o_j + nleft_j + (i - o_j) - (L[i] - Lb_j),
// which keeps the original order inside each child.
//   k_part_flags   : flag per position (column-major bins: one contiguous run
//                    of a single feature column per node) and left count per
//                    tile of 4096 positions.
//   k_part_scan    : exclusive scan of the tile counts (one block).
//   k_part_bounds  : Lb_j = L[o_j] for every node boundary, from the tile
//                    offset plus the flags of the boundary's own tile.
//   k_part_scatter : block scan of the tile's flags and the scatter; block 0
//                    also writes the child offsets and the next build list.
// No counter is shared between workgroups, so nothing serialises on atomics.
#include "sb_common.h"

namespace sb {
namespace {

constexpr int PT_THREADS = 256;
constexpr int PT_PER_THREAD = 16;
constexpr int PT_TILE = PT_THREADS * PT_PER_THREAD;  // 4096 positions

struct PartArgs {
  const uint8_t* bins_cm;
  int64_t ld_cm;
  const int32_t* row_in;
  const int32_t* off_in;
  const int32_t* best_f;
  const int32_t* best_b;
  int32_t* row_out;
  int32_t* off_out;
  int32_t* build_out;
  uint8_t* flags;
  int32_t* tile_cnt;
  int32_t* tile_off;  // n_tiles + 1 entries (last = total)
  int32_t* Lb;        // n_nodes + 1 entries
  int64_t n;
  int32_t m, n_nodes, n_tiles;
};

__device__ inline int64_t off_at(const PartArgs& a, int j) {
  int64_t v = a.off_in[j];
  return v < 0 ? 0 : (v > a.n ? a.n : v);
}

// node owning position i: largest j in [0, n_nodes) with off[j] <= i
__device__ inline int find_node(const PartArgs& a, int64_t i) {
  int lo = 0, hi = a.n_nodes;  // search over off[0..n_nodes]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (off_at(a, mid) <= i) lo = mid;
    else hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(PT_THREADS) k_part_flags(PartArgs a) {
  __shared__ int32_t wsum[PT_THREADS / 64];
  const int64_t i0 = (int64_t)blockIdx.x * PT_TILE + (int64_t)threadIdx.x * PT_PER_THREAD;
  const int64_t first = off_at(a, 0), last = off_at(a, a.n_nodes);
  int j = find_node(a, i0);
  int64_t jend = off_at(a, j + 1);
  int cnt_tile = 0;
  uint32_t packed[PT_PER_THREAD / 4];
#pragma unroll
  for (int w = 0; w < PT_PER_THREAD / 4; ++w) packed[w] = 0u;
#pragma unroll
  for (int r = 0; r < PT_PER_THREAD; ++r) {
    const int64_t i = i0 + r;
    uint32_t left = 0u;
    if (i < a.n && i >= first && i < last) {
      while (i >= jend && j < a.n_nodes - 1) {
        ++j;
        jend = off_at(a, j + 1);
      }
      int64_t row = a.row_in ? (int64_t)a.row_in[i] : i;
      row = row < 0 ? 0 : (row >= a.n ? a.n - 1 : row);
      const int32_t f = a.best_f[j];
      if (f < 0 || f >= a.m) {
        left = 1u;
      } else {
        left = a.bins_cm[(int64_t)f * a.ld_cm + row] <= a.best_b[j] ? 1u : 0u;
      }
      cnt_tile += (int)left;
    }
    packed[r >> 2] |= left << (8 * (r & 3));
  }
  // 16 flag bytes per thread, written as 4 words (tile base is 4096-aligned)
  if (i0 < a.n) {
    uint32_t* dst = reinterpret_cast<uint32_t*>(a.flags + i0);
#pragma unroll
    for (int w = 0; w < PT_PER_THREAD / 4; ++w) dst[w] = packed[w];
  }
  for (int off = 32; off > 0; off >>= 1) cnt_tile += __shfl_down(cnt_tile, off, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = cnt_tile;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < PT_THREADS / 64; ++w) s += wsum[w];
    a.tile_cnt[blockIdx.x] = s;
  }
}

// Exclusive scan of cnt[0..N) into out[0..N) by one 1024-thread block.
__device__ void block_excl_scan(const int32_t* cnt, int32_t* out, int N, int32_t* sh) {
  const int per = (N + 1023) / 1024;
  const int p0 = threadIdx.x * per;
  int32_t local = 0;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) local += cnt[p0 + i];
  sh[threadIdx.x] = local;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    int32_t v = threadIdx.x >= off ? sh[threadIdx.x - off] : 0;
    __syncthreads();
    sh[threadIdx.x] += v;
    __syncthreads();
  }
  int32_t run = threadIdx.x ? sh[threadIdx.x - 1] : 0;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) {
      out[p0 + i] = run;
      run += cnt[p0 + i];
    }
  __syncthreads();
}

__global__ void __launch_bounds__(1024) k_part_scan(PartArgs a) {
  __shared__ int32_t sh[1024];
  block_excl_scan(a.tile_cnt, a.tile_off, a.n_tiles, sh);
  if (threadIdx.x == 0) a.tile_off[a.n_tiles] = a.tile_off[a.n_tiles - 1] + a.tile_cnt[a.n_tiles - 1];
}

// Lb[j] = number of left rows at positions < off[j], j = 0..n_nodes.
__global__ void __launch_bounds__(PT_THREADS) k_part_bounds(PartArgs a) {
  __shared__ int32_t wsum[PT_THREADS / 64];
  const int j = blockIdx.x;
  const int64_t x = off_at(a, j);
  const int64_t t = x / PT_TILE;
  int cnt = 0;
  if (t < a.n_tiles) {
    const int64_t base = t * PT_TILE;
    for (int64_t i = base + threadIdx.x; i < x; i += PT_THREADS) cnt += a.flags[i];
  }
  for (int off = 32; off > 0; off >>= 1) cnt += __shfl_down(cnt, off, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < PT_THREADS / 64; ++w) s += wsum[w];
    a.Lb[j] = a.tile_off[t < a.n_tiles ? t : a.n_tiles] + (t < a.n_tiles ? s : 0);
  }
}

__global__ void __launch_bounds__(PT_THREADS) k_part_scatter(PartArgs a) {
  __shared__ int32_t sh[PT_THREADS];
  const int64_t i0 = (int64_t)blockIdx.x * PT_TILE + (int64_t)threadIdx.x * PT_PER_THREAD;
  uint32_t packed[PT_PER_THREAD / 4];
  int32_t mine = 0;
  if (i0 < a.n) {
    const uint32_t* src = reinterpret_cast<const uint32_t*>(a.flags + i0);
#pragma unroll
    for (int w = 0; w < PT_PER_THREAD / 4; ++w) {
      packed[w] = src[w];
      mine += __popc(packed[w]);  // flags are 0/1 bytes
    }
  } else {
#pragma unroll
    for (int w = 0; w < PT_PER_THREAD / 4; ++w) packed[w] = 0u;
  }
  // block exclusive scan of the per-thread left counts
  sh[threadIdx.x] = mine;
  __syncthreads();
  for (int off = 1; off < PT_THREADS; off <<= 1) {
    int32_t v = threadIdx.x >= off ? sh[threadIdx.x - off] : 0;
    __syncthreads();
    sh[threadIdx.x] += v;
    __syncthreads();
  }
  int64_t L = (int64_t)a.tile_off[blockIdx.x] + sh[threadIdx.x] - mine;
  if (blockIdx.x == 0) {
    for (int j = threadIdx.x; j < a.n_nodes; j += PT_THREADS) {
      const int64_t o0 = off_at(a, j), o1 = off_at(a, j + 1);
      const int64_t size = o1 > o0 ? o1 - o0 : 0;
      const int64_t nl = (int64_t)a.Lb[j + 1] - a.Lb[j];
      a.off_out[2 * j] = (int32_t)o0;
      a.off_out[2 * j + 1] = (int32_t)(o0 + nl);
      a.build_out[j] = (nl <= size - nl) ? 2 * j : 2 * j + 1;
    }
    if (threadIdx.x == 0) a.off_out[2 * a.n_nodes] = (int32_t)off_at(a, a.n_nodes);
  }
  if (i0 >= a.n) return;
  const int64_t first = off_at(a, 0), last = off_at(a, a.n_nodes);
  int j = find_node(a, i0);
  int64_t jstart = off_at(a, j), jend = off_at(a, j + 1);
#pragma unroll
  for (int r = 0; r < PT_PER_THREAD; ++r) {
    const int64_t i = i0 + r;
    const uint32_t left = (packed[r >> 2] >> (8 * (r & 3))) & 0xffu;
    if (i < a.n && i >= first && i < last) {
      while (i >= jend && j < a.n_nodes - 1) {
        ++j;
        jstart = jend;
        jend = off_at(a, j + 1);
      }
      int64_t row = a.row_in ? (int64_t)a.row_in[i] : i;
      row = row < 0 ? 0 : (row >= a.n ? a.n - 1 : row);
      const int64_t lrel = L - a.Lb[j];
      const int64_t nleft = a.Lb[j + 1] - a.Lb[j];
      int64_t dest = left ? jstart + lrel : jstart + nleft + (i - jstart) - lrel;
      dest = dest < 0 ? 0 : (dest >= a.n ? a.n - 1 : dest);
      a.row_out[dest] = (int32_t)row;
    }
    L += left;
  }
}

}  // namespace

// Workspace: [flags n][tile_cnt][tile_off][Lb]
int64_t partition_ws_bytes(int64_t n, int32_t n_nodes) {
  const int64_t tiles = (n + PT_TILE - 1) / PT_TILE;
  return align256(tiles * PT_TILE) + 2 * align256((tiles + 1) * 4) + align256((int64_t)(n_nodes + 1) * 4);
}

int32_t launch_partition(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm, const int32_t* row_in,
                         const int32_t* off_in, int32_t n_nodes, const int32_t* best_f, const int32_t* best_b,
                         int32_t* row_out, int32_t* off_out, int32_t* build_out, void* ws, hipStream_t st) {
  const int64_t tiles = (n + PT_TILE - 1) / PT_TILE;
  PartArgs a{};
  a.bins_cm = bins_cm;
  a.ld_cm = ld_cm;
  a.row_in = row_in;
  a.off_in = off_in;
  a.best_f = best_f;
  a.best_b = best_b;
  a.row_out = row_out;
  a.off_out = off_out;
  a.build_out = build_out;
  char* w = static_cast<char*>(ws);
  a.flags = reinterpret_cast<uint8_t*>(w);
  w += align256(tiles * PT_TILE);
  a.tile_cnt = reinterpret_cast<int32_t*>(w);
  w += align256((tiles + 1) * 4);
  a.tile_off = reinterpret_cast<int32_t*>(w);
  w += align256((tiles + 1) * 4);
  a.Lb = reinterpret_cast<int32_t*>(w);
  a.n = n;
  a.m = m;
  a.n_nodes = n_nodes;
  a.n_tiles = (int32_t)tiles;
  hipLaunchKernelGGL(k_part_flags, dim3((unsigned)tiles), dim3(PT_THREADS), 0, st, a);
  hipLaunchKernelGGL(k_part_scan, dim3(1), dim3(1024), 0, st, a);
  hipLaunchKernelGGL(k_part_bounds, dim3(n_nodes + 1), dim3(PT_THREADS), 0, st, a);
  hipLaunchKernelGGL(k_part_scatter, dim3((unsigned)tiles), dim3(PT_THREADS), 0, st, a);
  return check_launch("sb_partition_rows");
}

}  // namespace sb
