// Stable row partition of every node of a level (the split that turns leaf R
// into R_left = {bin <= b*} and R_right, Section 2).
//
// A global exclusive prefix L[i] of the "goes left" flags over the level's
// row positions gives every row its destination: with node j owning
// positions [o_j, o_{j+1}) and Lb_j = L[o_j] (= left rows of nodes before j),
//   left  row at i -> o_j + (L[i] - Lb_j)
//   right row at i -> o_j + nleft_j + (i - o_j) - (L[i] - Lb_j),
// which keeps the original order inside each child.
//   k_part_flags   : per tile of 4096 positions, the flags as 64-bit wave
//                    ballots (bit = lane = position) and the tile's left count.
//                    Lanes take consecutive positions, so the row-index reads
//                    are coalesced; the bin is one byte of the split feature's
//                    column.
//   k_part_bounds  : one block: tile offsets (scan of the counts), Lb_j at
//                    every node boundary (tile offset + popcounts of the
//                    ballots before it), child offsets and the next build
//                    list.
//   k_part_scatter : per tile, L[i] from the tile offset and the ballots,
//                    then the scatter of the row indices.
// No counter is shared between workgroups, so nothing serialises on atomics.
#include "sb_common.h"

namespace sb {
namespace {

constexpr int PT_THREADS = 256;
constexpr int PT_ITERS = 16;
constexpr int PT_TILE = PT_THREADS * PT_ITERS;  // 4096 positions
constexpr int PT_MASKS = PT_TILE / 64;          // 64 ballots per tile

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
  int64_t* next_pre;    // may be null: prefix of the built children's sizes, for the next level's histograms
  uint64_t* masks;      // n_tiles * PT_MASKS
  int32_t* tile_cnt;    // n_tiles
  int32_t* tile_off;    // n_tiles + 1 entries (last = total)
  int32_t* Lb;          // n_nodes + 1 entries
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

__device__ inline int32_t popc64(uint64_t x) { return __popcll(x); }

__global__ void __launch_bounds__(PT_THREADS) k_part_flags(PartArgs a) {
  __shared__ int32_t wsum[PT_THREADS / 64];
  const int64_t t0 = (int64_t)blockIdx.x * PT_TILE;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t first = off_at(a, 0), last = off_at(a, a.n_nodes);
  int64_t i = t0 + threadIdx.x;
  int j = find_node(a, i);
  int64_t jend = off_at(a, j + 1);
  int cnt = 0;
#pragma unroll 4
  for (int it = 0; it < PT_ITERS; ++it, i += PT_THREADS) {
    bool left = false;
    if (i < a.n && i >= first && i < last) {
      while (i >= jend && j < a.n_nodes - 1) {
        ++j;
        jend = off_at(a, j + 1);
      }
      int64_t row = a.row_in ? (int64_t)a.row_in[i] : i;
      row = row < 0 ? 0 : (row >= a.n ? a.n - 1 : row);
      const int32_t f = a.best_f[j];
      left = (f < 0 || f >= a.m) ? true : (int32_t)a.bins_cm[(int64_t)f * a.ld_cm + row] <= a.best_b[j];
    }
    const uint64_t mask = __ballot(left);
    if (lane == 0) {
      a.masks[(int64_t)blockIdx.x * PT_MASKS + it * (PT_THREADS / 64) + wave] = mask;
      cnt += popc64(mask);
    }
  }
  if (lane == 0) wsum[wave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < PT_THREADS / 64; ++w) s += wsum[w];
    a.tile_cnt[blockIdx.x] = s;
  }
}

// Exclusive scan over v(0..N-1) by one 1024-thread block; out(i, prefix) is
// called for every i, and the total is returned to every thread.
template <typename V, typename O>
__device__ int64_t block_excl_scan(int N, V v, O out, int64_t* sh) {
  const int per = (N + 1023) / 1024;
  const int p0 = threadIdx.x * per;
  int64_t local = 0;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) local += v(p0 + i);
  __syncthreads();
  sh[threadIdx.x] = local;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    int64_t x = threadIdx.x >= off ? sh[threadIdx.x - off] : 0;
    __syncthreads();
    sh[threadIdx.x] += x;
    __syncthreads();
  }
  int64_t run = threadIdx.x ? sh[threadIdx.x - 1] : 0;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) {
      out(p0 + i, run);
      run += v(p0 + i);
    }
  const int64_t total = sh[1023];
  __syncthreads();
  return total;
}

// Left rows of node j, clamped to its size.
__device__ inline int64_t node_left(const PartArgs& a, int j, int64_t* size_out) {
  const int64_t o0 = off_at(a, j), o1 = off_at(a, j + 1);
  const int64_t size = o1 > o0 ? o1 - o0 : 0;
  int64_t nl = (int64_t)a.Lb[j + 1] - a.Lb[j];
  *size_out = size;
  return nl < 0 ? 0 : (nl > size ? size : nl);
}

__global__ void __launch_bounds__(1024) k_part_bounds(PartArgs a) {
  __shared__ int64_t sh[1024];
  // 1. tile offsets
  const int64_t total = block_excl_scan(
      a.n_tiles, [&](int t) -> int64_t { return a.tile_cnt[t]; },
      [&](int t, int64_t pre) { a.tile_off[t] = (int32_t)pre; }, sh);
  if (threadIdx.x == 0) a.tile_off[a.n_tiles] = (int32_t)total;
  __syncthreads();
  // 2. Lb_j = left rows before each node boundary
  for (int j = threadIdx.x; j <= a.n_nodes; j += 1024) {
    const int64_t x = off_at(a, j);
    const int64_t t = x / PT_TILE;
    int64_t lb;
    if (t >= a.n_tiles) {
      lb = total;
    } else {
      const int w = (int)(x - t * PT_TILE);
      const uint64_t* mk = a.masks + t * PT_MASKS;
      lb = a.tile_off[t];
      for (int q = 0; q < (w >> 6); ++q) lb += popc64(mk[q]);
      if (w & 63) lb += popc64(mk[w >> 6] & ((uint64_t(1) << (w & 63)) - 1));
    }
    a.Lb[j] = (int32_t)lb;
  }
  __syncthreads();
  // 3. children and build list
  for (int j = threadIdx.x; j < a.n_nodes; j += 1024) {
    int64_t size;
    const int64_t nl = node_left(a, j, &size);
    const int64_t o0 = off_at(a, j);
    a.off_out[2 * j] = (int32_t)o0;
    a.off_out[2 * j + 1] = (int32_t)(o0 + nl);
    a.build_out[j] = (nl <= size - nl) ? 2 * j : 2 * j + 1;
  }
  if (threadIdx.x == 0) a.off_out[2 * a.n_nodes] = (int32_t)off_at(a, a.n_nodes);
  if (a.next_pre) {
    const int64_t total_built = block_excl_scan(
        a.n_nodes,
        [&](int j) -> int64_t {
          int64_t size;
          const int64_t nl = node_left(a, j, &size);
          return nl <= size - nl ? nl : size - nl;
        },
        [&](int j, int64_t pre) { a.next_pre[j] = pre; }, sh);
    if (threadIdx.x == 0) a.next_pre[a.n_nodes] = total_built;
  }
}

__global__ void __launch_bounds__(PT_THREADS) k_part_scatter(PartArgs a) {
  __shared__ uint64_t mk[PT_MASKS];
  __shared__ int32_t pre[PT_MASKS];
  const int64_t t0 = (int64_t)blockIdx.x * PT_TILE;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (threadIdx.x < PT_MASKS) mk[threadIdx.x] = a.masks[(int64_t)blockIdx.x * PT_MASKS + threadIdx.x];
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t r = a.tile_off[blockIdx.x];
    for (int q = 0; q < PT_MASKS; ++q) {
      pre[q] = r;
      r += popc64(mk[q]);
    }
  }
  __syncthreads();
  const int64_t first = off_at(a, 0), last = off_at(a, a.n_nodes);
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int64_t i = t0 + threadIdx.x;
  int j = find_node(a, i);
  int64_t jstart = off_at(a, j), jend = off_at(a, j + 1);
  int64_t lbj = a.Lb[j], nleft = (int64_t)a.Lb[j + 1] - lbj;
#pragma unroll 4
  for (int it = 0; it < PT_ITERS; ++it, i += PT_THREADS) {
    if (i < a.n && i >= first && i < last) {
      while (i >= jend && j < a.n_nodes - 1) {
        ++j;
        jstart = jend;
        jend = off_at(a, j + 1);
        lbj = a.Lb[j];
        nleft = (int64_t)a.Lb[j + 1] - lbj;
      }
      const int q = it * (PT_THREADS / 64) + wave;
      const uint64_t m = mk[q];
      const bool left = (m >> lane) & 1u;
      const int64_t L = (int64_t)pre[q] + popc64(m & below);
      int64_t row = a.row_in ? (int64_t)a.row_in[i] : i;
      row = row < 0 ? 0 : (row >= a.n ? a.n - 1 : row);
      const int64_t lrel = L - lbj;
      int64_t dest = left ? jstart + lrel : jstart + nleft + (i - jstart) - lrel;
      dest = dest < 0 ? 0 : (dest >= a.n ? a.n - 1 : dest);
      a.row_out[dest] = (int32_t)row;
    }
  }
}

}  // namespace

// Workspace: [masks][tile_cnt][tile_off][Lb]
int64_t partition_ws_bytes(int64_t n, int32_t n_nodes) {
  const int64_t tiles = (n + PT_TILE - 1) / PT_TILE;
  return align256(tiles * PT_MASKS * 8) + 2 * align256((tiles + 1) * 4) + align256((int64_t)(n_nodes + 1) * 4);
}

int32_t launch_partition(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm, const int32_t* row_in,
                         const int32_t* off_in, int32_t n_nodes, const int32_t* best_f, const int32_t* best_b,
                         int32_t* row_out, int32_t* off_out, int32_t* build_out, void* ws, hipStream_t st,
                         int64_t* next_pre) {
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
  a.next_pre = next_pre;
  char* w = static_cast<char*>(ws);
  a.masks = reinterpret_cast<uint64_t*>(w);
  w += align256(tiles * PT_MASKS * 8);
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
  hipLaunchKernelGGL(k_part_bounds, dim3(1), dim3(1024), 0, st, a);
  hipLaunchKernelGGL(k_part_scatter, dim3((unsigned)tiles), dim3(PT_THREADS), 0, st, a);
  return check_launch("sb_partition_rows");
}

}  // namespace sb
