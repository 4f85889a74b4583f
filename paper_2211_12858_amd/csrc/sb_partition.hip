// Stable row partition of every node of a level (the split that turns leaf R
// into R_left = {bin <= b*} and R_right, Section 2).
//
// A global exclusive prefix L[i] of the "goes left" flags over the level's
// row positions gives every row its destination: with node j owning
// positions [o_j, o_{j+1}) and Lb_j = L[o_j] (= left rows of nodes before j),
//   left  row at i -> o_j + (L[i] - Lb_j)
//   right row at i -> o_j + nleft_j + (i - o_j) - (L[i] - Lb_j),
// which keeps the original order inside each child.
//   k_part_flags   : per tile of PT_TILE positions, the flags as 64-bit wave
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
// For levels of up to PT_LDS_NODES nodes, every block first copies the
// level's node table (offsets, splits, left-count bases) into LDS, so that
// finding a position's node is a search in LDS rather than a chain of
// dependent global loads.
#include <mutex>

#include "sb_common.h"

namespace sb {
namespace {

// Scratch of sb_partition_rows_noalloc: the partition's workspace as a
// device array of the library, for callers that cannot allocate.  Each GPU
// the library runs on holds its own copy until the process ends.  Host code
// never passes the array's name to a kernel: it is a host-side stand-in, and
// the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[PARTITION_SCRATCH_BYTES];
constexpr int MAX_SCRATCH_DEVICES = 64;

constexpr int PT_THREADS = 256;
constexpr int PT_ITERS = 4;
constexpr int PT_TILE = PT_THREADS * PT_ITERS;  // positions per tile
constexpr int PT_MASKS = PT_TILE / 64;          // ballots per tile
static_assert(PT_MASKS >= 1 && PT_MASKS <= 64, "a tile's ballots are counted by one wave");

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
  // level loop: per (node, feature) best score and bin of the fused level
  // end; the flags kernel then picks each node's split and writes it (and
  // its score) to best_f / best_b / best_s
  const double* feat_s;
  const int32_t* feat_b;
  int32_t* out_f;
  int32_t* out_b;
  double* out_s;
  int64_t n;
  int32_t m, n_nodes, n_tiles;
};

__device__ inline int64_t off_at(const PartArgs& a, int j) {
  int64_t v = a.off_in[j];
  return v < 0 ? 0 : (v > a.n ? a.n : v);
}

// Node table of a flags or scatter block.  With SN the level's node offsets
// (clamped to [0, n]) and per-node values are staged in LDS once per block,
// so the node search and the per-node reads are LDS reads rather than
// chains of dependent global loads; levels of more than PT_LDS_NODES nodes
// read them from global memory.
constexpr int PT_LDS_NODES = 2048;
template <bool SN>
struct NodeTab {
  const int32_t* off;
  int64_t n;
  __device__ int64_t at(int j) const {
    if constexpr (SN) return off[j];
    const int64_t v = off[j];
    return v < 0 ? 0 : (v > n ? n : v);
  }
};

// node owning position i: largest j in [0, n_nodes) with off[j] <= i
template <bool SN>
__device__ inline int find_node(const NodeTab<SN>& t, int n_nodes, int64_t i) {
  int lo = 0, hi = n_nodes;  // search over off[0..n_nodes]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (t.at(mid) <= i) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Stage off[0..n_nodes] (clamped) into so; returns the table to search.
template <bool SN>
__device__ inline NodeTab<SN> stage_offsets(const PartArgs& a, int32_t* so) {
  NodeTab<SN> t{a.off_in, a.n};
  if constexpr (SN) {
    for (int j = threadIdx.x; j <= a.n_nodes; j += PT_THREADS) so[j] = (int32_t)off_at(a, j);
    t.off = so;
  }
  return t;
}

__device__ inline int32_t popc64(uint64_t x) { return __popcll(x); }

// Each thread handles the positions t0 + tid + 256*it, it < PT_ITERS.  The
// row indices of all its positions are loaded first, then their bins, so
// each thread keeps PT_ITERS independent loads in flight instead of a chain
// of dependent pairs.  Node offsets and splits come from the block's node table.
template <bool SN>
__global__ void __launch_bounds__(PT_THREADS) k_part_flags(PartArgs a) {
  __shared__ int32_t wsum[PT_THREADS / 64];
  extern __shared__ int32_t pt_nodes[];  // SN: [off: n_nodes + 1][f: n_nodes][b: n_nodes]
  const int64_t t0 = (int64_t)blockIdx.x * PT_TILE;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t row[PT_ITERS];
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t i = t0 + threadIdx.x + (int64_t)it * PT_THREADS;
    const int64_t ic = i < a.n ? i : a.n - 1;
    row[it] = a.row_in ? (int64_t)a.row_in[ic] : ic;
  }
  const NodeTab<SN> tab = stage_offsets<SN>(a, pt_nodes);
  const int32_t* bf = a.best_f;
  const int32_t* bb = a.best_b;
  if constexpr (SN) {
    int32_t* sf = pt_nodes + a.n_nodes + 1;
    int32_t* sb = sf + a.n_nodes;
    for (int j = threadIdx.x; j < a.n_nodes; j += PT_THREADS) {
      sf[j] = a.best_f[j];
      sb[j] = a.best_b[j];
    }
    __syncthreads();
    bf = sf;
    bb = sb;
  }
  const int64_t first = tab.at(0), last = tab.at(a.n_nodes);
  // node of each position (positions grow with it) and its split
  int32_t f_of[PT_ITERS], b_of[PT_ITERS];
  int j = find_node<SN>(tab, a.n_nodes, t0 + threadIdx.x);
  int64_t jend = tab.at(j + 1);
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t i = t0 + threadIdx.x + (int64_t)it * PT_THREADS;
    while (i >= jend && j < a.n_nodes - 1) {
      ++j;
      jend = tab.at(j + 1);
    }
    const int32_t f = bf[j];
    const bool live = i < a.n && i >= first && i < last;
    f_of[it] = (!live) ? -2 : ((f < 0 || f >= a.m) ? -1 : f);
    b_of[it] = bb[j];
  }
  uint32_t bin[PT_ITERS];
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t r = row[it] < 0 ? 0 : (row[it] >= a.n ? a.n - 1 : row[it]);
    bin[it] = f_of[it] >= 0 ? a.bins_cm[(int64_t)f_of[it] * a.ld_cm + r] : 0u;
  }
  int cnt = 0;
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    // terminal node (f = -1): every row goes left; positions outside the nodes (-2) are not flagged
    const bool left = f_of[it] == -1 || (f_of[it] >= 0 && (int32_t)bin[it] <= b_of[it]);
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
// called for every i, and the total is returned to every thread.  Each
// thread scans a contiguous run of per = ceil(N/1024) values; the per-thread
// totals are scanned with wave shuffles and one pass over the 16 wave totals.
template <typename V, typename O>
__device__ int64_t block_excl_scan(int N, V v, O out, int64_t* sh) {
  const int per = (N + 1023) / 1024;
  const int p0 = threadIdx.x * per;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t local = 0;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) local += v(p0 + i);
  int64_t incl = local;
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  __syncthreads();  // sh may still be read by a previous scan
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  int64_t wbase = 0, total = 0;
  for (int w = 0; w < 16; ++w) {
    const int64_t x = sh[w];
    if (w < wave) wbase += x;
    total += x;
  }
  int64_t run = wbase + incl - local;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) {
      out(p0 + i, run);
      run += v(p0 + i);
    }
  return total;
}

// Left rows of a node from its offsets and left-count bases, clamped to its size.
__device__ inline int64_t node_left(int64_t o0, int64_t o1, int64_t lb0, int64_t lb1, int64_t* size_out) {
  const int64_t size = o1 > o0 ? o1 - o0 : 0;
  const int64_t nl = lb1 - lb0;
  *size_out = size;
  return nl < 0 ? 0 : (nl > size ? size : nl);
}

// With SN the node offsets, the tile offsets and the left-count bases are
// also kept in LDS, so that the block's later steps read them there instead
// of going back to global memory (one memory latency each).
constexpr int PB_LDS_TILES = 8192;
template <bool SN>
__global__ void __launch_bounds__(1024) k_part_bounds(PartArgs a) {
  __shared__ int64_t sh[16];
  __shared__ int32_t s_off[SN ? PT_LDS_NODES + 1 : 1], s_lb[SN ? PT_LDS_NODES + 1 : 1];
  __shared__ int32_t s_toff[SN ? PB_LDS_TILES : 1];
  if constexpr (SN)
    for (int j = threadIdx.x; j <= a.n_nodes; j += 1024) s_off[j] = (int32_t)off_at(a, j);
  auto off = [&](int j) -> int64_t {
    if constexpr (SN) return s_off[j];
    else return off_at(a, j);
  };
  auto lb = [&](int j) -> int64_t {
    if constexpr (SN) return s_lb[j];
    else return a.Lb[j];
  };
  // 1. tile offsets
  const int64_t total = block_excl_scan(
      a.n_tiles, [&](int t) -> int64_t { return a.tile_cnt[t]; },
      [&](int t, int64_t pre) {
        a.tile_off[t] = (int32_t)pre;
        if constexpr (SN) s_toff[t] = (int32_t)pre;
      },
      sh);
  if (threadIdx.x == 0) a.tile_off[a.n_tiles] = (int32_t)total;
  __syncthreads();
  // 2. Lb_j = left rows before each node boundary: one wave per boundary,
  // lane q counts the flags of ballot q of the boundary's tile
  {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int j = wave; j <= a.n_nodes; j += 16) {
      const int64_t x = off(j);
      const int64_t t = x / PT_TILE;
      int64_t c = 0;
      if (t < a.n_tiles) {
        const int w = (int)(x - t * PT_TILE);
        const uint64_t mq = lane < PT_MASKS ? a.masks[t * PT_MASKS + lane] : 0;
        if (lane < (w >> 6)) c = popc64(mq);
        else if (lane == (w >> 6) && (w & 63)) c = popc64(mq & ((uint64_t(1) << (w & 63)) - 1));
      }
      for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
      if (lane == 0) {
        int64_t toff;
        if constexpr (SN) toff = t < a.n_tiles ? s_toff[t] : 0;
        else toff = t < a.n_tiles ? a.tile_off[t] : 0;
        const int32_t v = (int32_t)(t < a.n_tiles ? toff + c : total);
        a.Lb[j] = v;
        if constexpr (SN) s_lb[j] = v;
      }
    }
  }
  __syncthreads();
  // 3. children and build list
  for (int j = threadIdx.x; j < a.n_nodes; j += 1024) {
    int64_t size;
    const int64_t o0 = off(j);
    const int64_t nl = node_left(o0, off(j + 1), lb(j), lb(j + 1), &size);
    a.off_out[2 * j] = (int32_t)o0;
    a.off_out[2 * j + 1] = (int32_t)(o0 + nl);
    a.build_out[j] = (nl <= size - nl) ? 2 * j : 2 * j + 1;
  }
  if (threadIdx.x == 0) a.off_out[2 * a.n_nodes] = (int32_t)off(a.n_nodes);
  if (a.next_pre) {
    const int64_t total_built = block_excl_scan(
        a.n_nodes,
        [&](int j) -> int64_t {
          int64_t size;
          const int64_t nl = node_left(off(j), off(j + 1), lb(j), lb(j + 1), &size);
          return nl <= size - nl ? nl : size - nl;
        },
        [&](int j, int64_t pre) { a.next_pre[j] = pre; }, sh);
    if (threadIdx.x == 0) a.next_pre[a.n_nodes] = total_built;
  }
}

template <bool SN>
__global__ void __launch_bounds__(PT_THREADS) k_part_scatter(PartArgs a) {
  __shared__ uint64_t mk[PT_MASKS];
  __shared__ int32_t pre[PT_MASKS];
  extern __shared__ int32_t pt_nodes[];  // SN: [off: n_nodes + 1][Lb: n_nodes + 1]
  const int64_t t0 = (int64_t)blockIdx.x * PT_TILE;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t row[PT_ITERS];
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t i = t0 + threadIdx.x + (int64_t)it * PT_THREADS;
    const int64_t ic = i < a.n ? i : a.n - 1;
    row[it] = a.row_in ? (int64_t)a.row_in[ic] : ic;
  }
  // ballots of the tile and their exclusive prefix, by the first wave
  if (wave == 0) {
    const uint64_t m = lane < PT_MASKS ? a.masks[(int64_t)blockIdx.x * PT_MASKS + lane] : 0;
    const int32_t c = popc64(m);
    int32_t incl = c;
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    if (lane < PT_MASKS) {
      mk[lane] = m;
      pre[lane] = a.tile_off[blockIdx.x] + incl - c;
    }
  }
  const NodeTab<SN> tab = stage_offsets<SN>(a, pt_nodes);
  const int32_t* lb = a.Lb;
  if constexpr (SN) {
    int32_t* sl = pt_nodes + a.n_nodes + 1;
    for (int q = threadIdx.x; q <= a.n_nodes; q += PT_THREADS) sl[q] = a.Lb[q];
    lb = sl;
  }
  __syncthreads();
  const int64_t first = tab.at(0), last = tab.at(a.n_nodes);
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int64_t i = t0 + threadIdx.x;
  int j = find_node<SN>(tab, a.n_nodes, i);
  int64_t jstart = tab.at(j), jend = tab.at(j + 1);
  int64_t lbj = lb[j], nleft = (int64_t)lb[j + 1] - lbj;
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it, i += PT_THREADS) {
    if (i < a.n && i >= first && i < last) {
      while (i >= jend && j < a.n_nodes - 1) {
        ++j;
        jstart = jend;
        jend = tab.at(j + 1);
        lbj = lb[j];
        nleft = (int64_t)lb[j + 1] - lbj;
      }
      const int q = it * (PT_THREADS / 64) + wave;
      const uint64_t m = mk[q];
      const bool left = (m >> lane) & 1u;
      const int64_t L = (int64_t)pre[q] + popc64(m & below);
      const int64_t rw = row[it] < 0 ? 0 : (row[it] >= a.n ? a.n - 1 : row[it]);
      const int64_t lrel = L - lbj;
      int64_t dest = left ? jstart + lrel : jstart + nleft + (i - jstart) - lrel;
      dest = dest < 0 ? 0 : (dest >= a.n ? a.n - 1 : dest);
      a.row_out[dest] = (int32_t)rw;
    }
  }
}

// ---------------------------------------------------------------- two-kernel partition
// For levels of up to PT_LDS_NODES nodes and PB_LDS_TILES tiles the level's
// partition takes two kernels:
//   k_part_flags_pick : the flags and tile counts of k_part_flags; in the
//                       level loop it first picks the split of every node its
//                       tile touches from the fused level end's per-feature
//                       results (the argmax of k_score_node, same order), and
//                       block b writes the split and score of the nodes
//                       j = b (mod grid);
//   k_part_scan_scatter : every block scans the tile counts into LDS, derives
//                       the left-count bases Lb of the node boundaries it
//                       needs from the ballots, and scatters its tiles (one,
//                       or two from about 1.5M rows); block 0 also writes the
//                       child offsets, the build list and the built-size
//                       prefix.
// This replaces the one-block bounds kernel (and the node argmax kernel),
// whose launches and dependent load chains dominated the small levels.

// Exclusive scan over v(0..N-1) by one block of NT threads (NT / 64 waves),
// as block_excl_scan; sh holds NT / 64 values.  Thread t owns the run
// [t * per, (t + 1) * per) and reads each v(i) before it calls out(i, .), so
// out may overwrite v's storage in place.
template <int NT, typename V, typename O>
__device__ int64_t block_scan_nt(int N, V v, O out, int64_t* sh) {
  const int per = (N + NT - 1) / NT;
  const int p0 = threadIdx.x * per;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t local = 0;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) local += v(p0 + i);
  // every partial sum is a count of positions, below 2^31
  const int64_t incl = wave_incl_scan_i32((int32_t)local);
  __syncthreads();
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  int64_t wbase = 0, total = 0;
  for (int w = 0; w < NT / 64; ++w) {
    const int64_t x = sh[w];
    if (w < wave) wbase += x;
    total += x;
  }
  int64_t run = wbase + incl - local;
  for (int i = 0; i < per; ++i)
    if (p0 + i < N) {
      const int64_t x = v(p0 + i);
      out(p0 + i, run);
      run += x;
    }
  return total;
}

template <bool PICK>
__global__ void __launch_bounds__(PT_THREADS) k_part_flags_pick(PartArgs a) {
  __shared__ int32_t wsum[PT_THREADS / 64];
  extern __shared__ int32_t pt_nodes[];  // [off: n_nodes + 1][f: n_nodes][b: n_nodes]
  const int64_t t0 = (int64_t)blockIdx.x * PT_TILE;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t row[PT_ITERS];
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t i = t0 + threadIdx.x + (int64_t)it * PT_THREADS;
    const int64_t ic = i < a.n ? i : a.n - 1;
    row[it] = a.row_in ? (int64_t)a.row_in[ic] : ic;
  }
  const NodeTab<true> tab = stage_offsets<true>(a, pt_nodes);
  int32_t* sf = pt_nodes + a.n_nodes + 1;
  int32_t* sb = sf + a.n_nodes;
  if constexpr (PICK) {
    __syncthreads();  // offsets staged
    // the nodes this tile touches
    const int64_t last_pos = (t0 + PT_TILE < a.n ? t0 + PT_TILE : a.n) - 1;
    const int ja = find_node<true>(tab, a.n_nodes, t0), jb = find_node<true>(tab, a.n_nodes, last_pos);
    for (int j = ja + wave; j <= jb; j += PT_THREADS / 64) {
      int32_t f, b;
      double sc;
      wave_best_feature(a.feat_s + (int64_t)j * a.m, a.feat_b + (int64_t)j * a.m, a.m, &f, &b, &sc);
      if (lane == 0) {
        sf[j] = f;
        sb[j] = b;
      }
    }
    // this block's share of the node results
    for (int j = blockIdx.x + wave * gridDim.x; j < a.n_nodes; j += (PT_THREADS / 64) * gridDim.x) {
      int32_t f, b;
      double sc;
      wave_best_feature(a.feat_s + (int64_t)j * a.m, a.feat_b + (int64_t)j * a.m, a.m, &f, &b, &sc);
      if (lane == 0) {
        a.out_f[j] = f;
        a.out_b[j] = b;
        a.out_s[j] = sc;
      }
    }
  } else {
    for (int j = threadIdx.x; j < a.n_nodes; j += PT_THREADS) {
      sf[j] = a.best_f[j];
      sb[j] = a.best_b[j];
    }
  }
  __syncthreads();
  const int64_t first = tab.at(0), last = tab.at(a.n_nodes);
  int32_t f_of[PT_ITERS], b_of[PT_ITERS];
  int j = find_node<true>(tab, a.n_nodes, t0 + threadIdx.x);
  int64_t jend = tab.at(j + 1);
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t i = t0 + threadIdx.x + (int64_t)it * PT_THREADS;
    while (i >= jend && j < a.n_nodes - 1) {
      ++j;
      jend = tab.at(j + 1);
    }
    const int32_t f = sf[j];
    const bool live = i < a.n && i >= first && i < last;
    f_of[it] = (!live) ? -2 : ((f < 0 || f >= a.m) ? -1 : f);
    b_of[it] = sb[j];
  }
  uint32_t bin[PT_ITERS];
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const int64_t r = row[it] < 0 ? 0 : (row[it] >= a.n ? a.n - 1 : row[it]);
    bin[it] = f_of[it] >= 0 ? a.bins_cm[(int64_t)f_of[it] * a.ld_cm + r] : 0u;
  }
  int cnt = 0;
#pragma unroll
  for (int it = 0; it < PT_ITERS; ++it) {
    const bool left = f_of[it] == -1 || (f_of[it] >= 0 && (int32_t)bin[it] <= b_of[it]);
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

template <int TPB>
__global__ void __launch_bounds__(PT_THREADS) k_part_scan_scatter(PartArgs a) {
  constexpr int NM = PT_MASKS * TPB;  // ballots of the block's tiles
  static_assert(NM <= 64, "one wave scans the block's ballots");
  __shared__ uint64_t mk[NM];
  __shared__ int32_t pre[NM];
  __shared__ int64_t sh[PT_THREADS / 64];
  __shared__ int32_t span[2];
  extern __shared__ int32_t pt_lds[];  // [toff: n_tiles][off: n_nodes + 1][lb: n_nodes + 1]
  int32_t* s_toff = pt_lds;
  int32_t* s_off = s_toff + a.n_tiles;
  int32_t* s_lb = s_off + a.n_nodes + 1;
  const int64_t tile0 = (int64_t)blockIdx.x * TPB;  // the block's first tile
  const int64_t t0 = tile0 * PT_TILE;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t row[PT_ITERS * TPB];
#pragma unroll
  for (int it = 0; it < PT_ITERS * TPB; ++it) {
    const int64_t i = t0 + threadIdx.x + (int64_t)it * PT_THREADS;
    const int64_t ic = i < a.n ? i : a.n - 1;
    row[it] = a.row_in ? (int64_t)a.row_in[ic] : ic;
  }
  for (int j = threadIdx.x; j <= a.n_nodes; j += PT_THREADS) s_off[j] = (int32_t)off_at(a, j);
  uint64_t my_mask = 0;
  if (wave == 0 && lane < NM && tile0 + lane / PT_MASKS < a.n_tiles) my_mask = a.masks[tile0 * PT_MASKS + lane];
  // 1. exclusive prefix of the tile counts (every block its own copy): the
  // counts are staged into LDS with eight loads in flight per thread, then
  // each thread scans a contiguous run of them in place.  With two tiles per
  // block the entries are the counts of tile pairs (half the scan): entry e
  // is the prefix before tile TPB * e
  const int ns = TPB == 1 ? a.n_tiles : (a.n_tiles + 1) / 2;
  for (int t0s = 0; t0s < ns; t0s += 8 * PT_THREADS) {
    int32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = t0s + u * PT_THREADS + threadIdx.x;
      v[u] = 0;
      if (TPB == 1) {
        if (t < ns) v[u] = a.tile_cnt[t];
      } else if (t < ns) {
        // the slot past an odd last tile is allocated; its value is not used
        const int2 pr = reinterpret_cast<const int2*>(a.tile_cnt)[t];
        v[u] = pr.x + (2 * t + 1 < a.n_tiles ? pr.y : 0);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = t0s + u * PT_THREADS + threadIdx.x;
      if (t < ns) s_toff[t] = v[u];
    }
  }
  __syncthreads();
  const int64_t total = block_scan_nt<PT_THREADS>(
      ns, [&](int t) -> int64_t { return s_toff[t]; }, [&](int t, int64_t p) { s_toff[t] = (int32_t)p; }, sh);
  __syncthreads();  // s_toff complete
  // the block's ballots and their prefix
  if (wave == 0) {
    const int32_t c = popc64(my_mask);
    const int32_t incl = wave_incl_scan_i32(c);
    if (lane < NM) {
      mk[lane] = my_mask;
      pre[lane] = s_toff[blockIdx.x] + incl - c;
    }
  }
  __syncthreads();
  const NodeTab<true> tab{s_off, a.n};
  // 2. the node boundaries this block needs: all of them in block 0 (it
  // writes the level's bounds), else those of the nodes its tile touches
  if (threadIdx.x == 0) {
    if (blockIdx.x == 0) {
      span[0] = 0;
      span[1] = a.n_nodes;
    } else {
      const int64_t last_pos = (t0 + PT_TILE * TPB < a.n ? t0 + PT_TILE * TPB : a.n) - 1;
      span[0] = find_node<true>(tab, a.n_nodes, t0);
      span[1] = find_node<true>(tab, a.n_nodes, last_pos) + 1;
    }
  }
  __syncthreads();
  const int J0 = span[0], J1 = span[1];
  // Lb_j = left flags before position off[j]: the tile offset of its tile
  // plus the popcounts of the ballots before it.  PT_MASKS consecutive lanes
  // share a boundary (one ballot each, one row of 16 lanes) and add their
  // counts in registers, the sum ending in the row's last lane.
  static_assert(PT_MASKS == 16 && PT_THREADS % 64 == 0, "a boundary's ballots fill one row of 16 lanes");
  const int nb = J1 - J0 + 1;
  for (int e0 = 0; e0 < nb * PT_MASKS; e0 += PT_THREADS) {
    const int e = e0 + threadIdx.x;
    const int jb = J0 + e / PT_MASKS, q = e % PT_MASKS;
    int32_t c = 0;
    int64_t tx = 0;
    bool in = false;
    if (e < nb * PT_MASKS) {
      const int64_t x = s_off[jb];
      tx = x / PT_TILE;
      in = tx < a.n_tiles;
      if (in) {
        const int w = (int)(x - tx * PT_TILE);
        if (q < (w >> 6) || (q == (w >> 6) && (w & 63))) {
          const uint64_t mq = a.masks[tx * PT_MASKS + q];
          c = q < (w >> 6) ? popc64(mq) : popc64(mq & ((uint64_t(1) << (w & 63)) - 1));
        }
        if (TPB == 2 && q == 0 && (tx & 1)) c += a.tile_cnt[tx - 1];  // the pair's first tile
      }
    }
    c = row16_sum_i32(c);
    if (e < nb * PT_MASKS && q == PT_MASKS - 1) s_lb[jb] = in ? s_toff[tx / TPB] + c : (int32_t)total;
  }
  __syncthreads();
  // 3. block 0: child offsets, build list and the built-size prefix
  if (blockIdx.x == 0) {
    for (int j = threadIdx.x; j < a.n_nodes; j += PT_THREADS) {
      int64_t size;
      const int64_t o0 = s_off[j];
      const int64_t nl = node_left(o0, s_off[j + 1], s_lb[j], s_lb[j + 1], &size);
      a.off_out[2 * j] = (int32_t)o0;
      a.off_out[2 * j + 1] = (int32_t)(o0 + nl);
      a.build_out[j] = (nl <= size - nl) ? 2 * j : 2 * j + 1;
    }
    if (threadIdx.x == 0) a.off_out[2 * a.n_nodes] = s_off[a.n_nodes];
    if (a.next_pre) {
      const int64_t total_built = block_scan_nt<PT_THREADS>(
          a.n_nodes,
          [&](int j) -> int64_t {
            int64_t size;
            const int64_t nl = node_left(s_off[j], s_off[j + 1], s_lb[j], s_lb[j + 1], &size);
            return nl <= size - nl ? nl : size - nl;
          },
          [&](int j, int64_t p) { a.next_pre[j] = p; }, sh);
      if (threadIdx.x == 0) a.next_pre[a.n_nodes] = total_built;
    }
  }
  // 4. scatter of the tile
  const int64_t first = tab.at(0), last = tab.at(a.n_nodes);
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int64_t i = t0 + threadIdx.x;
  int j = find_node<true>(tab, a.n_nodes, i);
  int64_t jstart = tab.at(j), jend = tab.at(j + 1);
  int64_t lbj = s_lb[j], nleft = (int64_t)s_lb[j + 1] - lbj;
#pragma unroll
  for (int it = 0; it < PT_ITERS * TPB; ++it, i += PT_THREADS) {
    if (i < a.n && i >= first && i < last) {
      while (i >= jend && j < a.n_nodes - 1) {
        ++j;
        jstart = jend;
        jend = tab.at(j + 1);
        lbj = s_lb[j];
        nleft = (int64_t)s_lb[j + 1] - lbj;
      }
      const int q = it * (PT_THREADS / 64) + wave;
      const uint64_t m = mk[q];
      const bool left = (m >> lane) & 1u;
      const int64_t L = (int64_t)pre[q] + popc64(m & below);
      const int64_t rw = row[it] < 0 ? 0 : (row[it] >= a.n ? a.n - 1 : row[it]);
      const int64_t lrel = L - lbj;
      int64_t dest = left ? jstart + lrel : jstart + nleft + (i - jstart) - lrel;
      dest = dest < 0 ? 0 : (dest >= a.n ? a.n - 1 : dest);
      a.row_out[dest] = (int32_t)rw;
    }
  }
}

}  // namespace

int32_t partition_scratch(void** out) {
  static std::mutex mu;
  static void* addr[MAX_SCRATCH_DEVICES] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0)
    return fail(SB_E_DEVICE, "sb_partition_rows_noalloc: no current HIP device");
  if (dev >= MAX_SCRATCH_DEVICES)
    return fail(SB_E_UNSUPPORTED, "sb_partition_rows_noalloc: device index " + std::to_string(dev) + " >= 64");
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SB_E_DEVICE, std::string("sb_partition_rows_noalloc: hipGetSymbolAddress failed: ") +
                                   hipGetErrorString(e));
    addr[dev] = p;
  }
  *out = addr[dev];
  return SB_OK;
}

// Workspace: [masks][tile_cnt][tile_off][Lb]
int64_t partition_ws_bytes(int64_t n, int32_t n_nodes) {
  const int64_t tiles = (n + PT_TILE - 1) / PT_TILE;
  return align256(tiles * PT_MASKS * 8) + 2 * align256((tiles + 1) * 4) + align256((int64_t)(n_nodes + 1) * 4);
}

bool partition_picks_splits(int64_t n, int32_t n_nodes) {
  const int64_t tiles = (n + PT_TILE - 1) / PT_TILE;
  return n_nodes <= PT_LDS_NODES && tiles <= PB_LDS_TILES;
}

int32_t launch_partition(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm, const int32_t* row_in,
                         const int32_t* off_in, int32_t n_nodes, const int32_t* best_f, const int32_t* best_b,
                         int32_t* row_out, int32_t* off_out, int32_t* build_out, void* ws, hipStream_t st,
                         int64_t* next_pre, const double* feat_s, const int32_t* feat_b, double* best_s) {
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
  if (partition_picks_splits(n, n_nodes)) {
    const size_t lf = (size_t)(3 * n_nodes + 1) * 4, ls = (size_t)(tiles + 2 * (n_nodes + 1)) * 4;
    if (feat_s) {
      a.feat_s = feat_s;
      a.feat_b = feat_b;
      a.out_f = const_cast<int32_t*>(best_f);
      a.out_b = const_cast<int32_t*>(best_b);
      a.out_s = best_s;
      hipLaunchKernelGGL(k_part_flags_pick<true>, dim3((unsigned)tiles), dim3(PT_THREADS), lf, st, a);
    } else {
      hipLaunchKernelGGL(k_part_flags_pick<false>, dim3((unsigned)tiles), dim3(PT_THREADS), lf, st, a);
    }
    // from about 1.5M rows, two tiles per scatter block: every block scans
    // the tile counts, here in pairs, so the scan is half as long and half as
    // many blocks run it (2M rows: 14.4 -> 11.7 us per level; at 1M rows one
    // tile per block is faster)
    if (tiles >= 1536)
      hipLaunchKernelGGL(k_part_scan_scatter<2>, dim3((unsigned)((tiles + 1) / 2)), dim3(PT_THREADS), ls, st, a);
    else
      hipLaunchKernelGGL(k_part_scan_scatter<1>, dim3((unsigned)tiles), dim3(PT_THREADS), ls, st, a);
    return check_launch("sb_partition_rows");
  }
  if (feat_s) return fail(SB_E_UNSUPPORTED, "partition: picking splits needs <= 2048 nodes and <= 8192 tiles");
  if (n_nodes <= PT_LDS_NODES) {
    const size_t lf = (size_t)(3 * n_nodes + 1) * 4, ls = (size_t)(2 * n_nodes + 2) * 4;
    hipLaunchKernelGGL(k_part_flags<true>, dim3((unsigned)tiles), dim3(PT_THREADS), lf, st, a);
    if (tiles <= PB_LDS_TILES) hipLaunchKernelGGL(k_part_bounds<true>, dim3(1), dim3(1024), 0, st, a);
    else hipLaunchKernelGGL(k_part_bounds<false>, dim3(1), dim3(1024), 0, st, a);
    hipLaunchKernelGGL(k_part_scatter<true>, dim3((unsigned)tiles), dim3(PT_THREADS), ls, st, a);
  } else {
    hipLaunchKernelGGL(k_part_flags<false>, dim3((unsigned)tiles), dim3(PT_THREADS), 0, st, a);
    hipLaunchKernelGGL(k_part_bounds<false>, dim3(1), dim3(1024), 0, st, a);
    hipLaunchKernelGGL(k_part_scatter<false>, dim3((unsigned)tiles), dim3(PT_THREADS), 0, st, a);
  }
  return check_launch("sb_partition_rows");
}

}  // namespace sb
