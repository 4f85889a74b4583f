// Per-node histograms of one tree level (Section 3.4) and sibling subtraction.
//
// Design for gfx950 (measured: ds_add_f32 retires ~0.33 lanes/clk/CU while
// ds_add_u32 retires 10-14 lanes/clk/CU):
//  * every sketch value is quantised to an integer rint(v * 2^qexp[t]) of
//    magnitude <= 2^QBITS and accumulated with int32 LDS atomics;
//  * each LDS cell is a running sum modulo 2^32.  Its owner thread reads it
//    back every window of <= WINDOW_ROWS rows and adds the wrapped difference
//    into an int64 register total, so no cell can overflow;
//  * a workgroup owns one feature slice (F features, LDS = F*B*(k+1) int32
//    cells) and a contiguous range of the rows of the built nodes, taken in
//    build-list order; it writes one int64 partial per node it touched;
//  * k_hist_reduce sums the partials of each node (integer, so the result is
//    independent of the grid and of the order of the atomics) and writes the
//    fp64 histogram.  Sums of fixed-point values are exact in fp64, which
//    makes sibling subtraction exact as well.
// Workgroups that share a row range but own different slices are placed on
// the same XCD (dispatch is round-robin over the 8 XCDs by block index) so
// the rows they all read stay in that XCD's L2.
#include "sb_common.h"

namespace sb {

HistPlan hist_plan(int32_t m, int32_t n_bins, int32_t k, int32_t n_build) {
  HistPlan p{};
  p.c = k + 1;
  const int64_t quad_bytes = 4ll * n_bins * p.c * 4;
  int nq_max = (int)(HIST_LDS_BYTES / quad_bytes);
  const int quads_total = (m + 3) / 4;
  if (nq_max > quads_total) nq_max = quads_total;
  if (nq_max > 64) nq_max = 64;
  if (nq_max < 1) nq_max = 0;  // does not fit: caller rejects
  if (nq_max == 0) return p;
  p.slices = (quads_total + nq_max - 1) / nq_max;
  p.nq = (quads_total + p.slices - 1) / p.slices;
  p.f = 4 * p.nq;
  p.rows_wave = 64 / p.nq;
  p.cells = p.f * n_bins * p.c;
  int q = 256 / p.slices;
  if (q < 1) q = 1;
  p.q = q;
  p.q_pad = (q + 7) & ~7;
  p.slots = (int64_t)q + n_build;
  return p;
}

// Workspace: [pre: n_build+1 int64][partials: slices * slots * cells int64]
int64_t hist_ws_bytes(int32_t m, int32_t n_bins, int32_t k, int32_t n_build) {
  HistPlan p = hist_plan(m, n_bins, k, n_build);
  if (p.nq == 0) return -1;
  return align256((int64_t)(n_build + 1) * 8) + align256((int64_t)p.slices * p.slots * p.cells * 8);
}

namespace {

struct HistArgs {
  const uint8_t* bins;
  int64_t ld_bins;
  const float* GH;
  int64_t ld_gh;
  const int32_t* qexp;
  const int32_t* row_idx;
  const int32_t* node_off;
  const int32_t* build_list;
  int64_t* pre;
  int64_t* partial;
  double* H;
  int64_t n;
  int32_t m, n_bins, c, n_nodes, n_build;
  int32_t nq, f, slices, rows_wave, cells, q, cpt, steps_per_window;
  int64_t slots;
};

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

// Thread t owns the contiguous cells [t*MAXC, t*MAXC + MAXC) (MAXC =
// HIST_MAX_CELLS_PER_THREAD), so one base address plus immediate offsets
// reaches all of them.
__device__ inline void fold_cells(const int32_t* lds, int64_t* tot, int cells) {
  const int e0 = threadIdx.x * HIST_MAX_CELLS_PER_THREAD;
#pragma unroll
  for (int jj = 0; jj < HIST_MAX_CELLS_PER_THREAD; ++jj) {
    if (e0 + jj < cells) {
      const uint32_t cur = (uint32_t)lds[e0 + jj];
      const int32_t delta = (int32_t)(cur - (uint32_t)tot[jj]);
      tot[jj] += delta;
    }
  }
}

__global__ void __launch_bounds__(HIST_THREADS)
k_hist(HistArgs a) {
  extern __shared__ int32_t lds[];
  const int b = blockIdx.x;
  const int xcd = b & 7, g = b >> 3;
  const int q = (g / a.slices) * 8 + xcd;
  const int s = g % a.slices;
  if (q >= a.q) return;
  const int64_t T = a.pre[a.n_build];
  const int64_t v0 = (int64_t)q * T / a.q;
  const int64_t v1 = (int64_t)(q + 1) * T / a.q;
  if (v0 >= v1) return;

  // first built node whose range holds v0: largest p with pre[p] <= v0
  int lo = 0, hi = a.n_build;  // pre[lo] <= v0 < pre[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.pre[mid] <= v0) lo = mid;
    else hi = mid;
  }
  int p = lo;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int rr = lane / a.nq, qd = lane - rr * a.nq;
  const bool lane_on = rr < a.rows_wave;
  const int f0 = s * a.f;
  const int fq = f0 + 4 * qd;  // first feature of this lane's quad
  const int B = a.n_bins, c = a.c;
  const int rows_step = (HIST_THREADS / 64) * a.rows_wave;

  int64_t tot[HIST_MAX_CELLS_PER_THREAD];
#pragma unroll
  for (int jj = 0; jj < HIST_MAX_CELLS_PER_THREAD; ++jj) tot[jj] = 0;
  for (int e = tid; e < a.cells; e += HIST_THREADS) lds[e] = 0;
  __syncthreads();

  int64_t v = v0;
  while (v < v1) {
    const int32_t j = node_of(a, p);
    const int64_t pstart = a.pre[p];
    const int64_t vend = v1 < a.pre[p + 1] ? v1 : a.pre[p + 1];
    const int64_t seg0 = clamp_i32(a.node_off[j], 0, a.n);
    int steps = 0;
    for (int64_t vs = v; vs < vend; vs += rows_step) {
      const int64_t vv = vs + (int64_t)wave * a.rows_wave + rr;
      if (lane_on && vv < vend && fq < a.m) {
        const int64_t pos = seg0 + (vv - pstart);
        int64_t row = a.row_idx ? (int64_t)a.row_idx[pos] : pos;
        row = row < 0 ? 0 : (row >= a.n ? a.n - 1 : row);
        const uint32_t word = *reinterpret_cast<const uint32_t*>(a.bins + row * a.ld_bins + fq);
        int base[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          int bin = (int)((word >> (8 * u)) & 0xffu);
          bin = bin < B ? bin : B - 1;
          base[u] = ((4 * qd + u) * B + bin) * c;
        }
        const int nf = (a.m - fq) < 4 ? (a.m - fq) : 4;
        const float* ghr = a.GH + row * a.ld_gh;
        for (int t = 0; t < c; ++t) {
          const int32_t vq = (int32_t)rintf(ldexpf(ghr[t], a.qexp[t]));
          atomicAdd(&lds[base[0] + t], vq);
          if (nf > 1) atomicAdd(&lds[base[1] + t], vq);
          if (nf > 2) atomicAdd(&lds[base[2] + t], vq);
          if (nf > 3) atomicAdd(&lds[base[3] + t], vq);
        }
      }
      if (++steps == a.steps_per_window) {
        steps = 0;
        __syncthreads();
        fold_cells(lds, tot, a.cells);
      }
    }
    // end of this node's part: final fold, write the partial, reset
    __syncthreads();
    fold_cells(lds, tot, a.cells);
    int64_t* dst = a.partial + ((int64_t)s * a.slots + q + p) * a.cells;
#pragma unroll
    for (int jj = 0; jj < HIST_MAX_CELLS_PER_THREAD; ++jj) {
      const int e = tid * HIST_MAX_CELLS_PER_THREAD + jj;
      if (e < a.cells) {
        dst[e] = tot[jj];
        lds[e] = 0;
      }
      tot[jj] = 0;
    }
    __syncthreads();
    v = vend;
    ++p;
    while (p < a.n_build && a.pre[p + 1] <= v) ++p;
  }
}

__device__ inline int64_t group_of(int64_t x, int64_t T, int64_t Q) { return ((x + 1) * Q - 1) / T; }

// H[node][f][b][t] = sum of the partials of the row groups that covered the node.
__global__ void __launch_bounds__(256) k_hist_reduce(HistArgs a) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int p = blockIdx.y, s = blockIdx.z;
  if (e >= a.cells) return;
  const int32_t j = node_of(a, p);
  if (j < 0 || j >= a.n_nodes) return;
  const int bc = a.n_bins * a.c;
  const int fl = e / bc;
  const int rem = e - fl * bc;
  const int t = rem % a.c;
  const int f = s * a.f + fl;
  if (f >= a.m) return;
  const int64_t T = a.pre[a.n_build];
  const int64_t lo = a.pre[p], hi = a.pre[p + 1];
  int64_t sum = 0;
  if (hi > lo) {
    const int64_t qlo = group_of(lo, T, a.q), qhi = group_of(hi - 1, T, a.q);
    for (int64_t q = qlo; q <= qhi; ++q) {
      if (q * T / a.q < (q + 1) * T / a.q)
        sum += a.partial[((int64_t)s * a.slots + q + p) * a.cells + e];
    }
  }
  a.H[((int64_t)j * a.m + f) * bc + rem] = ldexp((double)sum, -a.qexp[t]);
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

}  // namespace

int32_t launch_build_histograms(const uint8_t* bins, int64_t n, int32_t m, int64_t ld_bins, int32_t n_bins,
                                const float* GH, int64_t ld_gh, int32_t k, const int32_t* qexp,
                                const int32_t* row_idx, const int32_t* node_off, int32_t n_nodes,
                                const int32_t* build_list, int32_t n_build, double* H, void* ws, hipStream_t st) {
  const HistPlan pl = hist_plan(m, n_bins, k, n_build);
  HistArgs a{};
  a.bins = bins;
  a.ld_bins = ld_bins;
  a.GH = GH;
  a.ld_gh = ld_gh;
  a.qexp = qexp;
  a.row_idx = row_idx;
  a.node_off = node_off;
  a.build_list = build_list;
  char* w = static_cast<char*>(ws);
  a.pre = reinterpret_cast<int64_t*>(w);
  a.partial = reinterpret_cast<int64_t*>(w + align256((int64_t)(n_build + 1) * 8));
  a.H = H;
  a.n = n;
  a.m = m;
  a.n_bins = n_bins;
  a.c = pl.c;
  a.n_nodes = n_nodes;
  a.n_build = n_build;
  a.nq = pl.nq;
  a.f = pl.f;
  a.slices = pl.slices;
  a.rows_wave = pl.rows_wave;
  a.cells = pl.cells;
  a.q = pl.q;
  a.cpt = (pl.cells + HIST_THREADS - 1) / HIST_THREADS;
  const int rows_step = (HIST_THREADS / 64) * pl.rows_wave;
  a.steps_per_window = WINDOW_ROWS / rows_step > 0 ? WINDOW_ROWS / rows_step : 1;
  a.slots = pl.slots;
  if (rows_step > WINDOW_ROWS) return fail(SB_E_UNSUPPORTED, "histogram step exceeds the fixed-point window");

  hipLaunchKernelGGL(k_hist_plan, dim3(1), dim3(1024), 0, st, a);
  const int grid = pl.q_pad * pl.slices;
  hipLaunchKernelGGL(k_hist, dim3(grid), dim3(HIST_THREADS), (size_t)pl.cells * 4, st, a);
  dim3 rg((pl.cells + 255) / 256, n_build, pl.slices);
  hipLaunchKernelGGL(k_hist_reduce, rg, dim3(256), 0, st, a);
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
