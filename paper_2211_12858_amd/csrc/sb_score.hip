// Split scoring (Section 2, "Finding the tree structure", eq. 4; hessian-free
// form S_G of Section 3 with the single hessian column as weight).
//
// k_score_feature: one wave per (node, feature).  Each lane owns a run of
//   consecutive bins; a per-lane prefix plus a wave scan (shuffles) gives
//   the inclusive prefix over bins of every channel.  H is laid out
//   [node][feature][channel][bin], so a wave reads each channel's bins as
//   one contiguous run.  Histogram values are fixed-point sums stored in
//   fp64, so these prefix sums are exact.  The lane then scores its
//   thresholds and the wave keeps the best (score descending, bin
//   ascending).
// k_score_node: one wave per node picks the best feature (score descending,
//   feature ascending).  Fixed reduction order: results do not depend on
//   timing.
#include <cmath>

#include "sb_common.h"

namespace sb {
namespace {

constexpr int MAX_BPL = 4;  // bins per lane: n_bins <= 256

__device__ inline double wave_incl_scan(double v) {
  const int lane = threadIdx.x & 63;
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

// better(a, b): score a beats score b, ties broken by the smaller index.
__device__ inline bool better(double sa, int ia, double sb_, int ib) {
  return sa > sb_ || (sa == sb_ && ia < ib);
}

__global__ void __launch_bounds__(256)
k_score_feature(const double* __restrict__ H, int n_nodes, int m, int B, int k, double lam, double mcw,
                double* __restrict__ ws_s, int32_t* __restrict__ ws_b) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int f = blockIdx.x * 4 + wave;
  const int j = blockIdx.y;
  if (f >= m) return;
  const int c = k + 1;
  const int bpl = (B + 63) / 64;
  const double* Hf = H + ((int64_t)j * m + f) * c * B;
  const int b0 = lane * bpl;

  // hessian channel
  double hl[MAX_BPL], sl[MAX_BPL], sr[MAX_BPL];
  double run = 0.0;
#pragma unroll
  for (int i = 0; i < MAX_BPL; ++i) {
    const int b = b0 + i;
    if (i < bpl && b < B) run += Hf[(int64_t)k * B + b];
    hl[i] = run;
    sl[i] = 0.0;
    sr[i] = 0.0;
  }
  double incl = wave_incl_scan(run);
  double excl = incl - run;
  const double Th = __shfl(incl, 63, 64);
#pragma unroll
  for (int i = 0; i < MAX_BPL; ++i) hl[i] += excl;

  for (int t = 0; t < k; ++t) {
    double gl[MAX_BPL];
    double r = 0.0;
#pragma unroll
    for (int i = 0; i < MAX_BPL; ++i) {
      const int b = b0 + i;
      if (i < bpl && b < B) r += Hf[(int64_t)t * B + b];
      gl[i] = r;
    }
    const double in = wave_incl_scan(r);
    const double ex = in - r;
    const double Tt = __shfl(in, 63, 64);
#pragma unroll
    for (int i = 0; i < MAX_BPL; ++i) {
      const double L = gl[i] + ex;
      const double R = Tt - L;
      sl[i] += L * L;
      sr[i] += R * R;
    }
  }

  double best_s = -INFINITY;
  int best_b = -1;
#pragma unroll
  for (int i = 0; i < MAX_BPL; ++i) {
    const int b = b0 + i;
    if (i < bpl && b <= B - 2) {
      const double HL = hl[i], HR = Th - hl[i];
      if (HL > mcw && HR > mcw) {
        const double S = sl[i] / (HL + lam) + sr[i] / (HR + lam);
        if (S > best_s) {
          best_s = S;
          best_b = b;
        }
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    const double os = __shfl_xor(best_s, off, 64);
    const int ob = __shfl_xor(best_b, off, 64);
    const bool take = (ob >= 0) && (best_b < 0 || better(os, ob, best_s, best_b));
    if (take) {
      best_s = os;
      best_b = ob;
    }
  }
  if (lane == 0) {
    ws_s[(int64_t)j * m + f] = best_s;
    ws_b[(int64_t)j * m + f] = best_b;
  }
}

__global__ void __launch_bounds__(64)
k_score_node(const double* __restrict__ ws_s, const int32_t* __restrict__ ws_b, int m, int32_t* __restrict__ bf,
             int32_t* __restrict__ bb, double* __restrict__ bs) {
  const int j = blockIdx.x;
  int32_t f, b;
  double s;
  wave_best_feature(ws_s + (int64_t)j * m, ws_b + (int64_t)j * m, m, &f, &b, &s);
  if (threadIdx.x == 0) {
    bf[j] = f;
    bb[j] = b;
    bs[j] = s;
  }
}

}  // namespace

int64_t score_ws_bytes(int32_t n_nodes, int32_t m) {
  return align256((int64_t)n_nodes * m * 8) + align256((int64_t)n_nodes * m * 4);
}

int32_t launch_score(const double* H, int32_t n_nodes, int32_t m, int32_t n_bins, int32_t k, double lambda,
                     double mcw, int32_t* best_f, int32_t* best_b, double* best_s, void* ws, hipStream_t st) {
  char* w = static_cast<char*>(ws);
  double* ws_s = reinterpret_cast<double*>(w);
  int32_t* ws_b = reinterpret_cast<int32_t*>(w + align256((int64_t)n_nodes * m * 8));
  hipLaunchKernelGGL(k_score_feature, dim3((m + 3) / 4, n_nodes), dim3(256), 0, st, H, n_nodes, m, n_bins, k, lambda,
                     mcw, ws_s, ws_b);
  hipLaunchKernelGGL(k_score_node, dim3(n_nodes), dim3(64), 0, st, ws_s, ws_b, m, best_f, best_b, best_s);
  return check_launch("sb_score_splits");
}

int32_t launch_score_node(const double* feat_s, const int32_t* feat_b, int32_t n_nodes, int32_t m, int32_t* best_f,
                          int32_t* best_b, double* best_s, hipStream_t st) {
  hipLaunchKernelGGL(k_score_node, dim3(n_nodes), dim3(64), 0, st, feat_s, feat_b, m, best_f, best_b, best_s);
  return check_launch("sb_grow_tree");
}

}  // namespace sb
