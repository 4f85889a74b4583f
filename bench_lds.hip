// LDS scatter-add rates on gfx950 for the histogram kernel's access patterns.
//
// Measurement source (not part of the library).  One workgroup per CU (256
// workgroups), 96 KB of 64-bit cells laid out [bin][pair][16 slots] as in the
// histogram kernel, uniformly random bins (murmur3 finalizer, 16 bins per
// "row" from four 32-bit hashes).  Each workgroup times its loop with
// s_memtime (shader clock) and s_memrealtime (100 MHz), so rates are per
// measured clock and the clock itself is reported.
//
// Build and run on one GPU:
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//         -o /tmp/bench_lds bench_lds.hip && /tmp/bench_lds
//
// Modes (lane l, step i, 64 lanes per wave):
//   rot F   : ds_add_u64 x3 (three channel pairs), lane l on slot (l + i) mod F
//             (F = 16 is the histogram kernel; F < 16 leaves slots unused)
//   wave    : ds_add_u64 x3, the whole wave on slot i (64 random bins, one bank pair)
//   col     : ds_add_u64 x3, cells [pair][feature][bin], whole wave on feature i
//             (the bank is chosen by the random bin)
//   u32     : ds_add_u32 x3 on the rotated slots (one channel per op)
//   f32     : ds_add_f32 x3 on the rotated slots (floating-point atomics)
//   write   : ds_write_b64 x3 on the rotated slots (no read-modify-write)
//   read    : ds_read_b64 x3 on the rotated slots
#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#define CK(x)                                                                            \
  do {                                                                                   \
    hipError_t e_ = (x);                                                                 \
    if (e_ != hipSuccess) {                                                              \
      printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);              \
      exit(1);                                                                           \
    }                                                                                    \
  } while (0)

enum { ROT = 0, WAVE = 1, COL = 2, U32 = 3, F32 = 4, WRITE = 5, READ = 6 };
constexpr int CELLS = 256 * 3 * 16;  // 64-bit cells, 96 KB
constexpr int GRID = 256;

__device__ inline uint32_t fmix(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  h *= 0xc2b2ae35u;
  h ^= h >> 16;
  return h;
}

typedef __attribute__((address_space(3))) unsigned long long lds_u64;
typedef __attribute__((address_space(3))) unsigned int lds_u32;
typedef __attribute__((address_space(3))) float lds_f32;

template <int MODE, int F, int NT>
__global__ void __launch_bounds__(NT) k_lds(int iters, unsigned long long* out, long long* tm) {
  extern __shared__ unsigned long long cells[];
  for (int i = threadIdx.x; i < CELLS; i += NT) cells[i] = 0;
  __syncthreads();
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t r = lane % F;
  const uint32_t seed = (blockIdx.x * NT + threadIdx.x) * 0x9E3779B9u;
  const uint32_t base = (uint32_t)(size_t)cells;
  unsigned long long acc = 0;
  long long t0 = 0, w0 = 0;
  if (threadIdx.x == 0) {
    t0 = __builtin_amdgcn_s_memtime();
    w0 = __builtin_amdgcn_s_memrealtime();
  }
  for (int it = 0; it < iters; ++it) {
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = fmix(seed + (uint32_t)it * 4u + j);
    const unsigned long long v = (unsigned long long)it * 0x100000001ull;
#pragma unroll
    for (int i = 0; i < F; ++i) {
      uint32_t fi = r + i;
      fi = fi >= (uint32_t)F ? fi - F : fi;
      if (MODE == WAVE || MODE == COL) fi = i;
      const uint32_t ww = fi < 8 ? (fi < 4 ? w[0] : w[1]) : (fi < 12 ? w[2] : w[3]);
      const uint32_t bin = (ww >> ((fi & 3) * 8)) & 255u;
      // [bin][pair][slot]: pair stride 128 bytes; [pair][feature][bin]: pair stride 32 KB
      const uint32_t addr = MODE == COL ? base + (fi * 256u + bin) * 8u : base + bin * 384u + fi * 8u;
      const uint32_t pstride = MODE == COL ? 16u * 256u * 8u : 128u;
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        const uint32_t a = addr + p * pstride;
        if (MODE == ROT || MODE == WAVE || MODE == COL) {
          __hip_atomic_fetch_add((lds_u64*)(size_t)a, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        } else if (MODE == U32) {
          __hip_atomic_fetch_add((lds_u32*)(size_t)a, (unsigned)it, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        } else if (MODE == F32) {
          __hip_atomic_fetch_add((lds_f32*)(size_t)a, 1.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        } else if (MODE == WRITE) {
          *(lds_u64*)(size_t)a = v + p;
        } else {
          acc += *(volatile lds_u64*)(size_t)a;
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    tm[2 * blockIdx.x] = __builtin_amdgcn_s_memtime() - t0;
    tm[2 * blockIdx.x + 1] = __builtin_amdgcn_s_memrealtime() - w0;
  }
  out[blockIdx.x * NT + threadIdx.x] = acc + cells[threadIdx.x];
}

template <int MODE, int F, int NT>
void run(const char* name, int iters, unsigned long long* out, long long* tm) {
  const size_t lds = CELLS * 8;
  for (int rep = 0; rep < 2; ++rep) hipLaunchKernelGGL((k_lds<MODE, F, NT>), dim3(GRID), dim3(NT), lds, 0, iters, out, tm);
  CK(hipGetLastError());
  CK(hipDeviceSynchronize());
  long long h[2 * GRID];
  CK(hipMemcpy(h, tm, sizeof(h), hipMemcpyDeviceToHost));
  double cyc = 0, wall = 0;
  for (int b = 0; b < GRID; ++b) {
    cyc += h[2 * b];
    wall += h[2 * b + 1];
  }
  cyc /= GRID;
  wall /= GRID;
  const double ghz = cyc / (wall * 1e-8) / 1e9;
  const double lane_ops = (double)NT * iters * F * 3;  // per workgroup
  const double per_op = (MODE == ROT || MODE == WAVE || MODE == COL || MODE == WRITE || MODE == READ) ? 2.0 : 1.0;
  printf("%-6s F=%2d threads=%4d  clock %.2f GHz  %6.2f clk per wave instruction  %6.2f channel-ops/clk/CU\n", name, F,
         NT, ghz, cyc / (lane_ops / 64.0), lane_ops * per_op / cyc);
}

int main() {
  unsigned long long* out;
  long long* tm;
  CK(hipMalloc(&out, (size_t)GRID * 1024 * 8));
  CK(hipMalloc(&tm, (size_t)GRID * 2 * 8));
  const int it = 400;
  run<ROT, 16, 768>("rot", it, out, tm);
  run<ROT, 16, 1024>("rot", it, out, tm);
  run<ROT, 16, 512>("rot", it, out, tm);
  run<ROT, 16, 256>("rot", it, out, tm);
  run<ROT, 15, 768>("rot", it, out, tm);
  run<ROT, 13, 768>("rot", it, out, tm);
  run<ROT, 12, 768>("rot", it, out, tm);
  run<ROT, 8, 768>("rot", it, out, tm);
  run<WAVE, 16, 768>("wave", it / 4, out, tm);
  run<COL, 16, 768>("col", it, out, tm);
  run<U32, 16, 768>("u32", it, out, tm);
  run<F32, 16, 768>("f32", it / 8, out, tm);
  run<WRITE, 16, 768>("write", it, out, tm);
  run<READ, 16, 768>("read", it, out, tm);
  CK(hipFree(out));
  CK(hipFree(tm));
  printf("done\n");
  return 0;
}
