// LDS scatter-add rates of the histogram kernel's access pattern on gfx950,
// with uniformly random bins (murmur3 finalizer of lane, feature and
// iteration), 768 threads and ~124 KB of cells per workgroup, one workgroup
// per CU.  Reported: channel-adds per clock per CU at the 2.4 GHz nominal
// clock.  Build and run (one GPU):
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//         -o lds_scatter lds_scatter.hip && ./lds_scatter
//  0: u32 atomics, lane = row, 6 channels at stride FB (= 0 mod 32 banks)
//  1: u32 atomics, lane = (row, channel), 10 rows x 6 channels per wave, stride FB+1
//  2: u64 atomics packing two channels (3 ops per row and feature)
//  3: ds_write_b32 (no atomic), lane = row, 6 channels
//  4: u32 atomics, conflict-free bins (lane-distinct), lane = row
//  5: u32 atomics, lane = row, channel stride FB+1 and feature stride B+1
//  6: u64 atomics, rotated feature order: cells [bin][pair][16 features],
//     lane l adds feature (i + l) mod 16 at step i (the histogram kernel's
//     layout for up to 6 channels)
//  7: the same cells with every lane on feature i at step i (same-feature order)
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <cstdint>

#define CK(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e_), __LINE__); exit(1);} } while (0)

constexpr int F = 20, B = 256, C = 6, FB = F * B;

__device__ inline uint32_t fmix(uint32_t h) {
  h ^= h >> 16; h *= 0x85ebca6bu; h ^= h >> 13; h *= 0xc2b2ae35u; h ^= h >> 16;
  return h;
}

template <int MODE>
__global__ void __launch_bounds__(768) k(int iters, int* out) {
  extern __shared__ int lds[];
  const int cells = C * (FB + 32) + 64;
  for (int i = threadIdx.x; i < cells; i += 768) lds[i] = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const uint32_t seed = (blockIdx.x * 768u + threadIdx.x) * 0x9E3779B9u;
  for (int it = 0; it < iters; ++it) {
    if (MODE == 1) {
      // lanes 0..59: row r = lane / 6, channel t = lane % 6; 10 rows per wave-iteration
      const int r = lane / 6, t = lane - 6 * (lane / 6);
      const bool on = lane < 60;
      const uint32_t rowseed = ((blockIdx.x * 768u + (threadIdx.x & ~63) + r) * 0x9E3779B9u) ^ (it * 0x632be5abu);
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int bin = fmix(rowseed + f) & 255;
        if (on) atomicAdd(lds + t * (FB + 1) + f * B + bin, (int)it);
      }
    } else if (MODE == 2) {
      unsigned long long* l64 = reinterpret_cast<unsigned long long*>(lds);
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int bin = fmix(seed + it * 131u + f) & 255;
#pragma unroll
        for (int t = 0; t < C / 2; ++t) atomicAdd(l64 + t * FB + f * B + bin, (unsigned long long)it);
      }
    } else if (MODE == 6 || MODE == 7) {
      // 16 features x 256 bins x 3 pairs = 12288 64-bit cells (96 KB)
      unsigned long long* l64 = reinterpret_cast<unsigned long long*>(lds);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int bin = fmix(seed + it * 131u + i) & 255;
        const int col = MODE == 6 ? ((i + lane) & 15) : i;
#pragma unroll
        for (int t = 0; t < C / 2; ++t) atomicAdd(l64 + bin * 48 + t * 16 + col, (unsigned long long)it);
      }
    } else {
#pragma unroll
      for (int f = 0; f < F; ++f) {
        int bin = fmix(seed + it * 131u + f) & 255;
        if (MODE == 4) bin = (lane * 5 + f + it) & 255;
        int* cell = MODE == 5 ? lds + f * (B + 1) + bin : lds + f * B + bin;
        const int stride = MODE == 5 ? FB + F + 1 : FB;
#pragma unroll
        for (int t = 0; t < C; ++t) {
          if (MODE == 3) cell[t * stride] = it;
          else atomicAdd(cell + t * stride, it);
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = lds[0] + lds[cells - 1];
}

int main() {
  int* out; CK(hipMalloc(&out, 1 << 20));
  hipEvent_t e0, e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  const int grid = 256, iters = 200;
  const size_t lds = (C * (FB + 32) + 64) * 4;  // 124 KB < 160 KB
  for (int mode = 0; mode < 8; ++mode) {
    auto L = [&]() {
      switch (mode) {
        case 0: hipLaunchKernelGGL(k<0>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 1: hipLaunchKernelGGL(k<1>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 2: hipLaunchKernelGGL(k<2>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 3: hipLaunchKernelGGL(k<3>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 4: hipLaunchKernelGGL(k<4>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 5: hipLaunchKernelGGL(k<5>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 6: hipLaunchKernelGGL(k<6>, dim3(grid), dim3(768), lds, 0, iters, out); break;
        case 7: hipLaunchKernelGGL(k<7>, dim3(grid), dim3(768), lds, 0, iters, out); break;
      }
    };
    L(); CK(hipGetLastError()); CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0)); L(); CK(hipEventRecord(e1)); CK(hipEventSynchronize(e1));
    float ms; CK(hipEventElapsedTime(&ms, e0, e1));
    // channel-adds: mode 1 does 10 rows x 6 ch per wave per iteration (60 of 64 lanes)
    double rows = (double)grid * 768 * iters * (mode == 1 ? 10.0 / 64.0 : 1.0);
    double adds = rows * (mode >= 6 ? 16 : F) * C;
    printf("mode %d: %.3f ms  %.2f channel-adds/clk/CU\n", mode, ms, adds / (ms * 1e-3) / (256.0 * 2.4e9));
  }
  printf("done\n");
  return 0;
}
