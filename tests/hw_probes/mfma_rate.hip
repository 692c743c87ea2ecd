// Sustained MFMA rate per SIMD (bf16, fp32 accumulation) under different
// dependency and operand patterns, at one and two waves per SIMD, with the
// shader clock measured in the kernel (s_memtime cycles over the 100 MHz
// s_memrealtime counter).  One workgroup per CU.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <cstdio>
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
#define MF(a, b, c) __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0)
constexpr int ITERS = 512;
template <int MODE>
__global__ __launch_bounds__(512) void k(float* out, int z, unsigned long long* clk) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[8192];  // 32 KB
  for (int i = threadIdx.x; i < 8192; i += 256) lds[i] = 0x3f803f80u ^ (i & z);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) { a[i] = (__bf16)(0.001f * (lane + i)); b[i] = (__bf16)(0.002f * (lane - i)); }
  f32x16 acc[16];
  for (int j = 0; j < 16; ++j) for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
  const uint32_t base = (lane & 31) * 288 + (lane >> 5) * 16;  // the kernels' row-read pattern (288-byte rows)
  f32x4 acc4[16];
  for (int j = 0; j < 16; ++j) for (int i = 0; i < 4; ++i) acc4[j][i] = 0.f;
  const unsigned long long t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < ITERS; ++it) {
    if constexpr (MODE == 1) {         // 2 chains
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[j & 1] = MF(a, b, acc[j & 1]);
    } else if constexpr (MODE == 2) {  // 1 chain
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[0] = MF(a, b, acc[0]);
    } else if constexpr (MODE == 3) {  // 4 chains, A from LDS right before use
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const bf16x8 x = *(const bf16x8*)((const char*)lds + base + (j & 7) * 32 + ((it & z) << 4));
        acc[j & 3] = MF(x, b, acc[j & 3]);
      }
    } else if constexpr (MODE == 5) {  // 16x16x32: 16 independent chains x 2 (same FLOPs as 16 32x32x16)
#pragma unroll
      for (int j = 0; j < 32; ++j) acc4[j & 15] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc4[j & 15], 0, 0, 0);
    } else {                            // 4 chains, A from LDS, all 16 reads issued first
      bf16x8 x[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) x[j] = *(const bf16x8*)((const char*)lds + base + (j & 7) * 32 + (j >> 3) * 9216 + ((it & z) << 4));
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[j & 3] = MF(x[j], b, acc[j & 3]);
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  if (blockIdx.x == 0 && threadIdx.x == 0) { clk[0] = t1 - t0; clk[1] = r1 - r0; }
  float s = 0.f;
  for (int j = 0; j < 16; ++j) for (int i = 0; i < 16; ++i) s += acc[j][i];
  for (int j = 0; j < 16; ++j) for (int i = 0; i < 4; ++i) s += acc4[j][i];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}
template <int MODE>
void run(int cus, float* d, const char* name, int threads, unsigned long long* clk) {
  hipEvent_t e0, e1; hipEventCreate(&e0); hipEventCreate(&e1);
  hipLaunchKernelGGL(k<MODE>, dim3(cus), dim3(threads), 0, 0, d, 0, clk);
  hipEventRecord(e0, 0);
  hipLaunchKernelGGL(k<MODE>, dim3(cus), dim3(threads), 0, 0, d, 0, clk);
  hipEventRecord(e1, 0);
  hipEventSynchronize(e1);
  float ms = 0; hipEventElapsedTime(&ms, e0, e1);
  unsigned long long c[2];
  hipMemcpy(c, clk, 16, hipMemcpyDeviceToHost);
  const int wps = threads / 256;  // waves per SIMD
  const double mfma_per_simd = (double)ITERS * 16 * wps;  // in 32x32x16 units
  const double tflops = (double)cus * 4 * mfma_per_simd * 32 * 32 * 16 * 2 / (ms * 1e-3) / 1e12;
  const double ghz = (double)c[0] / ((double)c[1] / 100e6) / 1e9;
  printf("%-44s waves/SIMD %d  %.3f ms  %.1f cycles per MFMA-unit per SIMD  %.0f TFLOP/s  (clock %.2f GHz)\n", name, wps, ms,
         (double)c[0] / (ITERS * 16 * wps), tflops, ghz);
}
int main() {
  int cus = 0; hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
  float* d; if (hipMalloc(&d, (size_t)cus * 512 * 4)) return 2;
  unsigned long long* clk; if (hipMalloc(&clk, 16)) return 2;
  for (int th : {256, 512}) {
    run<1>(cus, d, "2 chains, register operands", th, clk);
    run<2>(cus, d, "1 chain, register operands", th, clk);
    run<5>(cus, d, "16x16x32, 16 chains, register operands", th, clk);
    run<3>(cus, d, "4 chains, A read from LDS just before use", th, clk);
    run<4>(cus, d, "4 chains, 16 LDS reads issued first", th, clk);
  }
  return 0;
}
