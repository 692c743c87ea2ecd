// MFMA / VALU co-issue probe (gfx950): 32x32x16 bf16 MFMAs in four independent
// chains with NV independent VALU ops forced between consecutive MFMAs
// (sched_group_barrier), register operands only.  Reports shader cycles per
// MFMA of the timing wave (wave 0 of block 0, s_memtime) and the clock.
// KIND 0: v_fma_f32, 1: v_exp_f32, 2: alternating.  With two waves per SIMD
// the timing wave is the oldest one, which the arbiter favours, so those rows
// show that wave's rate, not the SIMD's.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <cstdio>
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
#define MF(a, b, c) __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0)
constexpr int ITERS = 256;
template <int NV, int KIND>
__global__ __launch_bounds__(512) void k(float* out, int z, unsigned long long* clk) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) { a[i] = (__bf16)(0.001f * (lane + i)); b[i] = (__bf16)(0.002f * (lane - i)); }
  f32x16 acc[4];
  for (int j = 0; j < 4; ++j) for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
  float x[32];
  for (int i = 0; i < 32; ++i) x[i] = 0.01f * (lane + i + z);
  const float c1 = 0.999f + z, c2 = 0.0001f * z;
  const unsigned long long t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < ITERS; ++it) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      acc[j & 3] = MF(a, b, acc[j & 3]);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        float& y = x[(j * NV + v) & 31];
        if constexpr (KIND == 0) y = __builtin_fmaf(y, c1, c2);
        else if constexpr (KIND == 1) y = __builtin_amdgcn_exp2f(-__builtin_fabsf(y));
        else { if (v & 1) y = __builtin_amdgcn_exp2f(-__builtin_fabsf(y)); else y = __builtin_fmaf(y, c1, c2); }
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if constexpr (NV > 0) __builtin_amdgcn_sched_group_barrier(0x002, NV, 0);
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  if (blockIdx.x == 0 && threadIdx.x == 0) { clk[0] = t1 - t0; clk[1] = r1 - r0; }
  float s = 0.f;
  for (int j = 0; j < 4; ++j) for (int i = 0; i < 16; ++i) s += acc[j][i];
  for (int i = 0; i < 32; ++i) s += x[i];
  out[blockIdx.x * 512 + threadIdx.x] = s;
}
template <int NV, int KIND>
void run(int cus, float* d, int threads, unsigned long long* clk) {
  hipEvent_t e0, e1; hipEventCreate(&e0); hipEventCreate(&e1);
  hipLaunchKernelGGL((k<NV, KIND>), dim3(cus), dim3(threads), 0, 0, d, 0, clk);
  hipEventRecord(e0, 0);
  hipLaunchKernelGGL((k<NV, KIND>), dim3(cus), dim3(threads), 0, 0, d, 0, clk);
  hipEventRecord(e1, 0);
  hipEventSynchronize(e1);
  float ms = 0; hipEventElapsedTime(&ms, e0, e1);
  unsigned long long c[2];
  hipMemcpy(c, clk, 16, hipMemcpyDeviceToHost);
  const int wps = threads / 256;
  const double ghz = (double)c[0] / ((double)c[1] / 100e6) / 1e9;
  printf("%s NV=%2d waves/SIMD %d: %.1f cycles per MFMA per SIMD (%.1f per wave-MFMA), clock %.2f GHz\n",
         KIND == 0 ? "fma " : KIND == 1 ? "exp " : "mix ", NV, wps, (double)c[0] / (ITERS * 16 * wps),
         (double)c[0] / (ITERS * 16), ghz);
}
template <int KIND>
void sweep(int cus, float* d, unsigned long long* clk) {
  for (int t : {256, 512}) {
    run<0, KIND>(cus, d, t, clk); run<2, KIND>(cus, d, t, clk); run<4, KIND>(cus, d, t, clk);
    run<6, KIND>(cus, d, t, clk); run<7, KIND>(cus, d, t, clk); run<8, KIND>(cus, d, t, clk);
    run<10, KIND>(cus, d, t, clk); run<12, KIND>(cus, d, t, clk); run<16, KIND>(cus, d, t, clk);
  }
}
int main() {
  int cus = 0; hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
  float* d; if (hipMalloc(&d, (size_t)cus * 512 * 4)) return 2;
  unsigned long long* clk; if (hipMalloc(&clk, 16)) return 2;
  sweep<0>(cus, d, clk); sweep<1>(cus, d, clk); sweep<2>(cus, d, clk);
  return 0;
}
