// Checks the assumed lane layout of v_mfma_f32_16x16x32_bf16:
//   A (16x32): lane l holds A[l % 16][8 (l / 16) + j], j = 0..7
//   B (32x16): lane l holds B[8 (l / 16) + j][l % 16]
//   D (16x16): lane l holds D[4 (l / 16) + i][l % 16], i = 0..3
// with small integers (exact in bf16 and fp32) against a host product.
#include <hip/hip_runtime.h>
#include <cstdio>
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
__global__ void k(const float* A, const float* B, float* D) {
  const int l = threadIdx.x;
  bf16x8 a, b;
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)A[(l % 16) * 32 + 8 * (l / 16) + j];
    b[j] = (__bf16)B[(8 * (l / 16) + j) * 16 + (l % 16)];
  }
  f32x4 c = {0.f, 0.f, 0.f, 0.f};
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  for (int i = 0; i < 4; ++i) D[(4 * (l / 16) + i) * 16 + (l % 16)] = c[i];
}
int main() {
  float hA[16 * 32], hB[32 * 16], hD[256], ref[256];
  unsigned s = 12345;
  auto rnd = [&]() { s = s * 1103515245u + 12345u; return (float)((int)((s >> 16) % 7) - 3); };
  for (auto& x : hA) x = rnd();
  for (auto& x : hB) x = rnd();
  for (int m = 0; m < 16; ++m) for (int n = 0; n < 16; ++n) {
    float acc = 0; for (int kk = 0; kk < 32; ++kk) acc += hA[m * 32 + kk] * hB[kk * 16 + n]; ref[m * 16 + n] = acc;
  }
  float *dA, *dB, *dD;
  if (hipMalloc(&dA, sizeof hA) || hipMalloc(&dB, sizeof hB) || hipMalloc(&dD, sizeof hD)) return 2;
  if (hipMemcpy(dA, hA, sizeof hA, hipMemcpyHostToDevice) || hipMemcpy(dB, hB, sizeof hB, hipMemcpyHostToDevice)) return 2;
  hipLaunchKernelGGL(k, dim3(1), dim3(64), 0, 0, dA, dB, dD);
  if (hipDeviceSynchronize() != hipSuccess) return 3;
  if (hipMemcpy(hD, dD, sizeof hD, hipMemcpyDeviceToHost)) return 3;
  int bad = 0;
  for (int i = 0; i < 256; ++i) if (hD[i] != ref[i]) ++bad;
  printf("mfma 16x16x32 bf16 layout: %s (%d of 256 differ)\n", bad ? "MISMATCH" : "as assumed", bad);
  return 0;
}
