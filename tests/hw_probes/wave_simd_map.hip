// Which SIMD each wave of a 512-thread workgroup runs on (HW_ID register,
// SIMD_ID field), over a grid of 2,048 such workgroups with 128 KB of LDS
// each (one workgroup per CU).  Prints the SIMD of waves 0-7 for the first
// workgroups and, over the grid, how often waves w and w+4 (and w and w+1)
// share a SIMD.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <vector>
constexpr int NWG = 2048;
__global__ __launch_bounds__(512) void k(int* out) {
  __shared__ int pad[32768];  // 128 KB
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    const unsigned hw = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 4);  // HW_REG_HW_ID, 32 bits
    pad[w] = (int)hw;
  }
  __syncthreads();
  if (threadIdx.x < 8) out[blockIdx.x * 8 + threadIdx.x] = pad[threadIdx.x];
}
int main() {
  int* d;
  if (hipMalloc(&d, NWG * 8 * sizeof(int)) != hipSuccess) return 1;
  hipLaunchKernelGGL(k, dim3(NWG), dim3(512), 0, 0, d);
  if (hipDeviceSynchronize() != hipSuccess) return 2;
  std::vector<int> h(NWG * 8);
  if (hipMemcpy(h.data(), d, h.size() * sizeof(int), hipMemcpyDeviceToHost) != hipSuccess) return 3;
  auto simd = [&](int g, int w) { return (h[g * 8 + w] >> 4) & 3; };
  for (int g = 0; g < 4; ++g) {
    printf("wg %d simd of waves 0-7:", g);
    for (int w = 0; w < 8; ++w) printf(" %d", simd(g, w));
    printf("  (hw_id wave0 0x%08x)\n", h[g * 8]);
  }
  long same4 = 0, same1 = 0, n4 = 0, n1 = 0;
  for (int g = 0; g < NWG; ++g) {
    for (int w = 0; w < 4; ++w, ++n4) same4 += simd(g, w) == simd(g, w + 4);
    for (int w = 0; w < 8; w += 2, ++n1) same1 += simd(g, w) == simd(g, w + 1);
  }
  printf("waves w, w+4 share a SIMD: %.3f; waves 2i, 2i+1: %.3f\n", (double)same4 / n4, (double)same1 / n1);
  (void)hipFree(d);
  return 0;
}
