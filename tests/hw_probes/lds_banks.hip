// Throughput and bank behaviour of the LDS read patterns the kernels use, on gfx950.
// LDS read throughput per access pattern: 4 waves per workgroup, 16 independent reads per batch.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <cstdio>
typedef short s4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
__device__ uint32_t addr_of(int pat, int lane) {
  const int r = lane & 31, h = lane >> 5, G = lane >> 4, sl = lane & 15;
  const int tr_row = 4 * (G >> 1) + (sl >> 2), tr_col = 16 * (G & 1) + 4 * (sl & 3);
  switch (pat) {
    case 0: return lane * 16;                      // b128 contiguous
    case 1: return r * 288 + h * 16;               // b128, rows of 288 B (D=128 + 16 pad)
    case 2: return r * 272 + h * 16;               // b128, rows of 272 B
    case 3: return r * 256 + h * 16;               // b128, rows of 256 B (no pad)
    case 4: return lane * 8;                       // tr, contiguous
    case 5: return tr_row * 288 + tr_col * 2;      // tr, rows of 288 B
    case 6: return tr_row * 272 + tr_col * 2;      // tr, rows of 272 B
    case 7: return tr_row * 256 + tr_col * 2;      // tr, rows of 256 B
    case 8: return tr_row * 320 + tr_col * 2;      // tr, rows of 320 B (D + 32)
    default: return r * 320 + h * 16;              // b128, rows of 320 B
  }
}
__global__ __launch_bounds__(256) void k(int pat, int z, uint32_t* sink) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[16384];  // 64 KB
  for (int i = threadIdx.x; i < 16384; i += 256) lds[i] = i;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const uint32_t a = addr_of(pat, lane);
  uint32_t acc = 0;
  for (int it = 0; it < 2048; ++it) {
    const uint32_t aa = a ^ (uint32_t)(it & z);
    if (pat < 4 || pat == 9) {
      u4 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = *(const u4*)((const char*)lds + aa + (u & 7) * 4096 + (u >> 3) * 32);
#pragma unroll
      for (int u = 0; u < 16; ++u) acc ^= v[u][0] ^ v[u][3];
    } else {
      s4 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        v[u] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)((__attribute__((address_space(3))) char*)lds + aa + (u & 7) * 4096 + (u >> 3) * 64));
#pragma unroll
      for (int u = 0; u < 16; ++u) acc ^= (uint32_t)v[u][0] ^ (uint32_t)v[u][3];
    }
  }
  sink[blockIdx.x * 256 + threadIdx.x] = acc;
}
int main() {
  int cus = 0;
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0);
  uint32_t* ds;
  if (hipMalloc(&ds, (size_t)cus * 256 * 4)) return 2;
  hipEvent_t e0, e1;
  hipEventCreate(&e0); hipEventCreate(&e1);
  for (int pat = 0; pat < 10; ++pat) {
    hipLaunchKernelGGL(k, dim3(cus), dim3(256), 0, 0, pat, 0, ds);  // warm
    hipEventRecord(e0, 0);
    hipLaunchKernelGGL(k, dim3(cus), dim3(256), 0, 0, pat, 0, ds);
    hipEventRecord(e1, 0);
    if (hipEventSynchronize(e1) != hipSuccess) { printf("fail\n"); return 3; }
    float ms = 0; hipEventElapsedTime(&ms, e0, e1);
    const double instr_per_cu = 4.0 * 2048 * 16;
    const double bytes = instr_per_cu * ((pat < 4 || pat == 9) ? 1024 : 512);
    printf("pattern %d: %.3f ms, %.2f ns per instruction per CU, %.1f B/ns per CU\n", pat, ms, ms * 1e6 / instr_per_cu, bytes / (ms * 1e6));
  }
  return 0;
}
