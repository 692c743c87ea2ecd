// Lane layout of buffer_load_dwordx4 ... lds (direct global-to-LDS copy): lane i lands at base + 16 i.
#include <hip/hip_runtime.h>
#include <stdint.h>
__device__ inline __amdgpu_buffer_rsrc_t mk(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__global__ void k(const uint32_t* src, uint32_t* out) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[1024];
  for (int i = threadIdx.x; i < 1024; i += 64) lds[i] = 0xdeadbeef;
  __syncthreads();
  auto r = mk(src, 4096);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)(lds + 64), 16, (uint32_t)((63 - threadIdx.x) * 16), 0, 0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int i = threadIdx.x; i < 1024; i += 64) out[i] = lds[i];
}
#include <cstdio>
int main() {
  uint32_t h[1024], o[1024];
  for (int i = 0; i < 1024; ++i) h[i] = i;
  uint32_t *ds, *dout;
  if (hipMalloc(&ds, 4096) || hipMalloc(&dout, 4096)) return 2;
  hipMemcpy(ds, h, 4096, hipMemcpyHostToDevice);
  hipLaunchKernelGGL(k, dim3(1), dim3(64), 0, 0, ds, dout);
  if (hipDeviceSynchronize() != hipSuccess) { printf("sync failed\n"); return 3; }
  hipMemcpy(o, dout, 4096, hipMemcpyDeviceToHost);
  int bad = 0, untouched = 0;
  for (int i = 0; i < 1024; ++i) {
    uint32_t want;
    if (i >= 64 && i < 64 + 256) { int lane = (i - 64) / 4, j = (i - 64) % 4; want = (63 - lane) * 4 + j; }
    else want = 0xdeadbeef;
    if (o[i] != want) { if (bad < 8) printf("i=%d got %x want %x\n", i, o[i], want); ++bad; }
    if (o[i] == 0xdeadbeef) ++untouched;
  }
  printf("lds dma layout: %s (mismatches %d, untouched %d)\n", bad ? "UNEXPECTED" : "lane*16 as expected", bad, untouched);
  return 0;
}
