// Practical HBM bandwidth of streaming kernels: a read-only pass (16 bytes per
// lane per load, non-temporal, one partial sum per thread written at the end)
// and a copy, over 2 GiB buffers, timed with HIP events (median of 10).
#include <hip/hip_runtime.h>
#include <cstdio>
#include <algorithm>
#include <vector>
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr size_t kBytes = size_t(2) << 30;
constexpr int kUnroll = 4;

__global__ __launch_bounds__(256) void read_k(const f32x4* __restrict__ src, float* __restrict__ out, size_t n4) {
  const size_t tid = (size_t)blockIdx.x * 256 + threadIdx.x, stride = (size_t)gridDim.x * 256;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (size_t i = tid; i < n4; i += stride * kUnroll) {
    f32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t k = i + u * stride;
      v[u] = k < n4 ? __builtin_nontemporal_load(src + k) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc += v[u];
  }
  out[tid] = acc[0] + acc[1] + acc[2] + acc[3];
}

__global__ __launch_bounds__(256) void copy_k(const f32x4* __restrict__ src, f32x4* __restrict__ dst, size_t n4) {
  const size_t tid = (size_t)blockIdx.x * 256 + threadIdx.x, stride = (size_t)gridDim.x * 256;
  for (size_t i = tid; i < n4; i += stride * kUnroll) {
    f32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t k = i + u * stride;
      v[u] = k < n4 ? __builtin_nontemporal_load(src + k) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t k = i + u * stride;
      if (k < n4) __builtin_nontemporal_store(v[u], dst + k);
    }
  }
}

int main() {
  const size_t n4 = kBytes / 16;
  f32x4 *a, *b;
  float* out;
  const int grids[] = {1024, 2048, 4096, 8192};
  if (hipMalloc(&a, kBytes) != hipSuccess || hipMalloc(&b, kBytes) != hipSuccess) return 1;
  if (hipMalloc(&out, (size_t)8192 * 256 * sizeof(float)) != hipSuccess) return 1;
  if (hipMemset(a, 0, kBytes) != hipSuccess || hipMemset(b, 0, kBytes) != hipSuccess) return 1;
  hipEvent_t e0, e1;
  (void)hipEventCreate(&e0);
  (void)hipEventCreate(&e1);
  for (int g : grids) {
    for (int kind = 0; kind < 2; ++kind) {
      std::vector<float> ms;
      for (int r = 0; r < 12; ++r) {
        (void)hipEventRecord(e0, 0);
        if (kind == 0) hipLaunchKernelGGL(read_k, dim3(g), dim3(256), 0, 0, a, out, n4);
        else hipLaunchKernelGGL(copy_k, dim3(g), dim3(256), 0, 0, a, b, n4);
        (void)hipEventRecord(e1, 0);
        if (hipEventSynchronize(e1) != hipSuccess) return 2;
        float t;
        (void)hipEventElapsedTime(&t, e0, e1);
        if (r >= 2) ms.push_back(t);
      }
      std::sort(ms.begin(), ms.end());
      const double t = ms[ms.size() / 2] * 1e-3;
      const double bytes = kind == 0 ? (double)kBytes : 2.0 * kBytes;
      printf("%-5s grid %5d x 256: %.3f ms, %.2f TB/s\n", kind == 0 ? "read" : "copy", g, t * 1e3, bytes / t / 1e12);
    }
  }
  (void)hipFree(a);
  (void)hipFree(b);
  (void)hipFree(out);
  return 0;
}
