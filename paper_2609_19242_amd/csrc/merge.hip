// J-way log-sum-exp merge of normalised partial attentions, gfx950.
//
// eq:csbp-lse-merge of arXiv 2609.19242 merges two partials; by
// eq:correctness-online-softmax-merge the same rule extends to J parts over
// disjoint key sets: m = max_j z_j, w_j = exp(z_j - m) (0 where z_j = -inf),
// O = sum_j w_j O_j / sum_j w_j, z = m + ln(sum_j w_j).  The paper's kernel
// folds one partial at a time into fp32 numerator / max / normaliser buffers
// in HBM; here one pass reads every partial once and keeps that state in
// registers, so the traffic is the algorithmic minimum (J reads, one write).
// Parts with w_j = 0 for a row (e.g. a key shard the row cannot see) are not
// read at all.
//
// Thread mapping: one thread per 8 consecutive head_dim elements of one
// (batch, row, head); a wavefront covers 64*8 contiguous elements, so every
// O_j read is a coalesced 16- or 32-byte-per-lane access.
#include "common.hpp"
#include "device.hpp"

namespace bdlm {

namespace {

template <typename TI>
__device__ inline void load8(const void* p, float* x) {
  if constexpr (sizeof(TI) == 2) {
    const u32x4 v = *(const u32x4*)p;
    const bf16x8 b = __builtin_bit_cast(bf16x8, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (float)b[e];
  } else {
    const f32x4 a0 = ((const f32x4*)p)[0], a1 = ((const f32x4*)p)[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = a0[e];
      x[4 + e] = a1[e];
    }
  }
}

template <typename TO>
__device__ inline void store8(void* p, const float* x) {
  if constexpr (sizeof(TO) == 2) {
    bf16x8 b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = to_bf16(x[e]);
    *(bf16x8*)p = b;
  } else {
    f32x4 a0, a1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a0[e] = x[e];
      a1[e] = x[4 + e];
    }
    ((f32x4*)p)[0] = a0;
    ((f32x4*)p)[1] = a1;
  }
}

template <int D, typename TI, typename TO>
__global__ __launch_bounds__(256) void merge_kernel(const MergeArgs a) {
  constexpr int CPR = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = a.batch * a.rows * a.heads * CPR;
  if (gid >= total) return;
  const int chunk = (int)(gid % CPR);
  const int64_t rh = gid / CPR;  // (b * rows + row) * heads + h
  const int h = (int)(rh % a.heads);
  const int64_t brow = rh / a.heads;
  const int64_t row = brow % a.rows, b = brow / a.rows;
  const int64_t lse_idx = (b * a.heads + h) * a.rows + row;
  const int64_t o_off = rh * D + chunk * 8;

  float m = -INFINITY;
  for (int j = 0; j < a.n_parts; ++j) m = fmaxf(m, a.lse_parts[j][lse_idx]);
  float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  if (m != -INFINITY) {
    for (int j = 0; j < a.n_parts; ++j) {
      const float z = a.lse_parts[j][lse_idx];
      if (z == -INFINITY) continue;  // w_j = 0: this part is not read
      const float wj = expf(z - m);
      float x[8];
      load8<TI>((const TI*)a.o_parts[j] + o_off, x);
      den += wj;
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] = fmaf(wj, x[e], num[e]);
    }
  }
  const bool empty = !(den > 0.f);
  const float inv = empty ? 0.f : 1.f / den;
#pragma unroll
  for (int e = 0; e < 8; ++e) num[e] *= inv;
  store8<TO>((TO*)a.o + o_off, num);
  if (chunk == 0) a.lse[lse_idx] = empty ? -INFINITY : m + logf(den);
}

template <int D>
hipError_t launch_d(const MergeArgs& a, int pt, int ot, hipStream_t s) {
  const int64_t total = a.batch * a.rows * a.heads * (D / 8);
  const dim3 grid((unsigned)((total + 255) / 256));
  if (pt == 0 && ot == 0) hipLaunchKernelGGL((merge_kernel<D, bf16, bf16>), grid, dim3(256), 0, s, a);
  if (pt == 0 && ot == 1) hipLaunchKernelGGL((merge_kernel<D, bf16, float>), grid, dim3(256), 0, s, a);
  if (pt == 1 && ot == 0) hipLaunchKernelGGL((merge_kernel<D, float, bf16>), grid, dim3(256), 0, s, a);
  if (pt == 1 && ot == 1) hipLaunchKernelGGL((merge_kernel<D, float, float>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int head_dim, int part_dtype, int out_dtype, hipStream_t s) {
  if (a.batch * a.rows * a.heads == 0) return hipSuccess;
  return head_dim == 128 ? launch_d<128>(a, part_dtype, out_dtype, s) : launch_d<64>(a, part_dtype, out_dtype, s);
}

}  // namespace bdlm
