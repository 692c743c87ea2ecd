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
// O_j read is a coalesced 16- or 32-byte-per-lane access.  At head_dim 128 the
// 16 threads of a (row, head) share the parts' z through lane broadcasts
// instead of each loading all of them.
#include "common.hpp"
#include "device.hpp"

namespace bdlm {
namespace {
// Parts whose loads are issued together per thread, and the cache policy of
// those loads: the partials are read exactly once, so they stream past the
// caches (non-temporal), as does the merged output.  Measured at the 256K CSBP
// share (17 bf16 partials, 10 read): 4 parts per group and non-temporal loads
// and stores 5.4 TB/s, against 4.4-4.6 TB/s with 8 per group and default policy.
constexpr int kPartGroup = 4;
constexpr int kNonTemporal = 2;  // buffer load cache-policy bits: nt
}  // namespace
}  // namespace bdlm

namespace bdlm {

namespace {

template <typename TO>
__device__ inline void store8(void* p, const float* x) {
  if constexpr (sizeof(TO) == 2) {
    bf16x8 b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = to_bf16(x[e]);
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, b), (u32x4*)p);
  } else {
    f32x4 a0, a1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a0[e] = x[e];
      a1[e] = x[4 + e];
    }
    __builtin_nontemporal_store(a0, (f32x4*)p);
    __builtin_nontemporal_store(a1, (f32x4*)p + 1);
  }
}

// z[j] = lane (j mod 16) of this lane's 16-lane row, from za (j < 16) or zb.
template <int J>
__device__ inline void row_broadcast_z(float (&z)[kMaxParts], float za, float zb, float& m) {
  if constexpr (J < kMaxParts) {
    const float src = J < 16 ? za : zb;
    z[J] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(src), 0x150 + (J & 15), 0xf, 0xf, false));
    m = fmaxf(m, z[J]);
    row_broadcast_z<J + 1>(z, za, zb, m);
  }
}

// Parts are processed in groups of kPartGroup with the group's loads issued
// before any is used.  With BUF (every
// part below 4 GiB) the loads go through buffer resources, and a part with
// w_j = 0 is given an out-of-range offset: no branch, and the hardware fetches
// nothing for it.
template <int D, typename TI, typename TO, bool BUF, bool DENSE>
__global__ __launch_bounds__(256) void merge_kernel(const MergeArgs a, uint32_t part_bytes) {
  constexpr int CPR = D / 8;
  constexpr int W = sizeof(TI) == 2 ? 1 : 2;  // 16-byte words per thread and part
  constexpr uint32_t kNone = 0xfffff000u;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = a.batch * a.rows * a.heads * CPR;
  if (gid >= total) return;
  const int chunk = (int)(gid % CPR);
  const int64_t rh = gid / CPR;  // (b * rows + row) * heads + h
  const int h = (int)(rh % a.heads);
  const int64_t brow = rh / a.heads;
  const int64_t row = brow % a.rows, b = brow / a.rows;
  // Element offsets of the parts' z and O and of the outputs; with DENSE both
  // batch strides equal rows (the 64-bit stride products would delay the loads
  // of this memory-bound kernel by a few percent).
  int64_t lse_idx, o_off, lse_out, out_off;
  if constexpr (DENSE) {
    lse_idx = lse_out = (b * a.heads + h) * a.rows + row;
    o_off = out_off = rh * D + chunk * 8;
  } else {
    lse_idx = (b * a.heads + h) * a.pstride + row;
    o_off = ((b * a.pstride + row) * a.heads + h) * D + chunk * 8;
    lse_out = (b * a.heads + h) * a.ostride + row;
    out_off = ((b * a.ostride + row) * a.heads + h) * D + chunk * 8;
  }
  const int n = a.n_parts;

  // The parts' z for this (row, head).
  float z[kMaxParts];
  float m = -INFINITY;
  if constexpr (CPR == 16) {
    // The 16 threads of a (row, head) are one 16-lane DPP row: lane c loads z
    // of parts c and c + 16, and each z_j reaches the row by a broadcast.
    static_assert(kMaxParts <= 32, "two z per lane");
    const float za = chunk < n ? a.lse_parts[chunk][lse_idx] : -INFINITY;
    const float zb = chunk + 16 < n ? a.lse_parts[chunk + 16][lse_idx] : -INFINITY;
    row_broadcast_z<0>(z, za, zb, m);
  } else {
#pragma unroll
    for (int j0 = 0; j0 < kMaxParts; j0 += 8) {
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) z[j0 + jj] = -INFINITY;
      if (j0 < n) {
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const int j = j0 + jj;
          const float v = a.lse_parts[j < n ? j : n - 1][lse_idx];
          z[j] = j < n ? v : -INFINITY;
          m = fmaxf(m, z[j]);
        }
      }
    }
  }
  float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  if (m != -INFINITY) {
    constexpr int PG = kPartGroup;
#pragma unroll
    for (int j0 = 0; j0 < kMaxParts; j0 += PG) {
      if (j0 >= n) break;
      u32x4 v[PG][W];
#pragma unroll
      for (int jj = 0; jj < PG; ++jj) {
        const int j = j0 + jj;
        const int jc = j < n ? j : n - 1;
        const bool live = j < n && z[j] != -INFINITY;
        if constexpr (BUF) {
          const auto rs = make_rsrc(a.o_parts[jc], part_bytes);
          const uint32_t off = live ? (uint32_t)(o_off * sizeof(TI)) : kNone;
#pragma unroll
          for (int q = 0; q < W; ++q)
            v[jj][q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * q, 0, kNonTemporal));
        } else {
          const u32x4* p = (const u32x4*)((const TI*)a.o_parts[jc] + o_off);
#pragma unroll
          for (int q = 0; q < W; ++q) v[jj][q] = live ? p[q] : u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int jj = 0; jj < PG; ++jj) {
        const int j = j0 + jj;
        const bool live = j < n && z[j] != -INFINITY;
        const float wj = live ? expf(z[j] - m) : 0.f;  // w_j = 0: the part was not read
        float x[8];
        if constexpr (sizeof(TI) == 2) {
          const bf16x8 bv = __builtin_bit_cast(bf16x8, v[jj][0]);
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = (float)bv[e];
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x[e] = __uint_as_float(v[jj][0][e]);
            x[4 + e] = __uint_as_float(v[jj][1][e]);
          }
        }
        den += wj;
#pragma unroll
        for (int e = 0; e < 8; ++e) num[e] = fmaf(wj, x[e], num[e]);
      }
    }
  }
  const bool empty = !(den > 0.f);
  const float inv = empty ? 0.f : 1.f / den;
#pragma unroll
  for (int e = 0; e < 8; ++e) num[e] *= inv;
  store8<TO>((TO*)a.o + out_off, num);
  if (chunk == 0) a.lse[lse_out] = empty ? -INFINITY : m + logf(den);
}

template <int D, bool BUF, bool DENSE>
void launch_dbd(const MergeArgs& a, int pt, int ot, uint32_t part_bytes, dim3 grid, hipStream_t s) {
  if (pt == 0 && ot == 0)
    hipLaunchKernelGGL((merge_kernel<D, bf16, bf16, BUF, DENSE>), grid, dim3(256), 0, s, a, part_bytes);
  if (pt == 0 && ot == 1)
    hipLaunchKernelGGL((merge_kernel<D, bf16, float, BUF, DENSE>), grid, dim3(256), 0, s, a, part_bytes);
  if (pt == 1 && ot == 0)
    hipLaunchKernelGGL((merge_kernel<D, float, bf16, BUF, DENSE>), grid, dim3(256), 0, s, a, part_bytes);
  if (pt == 1 && ot == 1)
    hipLaunchKernelGGL((merge_kernel<D, float, float, BUF, DENSE>), grid, dim3(256), 0, s, a, part_bytes);
}

template <int D, bool BUF>
hipError_t launch_db(const MergeArgs& a, int pt, int ot, uint32_t part_bytes, hipStream_t s) {
  const int64_t total = a.batch * a.rows * a.heads * (D / 8);
  const dim3 grid((unsigned)((total + 255) / 256));
  if (a.pstride == a.rows && a.ostride == a.rows) launch_dbd<D, BUF, true>(a, pt, ot, part_bytes, grid, s);
  else launch_dbd<D, BUF, false>(a, pt, ot, part_bytes, grid, s);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const MergeArgs& a, int pt, int ot, hipStream_t s) {
  const uint64_t bytes = (uint64_t)((a.batch - 1) * a.pstride + a.rows) * a.heads * D * (pt == 0 ? 2 : 4);
  if (bytes <= 0xffff0000ull) return launch_db<D, true>(a, pt, ot, (uint32_t)bytes, s);
  return launch_db<D, false>(a, pt, ot, 0u, s);
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, int head_dim, int part_dtype, int out_dtype, hipStream_t s) {
  if (a.batch * a.rows * a.heads == 0) return hipSuccess;
  return head_dim == 128 ? launch_d<128>(a, part_dtype, out_dtype, s) : launch_d<64>(a, part_dtype, out_dtype, s);
}

}  // namespace bdlm
