// BDLM attention forward for fp32 inputs (fp32 end to end), gfx950.
//
// The fp32 path serves small problems that need fp32 accuracy: inputs and
// outputs are fp32, while scores, exponentials and sums are carried in fp64 so
// the only rounding left is the final cast.  One thread owns one query row: it
// walks the visible key interval of every key range (the mask rules of
// common.hpp; arXiv 2609.19242 Sec. 3.2) with an online softmax, so masked keys
// are never touched and no tile classification is needed.  Output: normalised
// O and natural-log LSE; a row that sees no key gets O = 0 and LSE = -inf.
#include "common.hpp"

namespace bdlm {

namespace {

template <int D>
__global__ __launch_bounds__(kFwdRowsF32) void fwd_f32_kernel(const AttnArgs a) {
  const int T = a.total_tiles;
  const int tile = blockIdx.x % T;
  const int bh = blockIdx.x / T;
  const int h = bh % a.heads, b = bh / a.heads;
  int r = 0;
  while (r + 1 < a.n_q && tile >= a.qr[r + 1].tile0) ++r;
  const QRangeArg& qr = a.qr[r];
  const int row = (tile - qr.tile0) * kFwdRowsF32 + (int)threadIdx.x;
  if (row >= qr.len) return;
  const int64_t H = a.heads, HKV = a.kv_heads;
  const int kvh = h / a.group;
  const float* qp = (const float*)qr.q + (((int64_t)b * qr.bstride + row) * H + h) * D;
  float qv[D];
  double acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qv[d] = qp[d];
    acc[d] = 0.0;
  }
  double m = -INFINITY, l = 0.0;
  const double scale = (double)a.scale;
  const int pq = qr.pos0 + row;
  for (int j = 0; j < a.n_k; ++j) {
    const KRangeArg& kr = a.kr[j];
    int lo, hi;
    key_interval(qr.stream, pq, kr.stream, rule_of(a), lo, hi);
    lo = imax(lo, kr.pos0);
    hi = imin(hi, kr.pos0 + kr.len);
    for (int kp = lo; kp < hi; ++kp) {
      const int64_t off = (((int64_t)b * kr.bstride + (kp - kr.pos0)) * HKV + kvh) * D;
      const float* kv = (const float*)kr.k + off;
      const float* vv = (const float*)kr.v + off;
      double s = 0.0;
#pragma unroll
      for (int d = 0; d < D; ++d) s = fma((double)qv[d], (double)kv[d], s);
      s *= scale;
      if (s > m) {
        const double al = exp(m - s);
        l *= al;
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] *= al;
        m = s;
      }
      const double p = exp(s - m);
      l += p;
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] = fma(p, (double)vv[d], acc[d]);
    }
  }
  float* op = (float*)qr.o + (((int64_t)b * qr.bstride + row) * H + h) * D;
  const bool empty = !(l > 0.0);
  const double inv = empty ? 0.0 : 1.0 / l;
#pragma unroll
  for (int d = 0; d < D; ++d) op[d] = (float)(acc[d] * inv);
  qr.lse[((int64_t)b * H + h) * qr.bstride + row] = empty ? -INFINITY : (float)(m + log(l));
}

}  // namespace

hipError_t launch_fwd_f32(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int n = a.total_tiles * a.heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL((fwd_f32_kernel<128>), dim3(n), dim3(kFwdRowsF32), 0, s, a);
  else
    hipLaunchKernelGGL((fwd_f32_kernel<64>), dim3(n), dim3(kFwdRowsF32), 0, s, a);
  return hipGetLastError();
}

}  // namespace bdlm
