// BDLM attention backward for fp32 inputs, gfx950.
//
// Exact gradients from the saved O and LSE (arXiv 2609.19242 App. C; the
// query gradient eq:correctness-query-gradient and the key/value gradients
// summed over every query row, eq:correctness-clean-gradient):
//   P = exp(scale q.k - LSE),  dP = dO.v,  dS = P (dP - D),
//   dQ = scale sum_k dS k,  dK = scale sum_q dS q,  dV = sum_q P dO.
// Inputs and outputs are fp32; scores, exponentials and sums are carried in
// fp64.  Two deterministic passes walk the mask intervals of common.hpp directly:
// one thread per query row for dQ, one thread per (key row, KV head) for dK
// and dV (summing the query heads of its GQA group).  No atomics.
#include "common.hpp"

namespace bdlm {

namespace {

template <int D>
__global__ __launch_bounds__(128) void bwd_dq_f32_kernel(const AttnArgs a) {
  const int T = a.total_tiles;  // query tiles of kFwdRowsF32 rows
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
  const int64_t qoff = (((int64_t)b * qr.bstride + row) * H + h) * D;
  const float* qp = (const float*)qr.q + qoff;
  const float* dop = (const float*)qr.dO + qoff;
  float qv[D], dov[D];
  double dq[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qv[d] = qp[d];
    dov[d] = dop[d];
    dq[d] = 0.0;
  }
  const float lse = qr.lse[((int64_t)b * H + h) * qr.bstride + row];
  const double Dq = (double)qr.delta[((int64_t)b * H + h) * qr.len + row];
  const double scale = (double)a.scale;
  const int pq = qr.pos0 + row;
  if (lse != -INFINITY) {
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
        double s = 0.0, dp = 0.0;
#pragma unroll
        for (int d = 0; d < D; ++d) {
          s = fma((double)qv[d], (double)kv[d], s);
          dp = fma((double)dov[d], (double)vv[d], dp);
        }
        const double p = exp(s * scale - (double)lse);
        const double ds = p * (dp - Dq);
#pragma unroll
        for (int d = 0; d < D; ++d) dq[d] = fma(ds, (double)kv[d], dq[d]);
      }
    }
  }
  float* out = (float*)qr.dq + qoff;
#pragma unroll
  for (int d = 0; d < D; ++d) out[d] = (float)(dq[d] * scale);
}

template <int D>
__global__ __launch_bounds__(128) void bwd_dkv_f32_kernel(const AttnArgs a) {
  const int T = a.total_tiles;  // key tiles of kBwdKeysF32 rows
  const int tile = blockIdx.x % T;
  const int bk = blockIdx.x / T;
  const int kvh = bk % a.kv_heads, b = bk / a.kv_heads;
  int r = 0;
  while (r + 1 < a.n_k && tile >= a.kr[r + 1].tile0) ++r;
  const KRangeArg& kr = a.kr[r];
  const int row = (tile - kr.tile0) * kBwdKeysF32 + (int)threadIdx.x;
  if (row >= kr.len) return;
  const int64_t H = a.heads, HKV = a.kv_heads;
  const int64_t koff = (((int64_t)b * kr.bstride + row) * HKV + kvh) * D;
  const float* kp_ = (const float*)kr.k + koff;
  const float* vp_ = (const float*)kr.v + koff;
  float kv[D], vv[D];
  double dk[D], dv[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    kv[d] = kp_[d];
    vv[d] = vp_[d];
    dk[d] = 0.0;
    dv[d] = 0.0;
  }
  const double scale = (double)a.scale;
  const int pk = kr.pos0 + row;
  for (int hq = 0; hq < a.group; ++hq) {
    const int h = kvh * a.group + hq;
    for (int i = 0; i < a.n_q; ++i) {
      const QRangeArg& qr = a.qr[i];
      int lo, hi;
      query_interval(qr.stream, kr.stream, pk, rule_of(a), lo, hi);
      lo = imax(lo, qr.pos0);
      hi = imin(hi, qr.pos0 + qr.len);
      for (int pq = lo; pq < hi; ++pq) {
        const int qrow = pq - qr.pos0;
        const float lse = qr.lse[((int64_t)b * H + h) * qr.bstride + qrow];
        if (lse == -INFINITY) continue;
        const int64_t qoff = (((int64_t)b * qr.bstride + qrow) * H + h) * D;
        const float* qv = (const float*)qr.q + qoff;
        const float* dov = (const float*)qr.dO + qoff;
        double s = 0.0, dp = 0.0;
#pragma unroll
        for (int d = 0; d < D; ++d) {
          s = fma((double)qv[d], (double)kv[d], s);
          dp = fma((double)dov[d], (double)vv[d], dp);
        }
        const double p = exp(s * scale - (double)lse);
        const double ds = p * (dp - (double)qr.delta[((int64_t)b * H + h) * qr.len + qrow]);
#pragma unroll
        for (int d = 0; d < D; ++d) {
          dv[d] = fma(p, (double)dov[d], dv[d]);
          dk[d] = fma(ds, (double)qv[d], dk[d]);
        }
      }
    }
  }
  float* dkp = (float*)kr.dk + koff;
  float* dvp = (float*)kr.dv + koff;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    dkp[d] = (float)(dk[d] * scale);
    dvp[d] = (float)dv[d];
  }
}

}  // namespace

// a.total_tiles holds the key-tile count; the query-tile count is recomputed here.
hipError_t launch_bwd_f32(const AttnArgs& a, int head_dim, hipStream_t s) {
  AttnArgs aq = a;
  int tq = 0;
  for (int i = 0; i < a.n_q; ++i) {
    aq.qr[i].tile0 = tq;
    tq += (a.qr[i].len + kFwdRowsF32 - 1) / kFwdRowsF32;
  }
  aq.total_tiles = tq;
  const int nq = tq * a.heads * a.batch;
  const int nk = a.total_tiles * a.kv_heads * a.batch;
  if (nq > 0) {
    if (head_dim == 128) hipLaunchKernelGGL((bwd_dq_f32_kernel<128>), dim3(nq), dim3(128), 0, s, aq);
    else hipLaunchKernelGGL((bwd_dq_f32_kernel<64>), dim3(nq), dim3(128), 0, s, aq);
  }
  if (nk > 0) {
    if (head_dim == 128) hipLaunchKernelGGL((bwd_dkv_f32_kernel<128>), dim3(nk), dim3(128), 0, s, a);
    else hipLaunchKernelGGL((bwd_dkv_f32_kernel<64>), dim3(nk), dim3(128), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace bdlm
