// Backward pre-pass of the fp32 path, gfx950 (an HBM-bound elementwise pass).
//
// D[b][h][row] = sum_d dO * O in fp32: the row dot the softmax gradient
// dS = P * (dP - D) needs (arXiv 2609.19242 App. C reuses the saved O), and
// L2 = LSE * log2(e) (+inf for rows that see no key, so that exp2(s - L2) is 0
// for them), the per-row values the fp32 backward kernel reads.  (The bf16
// path computes D inside its dQ kernel.)  One thread per 8 consecutive
// head_dim elements; the D/8 threads of one (row, head) are adjacent lanes and
// reduce with cross-lane shuffles.
#include "common.hpp"
#include "device.hpp"

namespace bdlm {

namespace {

template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const AttnArgs a) {
  constexpr int CPR = D / 8;
  const QRangeArg& qr = a.qr[blockIdx.y];
  const int64_t H = a.heads;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)a.batch * qr.len * H * CPR;
  const bool ok = gid < total;
  const int64_t g = ok ? gid : 0;
  const int chunk = (int)(g % CPR);
  const int64_t rh = g / CPR;  // (b * len + row) * H + h
  const int h = (int)(rh % H);
  const int64_t brow = rh / H;
  const int64_t len = qr.len > 0 ? qr.len : 1;  // a range of no rows launches no thread with ok set
  const int64_t row = brow % len, b = brow / len;
  const int64_t off = ((b * qr.bstride + row) * H + h) * D + chunk * 8;
  float s = 0.f;
  if (ok) {
    const float* o = (const float*)qr.o + off;
    const float* d = (const float*)qr.dO + off;
#pragma unroll
    for (int e = 0; e < 8; ++e) s = fmaf(o[e], d[e], s);
  }
#pragma unroll
  for (int w = CPR / 2; w > 0; w >>= 1) s += __shfl_xor(s, w, CPR);
  if (!ok) return;
  if (chunk == 0) {
    const float z = qr.lse[(b * H + h) * qr.bstride + row];
    qr.delta[(b * H + h) * qr.len + row] = s;
    qr.l2[(b * H + h) * qr.len + row] = (z == -INFINITY) ? INFINITY : z * 1.44269504088896340736f;
  }
}

int64_t max_q_threads(const AttnArgs& a, int cpr) {
  int64_t m = 0;
  for (int i = 0; i < a.n_q; ++i) {
    const int64_t t = (int64_t)a.batch * a.qr[i].len * a.heads * cpr;
    m = t > m ? t : m;
  }
  return m;
}

}  // namespace

hipError_t launch_bwd_pre(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int64_t t = max_q_threads(a, head_dim / 8);
  if (t == 0) return hipSuccess;
  const dim3 grid((unsigned)((t + 255) / 256), a.n_q);
  if (head_dim == 128) hipLaunchKernelGGL((bwd_pre_kernel<128>), grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL((bwd_pre_kernel<64>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bdlm
