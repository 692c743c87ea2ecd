// dQ of the BDLM attention backward, query-major, bf16 inputs, fp32 accumulation, gfx950.
//
// For a query row i (arXiv 2609.19242 App. A, eq:correctness-query-gradient):
//   dQ_i = scale * sum_j dS_ij K_j,  dS_ij = P_ij (dO_i . V_j - D_i),
//   P_ij = exp(scale Q_i . K_j - LSE_i)
// over the keys j the mask lets row i see.  Each workgroup owns BM query rows
// of one head and walks their visible key tiles exactly like the forward
// (qtiles.hpp), so dQ needs no atomics and comes out in one deterministic
// pass: per key tile and wave, S^T = K Q^T and dP^T = V dO^T (K and V from LDS
// as A operands, the wave's Q and dO rows in registers as B operands), P and dS
// in registers (a lane owns one query row, so its LSE and D are scalars), and
// dQ^T += K^T dS^T with K^T read from the row-major K tile by LDS transpose
// reads, the same product shape as the forward's O^T += V^T P^T.
#include "qtiles.hpp"

namespace bdlm {

namespace {

constexpr float kLog2e = 1.44269504088896340736f;

template <int D, int NW, bool HILO>
__global__ __launch_bounds__(NW * 64) void bwd_dq_kernel(const AttnArgs a) {
  constexpr int BM = NW * 32, BN = 64, KS = D / 16, DT = D / 32;
  // K and V row reads at pitch PB; K^T transpose reads from a second copy of K at pitch PT.
  constexpr int PB = pitch_b128(D), PT = pitch_tr(D);
  constexpr int NT = NW * 64;
  constexpr int STAGE = BN * (2 * PB + PT);  // K tile, V tile, K tile again
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int G = lane >> 4, sl = lane & 15;

  const int n_wg = a.total_tiles * a.heads * a.batch;
  const QTileItem it = q_tile_item(a, xcd_remap(blockIdx.x, n_wg));
  const QRangeArg& qr = a.qr[it.r];
  const int kvh = it.h / a.group;
  const int row0 = it.t * BM;
  const int nvalid = imin(BM, qr.len - row0);
  const int64_t H = a.heads;

  // This wave's 32 query rows of Q and dO as MFMA B fragments.
  bf16x8 qf[KS], df[KS];
  {
    const int64_t qoff = (((int64_t)it.b * qr.bstride + row0) * H + it.h) * D;
    const uint32_t bytes = (uint32_t)(((int64_t)(nvalid - 1) * H * D + D) * 2);
    const auto rq = make_rsrc((const bf16*)qr.q + qoff, bytes);
    const auto rdo = make_rsrc((const bf16*)qr.dO + qoff, bytes);
    const uint32_t off = (uint32_t)(((int64_t)(w * 32 + l32) * H * D + 8 * half) * 2);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qf[s] = __builtin_bit_cast(bf16x8, buf_load16(rq, off + s * 32));
      df[s] = __builtin_bit_cast(bf16x8, buf_load16(rdo, off + s * 32));
    }
  }
  const int my_row = row0 + w * 32 + l32;
  const bool row_ok = my_row < qr.len;
  const int pq = qr.pos0 + imin(my_row, qr.len - 1);
  const int pq0 = qr.pos0 + row0, pq1 = qr.pos0 + row0 + nvalid - 1;
  // Rows past the range and rows that see no key get P = 0.
  float lse2 = INFINITY, dl = 0.f;
  if (row_ok) {
    const float z = qr.lse[((int64_t)it.b * H + it.h) * qr.bstride + my_row];
    lse2 = (z == -INFINITY) ? INFINITY : z * kLog2e;
    dl = qr.delta[((int64_t)it.b * H + it.h) * qr.len + my_row];
  }

  f32x16 acc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[d][i] = 0.f;
  const float c = a.scale_log2;

  int j = 0, t = 0, t1 = 0, f0 = 0, f1 = 0;
  bool have = find_key_tile(a, 0, qr.stream, pq0, pq1, BN, j, t, t1, f0, f1);
  KVTileLoader<D, BN, NT> ld;
  int cur = 0;
  int lane_lo = 0, lane_w = 0, lane_j = -1;
  if (have) {
    ld.load(a, j, t, it.b, kvh, tid);
    ld.template store<PB, PB, PT>(lds, lds + BN * PB, tid, lds + 2 * BN * PB);
  }
  __syncthreads();

  while (have) {
    int jn = j, tn = t + 1, t1n = t1, f0n = f0, f1n = f1;
    bool have_next = tn < t1;
    if (!have_next) have_next = find_key_tile(a, j + 1, qr.stream, pq0, pq1, BN, jn, tn, t1n, f0n, f1n);
    if (have_next) ld.load(a, jn, tn, it.b, kvh, tid);
    if (lane_j != j) {
      lane_key_interval(a, j, qr.stream, pq, lane_lo, lane_w);
      lane_j = j;
    }

    const bf16* Ks = lds + cur * STAGE;
    const bf16* Vs = Ks + BN * PB;
    const bf16* Kt = Ks + 2 * BN * PB;
    f32x16 sacc[2], dpacc[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        sacc[u][i] = 0.f;
        dpacc[u][i] = 0.f;
      }
      const bf16* kp = Ks + (u * 32 + l32) * PB + 8 * half;
      const bf16* vp = Vs + (u * 32 + l32) * PB + 8 * half;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        sacc[u] = mfma32(*(const bf16x8*)(kp + 16 * s), qf[s], sacc[u]);
        dpacc[u] = mfma32(*(const bf16x8*)(vp + 16 * s), df[s], dpacc[u]);
      }
    }

    if (!(t >= f0 && t < f1)) {
      const int base = a.kr[j].pos0 + t * BN + 4 * half - lane_lo;
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int kk = base + u * 32 + (i >> 2) * 8 + (i & 3);
          if ((unsigned)kk >= (unsigned)lane_w) sacc[u][i] = -INFINITY;
        }
    }

    // dS^T = P^T (dP^T - D) in the S^T register layout, rounded to bf16
    // (with HILO also the rounding residual, a second bf16 term).
    bf16x8 dsb[4], dsl[4];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = exp2f_fast(fmaf(sacc[u][i], c, -lse2));
        const float ds = p * (dpacc[u][i] - dl);
        const bf16 hi = to_bf16(ds);
        dsb[u * 2 + (i >> 3)][i & 7] = hi;
        if constexpr (HILO) dsl[u * 2 + (i >> 3)][i & 7] = to_bf16(ds - (float)hi);
      }

    // dQ^T[d][q] += sum_key K[key][d] dS[q][key]; key order per 16-key step as in the forward.
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bf16* kp = Kt + (16 * u + 4 * (G >> 1) + (sl >> 2)) * PT + 16 * (G & 1) + 4 * (sl & 3);
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const bf16x8 ka = cat(lds_read_tr(kp + 32 * d), lds_read_tr(kp + 32 * d + 8 * PT));
        acc[d] = mfma32(ka, dsb[u], acc[d]);
        if constexpr (HILO) acc[d] = mfma32(ka, dsl[u], acc[d]);
      }
    }

    if (have_next) {
      bf16* st = lds + (cur ^ 1) * STAGE;
      ld.template store<PB, PB, PT>(st, st + BN * PB, tid, st + 2 * BN * PB);
    }
    __syncthreads();
    cur ^= 1;
    j = jn; t = tn; t1 = t1n; f0 = f0n; f1 = f1n;
    have = have_next;
  }

  if (row_ok) {
    const int64_t orow = (((int64_t)it.b * qr.bstride + my_row) * H + it.h) * D;
    if (a.out_f32) {
      float* op = (float*)qr.dq + orow;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[d][g4 * 4 + e] * a.scale;
          *(f32x4*)(op + 32 * d + 8 * g4 + 4 * half) = v;
        }
    } else {
      bf16* op = (bf16*)qr.dq + orow;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = to_bf16(acc[d][g4 * 4 + e] * a.scale);
          *(bf16x4*)(op + 32 * d + 8 * g4 + 4 * half) = v;
        }
    }
  }
}

}  // namespace

// a.total_tiles / qr[i].tile0 / ntiles must describe kFwdRowsBf16-row query tiles.
hipError_t launch_bwd_dq_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  constexpr int NW = kFwdRowsBf16 / 32;
  const int n = a.total_tiles * a.heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128) {
    if (a.hilo) hipLaunchKernelGGL((bwd_dq_kernel<128, NW, true>), dim3(n), dim3(NW * 64), 0, s, a);
    else hipLaunchKernelGGL((bwd_dq_kernel<128, NW, false>), dim3(n), dim3(NW * 64), 0, s, a);
  } else {
    if (a.hilo) hipLaunchKernelGGL((bwd_dq_kernel<64, NW, true>), dim3(n), dim3(NW * 64), 0, s, a);
    else hipLaunchKernelGGL((bwd_dq_kernel<64, NW, false>), dim3(n), dim3(NW * 64), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace bdlm
