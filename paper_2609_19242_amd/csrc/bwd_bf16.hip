// dK and dV of the BDLM attention backward, key-major, bf16 inputs, fp32 accumulation, gfx950.
//
// Exact gradients from the saved O and LSE (arXiv 2609.19242 App. C fused
// backward; eq:correctness-corrupted-gradient and eq:correctness-clean-gradient):
// with P = exp(scale Q K^T + mask - LSE) and D = rowsum(dO * O) (pre pass),
//   dV = P^T dO,  dS = P * (dO V^T - D),  dK = scale dS^T Q,
// summed over every query row of every query range and over the query heads
// of the KV head's GQA group.  dQ comes from the query-major kernel in
// bwd_dq.hip, so this kernel needs no atomics.
//
// A workgroup owns 128 keys of one KV head (4 waves x 32 keys), holds their K
// and V rows in registers as MFMA operands and accumulates dK^T and dV^T in
// registers for the whole pass.  It walks the query heads of the group and,
// for each query range, the 32-row query steps that can see its keys (the
// query-side intervals of common.hpp give the span in closed form; steps every
// key sees completely skip the mask test).  Per step and wave:
//   S = Q K^T, dP = dO V^T          (Q, dO rows from LDS as A, K, V from registers as B)
//   dV^T += dO^T P, dK^T += Q^T dS  (dO^T, Q^T via LDS transpose reads; P, dS from registers)
// Q/dO/LSE/D of the next step are prefetched into registers at the top of the
// step and stored to the other LDS stage in its middle; one barrier per step.
#include "common.hpp"
#include "device.hpp"

namespace bdlm {

namespace {

constexpr float kLog2e = 1.44269504088896340736f;

// NH query heads of the GQA group are processed per step (same 32 query
// rows): their products and softmax are independent instruction streams the
// scheduler interleaves, so one head's MFMAs run while the other's VALU work
// issues -- with a single wave per SIMD nothing else could fill those gaps.
template <int D, bool HILO, int NH>
__global__ __launch_bounds__(256) void bwd_bf16_kernel(const AttnArgs a) {
  constexpr int BN = kBwdKeysBf16, BM = 32, PITCH = D + 16, KS = D / 16, DT = D / 32, NT = 256;
  constexpr int CPR = D / 8;
  constexpr int QCPT = NH * BM * CPR / NT;  // 16-byte chunks per thread per tensor and step
  static_assert(BN == 128 && (NH * BM * CPR) % NT == 0, "tile shape");
  __shared__ __attribute__((aligned(16))) bf16 q_lds[2][NH][BM * PITCH];
  __shared__ __attribute__((aligned(16))) bf16 do_lds[2][NH][BM * PITCH];
  __shared__ __attribute__((aligned(16))) float st_lds[2][NH][2][BM];  // [stage][head][lse*log2e | D][row]

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int G = lane >> 4, sl = lane & 15;
  const int64_t H = a.heads, HKV = a.kv_heads;

  // ---- work item: (batch, KV head, key range, key tile); heaviest tiles first per XCD
  const int T = a.total_tiles;
  const int logical = xcd_remap(blockIdx.x, T * a.kv_heads * a.batch);
  const int bk = logical / T;
  int order = logical - bk * T;
  const int b = bk / a.kv_heads, kvh = bk - (bk / a.kv_heads) * a.kv_heads;
  int r = a.order[0], t = order;
  for (int n = 0; n < a.n_k; ++n) {
    const int rr = a.order[n];
    const int nt = a.kr[rr].ntiles;
    if (order < nt) {
      r = rr;
      t = order;
      break;
    }
    order -= nt;
  }
  const KRangeArg& kr = a.kr[r];
  const int key0 = t * BN;
  const int nk = imin(BN, kr.len - key0);
  const bool ragged = nk < BN;
  const int mykey = w * 32 + l32;
  const bool key_ok = mykey < nk;
  const int pk = kr.pos0 + key0 + imin(mykey, nk - 1);
  const int kpos_first = kr.pos0 + key0, kpos_last = kr.pos0 + key0 + nk - 1;

  // ---- K, V rows of this wave's keys (B operands)
  bf16x8 kf[KS], vf[KS];
  {
    const int64_t eoff = (((int64_t)b * kr.bstride + key0) * HKV + kvh) * D;
    const uint32_t bytes = (uint32_t)(((int64_t)(nk - 1) * HKV * D + D) * 2);
    const auto rk = make_rsrc((const bf16*)kr.k + eoff, bytes);
    const auto rv = make_rsrc((const bf16*)kr.v + eoff, bytes);
    const uint32_t off = (uint32_t)(((int64_t)mykey * HKV * D + 8 * half) * 2);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kf[s] = __builtin_bit_cast(bf16x8, buf_load16(rk, off + 32 * s));
      vf[s] = __builtin_bit_cast(bf16x8, buf_load16(rv, off + 32 * s));
    }
  }

  f32x16 dka[DT], dva[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      dka[d][i] = 0.f;
      dva[d][i] = 0.f;
    }

  // ---- iteration: query ranges (outer), query heads of the group, 32-row steps.
  // The span of steps that can see this tile's keys depends only on the range.
  auto span = [&](int qi, int& s0, int& s1, int& f0, int& f1) -> bool {
    const QRangeArg& qr = a.qr[qi];
    int lo0, hi0, lo1, hi1;
    query_interval(qr.stream, kr.stream, kpos_first, a.M, a.intra, lo0, hi0);
    query_interval(qr.stream, kr.stream, kpos_last, a.M, a.intra, lo1, hi1);
    const int u0 = imax(lo0 - qr.pos0, 0), u1 = imin(hi1 - qr.pos0, qr.len);
    if (u1 <= u0) return false;
    s0 = u0 / BM;
    s1 = (u1 + BM - 1) / BM;
    const int i0 = imax(lo1 - qr.pos0, 0), i1 = imin(hi0 - qr.pos0, qr.len);
    f0 = f1 = 0;
    if (i1 > i0 && !ragged) {
      f0 = (i0 + BM - 1) / BM;
      f1 = i1 / BM;
    }
    return true;
  };
  auto first_range = [&](int qi, int& qo, int& s0, int& s1, int& f0, int& f1) -> bool {
    for (; qi < a.n_q; ++qi)
      if (span(qi, s0, s1, f0, f1)) {
        qo = qi;
        return true;
      }
    return false;
  };

  // Prefetch registers of the next step: Q and dO rows of the NH heads (the
  // heads are adjacent in memory, so a step's rows are NH*D contiguous
  // elements), and each lane's row's raw LSE and D for every head.
  u32x4 pq[QCPT], pdo[QCPT];
  float pz[NH], pd[NH];
  int prow_ok = 0;
  auto load_step = [&](int qi, int hp, int step) {
    const QRangeArg& qr = a.qr[qi];
    const int h0 = kvh * a.group + hp * NH;
    const int row0 = step * BM;
    const int nrows = imin(BM, qr.len - row0);
    const int64_t qoff = (((int64_t)b * qr.bstride + row0) * H + h0) * D;
    const uint32_t bytes = (uint32_t)(((int64_t)(nrows - 1) * H * D + NH * D) * 2);
    const auto rq = make_rsrc((const bf16*)qr.q + qoff, bytes);
    const auto rdo = make_rsrc((const bf16*)qr.dO + qoff, bytes);
#pragma unroll
    for (int n = 0; n < QCPT; ++n) {
      const int cidx = tid + n * NT;
      const int row = cidx / (NH * CPR), col = cidx % (NH * CPR);
      const uint32_t off = (uint32_t)(((int64_t)row * H * D + col * 8) * 2);
      pq[n] = buf_load16(rq, off);
      pdo[n] = buf_load16(rdo, off);
    }
#pragma unroll
    for (int j = 0; j < NH; ++j) {
      const auto rl = make_rsrc(qr.lse + ((int64_t)b * H + h0 + j) * qr.bstride + row0, (uint32_t)nrows * 4);
      const auto rd = make_rsrc(qr.delta + ((int64_t)b * H + h0 + j) * qr.len + row0, (uint32_t)nrows * 4);
      pz[j] = buf_load_f32(rl, (uint32_t)(tid & (BM - 1)) * 4);
      pd[j] = buf_load_f32(rd, (uint32_t)(tid & (BM - 1)) * 4);
    }
    prow_ok = (tid & (BM - 1)) < nrows;
  };
  auto store_step = [&](int stage) {
#pragma unroll
    for (int n = 0; n < QCPT; ++n) {
      const int cidx = tid + n * NT;
      const int row = cidx / (NH * CPR), col = cidx % (NH * CPR);
      const int j = col / CPR, cc = col % CPR;
      *(u32x4*)(&q_lds[stage][j][row * PITCH + cc * 8]) = pq[n];
      *(u32x4*)(&do_lds[stage][j][row * PITCH + cc * 8]) = pdo[n];
    }
    // Rows past the range end and rows that see no key get LSE = +inf (P = 0) and D = 0.
#pragma unroll
    for (int j = 0; j < NH; ++j) {
      if (tid < BM) st_lds[stage][j][0][tid] = (prow_ok && pz[j] != -INFINITY) ? pz[j] * kLog2e : INFINITY;
      else if (tid < 2 * BM) st_lds[stage][j][1][tid - BM] = prow_ok ? pd[j] : 0.f;
    }
  };

  const int npairs = a.group / NH;
  int qi = 0, hp = 0, s = 0, s0 = 0, s1 = 0, f0 = 0, f1 = 0;
  bool have = first_range(0, qi, s0, s1, f0, f1);
  s = s0;
  if (have) {
    load_step(qi, hp, s);
    store_step(0);
  }
  __syncthreads();

  // One barrier per step: Q/dO/LSE/D of step n+1 are stored to the other
  // stage during step n; that stage was last read before the previous barrier.
  int cur = 0, lane_range = -1, lane_qa = 0, lane_qw = 0;
  const float c = a.scale_log2;
  while (have) {
    int qin = qi, hpn = hp, sn = s + 1, s0n = s0, s1n = s1, f0n = f0, f1n = f1;
    bool have_next = true;
    if (sn >= s1) {
      if (hp + 1 < npairs) {
        hpn = hp + 1;
        sn = s0;
      } else {
        hpn = 0;
        have_next = first_range(qi + 1, qin, s0n, s1n, f0n, f1n);
        sn = s0n;
      }
    }
    // Unconditional prefetch (the last step re-reads its own rows) keeps the
    // loads at the top of the step, a full step ahead of their LDS store.
    if (have_next) load_step(qin, hpn, sn);
    else load_step(qi, hp, s);

    const QRangeArg& qr = a.qr[qi];
    if (lane_range != qi) {  // queries of range qi that see this lane's key
      int lo, hi;
      query_interval(qr.stream, kr.stream, pk, a.M, a.intra, lo, hi);
      lo = imax(lo, qr.pos0);
      hi = imin(hi, qr.pos0 + qr.len);
      lane_qa = lo;
      lane_qw = key_ok ? imax(hi - lo, 0) : 0;
      lane_range = qi;
    }
    const bool partial = !(s >= f0 && s < f1);
    const int mbase = qr.pos0 + s * BM + 4 * half - lane_qa;
    __builtin_amdgcn_sched_barrier(0);

    // S = Q K^T and dP = dO V^T for this wave's 32 keys, every head.
    f32x16 sacc[NH], dpacc[NH];
#pragma unroll
    for (int j = 0; j < NH; ++j) {
      const bf16* qs = &q_lds[cur][j][0];
      const bf16* dos = &do_lds[cur][j][0];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        sacc[j][i] = 0.f;
        dpacc[j][i] = 0.f;
      }
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        sacc[j] = mfma32(*(const bf16x8*)(qs + l32 * PITCH + 8 * half + 16 * k), kf[k], sacc[j]);
        dpacc[j] = mfma32(*(const bf16x8*)(dos + l32 * PITCH + 8 * half + 16 * k), vf[k], dpacc[j]);
      }
    }

    // P = exp2(S c - LSE log2 e) and dS = P (dP - D) per head; the mask only
    // on partly visible steps.
    bf16x8 pb[NH][2], pl[NH][2], dsb[NH][2], dsl[NH][2];
#pragma unroll
    for (int j = 0; j < NH; ++j) {
      if (partial) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if ((unsigned)(mbase + 8 * (i >> 2) + (i & 3)) >= (unsigned)lane_qw) sacc[j][i] = -INFINITY;
      }
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4 l2 = *(const f32x4*)(&st_lds[cur][j][0][8 * g4 + 4 * half]);
        const f32x4 dl = *(const f32x4*)(&st_lds[cur][j][1][8 * g4 + 4 * half]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * g4 + e;
          const float p = exp2f_fast(fmaf(sacc[j][i], c, -l2[e]));
          const float ds = p * (dpacc[j][i] - dl[e]);
          const bf16 phi = to_bf16(p);
          pb[j][i >> 3][i & 7] = phi;
          if constexpr (HILO) pl[j][i >> 3][i & 7] = to_bf16(p - (float)phi);
          const bf16 hi = to_bf16(ds);
          dsb[j][i >> 3][i & 7] = hi;
          if constexpr (HILO) dsl[j][i >> 3][i & 7] = to_bf16(ds - (float)hi);
        }
      }
    }

    // dV^T += dO^T P and dK^T += Q^T dS (queries are the contraction index),
    // one head and one 16-query half at a time with its transposed fragments.
#pragma unroll
    for (int j = 0; j < NH; ++j) {
      const bf16* qs = &q_lds[cur][j][0];
      const bf16* dos = &do_lds[cur][j][0];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int off = (16 * u + 4 * (G >> 1) + (sl >> 2)) * PITCH + 16 * (G & 1) + 4 * (sl & 3);
#pragma unroll
        for (int d = 0; d < DT; ++d) {
          const bf16x8 doT = cat(lds_read_tr(dos + off + 32 * d), lds_read_tr(dos + off + 32 * d + 8 * PITCH));
          const bf16x8 qT = cat(lds_read_tr(qs + off + 32 * d), lds_read_tr(qs + off + 32 * d + 8 * PITCH));
          dva[d] = mfma32(doT, pb[j][u], dva[d]);
          if constexpr (HILO) dva[d] = mfma32(doT, pl[j][u], dva[d]);
          dka[d] = mfma32(qT, dsb[j][u], dka[d]);
          if constexpr (HILO) dka[d] = mfma32(qT, dsl[j][u], dka[d]);
        }
      }
    }
    store_step(cur ^ 1);

    __syncthreads();
    cur ^= 1;
    qi = qin; hp = hpn; s = sn; s0 = s0n; s1 = s1n; f0 = f0n; f1 = f1n;
    have = have_next;
  }

  // ---- epilogue: dK = scale dK^T^T, dV (rounded to bf16); unseen keys get zeros
  if (key_ok) {
    const int64_t off = (((int64_t)b * kr.bstride + key0 + mykey) * HKV + kvh) * D;
    if (a.out_f32) {
      float* dkp = (float*)kr.dk + off;
      float* dvp = (float*)kr.dv + off;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          f32x4 vk, vv;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            vk[e] = dka[d][4 * g4 + e] * a.scale;
            vv[e] = dva[d][4 * g4 + e];
          }
          *(f32x4*)(dkp + 32 * d + 8 * g4 + 4 * half) = vk;
          *(f32x4*)(dvp + 32 * d + 8 * g4 + 4 * half) = vv;
        }
    } else {
      bf16* dkp = (bf16*)kr.dk + off;
      bf16* dvp = (bf16*)kr.dv + off;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          bf16x4 vk, vv;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            vk[e] = to_bf16(dka[d][4 * g4 + e] * a.scale);
            vv[e] = to_bf16(dva[d][4 * g4 + e]);
          }
          *(bf16x4*)(dkp + 32 * d + 8 * g4 + 4 * half) = vk;
          *(bf16x4*)(dvp + 32 * d + 8 * g4 + 4 * half) = vv;
        }
    }
  }
}

}  // namespace

template <int D, bool HILO>
void launch_nh(const AttnArgs& a, int n, hipStream_t s) {
  if (a.group % 2 == 0)
    hipLaunchKernelGGL((bwd_bf16_kernel<D, HILO, 2>), dim3(n), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_bf16_kernel<D, HILO, 1>), dim3(n), dim3(256), 0, s, a);
}

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int n = a.total_tiles * a.kv_heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128) {
    if (a.hilo) launch_nh<128, true>(a, n, s);
    else launch_nh<128, false>(a, n, s);
  } else {
    if (a.hilo) launch_nh<64, true>(a, n, s);
    else launch_nh<64, false>(a, n, s);
  }
  return hipGetLastError();
}

}  // namespace bdlm
