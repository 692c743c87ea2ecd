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

template <int D, bool HILO>
__global__ __launch_bounds__(256) void bwd_bf16_kernel(const AttnArgs a) {
  constexpr int BN = kBwdKeysBf16, BM = 32, PITCH = D + 16, KS = D / 16, DT = D / 32, NT = 256;
  constexpr int CPR = D / 8;
  constexpr int QCPT = BM * CPR / NT;
  static_assert(BN == 128 && (BM * CPR) % NT == 0, "tile shape");
  __shared__ __attribute__((aligned(16))) bf16 q_lds[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) bf16 do_lds[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) float st_lds[2][2][BM];  // [stage][lse*log2e | D][row]

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

  // ---- iteration over (query head of the group, query range) slots and their steps
  const int nslots = a.group * a.n_q;
  auto span = [&](int slot, int& s0, int& s1, int& f0, int& f1) -> bool {
    const QRangeArg& qr = a.qr[slot % a.n_q];
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
  auto find_from = [&](int slot, int& so, int& s0, int& s1, int& f0, int& f1) -> bool {
    for (; slot < nslots; ++slot)
      if (span(slot, s0, s1, f0, f1)) {
        so = slot;
        return true;
      }
    return false;
  };

  u32x4 pq[QCPT], pdo[QCPT];
  float pz = 0.f, pd = 0.f;  // raw LSE and D of row (tid % 32) of the prefetched step
  int prow_ok = 0;
  auto load_step = [&](int slot, int step) {
    const QRangeArg& qr = a.qr[slot % a.n_q];
    const int h = kvh * a.group + slot / a.n_q;
    const int row0 = step * BM;
    const int nrows = imin(BM, qr.len - row0);
    const int64_t qoff = (((int64_t)b * qr.bstride + row0) * H + h) * D;
    const uint32_t bytes = (uint32_t)(((int64_t)(nrows - 1) * H * D + D) * 2);
    const auto rq = make_rsrc((const bf16*)qr.q + qoff, bytes);
    const auto rdo = make_rsrc((const bf16*)qr.dO + qoff, bytes);
#pragma unroll
    for (int n = 0; n < QCPT; ++n) {
      const int cidx = tid + n * NT;
      const int row = cidx / CPR, col = cidx % CPR;
      const uint32_t off = (uint32_t)(((int64_t)row * H * D + col * 8) * 2);
      pq[n] = buf_load16(rq, off);
      pdo[n] = buf_load16(rdo, off);
    }
    // Branch-free: every lane reads row (tid % 32)'s LSE and D; the values
    // are only interpreted when stored, so nothing waits on them here.
    const auto rl = make_rsrc(qr.lse + ((int64_t)b * H + h) * qr.bstride + row0, (uint32_t)nrows * 4);
    const auto rd = make_rsrc(qr.delta + ((int64_t)b * H + h) * qr.len + row0, (uint32_t)nrows * 4);
    pz = buf_load_f32(rl, (uint32_t)(tid & (BM - 1)) * 4);
    pd = buf_load_f32(rd, (uint32_t)(tid & (BM - 1)) * 4);
    prow_ok = (tid & (BM - 1)) < nrows;
  };
  auto store_step = [&](int stage) {
#pragma unroll
    for (int n = 0; n < QCPT; ++n) {
      const int cidx = tid + n * NT;
      const int row = cidx / CPR, col = cidx % CPR;
      *(u32x4*)(&q_lds[stage][row * PITCH + col * 8]) = pq[n];
      *(u32x4*)(&do_lds[stage][row * PITCH + col * 8]) = pdo[n];
    }
    // Rows past the range end and rows that see no key get LSE = +inf (P = 0) and D = 0.
    if (tid < BM) st_lds[stage][0][tid] = (prow_ok && pz != -INFINITY) ? pz * kLog2e : INFINITY;
    else if (tid < 2 * BM) st_lds[stage][1][tid - BM] = prow_ok ? pd : 0.f;
  };

  int slot = 0, s = 0, s1 = 0, f0 = 0, f1 = 0;
  bool have = find_from(0, slot, s, s1, f0, f1);
  if (have) {
    load_step(slot, s);
    store_step(0);
  }
  __syncthreads();

  // One barrier per step: Q/dO/LSE/D of step n+1 are stored to the other
  // stage during step n; that stage was last read before the previous barrier.
  int cur = 0, lane_range = -1, lane_qa = 0, lane_qw = 0;
  const float c = a.scale_log2;
  while (have) {
    int slotn = slot, sn = s + 1, s1n = s1, f0n = f0, f1n = f1;
    bool have_next = sn < s1;
    if (!have_next) have_next = find_from(slot + 1, slotn, sn, s1n, f0n, f1n);
    // Unconditional prefetch (the last step re-reads its own rows) keeps the
    // loads at the top of the step, a full step ahead of their LDS store.
    if (have_next) load_step(slotn, sn);
    else load_step(slot, s);
    __builtin_amdgcn_sched_barrier(0);

    const int qi = slot % a.n_q;
    const QRangeArg& qr = a.qr[qi];
    const int h = kvh * a.group + slot / a.n_q;
    if (lane_range != qi) {  // queries of range qi that see this lane's key
      int lo, hi;
      query_interval(qr.stream, kr.stream, pk, a.M, a.intra, lo, hi);
      lo = imax(lo, qr.pos0);
      hi = imin(hi, qr.pos0 + qr.len);
      lane_qa = lo;
      lane_qw = key_ok ? imax(hi - lo, 0) : 0;
      lane_range = qi;
    }

    // S = Q K^T and dP = dO V^T for this wave's 32 keys (A operands read up front).
    const bf16* qs = &q_lds[cur][0];
    const bf16* dos = &do_lds[cur][0];
    f32x16 sacc, dpacc;
    {
      bf16x8 qa[KS], da[KS];
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        qa[k] = *(const bf16x8*)(qs + l32 * PITCH + 8 * half + 16 * k);
        da[k] = *(const bf16x8*)(dos + l32 * PITCH + 8 * half + 16 * k);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        sacc[i] = 0.f;
        dpacc[i] = 0.f;
      }
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        sacc = mfma32(qa[k], kf[k], sacc);
        dpacc = mfma32(da[k], vf[k], dpacc);
      }
    }
    // dO^T and Q^T fragments for dV and dK, and the rows' LSE and D.
    bf16x8 doT[2][DT], qT[2][DT];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int off = (16 * u + 4 * (G >> 1) + (sl >> 2)) * PITCH + 16 * (G & 1) + 4 * (sl & 3);
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        doT[u][d] = cat(lds_read_tr(dos + off + 32 * d), lds_read_tr(dos + off + 32 * d + 8 * PITCH));
        qT[u][d] = cat(lds_read_tr(qs + off + 32 * d), lds_read_tr(qs + off + 32 * d + 8 * PITCH));
      }
    }
    f32x4 l2[4], dl[4];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      l2[g4] = *(const f32x4*)(&st_lds[cur][0][8 * g4 + 4 * half]);
      dl[g4] = *(const f32x4*)(&st_lds[cur][1][8 * g4 + 4 * half]);
    }

    // P = exp2(S c - LSE log2 e), dS = P (dP - D); the mask only where needed.
    if (!(s >= f0 && s < f1)) {  // partly visible step: hide the masked pairs (P = 0)
      const int mbase = qr.pos0 + s * BM + 4 * half - lane_qa;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if ((unsigned)(mbase + 8 * (i >> 2) + (i & 3)) >= (unsigned)lane_qw) sacc[i] = -INFINITY;
    }
    bf16x8 pb[2], pl[2], dsb[2], dsl[2];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 4 * g4 + e;
        const float p = exp2f_fast(fmaf(sacc[i], c, -l2[g4][e]));
        const float ds = p * (dpacc[i] - dl[g4][e]);
        const bf16 phi = to_bf16(p);
        pb[i >> 3][i & 7] = phi;
        if constexpr (HILO) pl[i >> 3][i & 7] = to_bf16(p - (float)phi);
        const bf16 hi = to_bf16(ds);
        dsb[i >> 3][i & 7] = hi;
        if constexpr (HILO) dsl[i >> 3][i & 7] = to_bf16(ds - (float)hi);
      }
    }
    store_step(cur ^ 1);

    // dV^T += dO^T P and dK^T += Q^T dS (queries are the contraction index).
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        dva[d] = mfma32(doT[u][d], pb[u], dva[d]);
        if constexpr (HILO) dva[d] = mfma32(doT[u][d], pl[u], dva[d]);
        dka[d] = mfma32(qT[u][d], dsb[u], dka[d]);
        if constexpr (HILO) dka[d] = mfma32(qT[u][d], dsl[u], dka[d]);
      }

    __syncthreads();
    cur ^= 1;
    slot = slotn; s = sn; s1 = s1n; f0 = f0n; f1 = f1n;
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

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int n = a.total_tiles * a.kv_heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128) {
    if (a.hilo) hipLaunchKernelGGL((bwd_bf16_kernel<128, true>), dim3(n), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((bwd_bf16_kernel<128, false>), dim3(n), dim3(256), 0, s, a);
  } else {
    if (a.hilo) hipLaunchKernelGGL((bwd_bf16_kernel<64, true>), dim3(n), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((bwd_bf16_kernel<64, false>), dim3(n), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace bdlm
