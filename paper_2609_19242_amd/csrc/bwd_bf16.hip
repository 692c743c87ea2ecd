// Fused mask-aware BDLM attention backward, bf16 inputs, fp32 accumulation, gfx950.
//
// Exact gradients from the saved O and LSE (arXiv 2609.19242 App. C fused
// backward; eqs. eq:correctness-corrupted-gradient to
// eq:correctness-query-gradient): with P = exp(scale Q K^T + mask - LSE) and
// D = rowsum(dO * O) (from the pre pass),
//   dV = P^T dO,  dS = P * (dO V^T - D),  dK = scale dS^T Q,  dQ = scale dS K,
// where dK/dV sum over every query row of every query range and over the query
// heads of the KV head's GQA group.
//
// KV-major: a workgroup owns 128 keys of one KV head (4 waves x 32 keys), holds
// their K and V rows in registers as MFMA operands and accumulates dK^T and
// dV^T in registers for the whole pass.  It walks the query heads of the group
// and, for each query range, the 32-row query steps that can see its keys (the
// query-side intervals of common.hpp give the span in closed form; steps every
// key sees completely skip the mask test).  Per step and wave:
//   S = Q K^T, dP = dO V^T      (Q, dO rows from LDS as A, K, V from registers as B)
//   dV^T += dO^T P, dK^T += Q^T dS  (dO^T, Q^T via LDS transpose reads; P, dS from registers)
//   dQ[:, slice] += dS K        (dS^T staged in LDS, K tile in LDS, both via transpose reads)
// dQ partial sums go to an fp32 accumulator with global atomics; a post pass
// scales and rounds it.  Q/dO/LSE/D of the next step are prefetched into
// registers while the current step computes.
#include "common.hpp"
#include "device.hpp"

namespace bdlm {

namespace {

constexpr float kLog2e = 1.44269504088896340736f;

template <int D>
__global__ __launch_bounds__(256) void bwd_bf16_kernel(const AttnArgs a) {
  constexpr int BN = kBwdKeysBf16, BM = 32, PITCH = D + 16, KS = D / 16, DT = D / 32, NT = 256;
  constexpr int DSP = 48;  // dS^T row pitch: 32 queries + pad
  constexpr int CPR = D / 8;
  constexpr int QCPT = BM * CPR / NT;
  static_assert(BN == 128 && (BM * CPR) % NT == 0, "tile shape");
  constexpr int NSL = D / 32;           // dQ column slices of 32
  constexpr int NPART = 4 / NSL;        // waves per slice (split over keys)
  constexpr int QKSTEPS = (BN / 16) / NPART;
  __shared__ __attribute__((aligned(16))) bf16 k_lds[BN * PITCH];
  __shared__ __attribute__((aligned(16))) bf16 q_lds[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) bf16 do_lds[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) bf16 ds_lds[BN * DSP];
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

  // ---- K, V rows of this wave's keys (B operands) and the K tile in LDS
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
      *(bf16x8*)(k_lds + mykey * PITCH + 16 * s + 8 * half) = kf[s];
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
  float pst = 0.f;
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
    if (tid < 2 * BM) {
      const int row = row0 + (tid & (BM - 1));
      if (tid < BM) {
        const float z = row < qr.len ? qr.lse[((int64_t)b * H + h) * qr.bstride + row] : -INFINITY;
        pst = (z == -INFINITY) ? INFINITY : z * kLog2e;  // rows seeing nothing get P = 0
      } else {
        pst = row < qr.len ? qr.delta[((int64_t)b * H + h) * qr.len + row] : 0.f;
      }
    }
  };
  auto store_step = [&](int stage) {
#pragma unroll
    for (int n = 0; n < QCPT; ++n) {
      const int cidx = tid + n * NT;
      const int row = cidx / CPR, col = cidx % CPR;
      *(u32x4*)(&q_lds[stage][row * PITCH + col * 8]) = pq[n];
      *(u32x4*)(&do_lds[stage][row * PITCH + col * 8]) = pdo[n];
    }
    if (tid < 2 * BM) st_lds[stage][tid / BM][tid & (BM - 1)] = pst;
  };

  int slot = 0, s = 0, s1 = 0, f0 = 0, f1 = 0;
  bool have = find_from(0, slot, s, s1, f0, f1);
  if (have) {
    load_step(slot, s);
    store_step(0);
  }
  __syncthreads();

  int cur = 0, lane_range = -1, lane_qa = 0, lane_qw = 0;
  const float c = a.scale_log2;
  while (have) {
    int slotn = slot, sn = s + 1, s1n = s1, f0n = f0, f1n = f1;
    bool have_next = sn < s1;
    if (!have_next) have_next = find_from(slot + 1, slotn, sn, s1n, f0n, f1n);
    if (have_next) load_step(slotn, sn);

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

    // S = Q K^T and dP = dO V^T for this wave's 32 keys.
    f32x16 sacc, dpacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      sacc[i] = 0.f;
      dpacc[i] = 0.f;
    }
    {
      const bf16* qa = &q_lds[cur][l32 * PITCH + 8 * half];
      const bf16* da = &do_lds[cur][l32 * PITCH + 8 * half];
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        sacc = mfma32(*(const bf16x8*)(qa + 16 * k), kf[k], sacc);
        dpacc = mfma32(*(const bf16x8*)(da + 16 * k), vf[k], dpacc);
      }
    }

    // P = exp2(S c - LSE log2 e), dS = P (dP - D); the mask only where needed.
    const bool need_mask = !(s >= f0 && s < f1);
    const int mbase = qr.pos0 + s * BM + 4 * half - lane_qa;
    bf16x8 pb[2], dsb[2];
    bf16x4 dst[4];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const f32x4 l2 = *(const f32x4*)(&st_lds[cur][0][8 * g4 + 4 * half]);
      const f32x4 dl = *(const f32x4*)(&st_lds[cur][1][8 * g4 + 4 * half]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = 4 * g4 + e;
        float p = exp2f_fast(fmaf(sacc[i], c, -l2[e]));
        if (need_mask && (unsigned)(mbase + 8 * g4 + e) >= (unsigned)lane_qw) p = 0.f;
        const float ds = p * (dpacc[i] - dl[e]);
        pb[i >> 3][i & 7] = to_bf16(p);
        const bf16 dsh = to_bf16(ds);
        dsb[i >> 3][i & 7] = dsh;
        dst[g4][e] = dsh;
      }
    }

    // dV^T += dO^T P and dK^T += Q^T dS (queries are the contraction index).
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int qrow = 16 * u + 4 * (G >> 1) + (sl >> 2);
      const bf16* dop = &do_lds[cur][qrow * PITCH + 16 * (G & 1) + 4 * (sl & 3)];
      const bf16* qp = &q_lds[cur][qrow * PITCH + 16 * (G & 1) + 4 * (sl & 3)];
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const bf16x8 av = cat(lds_read_tr(dop + 32 * d), lds_read_tr(dop + 32 * d + 8 * PITCH));
        dva[d] = mfma32(av, pb[u], dva[d]);
        const bf16x8 aq = cat(lds_read_tr(qp + 32 * d), lds_read_tr(qp + 32 * d + 8 * PITCH));
        dka[d] = mfma32(aq, dsb[u], dka[d]);
      }
    }

    // dS^T to LDS for the dQ product.
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) *(bf16x4*)(ds_lds + mykey * DSP + 8 * g4 + 4 * half) = dst[g4];
    __syncthreads();

    {
      const int slice = w % NSL, part = w / NSL;
      f32x16 dqa;
#pragma unroll
      for (int i = 0; i < 16; ++i) dqa[i] = 0.f;
#pragma unroll
      for (int kk = 0; kk < QKSTEPS; ++kk) {
        const int krow = 16 * (part * QKSTEPS + kk) + 8 * (G >> 1) + (sl >> 2);
        const bf16* ap = ds_lds + krow * DSP + 16 * (G & 1) + 4 * (sl & 3);
        const bf16* bp = k_lds + krow * PITCH + 32 * slice + 16 * (G & 1) + 4 * (sl & 3);
        const bf16x8 av = cat(lds_read_tr(ap), lds_read_tr(ap + 4 * DSP));
        const bf16x8 bv = cat(lds_read_tr(bp), lds_read_tr(bp + 4 * PITCH));
        dqa = mfma32(av, bv, dqa);
      }
      const int row0 = s * BM;
      float* accp = qr.dqacc + (((int64_t)b * qr.len + row0) * H + h) * D + 32 * slice + l32;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int q = 8 * (i >> 2) + 4 * half + (i & 3);
        if (row0 + q < qr.len) unsafeAtomicAdd(accp + (int64_t)q * H * D, dqa[i]);
      }
    }

    if (have_next) store_step(cur ^ 1);
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
  if (head_dim == 128)
    hipLaunchKernelGGL((bwd_bf16_kernel<128>), dim3(n), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_bf16_kernel<64>), dim3(n), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bdlm
