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
// registers for the whole pass.  It walks the 32-row query steps that can see
// its keys, from the end of the query ranges down, and at each step every
// query range and every pair of query heads of the group (steps every key sees
// completely skip the mask test).  Per step and wave:
//   S = Q K^T, dP = dO V^T          (Q, dO rows from LDS as A, K, V from registers as B)
//   dV^T += dO^T P, dK^T += Q^T dS  (dO^T, Q^T via LDS transpose reads; P, dS from registers)
// A step's Q, dO, LSE*log2(e) and D go from global memory straight into one of
// three LDS stages (no register staging), two steps ahead of their use; one
// barrier per step.
#include "common.hpp"
#include "device.hpp"

namespace bdlm {

namespace {

template <int D, int NH>
struct BwdStage {
  // Rows of D elements, no padding; the 16-byte chunks of a row are permuted
  // by chunk_swz (device.hpp) so that neither access pattern has bank conflicts.
  bf16 q[NH * 32 * D];
  bf16 dO[NH * 32 * D];
  float l2[64];  // [head][row]: LSE * log2(e)  (64 floats: one copy instruction)
  float dl[64];  // [head][row]: D
};

// Global -> LDS copy plan of one step.  Each tensor (Q, dO) of a stage is
// NH * 32 rows of D / 8 16-byte chunks, TI copy instructions of 64
// consecutive slots (one per lane; a lane fetches the logical chunk that
// belongs in its physical slot).  Waves 0 and 1 copy Q, waves 2 and 3 copy
// dO, each wave one half of the tensor's instructions, so a wave's copies need
// no per-instruction choice of tensor; waves 2 and 3 also copy the
// LSE*log2(e) and D rows (one dword instruction each).  NMIN is the smallest
// per-wave instruction count of a step: waiting for vmcnt <= NMIN after
// issuing the next step leaves only that step's copies in flight.
template <int D, int NH>
struct CopyPlan {
  static constexpr int SLOTS = D / 8;
  static constexpr int TI = NH * 32 * SLOTS / 64;
  static constexpr int IPW = TI / 2;
  static constexpr int NMIN = IPW;
  static_assert(TI % 2 == 0, "whole copy instructions per wave");
};

// NQ: query-range slots the walk considers (2 when the call has at most two
// query ranges, else kMaxQ); fewer slots keep the walk state in fewer registers.
// HM: 0 single-term P and dS, 1 two-term on every step, 2 two-term on the
// 16-query halves of a step holding a probability of at least hilo_tau.
template <int D, int HM, int NH, int NQ>
__global__ __launch_bounds__(256) void bwd_bf16_kernel(const AttnArgs a) {
  constexpr int BN = kBwdKeysBf16, BM = 32, KS = D / 16, DT = D / 32;
  using Stage = BwdStage<D, NH>;
  using Plan = CopyPlan<D, NH>;
  constexpr uint32_t RB = D * 2, HB = BM * RB, TB = NH * HB;  // row, head and tensor bytes in a stage
  static_assert(BN == 128, "tile shape");
  static_assert(sizeof(Stage) % 256 == 0, "stage bases stay 256-byte aligned");
  __shared__ __attribute__((aligned(256))) Stage stages[3];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  const int G = lane >> 4, sl = lane & 15;
  const int64_t H = a.heads, HKV = a.kv_heads;

  // ---- work item: (batch, KV head, key range, key tile); heaviest tiles first per XCD
  const int T = a.total_tiles;
  const int logical = xcd_remap(blockIdx.x, T * a.kv_heads * a.batch);
  int bk, order;
  pair_and_rank(logical, T, a.kv_heads * a.batch, bk, order);
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
    // Keep the K/V operands in AGPRs: MFMAs read their A/B operands from AGPRs
    // directly, while the VGPRs go to the accumulators and the per-step tiles.
    // Left to itself the allocator spills them to AGPRs and copies each one
    // back before every use (64 register-file copies per step).
#pragma unroll
    for (int s = 0; s < KS; ++s) asm volatile("" : "+a"(kf[s]), "+a"(vf[s]));
  }

  f32x16 dka[DT], dva[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      dka[d][i] = 0.f;
      dva[d][i] = 0.f;
    }

  // ---- iteration order.  Per query range, the 32-row steps that can see this
  // tile's keys form a span [s0, s1) (the query-side intervals of common.hpp
  // give it in closed form) with a sub-span [f0, f1) that every key sees
  // completely.  Steps are walked from the highest index down; at each index
  // every range active there is visited (in range order), and in each range
  // every pair of query heads.  Visible query rows extend to the end of a range
  // for every key tile, so all workgroups resident on an XCD start on the same
  // rows and stay close together: their Q/dO reads are shared in L2.
  // Per range: steps [s0, s1), fully visible steps [f0, f1), the queries
  // [qa, qa + qw) of the range that see this lane's key, and the copy bases of
  // this wave (its tensor at the first row and first head of the group; for
  // waves 2 and 3 the LSE*log2(e) or D row of that head, and the bytes from
  // there to the end of the array).  Named slots (not an array) so that every
  // field stays in registers.
  struct Span {
    int s0, s1, f0, f1, pos0, qa, qw, len;
    const bf16* tb;
    const float* lb;
    uint32_t lrec;
  };
  static_assert(NQ == 2 || NQ == kMaxQ, "query-range slots");
  auto make_span = [&](int q) -> Span {
    Span sp{0, 0, 0, 0, 0, 0, 0, 0, nullptr, nullptr, 0u};
    if (q >= NQ || q >= a.n_q) return sp;
    const QRangeArg& qr = a.qr[q];
    sp.pos0 = qr.pos0;
    sp.len = qr.len;
    const int h0 = kvh * a.group;
    sp.tb = (const bf16*)(w < 2 ? qr.q : qr.dO) + ((int64_t)b * qr.bstride * H + h0) * D;
    const int64_t lrow = ((int64_t)b * H + h0) * qr.len;
    sp.lb = (w == 2 ? qr.l2 : qr.delta) + lrow;
    sp.lrec = (uint32_t)(((int64_t)a.batch * H * qr.len - lrow) * 4);
    int lo0, hi0, lo1, hi1;
    query_interval(qr.stream, kr.stream, kpos_first, rule_of(a), lo0, hi0);
    query_interval(qr.stream, kr.stream, kpos_last, rule_of(a), lo1, hi1);
    const int u0 = imax(lo0 - qr.pos0, 0), u1 = imin(hi1 - qr.pos0, qr.len);
    if (u1 > u0) {
      sp.s0 = u0 / BM;
      sp.s1 = (u1 + BM - 1) / BM;
      const int i0 = imax(lo1 - qr.pos0, 0), i1 = imin(hi0 - qr.pos0, qr.len);
      if (i1 > i0 && !ragged) {
        sp.f0 = (i0 + BM - 1) / BM;
        sp.f1 = i1 / BM;
      }
    }
    int lo, hi;
    query_interval(qr.stream, kr.stream, pk, rule_of(a), lo, hi);
    lo = imax(lo, qr.pos0);
    hi = imin(hi, qr.pos0 + qr.len);
    sp.qa = lo;
    sp.qw = key_ok ? imax(hi - lo, 0) : 0;
    return sp;
  };
  static_assert(kMaxQ == 4, "four range slots");
  const Span R0 = make_span(0), R1 = make_span(1), R2 = make_span(2), R3 = make_span(3);
  // Select by value (a select of member addresses would force the spans into memory).
  auto sel4 = [](int q, auto v0, auto v1, auto v2, auto v3) {
    if constexpr (NQ == 2) return q ? v1 : v0;
    else return q == 0 ? v0 : q == 1 ? v1 : q == 2 ? v2 : v3;
  };
#define BDLM_PICK(f, q) sel4((q), R0.f, R1.f, R2.f, R3.f)
  auto active = [](const Span& sp, int s) { return sp.s0 <= s && s < sp.s1; };
  // First range after q that is active at step s (kMaxQ if none).
  auto range_at = [&](int s, int q) -> int {
    return (q < 0 && active(R0, s)) ? 0 : (q < 1 && active(R1, s)) ? 1
         : (q < 2 && active(R2, s)) ? 2 : (q < 3 && active(R3, s)) ? 3 : kMaxQ;
  };
  // Highest step below s that some range covers (-1 if none).
  auto below = [](const Span& sp, int s) {
    const int cand = imin(s - 1, sp.s1 - 1);
    return cand >= sp.s0 ? cand : -1;
  };
  auto step_below = [&](int s) -> int {
    return imax(imax(below(R0, s), below(R1, s)), imax(below(R2, s), below(R3, s)));
  };
  // A cursor is (range, head pair, step); step < 0 once the walk is over.
  struct Cursor {
    int q, hp, s;
  };
  const int npairs = a.group / NH;
  auto advance = [&](Cursor c) __attribute__((always_inline)) -> Cursor {
    if (c.s < 0) return c;
    if (++c.hp < npairs) return c;
    c.hp = 0;
    const int qn = range_at(c.s, c.q);
    if (qn != kMaxQ) {
      c.q = qn;
      return c;
    }
    c.s = step_below(c.s);
    c.q = c.s >= 0 ? range_at(c.s, -1) : 0;
    return c;
  };

  // ---- copy plan: per-lane global byte offsets of this wave's instructions
  // inside one step's NH heads x 32 rows (constant over the walk; the step
  // moves the resource base).  Instruction i of the wave is instruction
  // (w & 1) * IPW + i of its tensor.
  const int wodd = w & 1;
  uint32_t voff[Plan::IPW];
#pragma unroll
  for (int i = 0; i < Plan::IPW; ++i) {
    const int slot = (wodd * Plan::IPW + i) * 64 + lane;
    const int row = slot / Plan::SLOTS, ch = (slot % Plan::SLOTS) ^ chunk_swz<D>(row);
    const int j = row / BM, rr = row % BM;
    voff[i] = (uint32_t)(((rr * H + j) * D + ch * 8) * 2);
  }
  // Issue the copies of step c into stage S (empty copies when c is past the end).
  auto copy_step = [&](Stage& S, const Cursor c) __attribute__((always_inline)) {
    const bool live = c.s >= 0;
    const int q = live ? c.q : 0;
    const int row0 = c.s * BM;
    const int len = BDLM_PICK(len, q);
    const int nrows = live ? imin(BM, len - row0) : 0;
    const int hoff = c.hp * NH;
    const uint32_t bytes = live ? (uint32_t)(((int64_t)(nrows - 1) * H + NH) * D * 2) : 0u;
    const auto rt = make_rsrc(BDLM_PICK(tb, q) + ((int64_t)row0 * H + hoff) * D, bytes);
    bf16* dst = (w < 2 ? S.q : S.dO) + wodd * Plan::IPW * 512;
#pragma unroll
    for (int i = 0; i < Plan::IPW; ++i) buf_to_lds<16>(rt, dst + i * 512, voff[i], 0);
    if (w >= 2) {
      // LSE*log2(e) (wave 2) or D (wave 3) of the NH heads' rows, [head][row]
      // floats.  Each resource ends with its array, so rows past the end of the
      // last head read zeros; other rows past the range end read finite values
      // of the next head (those rows are always masked).
      const int64_t loff = (int64_t)hoff * len + row0;
      const uint32_t lbytes = live ? BDLM_PICK(lrec, q) - (uint32_t)(loff * 4) : 0u;
      const auto rl = make_rsrc(BDLM_PICK(lb, q) + loff, lbytes);
      const uint32_t vo = NH == 2 ? (uint32_t)(((lane >> 5) * len + (lane & 31)) * 4) : (uint32_t)(lane * 4);
      buf_to_lds<4>(rl, w == 2 ? S.l2 : S.dl, vo, 0);
    }
  };

  const float c = a.scale_log2;
  // Per-lane parts of the swizzled LDS read addresses (device.hpp).
  const uint32_t yrow = swz_row_part<D>(l32, half);
  const uint32_t ytr0 = swz_tr_part<D>(G, sl, 0), ytr1 = swz_tr_part<D>(G, sl, 8);
  // One step of the walk on stage S: S = Q K^T, dP = dO V^T, P, dS, then
  // dV^T += dO^T P, dK^T += Q^T dS for every head of the pair.
  auto compute_step = [&](const Stage& S, const Cursor cu) __attribute__((always_inline)) {
    const bool partial = !(cu.s >= BDLM_PICK(f0, cu.q) && cu.s < BDLM_PICK(f1, cu.q));
    const int mbase = BDLM_PICK(pos0, cu.q) + cu.s * BM + 4 * half - BDLM_PICK(qa, cu.q);
    const int lane_qw = BDLM_PICK(qw, cu.q);

    // Row reads: lane (half, l32) reads logical chunk 2k + half of row l32,
    // i.e. zr ^ 32k; heads and the dO tensor are immediate offsets.
    const uint32_t zr = lds_addr(&S) + yrow;
    if constexpr (HM == 0) {
      f32x16 sacc[NH], dpacc[NH];
#pragma unroll
      for (int j = 0; j < NH; ++j) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          sacc[j][i] = 0.f;
          dpacc[j][i] = 0.f;
        }
#pragma unroll
        for (int k = 0; k < KS; ++k) {
          const uint32_t a = (zr ^ (32u * k)) + j * HB;
          sacc[j] = mfma32(lds_load16(a), kf[k], sacc[j]);
          dpacc[j] = mfma32(lds_load16(a + TB), vf[k], dpacc[j]);
        }
      }

      // P = exp2(S c - LSE log2 e) and dS = P (dP - D) per head; the mask only
      // on partly visible steps.  Rows past the range end read Q = dO = 0 and are
      // always masked.
      bf16x8 pb[NH][2], dsb[NH][2];
#pragma unroll
      for (int j = 0; j < NH; ++j) {
        if (partial) {
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if ((unsigned)(mbase + 8 * (i >> 2) + (i & 3)) >= (unsigned)lane_qw) sacc[j][i] = -INFINITY;
        }
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const f32x4 l2 = *(const f32x4*)(&S.l2[j * BM + 8 * g4 + 4 * half]);
          const f32x4 dl = *(const f32x4*)(&S.dl[j * BM + 8 * g4 + 4 * half]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = 4 * g4 + e;
            const float p = exp2f_fast(fmaf(sacc[j][i], c, -l2[e]));
            const float ds = p * (dpacc[j][i] - dl[e]);
            const bf16 phi = to_bf16(p);
            pb[j][i >> 3][i & 7] = phi;
            const bf16 hi = to_bf16(ds);
            dsb[j][i >> 3][i & 7] = hi;
          }
        }
      }

      // dV^T += dO^T P and dK^T += Q^T dS (queries are the contraction index),
      // one head and one 16-query half at a time with its transposed fragments.
      // Transpose reads: rows 16u + R0 (zt0) and 16u + R0 + 8 (zt1), logical
      // 8-byte piece 8d + 4 (G & 1) + (sl & 3) of the row, i.e. zt ^ 64d.
      const uint32_t zt0 = lds_addr(&S) + ytr0, zt1 = lds_addr(&S) + ytr1;
#pragma unroll
      for (int j = 0; j < NH; ++j) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
          for (int d = 0; d < DT; ++d) {
            const uint32_t a0 = (zt0 ^ (64u * d)) + j * HB + u * 16 * RB;
            const uint32_t a1 = (zt1 ^ (64u * d)) + j * HB + u * 16 * RB;
            const bf16x8 doT = cat(lds_read_tr_at(a0 + TB), lds_read_tr_at(a1 + TB));
            const bf16x8 qT = cat(lds_read_tr_at(a0), lds_read_tr_at(a1));
            dva[d] = mfma32(doT, pb[j][u], dva[d]);
            dka[d] = mfma32(qT, dsb[j][u], dka[d]);
          }
        }
      }
    } else if constexpr (HM == 1) {
      f32x16 sacc[NH], dpacc[NH];
#pragma unroll
      for (int j = 0; j < NH; ++j) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          sacc[j][i] = 0.f;
          dpacc[j][i] = 0.f;
        }
#pragma unroll
        for (int k = 0; k < KS; ++k) {
          const uint32_t a = (zr ^ (32u * k)) + j * HB;
          sacc[j] = mfma32(lds_load16(a), kf[k], sacc[j]);
          dpacc[j] = mfma32(lds_load16(a + TB), vf[k], dpacc[j]);
        }
      }

      // P = exp2(S c - LSE log2 e) and dS = P (dP - D) per head; the mask only
      // on partly visible steps.  Rows past the range end read Q = dO = 0 and are
      // always masked.
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
          const f32x4 l2 = *(const f32x4*)(&S.l2[j * BM + 8 * g4 + 4 * half]);
          const f32x4 dl = *(const f32x4*)(&S.dl[j * BM + 8 * g4 + 4 * half]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = 4 * g4 + e;
            const float p = exp2f_fast(fmaf(sacc[j][i], c, -l2[e]));
            const float ds = p * (dpacc[j][i] - dl[e]);
            const bf16 phi = to_bf16(p);
            pb[j][i >> 3][i & 7] = phi;
            pl[j][i >> 3][i & 7] = to_bf16(p - (float)phi);
            const bf16 hi = to_bf16(ds);
            dsb[j][i >> 3][i & 7] = hi;
            dsl[j][i >> 3][i & 7] = to_bf16(ds - (float)hi);
          }
        }
      }

      // dV^T += dO^T P and dK^T += Q^T dS (queries are the contraction index),
      // one head and one 16-query half at a time with its transposed fragments.
      // Transpose reads: rows 16u + R0 (zt0) and 16u + R0 + 8 (zt1), logical
      // 8-byte piece 8d + 4 (G & 1) + (sl & 3) of the row, i.e. zt ^ 64d.
      const uint32_t zt0 = lds_addr(&S) + ytr0, zt1 = lds_addr(&S) + ytr1;
#pragma unroll
      for (int j = 0; j < NH; ++j) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
          for (int d = 0; d < DT; ++d) {
            const uint32_t a0 = (zt0 ^ (64u * d)) + j * HB + u * 16 * RB;
            const uint32_t a1 = (zt1 ^ (64u * d)) + j * HB + u * 16 * RB;
            const bf16x8 doT = cat(lds_read_tr_at(a0 + TB), lds_read_tr_at(a1 + TB));
            const bf16x8 qT = cat(lds_read_tr_at(a0), lds_read_tr_at(a1));
            dva[d] = mfma32(doT, pb[j][u], dva[d]);
            dva[d] = mfma32(doT, pl[j][u], dva[d]);
            dka[d] = mfma32(qT, dsb[j][u], dka[d]);
            dka[d] = mfma32(qT, dsl[j][u], dka[d]);
          }
        }
      }
    } else {
      // S = Q K^T and dP = dO V^T of head j of the pair.
      auto scores = [&](int j, f32x16& sa, f32x16& dpa) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          sa[i] = 0.f;
          dpa[i] = 0.f;
        }
#pragma unroll
        for (int k = 0; k < KS; ++k) {
          const uint32_t a = (zr ^ (32u * k)) + j * HB;
          sa = mfma32(lds_load16(a), kf[k], sa);
          dpa = mfma32(lds_load16(a + TB), vf[k], dpa);
        }
      };
      // P = exp2(S c - LSE log2 e) and dS = P (dP - D) of head j, to bf16 (with
      // lo, the rounding residuals); the mask only on partly visible steps.
      // Rows past the range end read Q = dO = 0 and are always masked.
      auto probs = [&](int j, f32x16& sa, const f32x16& dpa, bf16x8 (&pp)[2], bf16x8 (&dd)[2], float (&pmax)[2],
                       auto lo) __attribute__((always_inline)) {
        if (partial) {
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if ((unsigned)(mbase + 8 * (i >> 2) + (i & 3)) >= (unsigned)lane_qw) sa[i] = -INFINITY;
        }
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const f32x4 l2 = *(const f32x4*)(&S.l2[j * BM + 8 * g4 + 4 * half]);
          const f32x4 dl = *(const f32x4*)(&S.dl[j * BM + 8 * g4 + 4 * half]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = 4 * g4 + e;
            const float p = exp2f_fast(fmaf(sa[i], c, -l2[e]));
            const float ds = p * (dpa[i] - dl[e]);
            if constexpr (decltype(lo)::value) {
              pp[i >> 3][i & 7] = to_bf16(p - (float)to_bf16(p));
              dd[i >> 3][i & 7] = to_bf16(ds - (float)to_bf16(ds));
            } else {
              pp[i >> 3][i & 7] = to_bf16(p);
              dd[i >> 3][i & 7] = to_bf16(ds);
              pmax[i >> 3] = fmaxf(pmax[i >> 3], p);
            }
          }
        }
      };

      // dV^T += dO^T P and dK^T += Q^T dS (queries are the contraction index),
      // one head and one 16-query half at a time with its transposed fragments.
      // Transpose reads: rows 16u + R0 (zt0) and 16u + R0 + 8 (zt1), logical
      // 8-byte piece 8d + 4 (G & 1) + (sl & 3) of the row, i.e. zt ^ 64d.
      const uint32_t zt0 = lds_addr(&S) + ytr0, zt1 = lds_addr(&S) + ytr1;
      auto products = [&](int j, const bf16x8 (&pp)[2], const bf16x8 (&dd)[2]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
          for (int d = 0; d < DT; ++d) {
            const uint32_t a0 = (zt0 ^ (64u * d)) + j * HB + u * 16 * RB;
            const uint32_t a1 = (zt1 ^ (64u * d)) + j * HB + u * 16 * RB;
            const bf16x8 doT = cat(lds_read_tr_at(a0 + TB), lds_read_tr_at(a1 + TB));
            const bf16x8 qT = cat(lds_read_tr_at(a0), lds_read_tr_at(a1));
            dva[d] = mfma32(doT, pp[u], dva[d]);
            dka[d] = mfma32(qT, dd[u], dka[d]);
          }
        }
      };
      // Two-term products, one head at a time: a 16-query half of the head
      // also carries P - bf16(P) and dS - bf16(dS) as second bf16 terms when
      // some probability in it reaches hilo_tau.
#pragma unroll
      for (int j = 0; j < NH; ++j) {
        f32x16 sa, dpa;
        scores(j, sa, dpa);
        bf16x8 pb[2], dsb[2];
        float pmax[2] = {0.f, 0.f};
        probs(j, sa, dpa, pb, dsb, pmax, std::false_type{});
        products(j, pb, dsb);
        const bool two0 = __builtin_amdgcn_ballot_w64(pmax[0] >= a.hilo_tau) != 0;
        const bool two1 = __builtin_amdgcn_ballot_w64(pmax[1] >= a.hilo_tau) != 0;
        if (two0 || two1) {
          bf16x8 pl[2], dsl[2];
          probs(j, sa, dpa, pl, dsl, pmax, std::true_type{});
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            if (u == 0 ? two0 : two1) {
#pragma unroll
              for (int d = 0; d < DT; ++d) {
                const uint32_t a0 = (zt0 ^ (64u * d)) + j * HB + u * 16 * RB;
                const uint32_t a1 = (zt1 ^ (64u * d)) + j * HB + u * 16 * RB;
                dva[d] = mfma32(cat(lds_read_tr_at(a0 + TB), lds_read_tr_at(a1 + TB)), pl[u], dva[d]);
                dka[d] = mfma32(cat(lds_read_tr_at(a0), lds_read_tr_at(a1)), dsl[u], dka[d]);
              }
            }
          }
        }
      }
    }
  };

  // ---- the walk: three LDS stages, copies two steps ahead.  At the barrier
  // closing a step, every wave has waited for its copies of the next step
  // (only the copies of the step after it stay in flight), and every wave has
  // finished reading the stage the following step's copies overwrite.
  Cursor c0;
  c0.s = step_below(kBig);
  c0.q = c0.s >= 0 ? range_at(c0.s, -1) : 0;
  c0.hp = 0;
  Cursor c1 = advance(c0), c2 = advance(c1);
  copy_step(stages[0], c0);
  copy_step(stages[1], c1);
  vm_wait_barrier<Plan::NMIN>();
  int cur = 0;
  while (c0.s >= 0) {
    const int nx2 = cur == 0 ? 2 : cur - 1;  // (cur + 2) % 3
    copy_step(stages[nx2], c2);
    compute_step(stages[cur], c0);
    vm_wait_barrier<Plan::NMIN>();
    cur = cur == 2 ? 0 : cur + 1;
    c0 = c1;
    c1 = c2;
    c2 = advance(c2);
  }
  // Copies still in flight target stages nobody reads; they must land before
  // the workgroup's LDS is released.
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
#undef BDLM_PICK

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

template <int D, int HM, int NQ>
void launch_nh(const AttnArgs& a, int n, hipStream_t s) {
  if (a.group % 2 == 0)
    hipLaunchKernelGGL((bwd_bf16_kernel<D, HM, 2, NQ>), dim3(n), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_bf16_kernel<D, HM, 1, NQ>), dim3(n), dim3(256), 0, s, a);
}

template <int D, int HM>
void launch_nq(const AttnArgs& a, int n, hipStream_t s) {
  if (a.n_q <= 2) launch_nh<D, HM, 2>(a, n, s);
  else launch_nh<D, HM, kMaxQ>(a, n, s);
}

template <int D>
void launch_hm(const AttnArgs& a, int n, hipStream_t s) {
  if (!(a.hilo & kHiloDkDv)) launch_nq<D, 0>(a, n, s);
  else if (!(a.hilo & kHiloAdaptive)) launch_nq<D, 1>(a, n, s);
  else launch_nq<D, 2>(a, n, s);
}

hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
  const int n = a.total_tiles * a.kv_heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128) launch_hm<128>(a, n, s);
  else launch_hm<64>(a, n, s);
  return hipGetLastError();
}

}  // namespace bdlm
