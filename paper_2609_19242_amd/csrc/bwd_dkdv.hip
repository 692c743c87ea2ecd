// dK and dV of the BDLM attention backward, key-major, bf16 inputs, fp32
// accumulation, head_dim 128, gfx950: the software-pipelined kernel.
//
// Exact gradients from the saved O and LSE (arXiv 2609.19242 App. C fused
// backward; eq:correctness-corrupted-gradient and eq:correctness-clean-gradient):
// with P = exp(scale Q K^T + mask - LSE) and D = rowsum(dO * O),
//   dV = P^T dO,  dS = P * (dO V^T - D),  dK = scale dS^T Q,
// summed over every query row that sees a key and over the query heads of the
// key's GQA group.  dQ comes from the query-major kernel (bwd_dq.hip).
//
// Work split as in bwd_bf16.hip: a workgroup owns 128 keys of one KV head (4
// waves x 32 keys, one wave per SIMD), holds their K and V rows in AGPRs as
// MFMA operands and accumulates dK^T and dV^T in AGPRs over the whole walk of
// visible 32-row query steps (every query range, two query heads per step).
//
// What differs is the schedule of a step.  With one wave per SIMD nothing
// hides a wave's own dependency chain S, dP -> softmax -> dV, dK, so the step
// is written as four blocks of 16 matrix products each, with the vector and
// scalar work placed under them and the order fixed by scheduling fences:
//   A: S_0 = Q_0 K^T, dP_0 = dO_0 V^T (head 0)  under  the LDS-DMA copies of
//      the step three ahead and the copy plan of the step after
//   B: S_1, dP_1 (head 1)      under  P_0 = exp2(c S_0), dS_0 = P_0 dP_0, and
//      the first operand reads of C
//   C: dV += dO_0^T P_0, dK += Q_0^T dS_0   under  P_1 = exp2(c S_1)
//   D: dV += dO_1^T P_1, dK += Q_1^T dS_1   under  dS_1 = P_1 dP_1, the next
//      step's accumulator starts, and its first row reads (issued before the
//      step's barrier: that stage is complete from the barrier before)
// Row operands are read four products ahead, transpose operands eight.  The
// walk's bookkeeping is vector work: the descriptors of 64 steps (block,
// range, partial flag, copy resource words) sit in the lanes of a few VGPRs,
// computed every 56 steps from a closed form (walk_plan, walk_step), and a
// step reads its own with readlane, so a step issues about 27 scalar
// instructions where a scalar cursor took over a hundred.
// S and dP accumulate on top of -LSE/scale and -D read from LDS (the dQ
// kernel, which runs first, writes that form), so the softmax is one multiply
// and one exp2 per score and dS one multiply; rows the mask hides start at
// -inf.  LDS holds four stages, filled by LDS-DMA copies three steps ahead,
// so the next step's data is resident while a step runs; the copies are
// issued as inline assembly, which keeps the compiler from waiting on them
// before every LDS transpose read (it cannot tell which stage a DMA writes).
// The dV/dK products are inline-assembly MFMAs on AGPR accumulators (the S/dP
// products use VGPR accumulators, which the softmax reads).
#include "common.hpp"
#include "device.hpp"

namespace bdlm {

namespace {

constexpr int kD = 128;                 // head_dim
constexpr int kKS = kD / 16;            // k-steps of 16 in a score product
constexpr int kDT = kD / 32;            // 32-wide d tiles of dK^T / dV^T
constexpr int kBM = 32;                 // query rows per step
constexpr int kNH = 2;                  // query heads per step
constexpr int kStages = 4;
constexpr uint32_t kRB = kD * 2;        // bytes per row
constexpr uint32_t kHB = kBM * kRB;     // bytes per head in a stage tile (8 KB)
constexpr uint32_t kTileB = kNH * kHB;  // Q (or dO) tile of a stage (16 KB)
// LDS: the four Q tiles, then the four dO tiles (each region 64 KB, so every
// read address is a per-lane register plus an immediate offset below 2^16),
// then per stage -LSE/scale and -D of the step's 2 x 32 rows.
constexpr uint32_t kQRegion = 0;
constexpr uint32_t kDoRegion = kStages * kTileB;                 // 65536
constexpr uint32_t kStatRegion = 2 * kStages * kTileB;           // 131072
constexpr uint32_t kStatB = 2 * kNH * kBM * 4;                   // 512 bytes per stage
constexpr uint32_t kSpareRegion = kStatRegion + kStages * kStatB; // empty copies of waves 0, 1
constexpr uint32_t kLdsBytes = kSpareRegion + 2 * 256;             // 133632
// Copy plan: a tensor tile of a step is 2 heads x 32 rows x 16 chunks = 1024
// 16-byte slots = 16 instructions of 64 lanes; waves 0-1 copy Q, waves 2-3 dO,
// 8 instructions each; one more dword instruction per wave copies the 64
// floats of -LSE/scale (wave 2) or -D (wave 3) (waves 0, 1: an empty copy).
constexpr int kIPW = 8;

__device__ __forceinline__ void mfma_agpr(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// The same with the two wait states a VALU write of an operand needs before an
// MFMA reads it (the compiler does not pad inline assembly for it).
__device__ __forceinline__ void mfma_agpr_padded(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// Buffer resource as four SGPRs for the inline-assembly copies.
__device__ __forceinline__ u32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  u32x4 r;
  r[0] = (uint32_t)p;
  r[1] = (uint32_t)(p >> 32) & 0xffffu;
  r[2] = bytes;
  r[3] = 0x00020000u;
  return r;
}
// Global -> LDS copy: lane i's 16 (or 4) bytes at voff land at LDS byte
// address m0 + 16 i (4 i); offsets past the resource's end write zeros.
__device__ __forceinline__ void dma16(u32x4 rsrc, uint32_t lds_byte, uint32_t voff) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc), "{m0}"(lds_byte)
               : "memory");
}
__device__ __forceinline__ void dma4(u32x4 rsrc, uint32_t lds_byte, uint32_t voff) {
  asm volatile("s_nop 0\n\tbuffer_load_dword %0, %1, 0 offen lds" ::"v"(voff), "s"(rsrc), "{m0}"(lds_byte)
               : "memory");
}

__device__ __forceinline__ void fence() { __builtin_amdgcn_sched_barrier(0); }

__device__ __forceinline__ f32x4 lds_f4(uint32_t a) {
  return *(__attribute__((address_space(3))) const f32x4*)(uintptr_t)a;
}

// Descriptors of step i of a key tile's walk (walk_step): its 32-row block,
// q | partial << 1, and words 0-2 of the buffer resources of its tensor rows
// (32 rows x 2 heads from block s of range q, head pair hp) and of its
// statistics row; steps past the end copy nothing and are not partial.  Plain
// scalar parameters: as a lambda over captured variables, the compiler turned
// the per-lane selects into indexed loads from a stack copy of the captures.
struct StepDesc {
  int s, flags;
  uint32_t t0, t1, t2, l0, l1, l2;
};
__device__ __forceinline__ StepDesc step_desc(const WalkPlan& wp, int i, int64_t H, bool stats_wave, int len_0,
                                              int len_1, int f0_0, int f0_1, int f1_0, int f1_1, uint32_t lrec_0,
                                              uint32_t lrec_1, uint64_t tb_0, uint64_t tb_1, uint64_t lb_0,
                                              uint64_t lb_1) {
  constexpr int BM = kBM, NH = kNH;
  const WalkStep ws = walk_step(wp, i);
  const bool live = ws.live;
  const int q = live ? ws.q : 0;
  const int blk = ws.s;
  const int row0 = live ? blk * BM : 0;
  const int len = q ? len_1 : len_0;
  const int nrows = imin(BM, len - row0);
  const int hoff = ws.hp * NH;
  StepDesc d;
  d.s = blk;
  const bool part = live && !(blk >= (q ? f0_1 : f0_0) && blk < (q ? f1_1 : f1_0));
  d.flags = q | (part ? 2 : 0);
  const uint64_t tp = (q ? tb_1 : tb_0) + (uint64_t)(((int64_t)row0 * H + hoff) * kD * 2);
  d.t0 = (uint32_t)tp;
  d.t1 = (uint32_t)(tp >> 32) & 0xffffu;
  d.t2 = live ? (uint32_t)((nrows - 1) * (int)H + NH) * kD * 2 : 0u;
  const int loff = live ? hoff * len + row0 : 0;
  const uint64_t lp = (q ? lb_1 : lb_0) + (uint64_t)loff * 4u;
  d.l0 = (uint32_t)lp;
  d.l1 = (uint32_t)(lp >> 32) & 0xffffu;
  d.l2 = (live && stats_wave) ? (q ? lrec_1 : lrec_0) - (uint32_t)loff * 4u : 0u;
  return d;
}

// ADAPT: a step also carries P - bf16(P) and dS - bf16(dS) of a head's
// 16-row half as second bf16 terms when some probability of that half reaches
// hilo_tau (8 more products: head 0's after block B, head 1's after block D,
// each while its P and dS are still in registers).
template <bool ADAPT>
__global__ __launch_bounds__(256) void dkdv_kernel(const AttnArgs a) {
  constexpr int BN = kBwdKeysBf16, BM = kBM, NH = kNH;
  static_assert(BN == 128, "tile shape");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLdsBytes];
  const uint32_t L0 = lds_addr(lds);

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

  // ---- K, V rows of this wave's keys (B operands of the score products), in AGPRs
  bf16x8 kf[kKS], vf[kKS];
  {
    const int64_t eoff = (((int64_t)b * kr.bstride + key0) * HKV + kvh) * kD;
    const uint32_t bytes = (uint32_t)(((int64_t)(nk - 1) * HKV * kD + kD) * 2);
    const auto rk = make_rsrc((const bf16*)kr.k + eoff, bytes);
    const auto rv = make_rsrc((const bf16*)kr.v + eoff, bytes);
    const uint32_t off = (uint32_t)(((int64_t)mykey * HKV * kD + 8 * half) * 2);
#pragma unroll
    for (int s = 0; s < kKS; ++s) {
      kf[s] = __builtin_bit_cast(bf16x8, buf_load16(rk, off + 32 * s));
      vf[s] = __builtin_bit_cast(bf16x8, buf_load16(rv, off + 32 * s));
    }
  }
  // dK^T / dV^T accumulators (AGPRs, written only by the inline-assembly MFMAs)
  f32x16 dka[kDT], dva[kDT];
#pragma unroll
  for (int d = 0; d < kDT; ++d) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      dka[d][i] = 0.f;
      dva[d][i] = 0.f;
    }
    asm volatile("" : "+a"(dka[d]), "+a"(dva[d]));
  }

  // ---- walk over (query range, head pair, step), steps from the end of the
  // ranges down (every range active at a step index, then the next index);
  // the call passes at most two query ranges (the ones with rows).
  struct Span {
    int s0, s1, f0, f1, pos0, qa, qw, len;
    const bf16* tb;
    const float* lb;
    uint32_t lrec;
  };
  auto make_span = [&](int q) __attribute__((always_inline)) -> Span {
    Span sp{0, 0, 0, 0, 0, 0, 0, 0, nullptr, nullptr, 0u};
    if (q >= a.n_q) return sp;
    const QRangeArg& qr = a.qr[q];
    sp.pos0 = qr.pos0;
    sp.len = qr.len;
    const int h0 = kvh * a.group;
    sp.tb = (const bf16*)(w < 2 ? qr.q : qr.dO) + ((int64_t)b * qr.bstride * H + h0) * kD;
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
  const Span R0 = make_span(0), R1 = make_span(1);
  auto sel2 = [](int q, auto v0, auto v1) { return q ? v1 : v0; };
#define BDLM_PICK(f, q) sel2((q), R0.f, R1.f)
  // The walk by step index (walk_plan, walk_step).
  const WalkPlan wp = walk_plan(R0.s0, R0.s1, R1.s0, R1.s1, a.group / NH);
  const int nsteps = wp.nsteps;

  // ---- copies.  Instruction i of a wave is instruction (w & 1) * kIPW + i of
  // its tensor; the per-lane global offsets are constant over the walk.
  const int wodd = w & 1;
  uint32_t voff[kIPW];
#pragma unroll
  for (int i = 0; i < kIPW; ++i) {
    const int slot = (wodd * kIPW + i) * 64 + lane;
    const int row = slot / 16, ch = (slot % 16) ^ chunk_swz<kD>(row);
    const int j = row / BM, rr = row % BM;
    voff[i] = (uint32_t)(((rr * H + j) * kD + ch * 8) * 2);
  }
  // A step's copies: kIPW 16-byte instructions of the wave's tensor and one
  // dword instruction of -LSE/scale (wave 2) or -D (wave 3); waves 0 and 1
  // issue an empty dword copy into a spare LDS row instead, so that every wave
  // has kIPW + 1 copies per step in flight.
  struct CopyPlan {
    u32x4 rt, rl;   // resources: the wave's tensor rows, its -LSE/scale or -D row
    uint32_t lvo;   // per-lane offset of the dword copy
  };
  // Step descriptors, 64 steps at a time: lane l of a batch holds step
  // base + l (step_desc); a step reads them back with one readlane each.
  // Steps past the walk's end copy nothing (zero-size resources) and are not
  // partial.
  const int len_0 = R0.len, len_1 = R1.len, f0_0 = R0.f0, f0_1 = R1.f0, f1_0 = R0.f1, f1_1 = R1.f1;
  const uint32_t lrec_0 = R0.lrec, lrec_1 = R1.lrec;
  const uint64_t tb_0 = (uint64_t)(uintptr_t)R0.tb, tb_1 = (uint64_t)(uintptr_t)R1.tb;
  const uint64_t lb_0 = (uint64_t)(uintptr_t)R0.lb, lb_1 = (uint64_t)(uintptr_t)R1.lb;
  auto make_batch = [&](int base) __attribute__((always_inline)) -> StepDesc {
    return step_desc(wp, base + lane, H, w >= 2, len_0, len_1, f0_0, f0_1, f1_0, f1_1, lrec_0, lrec_1, tb_0, tb_1,
                     lb_0, lb_1);
  };
  StepDesc bt;
  int bbase = 0;
  // Per-lane offsets of the dword copy for each range (rows of two heads).
  const uint32_t lvo0 = (uint32_t)(((lane >> 5) * R0.len + (lane & 31)) * 4);
  const uint32_t lvo1 = (uint32_t)(((lane >> 5) * R1.len + (lane & 31)) * 4);
  auto rl = [&](uint32_t v, int i) __attribute__((always_inline)) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, i - bbase);
  };
  // The copy resources of step i.
  auto copy_plan = [&](int i) __attribute__((always_inline)) -> CopyPlan {
    CopyPlan cp;
    cp.rt[0] = rl(bt.t0, i);
    cp.rt[1] = rl(bt.t1, i);
    cp.rt[2] = rl(bt.t2, i);
    cp.rt[3] = 0x00020000u;
    cp.rl[0] = rl(bt.l0, i);
    cp.rl[1] = rl(bt.l1, i);
    cp.rl[2] = rl(bt.l2, i);
    cp.rl[3] = 0x00020000u;
    cp.lvo = (rl((uint32_t)bt.flags, i) & 1) ? lvo1 : lvo0;
    return cp;
  };
  auto copy_issue = [&](const CopyPlan& cp, int st, int i) __attribute__((always_inline)) {
    if (i < kIPW) {
      dma16(cp.rt, L0 + (w < 2 ? kQRegion : kDoRegion) + st * kTileB + (wodd * kIPW + i) * 1024, voff[i]);
    } else {
      const uint32_t ldst =
          w >= 2 ? L0 + kStatRegion + st * kStatB + (w == 2 ? 0u : 256u) : L0 + kSpareRegion + w * 256;
      dma4(cp.rl, ldst, cp.lvo);
    }
  };
  // The resource words come from readlane, a vector instruction writing scalar
  // registers; a buffer access reading them needs five wait states after it,
  // which the compiler does not insert before inline assembly.  Every plan
  // therefore passes an s_nop 4 that takes its words as inputs before its copies.
  auto plan_ready = [](const CopyPlan& cp) __attribute__((always_inline)) {
    asm volatile("s_nop 4" ::"s"(cp.rt), "s"(cp.rl), "v"(cp.lvo));
  };
  auto copy_step = [&](int st, int i) __attribute__((always_inline)) {
    const CopyPlan cp = copy_plan(i);
    plan_ready(cp);
#pragma unroll
    for (int i = 0; i <= kIPW; ++i) copy_issue(cp, st, i);
  };

  const float c = a.scale_log2;
  // Per-lane read addresses (loop-invariant; stage, head and tensor are immediate offsets).
  // Row reads: lane (half, l32) reads logical chunk 2k + half of row l32.
  // (The dO addresses are laundered through an empty asm statement: otherwise
  // the compiler re-derives them from the Q addresses with an add per read.)
  uint32_t yq[kKS], yd[kKS];
#pragma unroll
  for (int k = 0; k < kKS; ++k) {
    yq[k] = (L0 + kQRegion + swz_row_part<kD>(l32, half)) ^ (32u * k);
    yd[k] = yq[k] + kDoRegion;
    asm volatile("" : "+v"(yd[k]));
  }
  // Transpose reads: rows 16u + R0 and 16u + R0 + 8 of the head's tile, 8-byte
  // piece 8d + 4 (G & 1) + (sl & 3).
  uint32_t tq0[kDT], tq1[kDT], td0[kDT], td1[kDT];
#pragma unroll
  for (int d = 0; d < kDT; ++d) {
    tq0[d] = (L0 + kQRegion + swz_tr_part<kD>(G, sl, 0)) ^ (64u * d);
    tq1[d] = (L0 + kQRegion + swz_tr_part<kD>(G, sl, 8)) ^ (64u * d);
    td0[d] = tq0[d] + kDoRegion;
    td1[d] = tq1[d] + kDoRegion;
    asm volatile("" : "+v"(td0[d]), "+v"(td1[d]));
  }
  // Accumulator starts of a step: for head j, register i of a lane holds query
  // row 8 (i / 4) + 4 half + i % 4 of the step.
  uint32_t ystat = L0 + kStatRegion + (uint32_t)(4 * half) * 4;
  asm volatile("" : "+v"(ystat));  // one base register; stage, head and row offsets stay immediate

  f32x16 sa[NH], da[NH];
  // The first row-read pairs of a step, issued at the end of the step before
  // (its stage is complete from the barrier before that step on).
  constexpr int RA = 4;  // row-read pairs in flight ahead of the score products
  bf16x8 nq[RA], nd[RA];
  // Load the starts of step i (stage st) and apply the mask of partly visible steps.
  auto load_starts = [&](int st, int si) __attribute__((always_inline)) {
    const uint32_t base = ystat + st * kStatB;
#pragma unroll
    for (int j = 0; j < NH; ++j)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4 l = lds_f4(base + (j * BM + 8 * g4) * 4);
        const f32x4 dd = lds_f4(base + 256 + (j * BM + 8 * g4) * 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sa[j][4 * g4 + e] = l[e];
          da[j][4 * g4 + e] = dd[e];
        }
      }
    const int fl = (int)rl((uint32_t)bt.flags, si), q = fl & 1;
    // Partly visible steps: hidden scores start at -inf.  The compare and the
    // selects are inline assembly inside a wave-uniform branch: as plain code
    // the compiler speculates them onto every step.
    if (fl & 2) {
      const int mbase = BDLM_PICK(pos0, q) + (int)rl((uint32_t)bt.s, si) * BM + 4 * half - BDLM_PICK(qa, q);
      const int lane_qw = BDLM_PICK(qw, q);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float x0 = sa[0][i], x1 = sa[1][i];
        uint32_t tmp;
        // hidden when (unsigned)(mbase + row offset of register i) >= lane_qw
        asm volatile(
            "v_add_u32 %2, %3, %4\n\t"
            "v_cmp_lt_u32 vcc, %2, %5\n\t"
            "v_mov_b32 %2, 0xff800000\n\t"
            "v_cndmask_b32 %0, %2, %0, vcc\n\t"
            "v_cndmask_b32 %1, %2, %1, vcc"
            : "+v"(x0), "+v"(x1), "=&v"(tmp)
            : "n"(8 * (i >> 2) + (i & 3)), "v"(mbase), "v"(lane_qw)
            : "vcc");
        sa[0][i] = x0;
        sa[1][i] = x1;
      }
    }
  };

  // The starts of head j of step `cu` (stage st) into s, d, with the mask of
  // partly visible steps (the values load_starts gives that head).
  auto load_head_starts = [&](int st, int si, int j, f32x16& s, f32x16& d) __attribute__((always_inline)) {
    const uint32_t base = ystat + st * kStatB;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const f32x4 l = lds_f4(base + (j * BM + 8 * g4) * 4);
      const f32x4 dd = lds_f4(base + 256 + (j * BM + 8 * g4) * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[4 * g4 + e] = l[e];
        d[4 * g4 + e] = dd[e];
      }
    }
    const int fl = (int)rl((uint32_t)bt.flags, si), q = fl & 1;
    if (fl & 2) {
      const int mbase = BDLM_PICK(pos0, q) + (int)rl((uint32_t)bt.s, si) * BM + 4 * half - BDLM_PICK(qa, q);
      const int lane_qw = BDLM_PICK(qw, q);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float x0 = s[i];
        uint32_t tmp;
        asm volatile(
            "v_add_u32 %1, %2, %3\n\t"
            "v_cmp_lt_u32 vcc, %1, %4\n\t"
            "v_mov_b32 %1, 0xff800000\n\t"
            "v_cndmask_b32 %0, %1, %0, vcc"
            : "+v"(x0), "=&v"(tmp)
            : "n"(8 * (i >> 2) + (i & 3)), "v"(mbase), "v"(lane_qw)
            : "vcc");
        s[i] = x0;
      }
    }
  };

  // One step on stage ST: the copies of step `cp` into stage CP go out under
  // its first products, the starts of step `nx` (stage NX) are loaded under its
  // last ones, and the walk advances under the softmax of head 0.
  constexpr int TA = 8;  // transpose-read pairs in flight ahead of the dV/dK products
  int i0 = 0;    // the current step
  CopyPlan cpl;  // copies of step i0 + 3, planned during the step before
  auto run_step = [&](auto st_c, auto nx_c, int cp_stage) __attribute__((always_inline)) {
    constexpr int ST = decltype(st_c)::value, NX = decltype(nx_c)::value;
    constexpr uint32_t SO = ST * kTileB;  // stage offset inside a tensor region
    // ---- A and B: S_j = Q_j K^T + start, dP_j = dO_j V^T + start, j = 0, 1 (32
    // products), the softmax of head 0 under the products of head 1.
    bf16x8 rq[RA + 1], rd[RA + 1];
    auto rowq = [&](int n) { return lds_load16(yq[n % kKS] + SO + (n / kKS) * kHB); };
    auto rowd = [&](int n) { return lds_load16(yd[n % kKS] + SO + (n / kKS) * kHB); };
#pragma unroll
    for (int n = 0; n < RA; ++n) {
      rq[n] = nq[n];
      rd[n] = nd[n];
    }
    // Transpose reads of blocks C and D: rows 16u .. 16u + 15 of head j.
    auto trd = [&](int j, int u, int d) {
      const uint32_t o = SO + j * kHB + u * 16 * kRB;
      return cat(lds_read_tr_at(td0[d] + o), lds_read_tr_at(td1[d] + o));
    };
    auto trq = [&](int j, int u, int d) {
      const uint32_t o = SO + j * kHB + u * 16 * kRB;
      return cat(lds_read_tr_at(tq0[d] + o), lds_read_tr_at(tq1[d] + o));
    };
    // product m of a head: m < 8 -> dV (u = m / 4, d = m % 4), else dK
    auto opnd = [&](int j, int m) { return m < 8 ? trd(j, m / 4, m % 4) : trq(j, (m - 8) / 4, (m - 8) % 4); };
    bf16x8 tf[TA + 1];
    bf16x8 pb[NH][2], dsb[NH][2];
    float pm[NH][2] = {{0.f, 0.f}, {0.f, 0.f}};  // ADAPT: largest P per head and 16-row half
#pragma unroll
    for (int n = 0; n < 2 * kKS; ++n) {
      if (n + RA < 2 * kKS) {
        rq[(n + RA) % (RA + 1)] = rowq(n + RA);
        rd[(n + RA) % (RA + 1)] = rowd(n + RA);
      }
      if (n >= 2 * kKS - TA) tf[n - (2 * kKS - TA)] = opnd(0, n - (2 * kKS - TA));  // block C's first operands
      const int j = n / kKS, k = n % kKS;
      sa[j] = mfma32(rq[n % (RA + 1)], kf[k], sa[j]);
      da[j] = mfma32(rd[n % (RA + 1)], vf[k], da[j]);
      if (n <= kIPW) copy_issue(cpl, cp_stage, n);
      if (n == kIPW + 3) cpl = copy_plan(i0 + 4);
      if (n == kIPW + 4) plan_ready(cpl);

      if (j == 1) {
        // softmax of head 0: two scores per product pair
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int i = 2 * k + e;
          const float p = exp2f_fast(sa[0][i] * c);
          da[0][i] = p * da[0][i];
          sa[0][i] = p;
          if constexpr (ADAPT) pm[0][i >> 3] = fmaxf(pm[0][i >> 3], p);
        }
        if (k & 1) {
          const int i0 = 2 * (k - 1);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pb[0][(i0 + e) >> 3][(i0 + e) & 7] = to_bf16(sa[0][i0 + e]);
            dsb[0][(i0 + e) >> 3][(i0 + e) & 7] = to_bf16(da[0][i0 + e]);
          }
        }
      }
      fence();
    }
    // ---- C and D: dV^T += dO_j^T P_j, dK^T += Q_j^T dS_j (queries are the
    // contraction index), head 0 under the softmax of head 1, head 1 under
    // dS_1 and the next step's starts.  Per product: two transpose reads.
    // ADAPT: the 16-row half u of head j also carries P - bf16(P) and
    // dS - bf16(dS) (from P_j and dS_j, still in sa[j], da[j]) as second bf16
    // terms when some probability of that half reaches hilo_tau: 4 dV and 4 dK
    // products more.
    auto second_terms = [&](int j) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (__builtin_amdgcn_ballot_w64(pm[j][u] >= a.hilo_tau) != 0) {
          bf16x8 pl, dl;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float p = sa[j][8 * u + e], ds = da[j][8 * u + e];
            pl[e] = to_bf16(p - (float)to_bf16(p));
            dl[e] = to_bf16(ds - (float)to_bf16(ds));
          }
#pragma unroll
          for (int d = 0; d < kDT; ++d) mfma_agpr_padded(dva[d], trd(j, u, d), pl);
#pragma unroll
          for (int d = 0; d < kDT; ++d) mfma_agpr_padded(dka[d], trq(j, u, d), dl);
        }
      }
    };
    if constexpr (ADAPT) {
      second_terms(0);
      fence();
    }
#pragma unroll
    for (int n = 0; n < 32; ++n) {
      if (n + TA < 32) tf[(n + TA) % (TA + 1)] = opnd((n + TA) / 16, (n + TA) % 16);
      const int j = n / 16, m = n % 16;
      if (m < 8) mfma_agpr(dva[m % 4], tf[n % (TA + 1)], pb[j][m / 4]);
      else mfma_agpr(dka[(m - 8) % 4], tf[n % (TA + 1)], dsb[j][(m - 8) / 4]);
      if (j == 0) {
        // P_1 = exp2(c S_1): one score per product
        sa[1][m] = exp2f_fast(sa[1][m] * c);
        if constexpr (ADAPT) pm[1][m >> 3] = fmaxf(pm[1][m >> 3], sa[1][m]);
        if (m & 1) {
          pb[1][m >> 3][(m - 1) & 7] = to_bf16(sa[1][m - 1]);
          pb[1][m >> 3][m & 7] = to_bf16(sa[1][m]);
        }
      } else if (m < 8) {
        // dS_1 = P_1 dP_1 under the dV products of head 1
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int i = 2 * m + e;
          da[1][i] = sa[1][i] * da[1][i];
        }
        if (m & 1) {
          const int i0 = 2 * (m - 1);
#pragma unroll
          for (int e = 0; e < 4; ++e) dsb[1][(i0 + e) >> 3][(i0 + e) & 7] = to_bf16(da[1][i0 + e]);
        }
      } else if (m == 8) {
        if constexpr (!ADAPT) load_starts(NX, i0 + 1);
        else load_head_starts(NX, i0 + 1, 0, sa[0], da[0]);
      }
      fence();
    }
    if constexpr (ADAPT) {
      // head 1's second terms need P_1 and dS_1, which its next starts
      // overwrite: both come after the products here
      second_terms(1);
      load_head_starts(NX, i0 + 1, 1, sa[1], da[1]);
      fence();
    }
#pragma unroll
    for (int i = 0; i < RA; ++i) {
      nq[i] = lds_load16(yq[i] + NX * kTileB);
      nd[i] = lds_load16(yd[i] + NX * kTileB);
    }
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(kIPW + 1) : "memory");
    ++i0;
  };

  // ---- the walk: four LDS stages, copies three steps ahead.  At the barrier
  // closing step i every wave has waited for its copies of step i + 2 (only
  // those of step i + 3 stay in flight) and has finished reading stage i,
  // which the copies issued next overwrite.
  // A batch covers steps bbase .. bbase + 63 and is renewed every 56 steps: an
  // iteration of the loop below starting at step i0 reads steps up to i0 + 7.
  bt = make_batch(0);
  cpl = copy_plan(3);
  plan_ready(cpl);
  copy_step(0, 0);
  copy_step(1, 1);
  copy_step(2, 2);
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(kIPW + 1) : "memory");  // steps 0 and 1 landed
  // K and V are pinned in AGPRs only now: pinning reads them, so their loads
  // (issued first) are waited for here, after the walk set-up and the first
  // copies, instead of before them.
#pragma unroll
  for (int s = 0; s < kKS; ++s) asm volatile("" : "+a"(kf[s]), "+a"(vf[s]));
  load_starts(0, 0);
#pragma unroll
  for (int i = 0; i < RA; ++i) {
    nq[i] = lds_load16(yq[i]);
    nd[i] = lds_load16(yd[i]);
  }
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  while (i0 < nsteps) {
    if (i0 - bbase >= 56) {
      bbase = i0;
      bt = make_batch(bbase);
    }
    run_step(I0{}, I1{}, 3);
    if (i0 >= nsteps) break;
    run_step(I1{}, I2{}, 0);
    if (i0 >= nsteps) break;
    run_step(I2{}, I3{}, 1);
    if (i0 >= nsteps) break;
    run_step(I3{}, I0{}, 2);
  }
  // Copies still in flight target stages nobody reads; they must land before
  // the workgroup's LDS is released.  The last dV/dK products must finish
  // before their accumulators are read.
  asm volatile("s_waitcnt vmcnt(0)\n\ts_nop 15\n\ts_nop 15" ::: "memory");
#undef BDLM_PICK

  // ---- epilogue: dK = scale dK^T^T, dV (bf16 or fp32); unseen keys get zeros
#pragma unroll
  for (int d = 0; d < kDT; ++d) asm volatile("" : "+a"(dka[d]), "+a"(dva[d]));
  if (a.out_f32) {
    if (key_ok) {
      const int64_t off = (((int64_t)b * kr.bstride + key0 + mykey) * HKV + kvh) * kD;
      float* dkp = (float*)kr.dk + off;
      float* dvp = (float*)kr.dv + off;
#pragma unroll
      for (int d = 0; d < kDT; ++d)
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
    }
  } else {
    // Each wave's 32 rows of dK and dV go through its own 16 KB of LDS (in the
    // Q stages, free once every wave has left the walk), so that a store
    // writes 4 whole rows instead of 16 bytes of each of 32 rows.  Chunk c
    // (16 bytes) of row r sits at chunk c ^ (r & 15): conflict-free reads.
    asm volatile("s_barrier" ::: "memory");
    const uint32_t sw = L0 + kQRegion + (uint32_t)w * 16384u;
#pragma unroll
    for (int d = 0; d < kDT; ++d)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        bf16x4 vk, vv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vk[e] = to_bf16(dka[d][4 * g4 + e] * a.scale);
          vv[e] = to_bf16(dva[d][4 * g4 + e]);
        }
        const uint32_t o = (uint32_t)l32 * 256u + (((uint32_t)(4 * d + g4) ^ (uint32_t)(l32 & 15)) * 16u) + 8u * half;
        lds_store8(sw + o, vk);
        lds_store8(sw + 8192u + o, vv);
      }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = i * 4 + (lane >> 4), c = lane & 15;
      const uint32_t o = (uint32_t)r * 256u + (((uint32_t)c ^ (uint32_t)(r & 15)) * 16u);
      const bf16x8 xk = lds_load16(sw + o), xv = lds_load16(sw + 8192u + o);
      if (w * 32 + r < nk) {
        const int64_t go = (((int64_t)b * kr.bstride + key0 + w * 32 + r) * HKV + kvh) * kD + c * 8;
        *(bf16x8*)((bf16*)kr.dk + go) = xk;
        *(bf16x8*)((bf16*)kr.dv + go) = xv;
      }
    }
  }
}

}  // namespace

hipError_t launch_bwd_dkdv(const AttnArgs& a, hipStream_t s) {
  const int n = a.total_tiles * a.kv_heads * a.batch;
  if (n == 0) return hipSuccess;
  // two query heads per step, at most two query ranges (the walk state stays in registers)
  if (a.group % 2 != 0 || a.n_q > 2) return hipErrorInvalidValue;
  if (!(a.hilo & kHiloDkDv)) hipLaunchKernelGGL(dkdv_kernel<false>, dim3(n), dim3(256), 0, s, a);
  else if (a.hilo & kHiloAdaptive) hipLaunchKernelGGL(dkdv_kernel<true>, dim3(n), dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace bdlm
