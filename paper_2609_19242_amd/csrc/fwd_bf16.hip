// Fused mask-aware BDLM attention forward, bf16 inputs, fp32 accumulation, gfx950.
//
// Computes, for every query row of the query ranges, softmax(scale Q K^T + mask) V
// and the row log-sum-exp over all key ranges (arXiv 2609.19242, Sec. 3.2 mask;
// eq:context-parallel-attention), flash-style with an online softmax, so the
// partial attention of App. C (one key range) is the same kernel with n_k = 1.
//
// Workgroup: NW waves, 32 query rows per wave (BM = 32*NW rows of one head):
// 8 waves and three K/V stages on long walks (one workgroup per CU), 4 waves
// and two stages on short ones (two workgroups per CU, so that one's start-up
// and barriers overlap the other's products).
// Per key tile (BN = 64 keys) each wave computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (K from LDS as the A operand, the wave's Q rows held
// in registers as B), so a lane owns one query row and 32 of the tile's keys;
// the row max (needed only when the lazily kept running max moves) takes one
// permlane32 swap and the row sum stays split across the two half-waves until
// the epilogue.  O^T += V^T P^T uses the probabilities straight from the S^T
// registers as the B operand, and V^T fragments come from the row-major V tile
// through LDS transpose reads.  K/V tiles arrive by LDS-DMA copies NS - 1
// tiles ahead into NS stages, one barrier per tile, their rows stored unpadded
// with a row-dependent XOR permutation of 16-byte chunks under which both the
// row reads and the transpose reads are free of bank conflicts.  A wave none
// of whose rows sees a partly visible tile skips it.
//
// Masking: each lane's visible keys in a key range are one position interval
// (the rules in common.hpp).  Tiles inside every lane's interval run without a
// mask test, tiles outside all of them are never visited, and the O(1) tiles
// per range in between test each element against the lane's interval.
#include "qtiles.hpp"

namespace bdlm {

namespace {

constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kSumLimit = 18446744073709551616.f;  // 2^64: a lane's tile sum of p above which m_run moves

template <int D, int NW, int NS, int HM>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void fwd_bf16_kernel(
    const AttnArgs a) {
  constexpr int BM = NW * 32, BN = 64, KS = D / 16, DT = D / 32;
  constexpr uint32_t RB = D * 2, TB = BN * RB;  // row and tile bytes in LDS
  constexpr int STAGE = 2 * BN * D;             // K tile + V tile (elements), swizzled rows
  // Copies: each tile is BN * D / 8 16-byte slots, TI instructions of 64 lanes;
  // waves 0 .. NW/2 - 1 copy K and the others V, IPW instructions each.
  constexpr int TI = BN * D / 8 / 64, IPW = TI / (NW / 2);
  static_assert(TI % (NW / 2) == 0, "whole copy instructions per wave");
  __shared__ __attribute__((aligned(256))) bf16 lds[NS * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  const int G = lane >> 4, sl = lane & 15;

  const int n_wg = a.total_tiles * a.heads * a.batch;
  const QTileItem it = q_tile_item(a, xcd_remap(blockIdx.x, n_wg));
  const QRangeArg& qr = a.qr[it.r];
  const int kvh = it.h / a.group;
  const int row0 = it.t * BM;
  const int nvalid = imin(BM, qr.len - row0);
  const int64_t H = a.heads, HKV = a.kv_heads;

  // This wave's 32 query rows as MFMA B fragments (rows past the range read as zero).
  bf16x8 qf[KS];
  {
    const bf16* qbase = (const bf16*)qr.q + (((int64_t)it.b * qr.bstride + row0) * H + it.h) * D;
    const auto rs = make_rsrc(qbase, (uint32_t)(((int64_t)(nvalid - 1) * H * D + D) * 2));
    const uint32_t off = (uint32_t)(((int64_t)(w * 32 + l32) * H * D + 8 * half) * 2);
#pragma unroll
    for (int s = 0; s < KS; ++s) qf[s] = __builtin_bit_cast(bf16x8, buf_load16(rs, off + s * 32));
  }
  const int my_row = row0 + w * 32 + l32;
  const int pq = qr.pos0 + imin(my_row, qr.len - 1);
  const int pq0 = qr.pos0 + row0, pq1 = qr.pos0 + row0 + nvalid - 1;

  f32x16 acc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[d][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float c = a.scale_log2;

  // Key tiles in visiting order: (key range j, tile t), the range's last
  // visible tile t1 and its fully visible tiles [f0, f1).  Wave-uniform.
  struct KCur {
    int j, t, t1, f0, f1;
    bool have;
  };
  auto next_tile = [&](KCur c) -> KCur {
    if (!c.have) return c;
    if (++c.t < c.t1) return c;
    c.have = find_key_tile(a, c.j + 1, qr.stream, pq0, pq1, BN, c.j, c.t, c.t1, c.f0, c.f1);
    return c;
  };
  // The copy cursor runs NS - 1 tiles ahead of the compute cursor and carries
  // the source pointer of its tile (this wave's tensor, batch and KV head
  // applied) and the rows left in its range, so that advancing inside a range
  // is one pointer increment; both are recomputed only when the range changes.
  struct CopyCur {
    KCur c;
    const bf16* src;
    int rows_left;
  };
  const bool kwave = w < NW / 2;
  auto copy_seek = [&](CopyCur cc) -> CopyCur {
    if (cc.c.have) {
      const KRangeArg& kr = a.kr[cc.c.j];
      cc.src = (const bf16*)(kwave ? kr.k : kr.v) +
               (((int64_t)it.b * kr.bstride + (int64_t)cc.c.t * BN) * HKV + kvh) * D;
      cc.rows_left = kr.len - cc.c.t * BN;
    }
    return cc;
  };
  auto copy_next = [&](CopyCur cc) -> CopyCur {
    if (!cc.c.have) return cc;
    if (++cc.c.t < cc.c.t1) {
      cc.src += (int64_t)BN * HKV * D;
      cc.rows_left -= BN;
      return cc;
    }
    cc.c.have = find_key_tile(a, cc.c.j + 1, qr.stream, pq0, pq1, BN, cc.c.j, cc.c.t, cc.c.t1, cc.c.f0, cc.c.f1);
    return copy_seek(cc);
  };
  // LDS-DMA copy of the cursor's tile into stage st (empty copies past the
  // last tile, so every wave issues IPW per tile); rows past the range end
  // read zeros.
  uint32_t voff[IPW];
  const int cw = w % (NW / 2);
#pragma unroll
  for (int i = 0; i < IPW; ++i) voff[i] = swz_src_offset<D>((cw * IPW + i) * 64 + lane, HKV * D);
  const bf16* const any_src = (const bf16*)a.kr[0].k;
  auto copy_tile = [&](bf16* st, const CopyCur& cc) __attribute__((always_inline)) {
    const int nrows = cc.c.have ? imin(BN, cc.rows_left) : 0;
    const uint32_t bytes = cc.c.have ? (uint32_t)(((nrows - 1) * (int)HKV * D + D) * 2) : 0u;
    const auto r = make_rsrc(cc.c.have ? cc.src : any_src, bytes);
    bf16* dst = st + (kwave ? 0 : BN * D) + cw * IPW * 512;
#pragma unroll
    for (int i = 0; i < IPW; ++i) buf_to_lds<16>(r, dst + i * 512, voff[i], 0);
  };
  // Per-lane parts of the swizzled read addresses (device.hpp).
  const uint32_t yrow = swz_row_part<D>(l32, half);
  const uint32_t ytr0 = swz_tr_part<D>(G, sl, 0), ytr1 = swz_tr_part<D>(G, sl, 8);

  // NS LDS stages, copies NS - 1 tiles ahead.  At the barrier closing a
  // tile, every wave has waited for its copies of the next tile (only those
  // of the NS - 2 tiles after it stay in flight) and has finished reading
  // the stage the following copies overwrite.  (The compiler makes each
  // tile's first transpose read wait for every copy in flight, so a third
  // stage gains nothing over two except a shorter wait at the barrier.)
  KCur c0;
  c0.have = find_key_tile(a, 0, qr.stream, pq0, pq1, BN, c0.j, c0.t, c0.t1, c0.f0, c0.f1);
  CopyCur cp = copy_seek(CopyCur{c0, any_src, 0});
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) {
    copy_tile(lds + s * STAGE, cp);
    cp = copy_next(cp);
  }
  vm_wait_barrier<IPW * (NS - 2)>();
  int cur = 0;
  int lane_lo = 0, lane_w = 0, lane_j = -1;
  while (c0.have) {
    copy_tile(lds + (cur == 0 ? NS - 1 : cur - 1) * STAGE, cp);
    const int j = c0.j, t = c0.t, f0 = c0.f0, f1 = c0.f1;
    if (lane_j != j) {  // this lane's visible key interval inside range j
      lane_key_interval(a, j, qr.stream, pq, lane_lo, lane_w);
      lane_j = j;
    }

    // On a partly visible tile, a wave none of whose rows sees any of the
    // tile's keys skips it (it still copies and meets the barrier).
    bool skip = false;
    if (!(t >= f0 && t < f1)) {
      const int kstart = a.kr[j].pos0 + t * BN - lane_lo;
      skip = __builtin_amdgcn_ballot_w64(lane_w > 0 && kstart < lane_w && kstart + BN > 0) == 0;
    }
    if (!skip) {
      // S^T = K Q^T: K rows 32u + l32 by row reads (K tile at the stage base).
      const uint32_t sb = lds_addr(lds + cur * STAGE);
      const uint32_t zr = sb + yrow;
      f32x16 sacc[2];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 16; ++i) sacc[u][i] = 0.f;
      {
        // K fragments are read LA k-steps ahead of their products; the
        // scheduling fences keep the compiler from sinking each read down to
        // the product that uses it (which left every MFMA waiting on an LDS
        // read issued one product earlier).
        constexpr int LA = 3;
        bf16x8 kf[LA + 1][2];
#pragma unroll
        for (int s = 0; s < LA; ++s)
#pragma unroll
          for (int u = 0; u < 2; ++u) kf[s][u] = lds_load16((zr ^ (32u * s)) + u * 32 * RB);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          if (s + LA < KS) {
#pragma unroll
            for (int u = 0; u < 2; ++u) kf[(s + LA) % (LA + 1)][u] = lds_load16((zr ^ (32u * (s + LA))) + u * 32 * RB);
          }
#pragma unroll
          for (int u = 0; u < 2; ++u) sacc[u] = mfma32(kf[s % (LA + 1)][u], qf[s], sacc[u]);
          __builtin_amdgcn_sched_barrier(0);
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

      // V^T operands of P V (V tile by transpose reads), product n = (16-key
      // step n / DT, d tile n % DT).  The first PA are read here, before the
      // softmax, whose vector work then covers their latency; the rest are
      // read PA products ahead.
      const uint32_t zt0 = sb + TB + ytr0, zt1 = sb + TB + ytr1;
      auto vop = [&](int n) {
        const int u = n / DT, d = n % DT;
        return cat(lds_read_tr_at((zt0 ^ (64u * d)) + u * 16 * RB), lds_read_tr_at((zt1 ^ (64u * d)) + u * 16 * RB));
      };
      constexpr int PA = 4, NP = 4 * DT;
      bf16x8 vr[PA + 1];
      if constexpr (HM != 1) {
#pragma unroll
        for (int n = 0; n < PA; ++n) vr[n] = vop(n);
      }

      // HM 2: a 16-key chunk of the tile also carries P - bf16(P) as a second
      // bf16 term when some lane's largest p in it reaches hilo_tau times the
      // lane's running sum.  The row sum only grows, so an element whose final
      // probability reaches hilo_tau always passes this test.
      float psum;
      bf16x8 pb[4], pl[4];
      float cmax[4];
      auto probs = [&](float m_use) __attribute__((always_inline)) {
        psum = 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k) cmax[k] = 0.f;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float p = exp2f_fast(fmaf(sacc[u][i], c, -m_use));
            psum += p;
            const bf16 hi = to_bf16(p);
            pb[u * 2 + (i >> 3)][i & 7] = hi;
            if constexpr (HM != 0) pl[u * 2 + (i >> 3)][i & 7] = to_bf16(p - (float)hi);
            if constexpr (HM == 2) cmax[u * 2 + (i >> 3)] = fmaxf(cmax[u * 2 + (i >> 3)], p);
          }
      };
      // Lazy rescaling: the running max m_run of a row moves only on the row's
      // first visible tile or when p = exp2(s c - m_run) summed over a lane's
      // part of the tile exceeds 2^64; the tile max is computed only then.
      // Otherwise the stale max stays (every p <= 2^64: no overflow in fp32
      // or bf16, and l_run, O and the final LSE all use the same m_run).  The
      // tests are wave-uniform, so the O rescale (64 multiplies per lane) and
      // the max are skipped for the whole wave on almost every tile.
      bool rescale = __builtin_amdgcn_ballot_w64(m_run == -INFINITY) != 0;
      if (!rescale) {
        probs(m_run);
        rescale = __builtin_amdgcn_ballot_w64(psum > kSumLimit) != 0;
      }
      if (rescale) {
        float mx = -INFINITY;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[u][i]);
        mx = fmaxf(mx, partner(mx));
        const float m_new = fmaxf(m_run, mx * c);
        const float alpha = exp2f_fast(m_run - ((m_new == -INFINITY) ? 0.f : m_new));
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < DT; ++d)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[d][i] *= alpha;
        m_run = m_new;
        probs((m_run == -INFINITY) ? 0.f : m_run);
      }
      const float lim = a.hilo_tau * l_run;
      l_run += psum;

      // O^T[d][q] += sum_key V[key][d] P[q][key]; the key order inside each
      // 16-key step follows the S^T register layout (see device.hpp).
      auto pv = [&](const bf16x8 (&pp)[4]) __attribute__((always_inline)) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int n = 0; n < NP; ++n) {
          if (n + PA < NP) vr[(n + PA) % (PA + 1)] = vop(n + PA);
          acc[n % DT] = mfma32(vr[n % (PA + 1)], pp[n / DT], acc[n % DT]);
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      if constexpr (HM == 1) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
          for (int d = 0; d < DT; ++d) {
            const bf16x8 va = cat(lds_read_tr_at((zt0 ^ (64u * d)) + u * 16 * RB),
                                  lds_read_tr_at((zt1 ^ (64u * d)) + u * 16 * RB));
            acc[d] = mfma32(va, pb[u], acc[d]);
            acc[d] = mfma32(va, pl[u], acc[d]);
          }
        }
      } else {
        pv(pb);
        if constexpr (HM == 2) {
          // second terms of the chunks that hold a large p (V^T fragments re-read)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (__builtin_amdgcn_ballot_w64(cmax[u] >= lim) != 0) {
#pragma unroll
              for (int d = 0; d < DT; ++d) {
                const bf16x8 va = cat(lds_read_tr_at((zt0 ^ (64u * d)) + u * 16 * RB),
                                      lds_read_tr_at((zt1 ^ (64u * d)) + u * 16 * RB));
                acc[d] = mfma32(va, pl[u], acc[d]);
              }
            }
          }
        }
      }
    }

    vm_wait_barrier<IPW * (NS - 2)>();
    cur = cur == NS - 1 ? 0 : cur + 1;
    c0 = next_tile(c0);
    cp = copy_next(cp);
  }
  // Copies still in flight target stages nobody reads; they must land before
  // the workgroup's LDS is released.
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)

  // Epilogue: O = O^T / l (bf16), LSE = ln(2) * (m + log2 l); empty rows O = 0, LSE = -inf.
  const float l_tot = l_run + partner(l_run);
  const bool empty = !(l_tot > 0.f);
  const float inv = empty ? 0.f : 1.f / l_tot;
  if (a.out_f32) {
    if (my_row < qr.len) {
      float* op = (float*)qr.o + (((int64_t)it.b * qr.bstride + my_row) * H + it.h) * D;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[d][g4 * 4 + e] * inv;
          *(f32x4*)(op + 32 * d + 8 * g4 + 4 * half) = v;
        }
    }
  } else {
    // bf16 O through LDS (the stages are free: every wave's copies have landed
    // and every wave has left the walk once all meet this barrier).
    asm volatile("s_barrier" ::: "memory");
    const int wrow0 = row0 + w * 32;
    store_rows_bf16_via_lds<D>(
        lds_addr(lds) + (uint32_t)w * (D * 64), [&](int d, int g4, int e) { return acc[d][g4 * 4 + e] * inv; },
        (bf16*)qr.o + (((int64_t)it.b * qr.bstride + wrow0) * H + it.h) * D, H * D, qr.len - wrow0, lane);
  }
  if (my_row < qr.len) {
    if (half == 0)
      qr.lse[((int64_t)it.b * H + it.h) * qr.bstride + my_row] =
          empty ? -INFINITY : (m_run + log2f(l_tot)) * kLn2;
  }
}

// HM of the kernel: 0 single-term P (dS), 1 two-term on every tile, 2
// two-term on the 16-key chunks holding a large probability.
// NW waves of 32 rows; NS = 3 stages (96 KB: one 8-wave workgroup per CU)
// or 2 (64 KB: two 4-wave workgroups per CU).
template <int D, int NW, int NS>
void launch_hm(const AttnArgs& a, int n, hipStream_t s) {
  const int hm = !(a.hilo & kHiloPv) ? 0 : (a.hilo & kHiloAdaptive) ? 2 : 1;
  if (hm == 0) hipLaunchKernelGGL((fwd_bf16_kernel<D, NW, NS, 0>), dim3(n), dim3(NW * 64), 0, s, a);
  else if (hm == 1) hipLaunchKernelGGL((fwd_bf16_kernel<D, NW, NS, 1>), dim3(n), dim3(NW * 64), 0, s, a);
  else hipLaunchKernelGGL((fwd_bf16_kernel<D, NW, NS, 2>), dim3(n), dim3(NW * 64), 0, s, a);
}

template <int D>
void launch_rows(const AttnArgs& a, int rows, int n, hipStream_t s) {
  if (rows == kQRowsShortBf16) launch_hm<D, kQRowsShortBf16 / 32, 2>(a, n, s);
  else launch_hm<D, kQRowsLongBf16 / 32, 3>(a, n, s);
}

}  // namespace

hipError_t launch_fwd_bf16(const AttnArgs& a, int head_dim, int rows, hipStream_t s) {
  const int n = a.total_tiles * a.heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128) launch_rows<128>(a, rows, n, s);
  else launch_rows<64>(a, rows, n, s);
  return hipGetLastError();
}

}  // namespace bdlm
