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
// reads, the same product shape as the forward's O^T += V^T P^T.  The kernel
// forms D_i = dO_i . O_i itself (the lane already holds half of dO_i) and
// leaves each row's statistics in the workspace for the dK/dV kernel, which
// runs after it.
#include "qtiles.hpp"

namespace bdlm {

namespace {

constexpr float kLog2e = 1.44269504088896340736f;

template <int D, int NW, int NST, int HM>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void bwd_dq_kernel(
    const AttnArgs a) {
  constexpr int BM = NW * 32, BN = 64, KS = D / 16, DT = D / 32;
  // K and V tiles with swizzled rows: K serves both its row reads (S^T) and
  // its transpose reads (K^T), V its row reads (dP^T).
  constexpr uint32_t RB = D * 2, TB = BN * RB;
  constexpr int STAGE = 2 * BN * D;
  // Copies: each tile is BN * D / 8 16-byte slots, TI instructions of 64 lanes;
  // waves 0 .. NW/2 - 1 copy K and the others V, IPW instructions each.
  constexpr int TI = BN * D / 8 / 64, IPW = TI / (NW / 2);
  static_assert(TI % (NW / 2) == 0, "whole copy instructions per wave");
  __shared__ __attribute__((aligned(256))) bf16 lds[NST * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  const int G = lane >> 4, sl = lane & 15;

  const int n_wg = a.total_tiles * a.heads * a.batch;
  const QTileItem it = q_tile_item(a, xcd_remap(blockIdx.x, n_wg));
  const QRangeArg& qr = a.qr[it.r];
  const int kvh = it.h / a.group;
  const int row0 = it.t * BM;
  const int nvalid = imin(BM, qr.len - row0);
  const int64_t H = a.heads;

  // This wave's 32 query rows of Q and dO as MFMA B fragments, and
  // D = rowsum(dO * O) of the lane's row: a lane holds half of the row's
  // elements (8-element chunks 2s + half), its partner lane the other half.
  bf16x8 qf[KS], df[KS];
  float dsum = 0.f;
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
    if (a.out_f32) {  // O in fp32: two 16-byte loads per chunk
      const auto ro = make_rsrc((const float*)qr.o + qoff, 2 * bytes);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f32x4 o0 = __builtin_bit_cast(f32x4, buf_load16(ro, 2 * off + s * 64));
        const f32x4 o1 = __builtin_bit_cast(f32x4, buf_load16(ro, 2 * off + s * 64 + 16));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          dsum = fmaf(o0[e], (float)df[s][e], dsum);
          dsum = fmaf(o1[e], (float)df[s][4 + e], dsum);
        }
      }
    } else {
      const auto ro = make_rsrc((const bf16*)qr.o + qoff, bytes);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8 o = __builtin_bit_cast(bf16x8, buf_load16(ro, off + s * 32));
#pragma unroll
        for (int e = 0; e < 8; ++e) dsum = fmaf((float)o[e], (float)df[s][e], dsum);
      }
    }
  }
  dsum += partner(dsum);
  const int my_row = row0 + w * 32 + l32;
  const bool row_ok = my_row < qr.len;
  const int pq = qr.pos0 + imin(my_row, qr.len - 1);
  const int pq0 = qr.pos0 + row0, pq1 = qr.pos0 + row0 + nvalid - 1;
  // Rows past the range and rows that see no key get P = 0.  The row's
  // statistics for the dK/dV kernel, which runs after this one, go to the
  // workspace: (LSE log2(e), D), or (-LSE / scale, -D) for the scheduled
  // kernel (stats form 1).
  float lse2 = INFINITY;
  const float dl = dsum;
  if (row_ok) {
    const float z = qr.lse[((int64_t)it.b * H + it.h) * qr.bstride + my_row];
    lse2 = (z == -INFINITY) ? INFINITY : z * kLog2e;
    if (half == 0) {
      const int64_t si = ((int64_t)it.b * H + it.h) * qr.len + my_row;
      if (a.stats_form) {
        qr.delta[si] = -dsum;
        qr.l2[si] = (z == -INFINITY) ? -INFINITY : -z / a.scale;
      } else {
        qr.delta[si] = dsum;
        qr.l2[si] = (z == -INFINITY) ? INFINITY : z * kLog2e;
      }
    }
  }

  f32x16 acc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[d][i] = 0.f;
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
  const int64_t HKV = a.kv_heads;
  // The copy cursor runs NST - 1 tiles ahead of the compute cursor and carries
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
  // One instruction covers 512 / D rows and the chunk swizzle repeats every
  // 16 rows, so instructions PI = D / 32 apart share their lane offsets and
  // read through a resource based 16 rows further on (its size cut by as much).
  constexpr int PI = IPW < D / 32 ? IPW : D / 32, NB = IPW / PI;
  static_assert(IPW % PI == 0, "whole offset periods per wave");
  uint32_t voff[PI];
  const int cw = w % (NW / 2);
#pragma unroll
  for (int i = 0; i < PI; ++i) voff[i] = swz_src_offset<D>((cw * IPW + i) * 64 + lane, HKV * D);
  const bf16* const any_src = (const bf16*)a.kr[0].k;
  auto copy_tile = [&](bf16* st, const CopyCur& cc) __attribute__((always_inline)) {
    const int nrows = cc.c.have ? imin(BN, cc.rows_left) : 0;
    bf16* dst = st + (kwave ? 0 : BN * D) + cw * IPW * 512;
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int nr = nrows - 16 * k;
      const uint32_t bytes = nr > 0 ? (uint32_t)(((nr - 1) * (int)HKV * D + D) * 2) : 0u;
      const auto r = make_rsrc(nr > 0 ? cc.src + (int64_t)16 * k * HKV * D : any_src, bytes);
#pragma unroll
      for (int i = 0; i < PI; ++i) buf_to_lds<16>(r, dst + (k * PI + i) * 512, voff[i], 0);
    }
  };
  // Per-lane parts of the swizzled read addresses (device.hpp).
  const uint32_t yrow = swz_row_part<D>(l32, half);
  const uint32_t ytr0 = swz_tr_part<D>(G, sl, 0), ytr1 = swz_tr_part<D>(G, sl, 8);

  // NST LDS stages, copies NST - 1 tiles ahead (as in the forward: 8 waves
  // and three stages on long walks, 4 waves and two on short ones).
  KCur c0;
  c0.have = find_key_tile(a, 0, qr.stream, pq0, pq1, BN, c0.j, c0.t, c0.t1, c0.f0, c0.f1);
  CopyCur cp = copy_seek(CopyCur{c0, any_src, 0});
#pragma unroll
  for (int s = 0; s < NST - 1; ++s) {
    copy_tile(lds + s * STAGE, cp);
    cp = copy_next(cp);
  }
  vm_wait_barrier<IPW * (NST - 2)>();
  int cur = 0;
  int lane_lo = 0, lane_w = 0, lane_j = -1;
  while (c0.have) {
    copy_tile(lds + (cur == 0 ? NST - 1 : cur - 1) * STAGE, cp);
    const int j = c0.j, t = c0.t, f0 = c0.f0, f1 = c0.f1;
    if (lane_j != j) {
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
      // S^T = K Q^T and dP^T = V dO^T: K and V rows 32u + l32 by row reads.
      const uint32_t sb = lds_addr(lds + cur * STAGE);
      const uint32_t zr = sb + yrow;
      f32x16 sacc[2], dpacc[2];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          sacc[u][i] = 0.f;
          dpacc[u][i] = -dl;  // dP^T - D accumulates from -D (one subtract less per score)
        }
      {
        // K and V fragments are read LA steps ahead of their products (steps
        // run over (u, s)); the scheduling fences keep the compiler from
        // sinking each read down to the product that uses it.
        constexpr int LA = 2, NS = 2 * KS;
        bf16x8 kf[LA + 1], vf[LA + 1];
        auto addr = [&](int n) { return (zr ^ (32u * (n % KS))) + (n / KS) * 32 * RB; };
#pragma unroll
        for (int n = 0; n < LA; ++n) {
          kf[n] = lds_load16(addr(n));
          vf[n] = lds_load16(addr(n) + TB);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int n = 0; n < NS; ++n) {
          if (n + LA < NS) {
            kf[(n + LA) % (LA + 1)] = lds_load16(addr(n + LA));
            vf[(n + LA) % (LA + 1)] = lds_load16(addr(n + LA) + TB);
          }
          const int u = n / KS, s = n % KS;
          sacc[u] = mfma32(kf[n % (LA + 1)], qf[s], sacc[u]);
          dpacc[u] = mfma32(vf[n % (LA + 1)], df[s], dpacc[u]);
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

      // dS^T = P^T (dP^T - D) in the S^T register layout, rounded to bf16; HM 1
      // adds dS - bf16(dS) as a second bf16 term on every tile, HM 2 on the
      // 16-key chunks that hold a probability of at least hilo_tau.
      bf16x8 dsb[4], dsl[4];
      float cmax[4] = {0.f, 0.f, 0.f, 0.f};  // HM 2: largest P per 16-key chunk
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = exp2f_fast(fmaf(sacc[u][i], c, -lse2));
          const float ds = p * dpacc[u][i];
          const bf16 hi = to_bf16(ds);
          dsb[u * 2 + (i >> 3)][i & 7] = hi;
          if constexpr (HM != 0) dsl[u * 2 + (i >> 3)][i & 7] = to_bf16(ds - (float)hi);
          if constexpr (HM == 2) cmax[u * 2 + (i >> 3)] = fmaxf(cmax[u * 2 + (i >> 3)], p);
        }

      // dQ^T[d][q] += sum_key K[key][d] dS[q][key]; key order per 16-key step as in the forward.
      const uint32_t zt0 = sb + ytr0, zt1 = sb + ytr1;  // K tile by transpose reads
      auto dsk = [&](const bf16x8 (&dd)[4]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
          for (int d = 0; d < DT; ++d) {
            const bf16x8 ka = cat(lds_read_tr_at((zt0 ^ (64u * d)) + u * 16 * RB),
                                  lds_read_tr_at((zt1 ^ (64u * d)) + u * 16 * RB));
            acc[d] = mfma32(ka, dd[u], acc[d]);
          }
        }
      };
      if constexpr (HM == 1) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
          for (int d = 0; d < DT; ++d) {
            const bf16x8 ka = cat(lds_read_tr_at((zt0 ^ (64u * d)) + u * 16 * RB),
                                  lds_read_tr_at((zt1 ^ (64u * d)) + u * 16 * RB));
            acc[d] = mfma32(ka, dsb[u], acc[d]);
            acc[d] = mfma32(ka, dsl[u], acc[d]);
          }
        }
      } else {
        dsk(dsb);
        if constexpr (HM == 2) {
          // second terms of the 16-key chunks holding a probability >= hilo_tau
          // (K^T fragments re-read)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (__builtin_amdgcn_ballot_w64(cmax[u] >= a.hilo_tau) != 0) {
#pragma unroll
              for (int d = 0; d < DT; ++d) {
                const bf16x8 ka = cat(lds_read_tr_at((zt0 ^ (64u * d)) + u * 16 * RB),
                                      lds_read_tr_at((zt1 ^ (64u * d)) + u * 16 * RB));
                acc[d] = mfma32(ka, dsl[u], acc[d]);
              }
            }
          }
        }
      }
    }

    vm_wait_barrier<IPW * (NST - 2)>();
    cur = cur == NST - 1 ? 0 : cur + 1;
    c0 = next_tile(c0);
    cp = copy_next(cp);
  }
  // Copies still in flight target stages nobody reads; they must land before
  // the workgroup's LDS is released.
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)

  if (a.out_f32) {
    if (row_ok) {
      float* op = (float*)qr.dq + (((int64_t)it.b * qr.bstride + my_row) * H + it.h) * D;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[d][g4 * 4 + e] * a.scale;
          *(f32x4*)(op + 32 * d + 8 * g4 + 4 * half) = v;
        }
    }
  } else if constexpr (HM != 2) {
    // bf16 dQ through LDS, as the forward's O.
    asm volatile("s_barrier" ::: "memory");
    const int wrow0 = row0 + w * 32;
    store_rows_bf16_via_lds<D>(
        lds_addr(lds) + (uint32_t)w * (D * 64), [&](int d, int g4, int e) { return acc[d][g4 * 4 + e] * a.scale; },
        (bf16*)qr.dq + (((int64_t)it.b * qr.bstride + wrow0) * H + it.h) * D, H * D, qr.len - wrow0, lane);
  } else if (row_ok) {
    // The adaptive two-term kernel stores directly: the staged form needs the
    // last few registers it has and made it spill.
    bf16* op = (bf16*)qr.dq + (((int64_t)it.b * qr.bstride + my_row) * H + it.h) * D;
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

// HM of the kernel: 0 single-term P (dS), 1 two-term on every tile, 2
// two-term on the 16-key chunks holding a large probability.
// NW waves of 32 rows; NS = 3 stages (96 KB: one 8-wave workgroup per CU)
// or 2 (64 KB: two 4-wave workgroups per CU).
template <int D, int NW, int NS>
void launch_hm(const AttnArgs& a, int n, hipStream_t s) {
  const int hm = !(a.hilo & kHiloDq) ? 0 : (a.hilo & kHiloAdaptive) ? 2 : 1;
  if (hm == 0) hipLaunchKernelGGL((bwd_dq_kernel<D, NW, NS, 0>), dim3(n), dim3(NW * 64), 0, s, a);
  else if (hm == 1) hipLaunchKernelGGL((bwd_dq_kernel<D, NW, NS, 1>), dim3(n), dim3(NW * 64), 0, s, a);
  else hipLaunchKernelGGL((bwd_dq_kernel<D, NW, NS, 2>), dim3(n), dim3(NW * 64), 0, s, a);
}

template <int D>
void launch_rows(const AttnArgs& a, int rows, int n, hipStream_t s) {
  if (rows == kQRowsShortBf16) launch_hm<D, kQRowsShortBf16 / 32, 2>(a, n, s);
  else launch_hm<D, kQRowsLongBf16 / 32, 3>(a, n, s);
}

}  // namespace

// a.total_tiles / qr[i].tile0 / ntiles must describe query tiles of `rows` rows.
hipError_t launch_bwd_dq_bf16(const AttnArgs& a, int head_dim, int rows, hipStream_t s) {
  const int n = a.total_tiles * a.heads * a.batch;
  if (n == 0) return hipSuccess;
  if (head_dim == 128) launch_rows<128>(a, rows, n, s);
  else launch_rows<64>(a, rows, n, s);
  return hipGetLastError();
}

}  // namespace bdlm
