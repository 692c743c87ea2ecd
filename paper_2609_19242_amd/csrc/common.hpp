// Internal definitions shared by the BDLM attention kernels and the C ABI layer.
//
// The mask of BDLM training (arXiv 2609.19242, Sec. 3.2 and App. A step 1) is
// expressed as intervals: for a query row at position pq of stream qs, the
// visible keys of stream ks form one interval of positions [lo, hi), and for a
// key row at position pk the queries that see it form one interval too.  Both
// ends are non-decreasing in the position, which is what makes tile
// classification a closed form: over a tile of query rows [pq0, pq1] the union
// of the visible key intervals is [lo(pq0), hi(pq1)) and their intersection is
// [lo(pq1), hi(pq0)).  Key tiles inside the intersection are fully visible
// (no mask test), tiles outside the union are skipped, and only the few in
// between evaluate the mask per element.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdlm {

enum : int { kClean = 0, kCorrupted = 1 };
enum : int { kIntraCausal = 0, kIntraBlock = 1 };

constexpr int kMaxQ = 4;
// Products that take their P or dS operand as two bf16 terms (the hilo mask of
// the problem; the values of the BDLM_HILO_* bits of the C ABI).
constexpr int kHiloPv = 1;    // forward P V
constexpr int kHiloDkDv = 2;  // backward P^T dO and dS^T Q (dK/dV kernel)
constexpr int kHiloDq = 4;    // backward dS K (dQ kernel)
constexpr int kHiloAdaptive = 8;  // the second term only on tiles where some probability reaches kHiloTau
constexpr float kHiloTau = 1.0f / 64;
constexpr int kMaxK = 32;
constexpr int kMaxParts = 32;
constexpr int kBig = 0x3fffffff;  // "to the end of the stream" (positions stay below 2^30)

__host__ __device__ inline int imax(int a, int b) { return a > b ? a : b; }
__host__ __device__ inline int imin(int a, int b) { return a < b ? a : b; }

// The mask's parameters.  block_size M and the clean-to-clean reading come
// from Sec. 3.2.  Two optional generalisations keep every visible set an
// interval with non-decreasing ends:
//  * window W > 0 (sliding-window layers, App. "Savings Breakdowns"): a query
//    sees only the last W positions of its clean context, i.e. clean keys in
//    [e - W, e) where e is the end of the context it would see without the
//    window (q + 1, the end of q's block, or the start of q's corrupted block);
//  * prefix (DFlash2 drafter attention, eq:dflash2-block-attention): the clean
//    context of corrupted block b ends at prefix[b] (the block's anchor a_b)
//    instead of at M b.  The table holds nblk = L / M entries, non-decreasing
//    and in [0, L]; entries are clamped into [0, L] when read, so a table that
//    breaks the contract changes the mask but never addresses out of bounds.
struct MaskRule {
  int M, intra, window, nblk, L;
  const int* prefix;  // device (kernels) or host (host code) table, or null
};

// End of the clean context of corrupted block b.
__host__ __device__ inline int clean_end_of_block(const MaskRule& r, int b) {
  if (!r.prefix) return b * r.M;
  const int v = r.prefix[imin(imax(b, 0), r.nblk - 1)];
  return imin(imax(v, 0), r.L);
}

// First corrupted block whose clean context ends after position x (nblk if none).
__host__ __device__ inline int first_block_ending_after(const MaskRule& r, int x) {
  if (!r.prefix) return imin(x / r.M + 1, r.nblk);
  int lo = 0, hi = r.nblk;  // invariant: the answer lies in [lo, hi]
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (clean_end_of_block(r, mid) > x) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

// Visible key positions [lo, hi) for a query of stream qs at position pq,
// over keys of stream ks.  Empty when hi <= lo.
__host__ __device__ inline void key_interval(int qs, int pq, int ks, const MaskRule& r, int& lo, int& hi) {
  const int M = r.M, bq = pq / M;
  if (qs == kClean) {
    lo = 0;
    hi = (ks == kClean) ? (r.intra == kIntraBlock ? (bq + 1) * M : pq + 1) : 0;
  } else if (ks == kCorrupted) {  // own corrupted block, bidirectional
    lo = bq * M;
    hi = lo + M;
  } else {  // clean context of the block: the clean prefix of the earlier blocks
    lo = 0;
    hi = clean_end_of_block(r, bq);
  }
  if (ks == kClean && r.window > 0) lo = imax(lo, hi - r.window);
}

// Query positions [lo, hi) of stream qs that see a key of stream ks at
// position pk (the same rules read from the key side).
__host__ __device__ inline void query_interval(int qs, int ks, int pk, const MaskRule& r, int& lo, int& hi) {
  const int M = r.M, bk = pk / M, W = r.window;
  if (qs == kClean) {
    if (ks == kClean) {
      lo = (r.intra == kIntraBlock) ? bk * M : pk;
      // with a window: e(q) <= pk + W, e(q) = q + 1 or the end of q's block
      hi = W <= 0 ? kBig : (r.intra == kIntraBlock ? M * ((pk + W) / M) : pk + W);
    } else {
      lo = kBig;
      hi = kBig;
    }
  } else if (ks == kCorrupted) {
    lo = bk * M;
    hi = lo + M;
  } else {
    // blocks whose clean context [e - W, e) holds pk: e > pk and e <= pk + W
    lo = first_block_ending_after(r, pk) * M;
    hi = W <= 0 ? kBig : first_block_ending_after(r, pk + W) * M;
  }
}


// One query range as the kernels see it.  Pointers are to element 0 of the
// range for batch element 0; row i of batch b is at row (b * bstride + i).
struct QRangeArg {
  int32_t stream;
  int32_t pos0;
  int32_t len;
  int32_t ntiles;     // tiles of this range at the kernel's tile height
  int64_t bstride;    // rows between batch elements
  int32_t tile0;      // first tile of this range in the flattened tile list
  int32_t pad;
  const void* q;
  void* o;
  float* lse;
  const void* dO;
  void* dq;
  float* l2;          // LSE * log2(e), +inf where LSE = -inf, [batch][heads][len]
  float* delta;       // D = rowsum(dO * O), [batch][heads][len]
};

struct KRangeArg {
  int32_t stream;
  int32_t pos0;
  int32_t len;
  int32_t ntiles;
  int64_t bstride;
  int32_t tile0;
  int32_t pad;
  const void* k;
  const void* v;
  void* dk;
  void* dv;
};

struct AttnArgs {
  int32_t n_q, n_k;
  int32_t batch, heads, kv_heads, group;
  int32_t M, intra;
  int32_t window;      // clean keys per query at most (0: no limit)
  int32_t nblk;        // blocks per stream, L / M
  int32_t L;
  int32_t stats_form;  // bwd workspace per query row: 0 = (LSE log2(e), D), 1 = (-LSE / scale, -D)
  const int* prefix;   // clean context end per corrupted block (device), or null
  float scale;        // softmax scale
  float scale_log2;   // scale * log2(e): scores are kept in the base-2 domain
  int32_t total_tiles;   // flattened tiles (query tiles for fwd, key tiles for bwd)
  int32_t interleave;    // fwd: query ranges have equal tile counts, visit them round-robin
  int32_t out_f32;       // O, dQ, dK, dV are fp32 (else the input dtype)
  int32_t hilo;          // kHilo* bits: products whose P or dS operand is bf16 hi + lo
  float hilo_tau;        // those products take the second term only on tiles where some P reaches this (0: all tiles)
  int32_t order[kMaxK];  // bwd: visiting order of key ranges (heaviest first)
  QRangeArg qr[kMaxQ];
  KRangeArg kr[kMaxK];
};

struct MergeArgs {
  int32_t n_parts;
  int32_t heads;
  int64_t rows;
  int64_t batch;
  int64_t pstride, ostride;  // rows between batch elements in the parts and in the output (>= rows)
  const void* o_parts[kMaxParts];
  const float* lse_parts[kMaxParts];
  void* o;
  float* lse;
};

__host__ __device__ inline MaskRule rule_of(const AttnArgs& a) {
  return MaskRule{a.M, a.intra, a.window, a.nblk, a.L, a.prefix};
}

// Blocks are dispatched round-robin over the 8 XCDs of an MI355X.  Remap the
// hardware block id so that consecutive logical ids run on the same XCD (and
// share its L2): XCD x gets the logical span [x*n/8, (x+1)*n/8).
__device__ inline int xcd_remap(int wg, int n) {
  const int q = n >> 3, r = n & 7;
  const int xcd = wg & 7, slot = wg >> 3;
  return (xcd < r) ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}

// Logical work id (after xcd_remap) -> (pair, rank) for the key-major dK/dV
// kernels: T key tiles per (batch, KV head) pair, nbk pairs, the tiles of a
// pair numbered heaviest first.  When the pairs divide evenly over the 8 XCDs,
// the m pairs of one XCD are interleaved tile by tile, so that the heaviest
// tiles of all of them start first on the XCD's CUs (one pair after the other
// left the second pair's heaviest tiles to start late and end last: 7-8% of
// the kernel at batch 2 and 4, 4K keys).  Otherwise pairs follow one another.
// (The query-major kernels keep pairs in sequence: there interleaving puts the
// K/V of several heads in one XCD's L2 at once and was slower.)
__device__ inline void pair_and_rank(int logical, int T, int nbk, int& bk, int& rank) {
  if (nbk > 8 && nbk % 8 == 0) {
    const int m = nbk >> 3, span = m * T;
    const int x = logical / span, local = logical - x * span;
    rank = local / m;
    bk = x * m + (local - rank * m);
  } else {
    bk = logical / T;
    rank = logical - bk * T;
  }
}

// Launchers (defined in the .hip files).  All return hipSuccess or the launch error.
hipError_t launch_fwd_bf16(const AttnArgs& a, int head_dim, int rows, hipStream_t s);
hipError_t launch_fwd_f32(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_merge(const MergeArgs& a, int head_dim, int part_dtype, int out_dtype, hipStream_t s);
hipError_t launch_bwd_pre(const AttnArgs& a, int head_dim, hipStream_t s);  // fp32 path
hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_dkdv(const AttnArgs& a, hipStream_t s);
hipError_t launch_bwd_dq_bf16(const AttnArgs& a, int head_dim, int rows, hipStream_t s);
hipError_t launch_bwd_f32(const AttnArgs& a, int head_dim, hipStream_t s);

// The walk of a key tile of the scheduled dK/dV kernel over its visible query
// rows, by step index.  The rows come as up to two query ranges; range r is
// seen by the tile's keys in the 32-row blocks [a_r, b_r) (a_r = b_r = 0 when
// empty).  Step i is (range q, block s, head pair hp): blocks from the top
// down, at each block every range active there (range 0 first), each with its
// npairs head pairs in order.  The block axis splits at the four range ends
// into at most three segments with a fixed set of active ranges: segment k
// covers blocks [p_{k+1}, p_k) with cnt_k active ranges (the first q0_k), so
// step i follows from its segment in closed form.
struct WalkPlan {
  int p0, p1, p2, p3;  // range ends, descending
  int st1, st2, nsteps;  // first steps of segments 1 and 2; steps in all
  int cnt0, cnt1, cnt2, q00, q01, q02, npairs;
};
__host__ __device__ inline WalkPlan walk_plan(int a0, int b0, int a1, int b1, int npairs) {
  WalkPlan w;
  int p0 = b0, p1 = a0, p2 = b1, p3 = a1;
  auto cx = [](int& x, int& y) {
    const int hi = imax(x, y), lo = imin(x, y);
    x = hi;
    y = lo;
  };
  cx(p0, p1);
  cx(p2, p3);
  cx(p0, p2);
  cx(p1, p3);
  cx(p1, p2);
  auto act = [](int a, int b, int blk) { return a <= blk && blk < b ? 1 : 0; };
  w.p0 = p0;
  w.p1 = p1;
  w.p2 = p2;
  w.p3 = p3;
  w.cnt0 = act(a0, b0, p1) + act(a1, b1, p1);
  w.cnt1 = act(a0, b0, p2) + act(a1, b1, p2);
  w.cnt2 = act(a0, b0, p3) + act(a1, b1, p3);
  w.q00 = act(a0, b0, p1) ? 0 : 1;
  w.q01 = act(a0, b0, p2) ? 0 : 1;
  w.q02 = act(a0, b0, p3) ? 0 : 1;
  w.npairs = npairs;
  w.st1 = (p0 - p1) * w.cnt0 * npairs;
  w.st2 = w.st1 + (p1 - p2) * w.cnt1 * npairs;
  w.nsteps = w.st2 + (p2 - p3) * w.cnt2 * npairs;
  return w;
}
struct WalkStep {
  int q, s, hp;
  bool live;  // i < nsteps (q, s, hp are meaningless otherwise)
};
__host__ __device__ inline WalkStep walk_step(const WalkPlan& w, int i) {
  const bool k1 = i >= w.st1, k2 = i >= w.st2;
  const int top = (k2 ? w.p2 : k1 ? w.p1 : w.p0) - 1;
  const int cnt = k2 ? w.cnt2 : k1 ? w.cnt1 : w.cnt0;
  const int q0 = k2 ? w.q02 : k1 ? w.q01 : w.q00;
  const int off = i - (k2 ? w.st2 : k1 ? w.st1 : 0);
  const int per = imax(cnt * w.npairs, 1);
  const int sr = off / per, rem = off - sr * per;
  const int ridx = rem >= w.npairs ? 1 : 0;
  WalkStep st;
  st.live = i >= 0 && i < w.nsteps;
  st.hp = rem - ridx * w.npairs;
  st.q = cnt == 2 ? ridx : q0;
  st.s = top - sr;
  return st;
}

// The dK/dV kernel of bwd_dkdv.hip (head_dim 128, single-term or adaptive
// two-term dK/dV products, an even GQA group, at most two query ranges with
// rows) starts its score and dP accumulators at -LSE/scale and -D, so the backward
// workspace holds those (stats form 1); the general kernel of bwd_bf16.hip and
// the fp32 kernel read LSE log2(e) and D (form 0).
inline bool dkdv_uses_scheduled_kernel(int dtype_bf16, int head_dim, int hilo, int group, int n_q) {
  const bool terms_ok = !(hilo & kHiloDkDv) || (hilo & kHiloAdaptive);
  return dtype_bf16 && head_dim == 128 && terms_ok && group % 2 == 0 && n_q <= 2;
}

// Tile heights the launchers use (the C ABI fills ntiles/tile0 with them).
// The bf16 forward and dQ kernels take 256 query rows per workgroup (8 waves,
// one workgroup per CU) when some row of the call can see many keys, and 128
// (4 waves, two workgroups per CU) when none can see more than the kernel's
// short-walk limit: on short walks one workgroup's start-up and barriers
// overlap the other's products, which outweighs copying every K/V tile for
// half as many rows; on long walks the extra copies cost more.
constexpr int kQRowsLongBf16 = 256;
constexpr int kQRowsShortBf16 = 128;
constexpr int64_t kFwdShortWalk = 16384;  // keys a row may see for the 128-row forward
constexpr int64_t kDqShortWalk = 8192;    // ... and for the 128-row dQ kernel
constexpr int kFwdRowsF32 = 128;
constexpr int kBwdKeysBf16 = 128;  // key rows per backward workgroup (4 waves x 32)
constexpr int kBwdKeysF32 = 128;

}  // namespace bdlm
