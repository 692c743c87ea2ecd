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
constexpr int kMaxK = 32;
constexpr int kMaxParts = 32;
constexpr int kBig = 0x3fffffff;  // "to the end of the stream" (positions stay below 2^30)

// Visible key positions [lo, hi) for a query of stream qs at position pq,
// over keys of stream ks (block size M).  Empty when hi <= lo.
__host__ __device__ inline void key_interval(int qs, int pq, int ks, int M, int intra, int& lo, int& hi) {
  const int bq = pq / M;
  if (qs == kClean) {
    lo = 0;
    hi = (ks == kClean) ? (intra == kIntraBlock ? (bq + 1) * M : pq + 1) : 0;
  } else if (ks == kCorrupted) {  // own corrupted block, bidirectional
    lo = bq * M;
    hi = lo + M;
  } else {  // clean prefix of the earlier blocks
    lo = 0;
    hi = bq * M;
  }
}

// Query positions [lo, hi) of stream qs that see a key of stream ks at
// position pk (the same rules read from the key side).
__host__ __device__ inline void query_interval(int qs, int ks, int pk, int M, int intra, int& lo, int& hi) {
  const int bk = pk / M;
  if (qs == kClean) {
    if (ks == kClean) {
      lo = (intra == kIntraBlock) ? bk * M : pk;
      hi = kBig;
    } else {
      lo = kBig;
      hi = kBig;
    }
  } else if (ks == kCorrupted) {
    lo = bk * M;
    hi = lo + M;
  } else {
    lo = (bk + 1) * M;
    hi = kBig;
  }
}

__host__ __device__ inline int imax(int a, int b) { return a > b ? a : b; }
__host__ __device__ inline int imin(int a, int b) { return a < b ? a : b; }

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
  float scale;        // softmax scale
  float scale_log2;   // scale * log2(e): scores are kept in the base-2 domain
  int32_t total_tiles;   // flattened tiles (query tiles for fwd, key tiles for bwd)
  int32_t interleave;    // fwd: query ranges have equal tile counts, visit them round-robin
  int32_t out_f32;       // O, dQ, dK, dV are fp32 (else the input dtype)
  int32_t hilo;          // P and dS enter their products as bf16 hi + lo
  int32_t order[kMaxK];  // bwd: visiting order of key ranges (heaviest first)
  QRangeArg qr[kMaxQ];
  KRangeArg kr[kMaxK];
};

struct MergeArgs {
  int32_t n_parts;
  int32_t heads;
  int64_t rows;
  int64_t batch;
  const void* o_parts[kMaxParts];
  const float* lse_parts[kMaxParts];
  void* o;
  float* lse;
};

// Blocks are dispatched round-robin over the 8 XCDs of an MI355X.  Remap the
// hardware block id so that consecutive logical ids run on the same XCD (and
// share its L2): XCD x gets the logical span [x*n/8, (x+1)*n/8).
__device__ inline int xcd_remap(int wg, int n) {
  const int q = n >> 3, r = n & 7;
  const int xcd = wg & 7, slot = wg >> 3;
  return (xcd < r) ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
}

// Launchers (defined in the .hip files).  All return hipSuccess or the launch error.
hipError_t launch_fwd_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_fwd_f32(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_merge(const MergeArgs& a, int head_dim, int part_dtype, int out_dtype, hipStream_t s);
hipError_t launch_bwd_pre(const AttnArgs& a, int head_dim, int dtype, hipStream_t s);
hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_dq_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_bwd_f32(const AttnArgs& a, int head_dim, hipStream_t s);

// Tile heights the launchers use (the C ABI fills ntiles/tile0 with them).
constexpr int kFwdRowsBf16 = 256;  // query rows per forward / dQ workgroup (8 waves x 32)
constexpr int kFwdRowsF32 = 128;
constexpr int kBwdKeysBf16 = 128;  // key rows per backward workgroup (4 waves x 32)
constexpr int kBwdKeysF32 = 128;

}  // namespace bdlm
