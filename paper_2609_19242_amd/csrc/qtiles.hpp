// Query-major tiling shared by the forward and the dQ kernel.
//
// A workgroup owns BM consecutive query rows of one query range and one query
// head and walks the key tiles (BN rows) of every key range that any of its
// rows can see.  The visible keys of a query row form one position interval
// (common.hpp), whose ends are non-decreasing in the query position, so for
// the tile's rows [pq0, pq1] the union of the intervals is [lo(pq0), hi(pq1))
// and the intersection is [lo(pq1), hi(pq0)): key tiles outside the union are
// never visited and key tiles inside the intersection need no mask test.
#pragma once

#include "common.hpp"
#include "device.hpp"

namespace bdlm {

struct QTileItem {
  int b, h, r, t;  // batch, query head, query range, tile within the range
};

// Logical work id -> (batch, query head, query range, tile).  Logical ids are
// grouped by KV head (after xcd_remap one XCD serves one KV head, so its L2
// holds that head's K/V), the query heads of a group are interleaved, and the
// tiles of each range run from the last (longest key prefix) to the first.
__device__ inline QTileItem q_tile_item(const AttnArgs& a, int logical) {
  const int per_kv = a.group * a.total_tiles;
  const int bk = logical / per_kv;
  const int rank = logical - bk * per_kv;
  QTileItem it;
  it.b = bk / a.kv_heads;
  const int kvh = bk - it.b * a.kv_heads;
  const int order = rank / a.group;
  it.h = kvh * a.group + (rank - order * a.group);
  if (a.interleave) {
    it.r = order % a.n_q;
    it.t = a.qr[it.r].ntiles - 1 - order / a.n_q;
  } else {
    int r = 0;
    while (r + 1 < a.n_q && order >= a.qr[r + 1].tile0) ++r;
    it.r = r;
    it.t = a.qr[r].ntiles - 1 - (order - a.qr[r].tile0);
  }
  return it;
}

// Key tiles [t0, t1) of key range j that any query position in [pq0, pq1]
// can see, and the sub-span [f0, f1) every one of them sees completely.
__device__ inline void key_tile_span(const AttnArgs& a, int j, int qs, int pq0, int pq1, int BN,
                                     int& t0, int& t1, int& f0, int& f1) {
  const KRangeArg& kr = a.kr[j];
  int lo0, hi0, lo1, hi1;
  key_interval(qs, pq0, kr.stream, rule_of(a), lo0, hi0);
  key_interval(qs, pq1, kr.stream, rule_of(a), lo1, hi1);
  const int u0 = imax(lo0 - kr.pos0, 0), u1 = imin(hi1 - kr.pos0, kr.len);
  t0 = t1 = f0 = f1 = 0;
  if (u1 <= u0) return;
  t0 = u0 / BN;
  t1 = (u1 + BN - 1) / BN;
  const int i0 = imax(lo1 - kr.pos0, 0), i1 = imin(hi0 - kr.pos0, kr.len);
  if (i1 > i0) {
    f0 = (i0 + BN - 1) / BN;
    f1 = i1 / BN;
  }
}

// First key tile at or after key range jj that the query tile can see.
__device__ inline bool find_key_tile(const AttnArgs& a, int jj, int qs, int pq0, int pq1, int BN,
                                     int& jo, int& to, int& t1o, int& f0o, int& f1o) {
  for (; jj < a.n_k; ++jj) {
    int a0, a1, b0, b1;
    key_tile_span(a, jj, qs, pq0, pq1, BN, a0, a1, b0, b1);
    if (a1 > a0) {
      jo = jj;
      to = a0;
      t1o = a1;
      f0o = b0;
      f1o = b1;
      return true;
    }
  }
  return false;
}

// This lane's visible key interval [lo, lo + w) inside key range j (w may be 0).
__device__ inline void lane_key_interval(const AttnArgs& a, int j, int qs, int pq, int& lo, int& w) {
  const KRangeArg& kr = a.kr[j];
  int l, h;
  key_interval(qs, pq, kr.stream, rule_of(a), l, h);
  l = imax(l, kr.pos0);
  h = imin(h, kr.pos0 + kr.len);
  lo = l;
  w = imax(h - l, 0);
}

}  // namespace bdlm
