// C ABI of the BDLM attention library: argument validation, kernel argument
// construction and launches.  Declarations and contracts: include/bdlm_attn.h.
#include "bdlm_attn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

static_assert(BDLM_HILO_PV == bdlm::kHiloPv && BDLM_HILO_DKDV == bdlm::kHiloDkDv && BDLM_HILO_DQ == bdlm::kHiloDq &&
                  BDLM_HILO_ADAPTIVE == bdlm::kHiloAdaptive,
              "hilo bits of the C ABI and the kernels agree");

using namespace bdlm;

namespace {

thread_local std::string g_err;

bdlm_status fail(bdlm_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

bdlm_status hip_fail(hipError_t e, const char* what) {
  return fail(BDLM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- per-thread kernel timing (bdlm_timing_enable / bdlm_timing_collect)
enum KernelId { kKFwdBf16 = 0, kKFwdF32, kKMerge, kKBwdPre, kKBwdBf16, kKBwdDq, kKBwdF32, kKCount };
const char* const kKernelNames[kKCount] = {"fwd_bf16", "fwd_f32", "lse_merge", "bwd_pre", "bwd_dkdv_bf16",
                                           "bwd_dq_bf16", "bwd_f32"};
struct TimingRec {
  int id;
  hipEvent_t a, b;
};
thread_local bool g_timing = false;
thread_local std::vector<TimingRec> g_recs;
thread_local std::vector<hipEvent_t> g_event_pool;

hipEvent_t pool_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Launch through f(), bracketed by events when timing is on.
template <class F>
hipError_t timed(int id, hipStream_t s, F&& f) {
  if (!g_timing) return f();
  TimingRec r{id, pool_event(), pool_event()};
  if (!r.a || !r.b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(r.a, s);
  if (e != hipSuccess) return e;
  e = f();
  if (e != hipSuccess) return e;
  e = hipEventRecord(r.b, s);
  if (e != hipSuccess) return e;
  g_recs.push_back(r);
  return hipSuccess;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxPos = (int64_t)1 << 30;

bdlm_status check_problem(const bdlm_problem* p) {
  if (!p) return fail(BDLM_ERR_INVALID, "problem is null");
  if (p->batch < 1) return fail(BDLM_ERR_INVALID, "batch must be >= 1 (got %lld)", (long long)p->batch);
  if (p->L < 1 || p->L >= kMaxPos) return fail(BDLM_ERR_INVALID, "L must be in [1, 2^30) (got %lld)", (long long)p->L);
  if (p->block_size < 1 || p->L % p->block_size != 0)
    return fail(BDLM_ERR_INVALID, "block_size must be >= 1 and divide L (L=%lld, block_size=%lld)",
                (long long)p->L, (long long)p->block_size);
  if (p->heads < 1 || p->kv_heads < 1 || p->heads % p->kv_heads != 0)
    return fail(BDLM_ERR_INVALID, "heads (%d) must be a positive multiple of kv_heads (%d)", p->heads, p->kv_heads);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(BDLM_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", p->head_dim);
  if (p->dtype != BDLM_BF16 && p->dtype != BDLM_F32)
    return fail(BDLM_ERR_UNSUPPORTED, "dtype %d not supported", p->dtype);
  if (p->clean_intra != BDLM_CLEAN_INTRA_CAUSAL && p->clean_intra != BDLM_CLEAN_INTRA_BLOCK)
    return fail(BDLM_ERR_INVALID, "clean_intra %d is not a bdlm_clean_intra value", p->clean_intra);
  if (!std::isfinite(p->scale)) return fail(BDLM_ERR_INVALID, "scale is not finite");
  if (p->out_f32 != 0 && p->out_f32 != 1) return fail(BDLM_ERR_INVALID, "out_f32 must be 0 or 1");
  if (p->hilo < 0 || p->hilo > (BDLM_HILO_ALL | BDLM_HILO_ADAPTIVE))
    return fail(BDLM_ERR_INVALID, "hilo must be a mask of BDLM_HILO_* bits (0..%d, got %d)",
                BDLM_HILO_ALL | BDLM_HILO_ADAPTIVE, p->hilo);
  if (p->window < 0 || p->window >= kMaxPos)
    return fail(BDLM_ERR_INVALID, "window must be in [0, 2^30) (got %lld)", (long long)p->window);
  if (p->clean_prefix && (reinterpret_cast<uintptr_t>(p->clean_prefix) & 3u) != 0)
    return fail(BDLM_ERR_INVALID, "clean_prefix is not 4-byte aligned");
  return BDLM_OK;
}

MaskRule host_rule(const bdlm_problem* p, const int* prefix) {
  return MaskRule{(int)p->block_size, p->clean_intra, (int)p->window, (int)(p->L / p->block_size), (int)p->L, prefix};
}

bdlm_status check_range(const bdlm_problem* p, const bdlm_range& r, const char* what, int idx) {
  if (r.stream != BDLM_CLEAN && r.stream != BDLM_CORRUPTED)
    return fail(BDLM_ERR_INVALID, "%s range %d: stream %d is not a bdlm_stream value", what, idx, r.stream);
  if (r.reserved != 0) return fail(BDLM_ERR_INVALID, "%s range %d: reserved field must be 0", what, idx);
  if (r.pos0 < 0 || r.len < 0 || r.pos0 + r.len > p->L)
    return fail(BDLM_ERR_INVALID, "%s range %d: positions [%lld, %lld) outside [0, L=%lld)", what, idx,
                (long long)r.pos0, (long long)(r.pos0 + r.len), (long long)p->L);
  if (r.batch_stride != 0 && r.batch_stride < r.len)
    return fail(BDLM_ERR_INVALID, "%s range %d: batch_stride %lld < len %lld", what, idx, (long long)r.batch_stride,
                (long long)r.len);
  if ((r.batch_stride ? r.batch_stride : r.len) >= kMaxPos)
    return fail(BDLM_ERR_UNSUPPORTED, "%s range %d: batch_stride must be < 2^30", what, idx);
  return BDLM_OK;
}

bdlm_status check_ptr(const void* ptr, const char* what, int idx) {
  if (!ptr) return fail(BDLM_ERR_INVALID, "%s pointer of range %d is null", what, idx);
  if (!aligned16(ptr)) return fail(BDLM_ERR_INVALID, "%s pointer of range %d is not 16-byte aligned", what, idx);
  return BDLM_OK;
}

float resolved_scale(const bdlm_problem* p) {
  return p->scale > 0.f ? p->scale : 1.0f / std::sqrt((float)p->head_dim);
}

void fill_common(AttnArgs& a, const bdlm_problem* p) {
  a = AttnArgs{};
  a.batch = (int32_t)p->batch;
  a.heads = p->heads;
  a.kv_heads = p->kv_heads;
  a.group = p->heads / p->kv_heads;
  a.M = (int32_t)p->block_size;
  a.intra = p->clean_intra;
  a.window = (int32_t)p->window;
  a.nblk = (int32_t)(p->L / p->block_size);
  a.L = (int32_t)p->L;
  a.prefix = p->clean_prefix;
  a.scale = resolved_scale(p);
  a.scale_log2 = a.scale * 1.44269504088896340736f;
  a.out_f32 = (p->dtype == BDLM_F32 || p->out_f32) ? 1 : 0;
  a.hilo = p->hilo;
  a.hilo_tau = (p->hilo & BDLM_HILO_ADAPTIVE) ? kHiloTau : 0.f;
}

void fill_q(QRangeArg& d, const bdlm_range& r) {
  d.stream = r.stream;
  d.pos0 = (int32_t)r.pos0;
  d.len = (int32_t)r.len;
  d.bstride = r.batch_stride ? r.batch_stride : r.len;
}

void fill_k(KRangeArg& d, const bdlm_range& r) {
  d.stream = r.stream;
  d.pos0 = (int32_t)r.pos0;
  d.len = (int32_t)r.len;
  d.bstride = r.batch_stride ? r.batch_stride : r.len;
}

bdlm_status check_counts(int32_t n_q, int32_t n_k, const void* qr, const void* kr) {
  if (n_q < 1 || !qr) return fail(BDLM_ERR_INVALID, "need at least one query range (n_q=%d)", n_q);
  if (n_k < 1 || !kr) return fail(BDLM_ERR_INVALID, "need at least one key range (n_k=%d)", n_k);
  if (n_q > kMaxQ) return fail(BDLM_ERR_UNSUPPORTED, "n_q=%d exceeds %d", n_q, kMaxQ);
  if (n_k > kMaxK) return fail(BDLM_ERR_UNSUPPORTED, "n_k=%d exceeds %d", n_k, kMaxK);
  return BDLM_OK;
}

// Tiles of `rows` rows over the ranges; returns the total or -1 when too many blocks.
template <typename R>
int64_t tile_ranges(R* rr, int n, int rows) {
  int64_t tot = 0;
  for (int i = 0; i < n; ++i) {
    rr[i].tile0 = (int32_t)tot;
    rr[i].ntiles = (rr[i].len + rows - 1) / rows;
    tot += rr[i].ntiles;
  }
  return tot;
}

// Query rows per bf16 forward / dQ workgroup: the short tile when the longest
// key range (with a sliding window: the window plus one block, as a row sees
// no more clean keys than the window and no corrupted keys outside its own
// block) is at most the kernel's short-walk limit.  A throughput choice only.
int bf16_query_rows(const bdlm_problem* p, int n_k, const bdlm_range* k_ranges, int64_t short_walk) {
  int64_t walk = 0;
  for (int j = 0; j < n_k; ++j) walk = std::max<int64_t>(walk, k_ranges[j].len);
  if (p->window > 0) walk = std::min<int64_t>(walk, p->window + p->block_size);
  return walk <= short_walk ? kQRowsShortBf16 : kQRowsLongBf16;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bdlm_status check_grid(int64_t tiles, int64_t mult) {
  if (tiles * mult >= ((int64_t)1 << 31))
    return fail(BDLM_ERR_UNSUPPORTED, "problem needs %lld workgroups (limit 2^31)", (long long)(tiles * mult));
  return BDLM_OK;
}

}  // namespace

extern "C" {

const char* bdlm_last_error(void) { return g_err.c_str(); }

bdlm_status bdlm_attn_fwd(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges, const void* const* q,
                          void* const* o, float* const* lse, int32_t n_k, const bdlm_range* k_ranges,
                          const void* const* k, const void* const* v, hipStream_t stream) {
  bdlm_status st;
  if ((st = check_problem(p)) != BDLM_OK) return st;
  if ((st = check_counts(n_q, n_k, q_ranges, k_ranges)) != BDLM_OK) return st;
  if (!q || !o || !lse || !k || !v) return fail(BDLM_ERR_INVALID, "pointer array is null");
  AttnArgs a;
  fill_common(a, p);
  a.n_q = n_q;
  a.n_k = n_k;
  for (int i = 0; i < n_q; ++i) {
    if ((st = check_range(p, q_ranges[i], "query", i)) != BDLM_OK) return st;
    if (q_ranges[i].len > 0) {
      if ((st = check_ptr(q[i], "q", i)) != BDLM_OK) return st;
      if ((st = check_ptr(o[i], "o", i)) != BDLM_OK) return st;
      if (!lse[i]) return fail(BDLM_ERR_INVALID, "lse pointer of range %d is null", i);
    }
    fill_q(a.qr[i], q_ranges[i]);
    a.qr[i].q = q[i];
    a.qr[i].o = o[i];
    a.qr[i].lse = lse[i];
  }
  for (int j = 0; j < n_k; ++j) {
    if ((st = check_range(p, k_ranges[j], "key", j)) != BDLM_OK) return st;
    if (k_ranges[j].len > 0) {
      if ((st = check_ptr(k[j], "k", j)) != BDLM_OK) return st;
      if ((st = check_ptr(v[j], "v", j)) != BDLM_OK) return st;
    }
    fill_k(a.kr[j], k_ranges[j]);
    a.kr[j].k = k[j];
    a.kr[j].v = v[j];
  }
  const int rows = p->dtype == BDLM_BF16 ? bf16_query_rows(p, n_k, k_ranges, kFwdShortWalk) : kFwdRowsF32;
  const int64_t tiles = tile_ranges(a.qr, n_q, rows);
  if ((st = check_grid(tiles, (int64_t)p->heads * p->batch)) != BDLM_OK) return st;
  a.total_tiles = (int32_t)tiles;
  a.interleave = 1;
  for (int i = 1; i < n_q; ++i)
    if (a.qr[i].ntiles != a.qr[0].ntiles) a.interleave = 0;
  const hipError_t e = p->dtype == BDLM_BF16
                           ? timed(kKFwdBf16, stream, [&] { return launch_fwd_bf16(a, p->head_dim, rows, stream); })
                           : timed(kKFwdF32, stream, [&] { return launch_fwd_f32(a, p->head_dim, stream); });
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  return BDLM_OK;
}

bdlm_status bdlm_attn_partial_fwd(const bdlm_problem* p, bdlm_range qr, const void* q, void* o, float* lse,
                                  bdlm_range kr, const void* k, const void* v, hipStream_t stream) {
  const void* qa[1] = {q};
  void* oa[1] = {o};
  float* la[1] = {lse};
  const void* ka[1] = {k};
  const void* va[1] = {v};
  return bdlm_attn_fwd(p, 1, &qr, qa, oa, la, 1, &kr, ka, va, stream);
}

bdlm_status bdlm_lse_merge(int64_t batch, int64_t rows, int32_t heads, int32_t head_dim, int32_t n_parts,
                           const void* const* o_parts, const float* const* lse_parts, int32_t part_dtype, void* o,
                           float* lse, int32_t out_dtype, hipStream_t stream) {
  return bdlm_lse_merge_strided(batch, rows, heads, head_dim, n_parts, o_parts, lse_parts, part_dtype, 0, o, lse,
                                out_dtype, 0, stream);
}

bdlm_status bdlm_lse_merge_strided(int64_t batch, int64_t rows, int32_t heads, int32_t head_dim, int32_t n_parts,
                                   const void* const* o_parts, const float* const* lse_parts, int32_t part_dtype,
                                   int64_t part_batch_stride, void* o, float* lse, int32_t out_dtype,
                                   int64_t out_batch_stride, hipStream_t stream) {
  if (batch < 1 || rows < 0 || heads < 1)
    return fail(BDLM_ERR_INVALID, "bad merge shape batch=%lld rows=%lld heads=%d", (long long)batch,
                (long long)rows, heads);
  const int64_t ps = part_batch_stride == 0 ? rows : part_batch_stride;
  const int64_t os = out_batch_stride == 0 ? rows : out_batch_stride;
  if (ps < rows || os < rows)
    return fail(BDLM_ERR_INVALID, "merge batch strides %lld / %lld below rows=%lld", (long long)part_batch_stride,
                (long long)out_batch_stride, (long long)rows);
  if (ps > kMaxPos || os > kMaxPos)
    return fail(BDLM_ERR_UNSUPPORTED, "merge batch stride above 2^30");
  if (head_dim != 64 && head_dim != 128)
    return fail(BDLM_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", head_dim);
  constexpr int64_t kMaxUnits = ((int64_t)1 << 31) - 1;  // (row, head) pairs: the grid stays below 2^31 workgroups
  if (rows > 0 && (batch > kMaxUnits / rows || (int64_t)heads > kMaxUnits / (batch * rows)))
    return fail(BDLM_ERR_UNSUPPORTED, "merge of batch=%lld x rows=%lld x heads=%d exceeds 2^31 (row, head) pairs",
                (long long)batch, (long long)rows, heads);
  if (n_parts < 1) return fail(BDLM_ERR_INVALID, "n_parts must be >= 1");
  if (n_parts > kMaxParts) return fail(BDLM_ERR_UNSUPPORTED, "n_parts=%d exceeds %d", n_parts, kMaxParts);
  if ((part_dtype != BDLM_BF16 && part_dtype != BDLM_F32) || (out_dtype != BDLM_BF16 && out_dtype != BDLM_F32))
    return fail(BDLM_ERR_UNSUPPORTED, "merge dtypes %d -> %d not supported", part_dtype, out_dtype);
  if (!o_parts || !lse_parts) return fail(BDLM_ERR_INVALID, "pointer array is null");
  MergeArgs a{};
  a.n_parts = n_parts;
  a.heads = heads;
  a.rows = rows;
  a.batch = batch;
  a.pstride = ps;
  a.ostride = os;
  if (rows > 0) {
    bdlm_status st;
    if ((st = check_ptr(o, "o", 0)) != BDLM_OK) return st;
    if (!lse) return fail(BDLM_ERR_INVALID, "lse output is null");
    for (int j = 0; j < n_parts; ++j) {
      if ((st = check_ptr(o_parts[j], "o_parts", j)) != BDLM_OK) return st;
      if (!lse_parts[j]) return fail(BDLM_ERR_INVALID, "lse pointer of part %d is null", j);
      if (o_parts[j] == o || lse_parts[j] == lse) return fail(BDLM_ERR_INVALID, "output aliases part %d", j);
    }
  }
  for (int j = 0; j < n_parts; ++j) {
    a.o_parts[j] = o_parts[j];
    a.lse_parts[j] = lse_parts[j];
  }
  a.o = o;
  a.lse = lse;
  const hipError_t e =
      timed(kKMerge, stream, [&] { return launch_merge(a, head_dim, part_dtype, out_dtype, stream); });
  if (e != hipSuccess) return hip_fail(e, "merge launch");
  return BDLM_OK;
}

size_t bdlm_attn_bwd_workspace_bytes(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges) {
  if (!p || !q_ranges || n_q < 1 || n_q > kMaxQ || p->batch < 1 || p->heads < 1 || p->head_dim < 1) return 0;
  size_t tot = 0;
  for (int i = 0; i < n_q; ++i) {
    const size_t rows = (size_t)p->batch * (size_t)(q_ranges[i].len > 0 ? q_ranges[i].len : 0);
    tot += 2 * align256(rows * p->heads * sizeof(float));  // LSE * log2(e), then D = rowsum(dO * O)
  }
  return tot;
}

}  // extern "C"

namespace {

// ---- the allocation-free backward's workspace: a file-scope device array.
// Each GPU the library runs on holds its own copy until the process ends; its
// address on the current device is looked up once per device and kept.
constexpr size_t kScratchBytes = BDLM_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

bdlm_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(BDLM_ERR_UNSUPPORTED, "device %d: the scratch table holds %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return BDLM_OK;
}

// The backward with its D / LSE*log2(e) arrays in `workspace`, or (workspace
// == nullptr and use_scratch) in the current device's scratch array.  Every
// argument is validated before the first HIP call.
bdlm_status attn_bwd_impl(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges, const void* const* q,
                          const void* const* o, const float* const* lse, const void* const* dO, void* const* dq,
                          int32_t n_k, const bdlm_range* k_ranges, const void* const* k, const void* const* v,
                          void* const* dk, void* const* dv, void* workspace, size_t workspace_bytes,
                          bool use_scratch, hipStream_t stream) {
  bdlm_status st;
  if ((st = check_problem(p)) != BDLM_OK) return st;
  if ((st = check_counts(n_q, n_k, q_ranges, k_ranges)) != BDLM_OK) return st;
  if (!q || !o || !lse || !dO || !dq || !k || !v || !dk || !dv) return fail(BDLM_ERR_INVALID, "pointer array is null");
  for (int i = 0; i < n_q; ++i)
    if ((st = check_range(p, q_ranges[i], "query", i)) != BDLM_OK) return st;
  const size_t need = bdlm_attn_bwd_workspace_bytes(p, n_q, q_ranges);
  if (use_scratch) {
    if (need > kScratchBytes)
      return fail(BDLM_ERR_UNSUPPORTED,
                  "the allocation-free backward needs %zu bytes of scratch for these query ranges; its limit is %zu "
                  "(2 x batch x rows x heads fp32 values per query range, each array rounded up to 256 bytes)",
                  need, kScratchBytes);
  } else if (need > 0 && (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u))) {
    return fail(BDLM_ERR_WORKSPACE, "workspace needs %zu bytes, 256-byte aligned (got %zu at %p)", need,
                workspace_bytes, workspace);
  }
  AttnArgs a;
  fill_common(a, p);
  a.n_q = n_q;
  a.n_k = n_k;
  int n_q_rows = 0;  // query ranges with rows (empty ones add no work to dK/dV)
  for (int i = 0; i < n_q; ++i) n_q_rows += q_ranges[i].len > 0 ? 1 : 0;
  a.stats_form = dkdv_uses_scheduled_kernel(p->dtype == BDLM_BF16, p->head_dim, p->hilo, a.group, n_q_rows) ? 1 : 0;
  size_t ws_off[kMaxQ] = {};
  size_t off = 0;
  for (int i = 0; i < n_q; ++i) {
    const bdlm_range& r = q_ranges[i];
    if (r.len > 0) {
      if ((st = check_ptr(q[i], "q", i)) != BDLM_OK) return st;
      if ((st = check_ptr(o[i], "o", i)) != BDLM_OK) return st;
      if ((st = check_ptr(dO[i], "dO", i)) != BDLM_OK) return st;
      if ((st = check_ptr(dq[i], "dq", i)) != BDLM_OK) return st;
      if (!lse[i]) return fail(BDLM_ERR_INVALID, "lse pointer of range %d is null", i);
    }
    fill_q(a.qr[i], r);
    a.qr[i].q = q[i];
    a.qr[i].o = const_cast<void*>(o[i]);
    a.qr[i].lse = const_cast<float*>(lse[i]);
    a.qr[i].dO = dO[i];
    a.qr[i].dq = dq[i];
    const size_t rows = (size_t)p->batch * (size_t)r.len;
    const size_t arr = align256(rows * p->heads * sizeof(float));
    if (arr > ((size_t)1 << 30))
      return fail(BDLM_ERR_UNSUPPORTED, "query range %d: batch * len * heads = %zu rows exceeds 2^28", i,
                  rows * p->heads);
    ws_off[i] = off;  // l2 at off, D at off + arr (pointers set once the base is known)
    off += 2 * arr;
  }
  for (int j = 0; j < n_k; ++j) {
    if ((st = check_range(p, k_ranges[j], "key", j)) != BDLM_OK) return st;
    if (k_ranges[j].len > 0) {
      if ((st = check_ptr(k[j], "k", j)) != BDLM_OK) return st;
      if ((st = check_ptr(v[j], "v", j)) != BDLM_OK) return st;
      if ((st = check_ptr(dk[j], "dk", j)) != BDLM_OK) return st;
      if ((st = check_ptr(dv[j], "dv", j)) != BDLM_OK) return st;
    }
    fill_k(a.kr[j], k_ranges[j]);
    a.kr[j].k = k[j];
    a.kr[j].v = v[j];
    a.kr[j].dk = dk[j];
    a.kr[j].dv = dv[j];
  }
  const int keys = p->dtype == BDLM_BF16 ? kBwdKeysBf16 : kBwdKeysF32;
  const int64_t tiles = tile_ranges(a.kr, n_k, keys);
  if ((st = check_grid(tiles, (int64_t)p->kv_heads * p->batch)) != BDLM_OK) return st;
  a.total_tiles = (int32_t)tiles;
  // The dQ kernel walks query tiles (of its own height).
  AttnArgs aq = a;
  const int dq_rows = bf16_query_rows(p, n_k, k_ranges, kDqShortWalk);
  if (p->dtype == BDLM_BF16) {
    const int64_t qt = tile_ranges(aq.qr, n_q, dq_rows);
    if ((st = check_grid(qt, (int64_t)p->heads * p->batch)) != BDLM_OK) return st;
    aq.total_tiles = (int32_t)qt;
    aq.interleave = 1;
    for (int i = 1; i < n_q; ++i)
      if (aq.qr[i].ntiles != aq.qr[0].ntiles) aq.interleave = 0;
  }
  // Validation done: place D and LSE*log2(e).
  char* base = static_cast<char*>(workspace);
  if (use_scratch && need > 0) {
    void* sp = nullptr;
    if ((st = scratch_of_current_device(&sp)) != BDLM_OK) return st;
    base = static_cast<char*>(sp);
  }
  for (int i = 0; i < n_q; ++i) {
    const size_t arr = align256((size_t)p->batch * (size_t)q_ranges[i].len * p->heads * sizeof(float));
    float* l2 = need > 0 ? reinterpret_cast<float*>(base + ws_off[i]) : nullptr;
    float* dl = need > 0 ? reinterpret_cast<float*>(base + ws_off[i] + arr) : nullptr;
    a.qr[i].l2 = aq.qr[i].l2 = l2;
    a.qr[i].delta = aq.qr[i].delta = dl;
  }
  // Visit key ranges heaviest first: clean ranges by ascending position (their
  // early keys are seen by the most queries), then corrupted ranges.
  int n = 0;
  for (int pass = 0; pass < 2; ++pass) {
    const int want = pass == 0 ? BDLM_CLEAN : BDLM_CORRUPTED;
    bool used[kMaxK] = {false};
    for (int c = 0; c < n_k; ++c) {
      int best = -1;
      for (int j = 0; j < n_k; ++j)
        if (!used[j] && k_ranges[j].stream == want && (best < 0 || k_ranges[j].pos0 < k_ranges[best].pos0)) best = j;
      if (best < 0) break;
      used[best] = true;
      a.order[n++] = best;
    }
  }
  hipError_t e = hipSuccess;
  if (p->dtype == BDLM_BF16) {
    // The dQ kernel computes D = rowsum(dO * O) itself and leaves each row's
    // statistics in the workspace for the dK/dV kernel, so it runs first.
    for (int j = 0; j < n_k; ++j) aq.order[j] = a.order[j];
    e = timed(kKBwdDq, stream, [&] { return launch_bwd_dq_bf16(aq, p->head_dim, dq_rows, stream); });
    if (e != hipSuccess) return hip_fail(e, "backward dQ launch");
    e = timed(kKBwdBf16, stream, [&] {
      if (!a.stats_form) return launch_bwd_bf16(a, p->head_dim, stream);
      // The scheduled kernel walks at most two query ranges: pass it the ranges
      // that have rows, in call order (the order the walk accumulates in).
      AttnArgs ak = a;
      ak.n_q = 0;
      for (int i = 0; i < n_q; ++i)
        if (a.qr[i].len > 0) ak.qr[ak.n_q++] = a.qr[i];
      return launch_bwd_dkdv(ak, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "backward dK/dV launch");
  } else {
    e = timed(kKBwdPre, stream, [&] { return launch_bwd_pre(a, p->head_dim, stream); });
    if (e != hipSuccess) return hip_fail(e, "backward pre-pass launch");
    e = timed(kKBwdF32, stream, [&] { return launch_bwd_f32(a, p->head_dim, stream); });
    if (e != hipSuccess) return hip_fail(e, "backward launch");
  }
  return BDLM_OK;
}

}  // namespace

extern "C" {

bdlm_status bdlm_attn_bwd(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges, const void* const* q,
                          const void* const* o, const float* const* lse, const void* const* dO, void* const* dq,
                          int32_t n_k, const bdlm_range* k_ranges, const void* const* k, const void* const* v,
                          void* const* dk, void* const* dv, void* workspace, size_t workspace_bytes,
                          hipStream_t stream) {
  return attn_bwd_impl(p, n_q, q_ranges, q, o, lse, dO, dq, n_k, k_ranges, k, v, dk, dv, workspace,
                       workspace_bytes, false, stream);
}

bdlm_status bdlm_attn_bwd_noalloc(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges,
                                  const void* const* q, const void* const* o, const float* const* lse,
                                  const void* const* dO, void* const* dq, int32_t n_k, const bdlm_range* k_ranges,
                                  const void* const* k, const void* const* v, void* const* dk, void* const* dv,
                                  hipStream_t stream) {
  return attn_bwd_impl(p, n_q, q_ranges, q, o, lse, dO, dq, n_k, k_ranges, k, v, dk, dv, nullptr, 0, true, stream);
}

bdlm_status bdlm_timing_enable(int32_t on) {
  g_timing = on != 0;
  return BDLM_OK;
}

int32_t bdlm_timing_collect(int32_t max_records, int32_t* kernel_ids, float* ms) {
  int32_t n = 0;
  hipError_t err = hipSuccess;
  for (const TimingRec& r : g_recs) {
    if (err == hipSuccess && n < max_records && kernel_ids && ms) {
      float t = 0.f;
      err = hipEventSynchronize(r.b);
      if (err == hipSuccess) err = hipEventElapsedTime(&t, r.a, r.b);
      if (err == hipSuccess) {
        kernel_ids[n] = r.id;
        ms[n] = t;
        ++n;
      }
    }
    g_event_pool.push_back(r.a);
    g_event_pool.push_back(r.b);
  }
  g_recs.clear();
  if (err != hipSuccess) return (int32_t)hip_fail(err, "timing collect");
  return n;
}

const char* bdlm_kernel_name(int32_t kernel_id) {
  return (kernel_id >= 0 && kernel_id < kKCount) ? kKernelNames[kernel_id] : "unknown";
}

int64_t bdlm_visible_pairs(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges, int32_t n_k,
                           const bdlm_range* k_ranges) {
  if (check_problem(p) != BDLM_OK) return -1;
  if (check_counts(n_q, n_k, q_ranges, k_ranges) != BDLM_OK) return -1;
  for (int i = 0; i < n_q; ++i)
    if (check_range(p, q_ranges[i], "query", i) != BDLM_OK) return -1;
  for (int j = 0; j < n_k; ++j)
    if (check_range(p, k_ranges[j], "key", j) != BDLM_OK) return -1;
  // A clean-context table lives in device memory: read it back (synchronously)
  // and check its contract, which the asynchronous calls cannot.
  std::vector<int> table;
  if (p->clean_prefix) {
    table.resize((size_t)(p->L / p->block_size));
    if (hipMemcpy(table.data(), p->clean_prefix, table.size() * sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
      return -1;
    for (size_t b = 0; b < table.size(); ++b)
      if (table[b] < 0 || table[b] > p->L || (b > 0 && table[b] < table[b - 1])) return -1;
  }
  const MaskRule rule = host_rule(p, p->clean_prefix ? table.data() : nullptr);
  int64_t tot = 0;
  for (int i = 0; i < n_q; ++i)
    for (int64_t r = 0; r < q_ranges[i].len; ++r) {
      const int pq = (int)(q_ranges[i].pos0 + r);
      for (int j = 0; j < n_k; ++j) {
        int lo, hi;
        key_interval(q_ranges[i].stream, pq, k_ranges[j].stream, rule, lo, hi);
        lo = imax(lo, (int)k_ranges[j].pos0);
        hi = imin(hi, (int)(k_ranges[j].pos0 + k_ranges[j].len));
        if (hi > lo) tot += hi - lo;
      }
    }
  return tot;
}

}  // extern "C"
