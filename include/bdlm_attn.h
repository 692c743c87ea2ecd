/*
 * bdlm_attn.h -- C ABI of the BDLM attention library for MI355X (gfx950).
 *
 * Block-diffusion LM training evaluates attention over a length-2L sequence:
 * a clean copy x and a corrupted copy x_t of L tokens, both split into blocks
 * of block_size tokens (arXiv 2609.19242, Sec. 3.2).  With 0-based positions
 * and blk(p) = p / block_size, a query row may attend to a key row when
 *
 *   clean query q,     clean key k:     k <= q                (token-causal; the paper's rule,
 *                                                              App. A eq:correctness-clean-attention)
 *                                       blk(k) <= blk(q)      (BDLM_CLEAN_INTRA_BLOCK reading)
 *   corrupted query q, corrupted key k: blk(k) == blk(q)      (own block, bidirectional)
 *   corrupted query q, clean key k:     blk(k) <  blk(q)      (clean prefix of earlier blocks)
 *   clean query,       corrupted key:   never
 *
 * (eq:correctness-corrupted-attention).  The library computes masked softmax
 * attention under this mask, its log-sum-exp, partial attention over one key
 * range, the J-way log-sum-exp merge of partials (eq:csbp-lse-merge), and the
 * exact backward from the saved output and LSE (App. C, fused backward).
 *
 * Mask generalisations (both keep every visible set an interval of positions):
 *  - window W > 0 (the sliding-window attention layers of the paper's
 *    DiffusionGemma runs, App. "Savings Breakdowns"): with e the end of the
 *    clean context the rules above give a query (q + 1 for a clean query under
 *    the token-causal rule, the end of its block under BDLM_CLEAN_INTRA_BLOCK,
 *    the start of its block for a corrupted query), only clean keys k with
 *    e - W <= k < e stay visible.  Corrupted keys are unaffected.
 *  - clean_prefix (the DFlash2 drafter attention, App. "DFlash2 Drafter
 *    Training Methodology", eq:dflash2-block-attention): corrupted block b is a
 *    draft block whose clean context (the target features) ends at
 *    clean_prefix[b] = a_b instead of at block_size * b; it still sees its own
 *    block bidirectionally.  The table must be non-decreasing with entries in
 *    [0, L] (draft blocks ordered by anchor: their losses are independent, so
 *    the order is free).  The asynchronous calls cannot check the contents:
 *    entries are clamped into [0, L] when read, and a decreasing table gives an
 *    unspecified mask (never an out-of-bounds access).  bdlm_visible_pairs
 *    checks the table and returns -1 when it breaks the contract.
 *
 * Rows and ranges.  A tensor's rows are described by bdlm_range records: a
 * range is `len` consecutive rows of one stream holding global positions
 * [pos0, pos0 + len).  Per batch element b, row i of a range lives at row
 * (b * batch_stride + i) of the pointer given for that range, where
 * batch_stride >= len (0 means len).  The packed joint layout [x_t ; x] of a
 * [batch][2L][heads][head_dim] tensor is two ranges {CORRUPTED, 0, L} at row 0
 * and {CLEAN, 0, L} at row L, both with batch_stride 2L.
 *
 * Layouts (all row-major, head_dim innermost, 16-byte aligned pointers):
 *   Q, O, dO, dQ : [batch][rows][heads][head_dim]
 *   K, V, dK, dV : [batch][rows][kv_heads][head_dim]
 *   Q, K, V, dO are in the problem's dtype; O, dQ, dK, dV are in that dtype,
 *   or fp32 when out_f32 = 1 (bdlm_attn_bwd reads O in the same type).
 *   LSE          : [batch][heads][rows] fp32, natural log; for a range with
 *                  batch stride R, element (b, h, i) is at b*heads*R + h*R + i.
 * Query head h reads KV head h / (heads / kv_heads).
 *
 * Ownership and execution.  Every buffer is device memory owned by the caller;
 * the library allocates and frees nothing.  Each call validates its arguments
 * on the host, then enqueues kernels on `stream` and returns without
 * synchronising.  Pointer arrays (`const void* const* q` ...) are host arrays
 * of device pointers, read during the call only.
 *
 * Errors.  A call returns BDLM_OK or a negative status.  Invalid or
 * unsupported arguments are rejected before anything is enqueued; a failed
 * launch returns BDLM_ERR_HIP.  bdlm_last_error() returns a message for the
 * calling thread's last failure.  No C++ exception crosses this interface.
 */
#ifndef BDLM_ATTN_H
#define BDLM_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BDLM_OK = 0,
  BDLM_ERR_INVALID = -1,     /* malformed argument: sizes, ranges, null or misaligned pointers */
  BDLM_ERR_UNSUPPORTED = -2, /* well-formed but not implemented: head_dim, dtype, too many ranges */
  BDLM_ERR_HIP = -3,         /* a HIP call or kernel launch failed */
  BDLM_ERR_WORKSPACE = -4    /* workspace missing or smaller than bdlm_attn_bwd_workspace_bytes */
} bdlm_status;

typedef enum { BDLM_BF16 = 0, BDLM_F32 = 1 } bdlm_dtype;
typedef enum { BDLM_CLEAN = 0, BDLM_CORRUPTED = 1 } bdlm_stream;
typedef enum {
  BDLM_CLEAN_INTRA_CAUSAL = 0, /* clean query at position q sees clean keys at positions <= q */
  BDLM_CLEAN_INTRA_BLOCK = 1   /* clean query sees every clean key of its own and earlier blocks */
} bdlm_clean_intra;

/* Bits of bdlm_problem.hilo: which products carry P or dS as two bf16 terms. */
#define BDLM_HILO_PV 1   /* forward O += P V */
#define BDLM_HILO_DKDV 2 /* backward dV += P^T dO and dK += dS^T Q */
#define BDLM_HILO_DQ 4   /* backward dQ += dS K */
#define BDLM_HILO_ALL 7
/* With any of the bits above: a selected product carries the second term only where some
   probability P of the block of operands it contracts reaches 1/64, and a single bf16 term
   elsewhere.  The blocks are one wave's 32 query rows x 16 keys (P V, dS K) or 32 keys x 16 query
   rows of one query head (P^T dO, dS^T Q); the forward tests P against the row's running sum,
   which can only over-select.  An element left single-term has P < 1/64, so its rounding error is
   below 2^-15 in P and below 2^-15 |dP - D| in dS.  Same results as the all-tiles form up to
   rounding; fewer matrix products where large probabilities are rare. */
#define BDLM_HILO_ADAPTIVE 8

/* Limits of one call (kernel-argument capacity). */
#define BDLM_MAX_Q_RANGES 4
#define BDLM_MAX_K_RANGES 32
#define BDLM_MAX_MERGE_PARTS 32

/* Shape and mask description shared by every attention call. */
typedef struct {
  int64_t batch;      /* independent sequences, >= 1 */
  int64_t L;          /* tokens per copy: positions of both streams lie in [0, L) */
  int64_t block_size; /* tokens per block (the paper's M = L / B); L % block_size == 0 */
  int32_t heads;      /* query heads, a multiple of kv_heads */
  int32_t kv_heads;   /* key/value heads */
  int32_t head_dim;   /* 64 or 128 */
  int32_t dtype;      /* bdlm_dtype of Q, K, V and dO (and of the outputs unless out_f32) */
  float scale;        /* softmax scale; <= 0 selects 1 / sqrt(head_dim) */
  int32_t clean_intra;/* bdlm_clean_intra */
  int32_t out_f32;    /* 0: O, dQ, dK, dV in `dtype`; 1: in fp32 (the fp32 accumulators, unrounded) */
  int32_t hilo;       /* bf16 path: a mask of BDLM_HILO_* bits.  A product whose bit is clear takes
                         its operand P (softmax probabilities) or dS = P (dP - D) rounded to bf16;
                         a product whose bit is set takes it as a two-term bf16 sum hi + lo (about
                         16 significant bits, twice the matrix work of that product), on every
                         tile or, with BDLM_HILO_ADAPTIVE, only on tiles holding a large P.  For
                         inputs with large scores or |dS|, e.g. keys of large norm.  Ignored by
                         the fp32 path. */
  int64_t window;     /* 0: no limit.  > 0: a query sees only the last `window` positions of its clean
                         context (sliding-window layers; see "Mask generalisations" above) */
  const int32_t* clean_prefix; /* NULL, or a device array of L / block_size ints: the end of the clean
                         context of corrupted block b (DFlash2 anchors; see above).  Read by the kernels
                         during the call's execution; bdlm_visible_pairs reads it synchronously. */
} bdlm_problem;

/* A run of rows of one stream (see "Rows and ranges" above). */
typedef struct {
  int32_t stream;       /* bdlm_stream */
  int32_t reserved;     /* must be 0 */
  int64_t pos0;         /* global position of the range's first row, >= 0 */
  int64_t len;          /* rows, >= 0; pos0 + len <= L */
  int64_t batch_stride; /* rows between batch elements in this range's tensors; 0 means len */
} bdlm_range;

/*
 * Fused forward (Sec. 3.2 mask; eq:context-parallel-attention).
 * For every row of the n_q query ranges: O = softmax(scale * Q K^T + mask) V
 * and LSE = log sum exp(scale * Q K^T + mask), over all rows of the n_k key
 * ranges, in one pass with online softmax across ranges.  Tiles the mask
 * hides are skipped; only tiles it partly hides evaluate it.
 *   q[i], o[i], lse[i] : query range i's Q (in), O (out), LSE (out)
 *   k[j], v[j]         : key range j's K and V (in)
 * A query row that sees no key gets O = 0 and LSE = -inf.
 * Limits: 1 <= n_q <= BDLM_MAX_Q_RANGES, 1 <= n_k <= BDLM_MAX_K_RANGES.
 */
bdlm_status bdlm_attn_fwd(const bdlm_problem* p,
                          int32_t n_q, const bdlm_range* q_ranges,
                          const void* const* q, void* const* o, float* const* lse,
                          int32_t n_k, const bdlm_range* k_ranges,
                          const void* const* k, const void* const* v,
                          hipStream_t stream);

/*
 * Partial forward of one query range over one key range (App. A, step 2,
 * eq:correctness-online-softmax-merge; the per-launch normalised output O_j and
 * LSE z_j of App. C).  Same arithmetic as bdlm_attn_fwd restricted to key range
 * kr: O_j is normalised over the visible keys of kr only; rows that see none of
 * them get O_j = 0 exactly and z_j = -inf, so merging them is a no-op.
 *   q, o, lse : query range qr's Q (in), O_j (out), z_j (out)
 *   k, v      : key range kr's K and V (in)
 */
bdlm_status bdlm_attn_partial_fwd(const bdlm_problem* p,
                                  bdlm_range qr, const void* q, void* o, float* lse,
                                  bdlm_range kr, const void* k, const void* v,
                                  hipStream_t stream);

/*
 * J-way log-sum-exp merge of normalised partials over disjoint key sets
 * (eq:csbp-lse-merge generalised by eq:correctness-online-softmax-merge):
 *   m = max_j z_j,  w_j = exp(z_j - m) (0 where z_j = -inf),
 *   O = sum_j w_j O_j / sum_j w_j,  z = m + log(sum_j w_j),
 * in fp32 registers, one pass over the J inputs.  A row with every z_j = -inf
 * gets O = 0 and z = -inf.
 *   o_parts[j] : [batch][rows][heads][head_dim] in part_dtype
 *   lse_parts[j] : [batch][heads][rows] fp32
 *   o : [batch][rows][heads][head_dim] in out_dtype;  lse : [batch][heads][rows] fp32
 * o and lse may alias neither input.  1 <= n_parts <= BDLM_MAX_MERGE_PARTS;
 * batch * rows * heads < 2^31 (else BDLM_ERR_UNSUPPORTED, nothing launched).
 */
bdlm_status bdlm_lse_merge(int64_t batch, int64_t rows, int32_t heads, int32_t head_dim,
                           int32_t n_parts, const void* const* o_parts,
                           const float* const* lse_parts, int32_t part_dtype,
                           void* o, float* lse, int32_t out_dtype, hipStream_t stream);

/*
 * bdlm_lse_merge over rows laid out with batch strides, as the attention calls
 * write them (bdlm_range.batch_stride): part element (b, i, h, :) of O_j is at
 * row b * part_batch_stride + i of o_parts[j], z_j(b, h, i) at
 * (b * heads + h) * part_batch_stride + i of lse_parts[j]; the outputs likewise
 * with out_batch_stride.  A stride of 0 means rows (dense, as bdlm_lse_merge).
 * Strides below rows give BDLM_ERR_INVALID, above 2^30 BDLM_ERR_UNSUPPORTED;
 * otherwise the contract of bdlm_lse_merge, which is this call with both
 * strides 0.  Padding rows between batch elements are neither read nor written.
 */
bdlm_status bdlm_lse_merge_strided(int64_t batch, int64_t rows, int32_t heads, int32_t head_dim,
                                   int32_t n_parts, const void* const* o_parts,
                                   const float* const* lse_parts, int32_t part_dtype,
                                   int64_t part_batch_stride, void* o, float* lse,
                                   int32_t out_dtype, int64_t out_batch_stride,
                                   hipStream_t stream);

/* Workspace bytes bdlm_attn_bwd needs for these query ranges: per range two
 * fp32 arrays of batch * len * heads values (each rounded up to 256 bytes),
 * LSE * log2(e) and the row dots D = rowsum(dO * O).  Ranges whose
 * batch * len * heads exceeds 2^28 are rejected by bdlm_attn_bwd. */
size_t bdlm_attn_bwd_workspace_bytes(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges);

/*
 * Backward from the saved (final, merged) O and LSE (App. C fused backward;
 * eqs. eq:correctness-corrupted-gradient .. eq:correctness-query-gradient).
 * With P = exp(scale * Q K^T + mask - LSE) and D = rowsum(dO * O):
 *   dV = P^T dO,  dS = P * (dO V^T - D),  dQ = scale * dS K,  dK = scale * dS^T Q,
 * summed over every query row of every query range, and over the query heads
 * of each KV head.  dq[i] like q[i]; dk[j], dv[j] like k[j]; all overwritten.
 * Key rows no query sees get dK = dV = 0.
 * workspace: device memory of at least bdlm_attn_bwd_workspace_bytes(), 256-byte
 * aligned, contents ignored on entry.
 */
bdlm_status bdlm_attn_bwd(const bdlm_problem* p,
                          int32_t n_q, const bdlm_range* q_ranges,
                          const void* const* q, const void* const* o, const float* const* lse,
                          const void* const* dO, void* const* dq,
                          int32_t n_k, const bdlm_range* k_ranges,
                          const void* const* k, const void* const* v,
                          void* const* dk, void* const* dv,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * bdlm_attn_bwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, arithmetic, kernels and results as
 * bdlm_attn_bwd; D and LSE * log2(e) live in a library-owned device array of
 * BDLM_NOALLOC_SCRATCH_BYTES bytes instead (one per GPU, held until the process
 * ends).  The call allocates nothing.  Query ranges that need more than the
 * array holds (bdlm_attn_bwd_workspace_bytes() > BDLM_NOALLOC_SCRATCH_BYTES,
 * i.e. more than about 8M (batch x row x head) entries) are rejected with
 * BDLM_ERR_UNSUPPORTED before anything is enqueued.  The array of the device
 * current at the call is used, so `stream` must belong to that device.  Every
 * call on one GPU shares its array: calls that overlap in time on one GPU
 * (other streams, other threads) race and must be serialised by the caller.
 */
#define BDLM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
bdlm_status bdlm_attn_bwd_noalloc(const bdlm_problem* p,
                                  int32_t n_q, const bdlm_range* q_ranges,
                                  const void* const* q, const void* const* o, const float* const* lse,
                                  const void* const* dO, void* const* dq,
                                  int32_t n_k, const bdlm_range* k_ranges,
                                  const void* const* k, const void* const* v,
                                  void* const* dk, void* const* dv, hipStream_t stream);

/*
 * Number of valid query-key pairs of the mask per (batch element, query head),
 * summed over the given ranges (the paper's unit of attention work, App. B
 * eq:block-work-by-position).  Host only; returns -1 on invalid arguments.
 */
int64_t bdlm_visible_pairs(const bdlm_problem* p, int32_t n_q, const bdlm_range* q_ranges,
                           int32_t n_k, const bdlm_range* k_ranges);

/*
 * Kernel timing (observability).  While enabled for the calling thread, every
 * kernel the library enqueues is bracketed by two hipEvents recorded on its
 * stream.  bdlm_timing_collect() waits for the recorded events, writes up to
 * max_records (kernel id, milliseconds) pairs in launch order, forgets them and
 * returns how many it wrote (or a negative status).  bdlm_kernel_name() maps an
 * id to a name.  Disabled by default; events are created on first use and
 * reused.
 */
bdlm_status bdlm_timing_enable(int32_t on);
int32_t bdlm_timing_collect(int32_t max_records, int32_t* kernel_ids, float* ms);
const char* bdlm_kernel_name(int32_t kernel_id);

/* Message for the calling thread's last failed call ("" if none). */
const char* bdlm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* BDLM_ATTN_H */
