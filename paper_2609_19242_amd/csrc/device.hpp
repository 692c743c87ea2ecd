// gfx950 device helpers: vector types, MFMA, buffer loads, LDS transpose reads.
//
// Lane layouts (checked on the GPU):
//  * v_mfma_f32_32x32x16_bf16 -- A (32x16): lane l holds row l%32, k = 8*(l/32)+j;
//    B (16x32): lane l holds column l%32, k = 8*(l/32)+j;  C (32x32): lane l,
//    register i holds column l%32, row 8*(i/4) + 4*(l/32) + i%4.
//  * ds_read_b64_tr_b16 -- inside each group of 16 lanes, lane i receives
//    element i%4 of the 8-byte rows addressed by lanes i/4, i/4+4, i/4+8,
//    i/4+12.  Addressing row R(s/4), column c0 + 4*(s%4) from source lane s
//    therefore hands lane i the column c0 + i of rows R(0..3): a transposed
//    4x16 fragment, which is how row-major V, Q and dO tiles in LDS become the
//    k-major MFMA operands the products P V, dO^T P and Q^T dS need.
//  * v_permlane32_swap with both operands x: result[0] holds x of lanes 0..31
//    in both halves, result[1] holds x of lanes 32..63 in both halves.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdlm {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef short short4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Raw buffer resource over [base, base + bytes): loads past the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

__device__ __forceinline__ float buf_load_f32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
}

// Global -> LDS copy that bypasses registers: lane i of the wave writes its
// BYTES (4 or 16) to lds + i * BYTES (lds is wave-uniform); offsets past the
// resource's end write zeros and fetch nothing.  Completion counts against
// vmcnt like any vector-memory load.
template <int BYTES>
__device__ __forceinline__ void buf_to_lds(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff, uint32_t soff) {
  static_assert(BYTES == 4 || BYTES == 16, "LDS copy width");
  auto* dst = (__attribute__((address_space(3))) void*)lds;
  if constexpr (BYTES == 16) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
  else __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 4, voff, soff, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are in flight,
// then a workgroup barrier.  Used where LDS written by buf_to_lds copies of
// every wave must be complete; the memory clobber keeps LDS accesses on their
// side of the barrier.
template <int N>
__device__ __forceinline__ void vm_wait_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// ---- swizzled LDS tiles of bf16 rows.
//
// Tiles of D-element bf16 rows (Q, dO, K or V) are stored in LDS unpadded;
// logical 16-byte chunk c of row r sits in physical chunk c ^ chunk_swz<D>(r).
// The kernels read such a tile in two patterns: 64-lane ds_read_b128 row reads
// (16 lanes per LDS cycle: 16 consecutive rows, one chunk each) and
// ds_read_b64_tr_b16 transpose reads (32 lanes per cycle: 4 consecutive rows,
// 64 bytes each).  With 256-byte rows (D = 128) the 16 rows of a row read land
// in 16 distinct chunk columns and the 4 rows of a transpose read in 4
// disjoint quarter-rows, so both are conflict-free (64 banks x 4 bytes); for
// D = 64 (128-byte rows, two rows per bank period) the same holds with the
// second function.  Padding alone cannot do both: 272-byte rows are 4-way on
// transpose reads, 320-byte rows 4-way on row reads, 288-byte rows 2-way on
// each.  The function depends on r mod 16 only.  Copies into such a tile go
// through LDS DMA (buf_to_lds), where lane i fills physical slot i of its
// instruction: the lane fetches the logical chunk that belongs there.
template <int D>
__host__ __device__ constexpr int chunk_swz(int r) {
  return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
}

// Global byte offset of the logical chunk stored in physical slot `slot` of a
// swizzled tile whose row r lives at global element offset r * row_stride.
template <int D>
__device__ __forceinline__ uint32_t swz_src_offset(int slot, int64_t row_stride) {
  const int row = slot / (D / 8), ch = (slot % (D / 8)) ^ chunk_swz<D>(row);
  return (uint32_t)((row * row_stride + ch * 8) * 2);
}

// 32-bit LDS addresses.  Tile bases are 256-byte aligned, so XOR-ing chunk
// bits into a row address never carries into the row bits.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}
__device__ __forceinline__ void lds_store8(uint32_t a, bf16x4 v) {
  *(__attribute__((address_space(3))) bf16x4*)(uintptr_t)a = v;
}
__device__ __forceinline__ bf16x8 lds_load16(uint32_t a) {
  return *(__attribute__((address_space(3))) const bf16x8*)(uintptr_t)a;
}
// Transposed 8-byte LDS read at LDS address a (see the header comment).
__device__ __forceinline__ bf16x4 lds_read_tr_at(uint32_t a) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                        (__attribute__((address_space(3))) short4_t*)(uintptr_t)a));
}

// Per-lane parts of the swizzled read addresses.  Row reads: lane (half, l32)
// reads logical chunk 2k + half of row l32 at (base + row_part) ^ 32k.
// Transpose reads of the MFMA fragment layout: the lane reads rows 16u + r0
// and 16u + r0 + 8 (r0 = 4 (G >> 1) + (sl >> 2)), 8-byte piece
// 8d + 4 (G & 1) + (sl & 3), at (base + tr_part(0 or 8)) ^ 64d; row offsets
// that are multiples of 16 rows are plain additions.
template <int D>
__device__ __forceinline__ uint32_t swz_row_part(int l32, int half) {
  return l32 * (2 * D) + ((half ^ chunk_swz<D>(l32)) * 16);
}
template <int D>
__device__ __forceinline__ uint32_t swz_tr_part(int G, int sl, int plus) {
  const int r = 4 * (G >> 1) + (sl >> 2) + plus, ch = 2 * (G & 1) + ((sl >> 1) & 1);
  return r * (2 * D) + ((ch ^ chunk_swz<D>(r)) * 16) + 8 * (sl & 1);
}

__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// x of the lane l ^ 32 (the other half of the wavefront).
__device__ __forceinline__ float partner(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const uint32_t lane = __lane_id();
  return __uint_as_float(lane < 32 ? r[1] : r[0]);
}

__device__ __forceinline__ float exp2f_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16 to_bf16(float x) { return (bf16)x; }

}  // namespace bdlm

namespace bdlm {
// fp32 atomic add through a buffer resource: offsets past the resource's end
// are dropped by the hardware, so callers need no per-lane bounds branch.
__device__ __forceinline__ void buf_atomic_add(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float v) {
  __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(v, r, byte_off, 0, 0);
}

// A wave's 32 rows x D columns held the MFMA-accumulator way (the lanes l32
// and l32 + 32 own row l32; element e of fragment (dt, g4) is column
// 32 dt + 8 g4 + 4 half + e), written to global memory as bf16 through the
// wave's D * 64 bytes of LDS at sw: the lanes store their 8-byte pieces, then
// every global store writes 64 / (D / 8) whole rows instead of 16 bytes of
// each of 32 rows.  16-byte chunk c of row r sits at chunk c ^ (r % (D / 8)),
// so the row reads are conflict-free.  Row r goes to rows + r * row_stride
// (elements) when r < nrows.  Nobody else may use those LDS bytes meanwhile.
template <int D, class V>
__device__ __forceinline__ void store_rows_bf16_via_lds(uint32_t sw, V&& value, bf16* rows, int64_t row_stride,
                                                        int nrows, int lane) {
  constexpr int CH = D / 8, RPI = 64 / CH;
  const int l32 = lane & 31, half = lane >> 5;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      bf16x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = to_bf16(value(dt, g4, e));
      const uint32_t c = (uint32_t)((4 * dt + g4) ^ (l32 & (CH - 1)));
      lds_store8(sw + (uint32_t)l32 * (D * 2) + c * 16u + 8u * half, v);
    }
#pragma unroll
  for (int i = 0; i < 32 / RPI; ++i) {
    const int r = i * RPI + lane / CH, c = lane % CH;
    const bf16x8 x = lds_load16(sw + (uint32_t)r * (D * 2) + (uint32_t)(c ^ (r & (CH - 1))) * 16u);
    if (r < nrows) *(bf16x8*)(rows + r * row_stride + c * 8) = x;
  }
}

}  // namespace bdlm
