// Device-side building blocks shared by the LoRA-linear kernels (gfx950 only).
//
// Matrix-core primitives (bf16 in, fp32 accumulate):
//   v_mfma_f32_32x32x16_bf16 -- the GEMM workhorse.  With lane l, c = l % 32,
//     g = l / 32:  A operand (32 x 16, M x K): lane holds row c, k = 8g .. 8g+7;
//     B operand (16 x 32, K x N): lane holds column c, k = 8g .. 8g+7;
//     result (32 x 32): lane holds column c, rows 8(q/4) + 4g + q%4, q = 0..15.
//     On gfx950 it issues at the full bf16 rate (1024 flop/clk per SIMD).
//   v_mfma_f32_16x16x32_bf16 -- used by the small rank-r kernels.  With
//     c = l % 16, g = l / 16: A holds row c, k = 8g .. 8g+7; B holds column c,
//     the same k; the result holds column c, rows 4g .. 4g+3.  It issues at
//     about half the flop rate of the 32x32 form.
// Both operands carry k in the same positions, so any matrix stored with k
// contiguous is read with one 16-byte load per lane.
//
// LDS tiles come in two forms:
//   * k-contiguous tiles: rows of 64 bf16 (128 bytes = 8 chunks of 16 bytes).
//     Chunk q of row p is stored at chunk position q ^ ((p >> 1) & 7), so the
//     16 lanes that read one 16-byte chunk from 16 consecutive rows hit
//     distinct banks.
//   * mn-contiguous tiles (k is the row index): rows of COLS bf16, read with
//     ds_read_b64_tr_b16, which hands lane i of each 16-lane group column i of
//     a 4 x 16 block of rows (4 consecutive k of one operand column); two such
//     reads give a lane its 8 k.  The chunk swizzle depends on which lanes
//     share a read cycle: mc16_* for the 16x16x32 operand layout,
//     mc32_* (chunk q of row p at q ^ 4(p & 3)) for the 32x32x16 one.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

// Lambdas inside kernels are forced inline: the fragment registers written
// by the inline-assembly LDS reads below must stay in registers between the
// read and its wait, which an outlined call (its operands passed through
// scratch) would break.
#define LORA_INLINE __attribute__((always_inline))

namespace lora {

typedef uint16_t u16;
typedef short short8 __attribute__((ext_vector_type(8)));
typedef short short4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef int int4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4v lds_short4v;

// A buffer offset at or beyond every resource size used here: loads at it
// return zero.  Resource sizes are capped below it.
constexpr uint32_t kOOB = 0x80000000u;
constexpr uint32_t kMaxRecords = 0x7FFFFF00u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint64_t nbytes) {
  uint32_t n = nbytes > kMaxRecords ? kMaxRecords : (uint32_t)nbytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

// 16-byte load through a buffer resource; out-of-range offsets read as zero.
__device__ __forceinline__ int4v buf_load16(__amdgpu_buffer_rsrc_t rs, uint32_t byte_off) {
  return __builtin_bit_cast(int4v, __builtin_amdgcn_raw_buffer_load_b128(rs, byte_off, 0, 0));
}

__device__ __forceinline__ floatx4 mfma16x16x32(short8 a, short8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16((bf16x8)a, (bf16x8)b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx16 mfma32x32x16(short8 a, short8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16((bf16x8)a, (bf16x8)b, c, 0, 0, 0);
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// The lane's index in its wave from the mbcnt instructions (no input
// registers): for code after a long loop to recompute lane-derived values
// instead of keeping threadIdx-derived ones live across the loop.
__device__ __forceinline__ int lane_fresh() {
  return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Global -> LDS copy of 16 bytes per lane through a buffer resource (offset
// voff + soff): lane l's bytes land at lds_base + 16 l (lds_base wave-uniform).
// Out-of-range offsets write zeros.  Completion is counted by vmcnt.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff, void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds_base, 16, voff, soff, 0,
                                           0);
}

// The same with 4 bytes per lane: lane l's bytes land at lds_base + 4 l.
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff, void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds_base, 4, voff, soff, 0,
                                           0);
}

// s_waitcnt on the vector-memory count only: wait until at most N of this
// wave's vector-memory operations (global -> LDS copies included) are
// outstanding.  gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits
// 15:14, expcnt (bits 6:4) and lgkmcnt (bits 11:8) left at their maxima.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for pipelines fed by global -> LDS copies: waits until at
// most N of this wave's copies are outstanding and all of its LDS accesses
// are done, then s_barrier.  (__syncthreads would also wait for the copies
// still in flight for later stages.)  The asm statement keeps the compiler
// from moving memory accesses across the barrier.
template <int N>
__device__ __forceinline__ void copy_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
  asm volatile("s_barrier" ::: "memory");
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// LDS reads issued as inline assembly: the compiler does not see them as LDS
// accesses, so it neither waits for outstanding global -> LDS copies before
// them nor for their results; the caller waits (s_waitcnt lgkmcnt) before the
// first use, in an asm statement that takes the destinations as operands.
template <int OFF>
__device__ __forceinline__ void ds_read_tr_b64_asm(short4v& d, uint32_t addr) {
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(d) : "v"(addr), "i"(OFF));
}
template <int OFF>
__device__ __forceinline__ void ds_read_b128_asm(short8& d, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(d) : "v"(addr), "i"(OFF));
}

// 4-byte load through a buffer resource; out-of-range offsets read as zero.
__device__ __forceinline__ float buf_load4f(__amdgpu_buffer_rsrc_t rs, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, byte_off, 0, 0));
}

// 8-byte load through a buffer resource (byte_off a multiple of 8).
__device__ __forceinline__ uint2 buf_load8(__amdgpu_buffer_rsrc_t rs, uint32_t byte_off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, byte_off, 0, 0);
  return uint2{(uint32_t)v[0], (uint32_t)v[1]};
}

// 1-byte load through a buffer resource; out-of-range offsets read as zero.
__device__ __forceinline__ uint32_t buf_load_u8(__amdgpu_buffer_rsrc_t rs, uint32_t byte_off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rs, byte_off, 0, 0);
}

// Dropout on an operand fragment: element e of the 8 bf16 values in v is kept
// when bit e of `bits` is set and zeroed otherwise.
__device__ __forceinline__ short8 keep_mask8(short8 v, uint32_t bits) {
  int4v w = __builtin_bit_cast(int4v, v);
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const uint32_t lo = 0u - ((bits >> (2 * h)) & 1u), hi = 0u - ((bits >> (2 * h + 1)) & 1u);
    w[h] &= (int)((lo & 0xFFFFu) | (hi << 16));
  }
  return __builtin_bit_cast(short8, w);
}

__device__ __forceinline__ u16 f32_to_bf16(float f) {  // round to nearest even (v_cvt_pk_bf16_f32)
  return __builtin_bit_cast(u16, (__bf16)f);
}
__device__ __forceinline__ float bf16_to_f32(u16 h) {
  return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// ---- k-contiguous LDS tiles (rows of 128 bytes) ----------------------------
__device__ __forceinline__ int kc_swz(int row) { return (row >> 1) & 7; }

__device__ __forceinline__ uint32_t kc_offset(int row, int chunk) {
  return (uint32_t)(row * 128 + ((chunk ^ kc_swz(row)) << 4));
}

__device__ __forceinline__ short8 kc_read(const char* tile, int row, int chunk) {
  return *reinterpret_cast<const short8*>(tile + kc_offset(row, chunk));
}

// ---- mn-contiguous LDS tiles (rows of COLS bf16, COLS >= 128) --------------
__device__ __forceinline__ int mc16_swz(int row) { return 2 * (row & 3) + 8 * ((row >> 3) & 1); }
__device__ __forceinline__ int mc32_swz(int row) { return 4 * (row & 3); }

template <int COLS>
__device__ __forceinline__ uint32_t mc16_offset(int row, int chunk) {
  return (uint32_t)(row * (COLS * 2) + ((chunk ^ mc16_swz(row)) << 4));
}
template <int COLS>
__device__ __forceinline__ uint32_t mc32_offset(int row, int chunk) {
  return (uint32_t)(row * (COLS * 2) + ((chunk ^ mc32_swz(row)) << 4));
}

__device__ __forceinline__ short8 join4(short4v lo, short4v hi) {
  return short8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// 16x16x32 operand (16 columns x 32 k) from an mn-contiguous tile whose rows
// are k: lane (g = l/16, c = l%16) receives column col0 + c, k rows
// krow0 + 8g .. 8g+7.
template <int COLS>
__device__ __forceinline__ short8 mc16_read_tr(const char* tile, int krow0, int col0, int lane) {
  const int g = lane >> 4, j = lane & 15;
  const int e = j >> 2, q = j & 3;            // this lane addresses row e of 4, 4-column piece q
  const int col = col0 + 4 * q;
  const int r0 = krow0 + 8 * g + e;
  const char* p0 = tile + mc16_offset<COLS>(r0, col >> 3) + (col & 7) * 2;
  const char* p1 = tile + mc16_offset<COLS>(r0 + 4, col >> 3) + (col & 7) * 2;
  return join4(__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p0),
               __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p1));
}

// 32x32x16 operand (32 columns x 16 k) from an mn-contiguous tile whose rows
// are k: lane (g = l/32, c = l%32) receives column col0 + c, k rows
// krow0 + 8g .. 8g+7.  Lanes 16h .. 16h+15 of each half-wave cover columns
// col0 + 16(h%2) .. +15.
template <int COLS>
__device__ __forceinline__ short8 mc32_read_tr(const char* tile, int krow0, int col0, int lane) {
  const int g = lane >> 5, h = (lane >> 4) & 1, j = lane & 15;
  const int e = j >> 2, q = j & 3;
  const int col = col0 + 16 * h + 4 * q;
  const int r0 = krow0 + 8 * g + e;
  const char* p0 = tile + mc32_offset<COLS>(r0, col >> 3) + (col & 7) * 2;
  const char* p1 = tile + mc32_offset<COLS>(r0 + 4, col >> 3) + (col & 7) * 2;
  return join4(__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p0),
               __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)p1));
}

// Output block store.  A wave holds a 32 x 64 block of fp32 outputs in the
// v_mfma_f32_32x32x16 result layout (v0: columns 0..31, v1: columns 32..63;
// lane (g, c) holds row c, columns 8 (q / 4) + 4 g + q % 4).  Stored directly,
// every store instruction would touch 32 rows with 16 bytes each.  Instead
// the block goes through a wave-private LDS region of 32 rows of 64 bf16
// (kYsPitch bytes per row, conflict-free for both access patterns) and is
// written back with 16 bytes per lane, 8 whole 128-byte row segments per
// store.  dst points at the block's (row 0, column 0), ld is the row pitch in
// elements; rows >= nrows and columns >= ncols (a multiple of 8) are not
// written.  The caller provides kYsBytes of LDS that no other wave touches
// meanwhile; the fences order this wave's accesses to it.
constexpr int kYsPitch = 144, kYsBytes = 32 * kYsPitch;

__device__ __forceinline__ void store_block_32x64(const floatx16& v0, const floatx16& v1, char* ys, u16* dst,
                                                  size_t ld, int nrows, int ncols, int lane) {
  const int g = lane >> 5, c = lane & 31;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");   // earlier reads of the region
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const floatx16& a = h ? v1 : v0;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const uint32_t lo = (uint32_t)f32_to_bf16(a[4 * qq]) | ((uint32_t)f32_to_bf16(a[4 * qq + 1]) << 16);
      const uint32_t hi = (uint32_t)f32_to_bf16(a[4 * qq + 2]) | ((uint32_t)f32_to_bf16(a[4 * qq + 3]) << 16);
      *reinterpret_cast<uint2*>(ys + c * kYsPitch + (32 * h + 8 * qq + 4 * g) * 2) = uint2{lo, hi};
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  const int ch = lane & 7, r8 = lane >> 3;
  int4v v[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) v[p] = *reinterpret_cast<const int4v*>(ys + (8 * p + r8) * kYsPitch + ch * 16);
  if (8 * ch < ncols) {
#pragma unroll
    for (int p = 0; p < 4; ++p)
      if (8 * p + r8 < nrows) *reinterpret_cast<int4v*>(dst + (size_t)(8 * p + r8) * ld + 8 * ch) = v[p];
  }
}

// Tile workgroup index -> tile coordinates.  Workgroups are dealt to the 8
// XCDs round robin (block b runs on XCD b % 8); the first step renumbers blocks so each
// XCD receives a contiguous range of tile ids, the second walks tiles in
// groups of `group` tile-rows so neighbours share operand panels in that XCD's L2.
__device__ __forceinline__ void tile_coords(int tiles_m, int tiles_n, int group, int b, int& tm, int& tn) {
  const int nb = tiles_m * tiles_n;  // b: this workgroup's index among the tile workgroups
  const int xcd = b & 7, idx = b >> 3;
  const int per = nb >> 3, rem = nb & 7;
  const int lid = (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
  const int gsize = group * tiles_n;
  const int gi = lid / gsize;
  const int first_m = gi * group;
  const int gm = min(tiles_m - first_m, group);
  const int in = lid - gi * gsize;
  tm = first_m + in % gm;
  tn = in / gm;
}

}  // namespace lora
