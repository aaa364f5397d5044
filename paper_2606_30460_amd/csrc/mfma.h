// CDNA4 (gfx950) matrix-core helpers shared by the attention kernels.
//
// v_mfma_f32_32x32x16_bf16 computes C[32x32] += A[32x16] * B[16x32] for one
// 64-lane wave, fp32 accumulation.  Lane l (l32 = l % 32, hi = l / 32):
//   A operand: row l32 of A, eight consecutive k values of half `hi`;
//   B operand: column l32 of B, eight k values of half `hi` (same k order
//              as A, so any fixed permutation of k applied to both operands
//              leaves the product unchanged);
//   C/D:       column l32 of C, rows 8*(j/4) + 4*hi + (j%4) in register j.
#pragma once

#include <hip/hip_runtime.h>

namespace hsap {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef _Float16 h16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row index (within a 32-row C block) held by register j of a lane in half hi.
__device__ __forceinline__ constexpr int c_row(int j, int hi) { return 8 * (j >> 2) + 4 * hi + (j & 3); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bf16x8 cat4(const bf16x4& a, const bf16x4& b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// v_permlane32_swap with both operands x: lane l < 32 receives (x[l], x[l+32]),
// lane l >= 32 receives (x[l-32], x[l]).  So the pair holds x[l] and x[l ^ 32]
// in every lane, without an LDS round trip.
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane j supplies the LDS
// address of four consecutive 16-bit values c_j[0..3]; lane i receives
// c_{i/4 + 4k}[i % 4] for k = 0..3.  If lane j points at row (j / 4) of a
// 4-row block, columns 4 * (j % 4) .. +3, lane i gets column i of the four
// rows: a 4 x 16 tile read transposed.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
__device__ __forceinline__ bf16x4 ds_read_tr16(const __bf16* lds_ptr) {
  const s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(lds_ptr));
  return __builtin_bit_cast(bf16x4, r);
}

// Workgroup barrier for LDS producer/consumer hand-offs.  It waits for this
// wave's LDS operations only (lgkmcnt), not for its global loads, stores or
// atomics (vmcnt): prefetches and fire-and-forget atomics stay in flight
// across the barrier.  Must only order LDS traffic.  The asm's memory
// clobber keeps the compiler from moving memory operations across it.
__device__ __forceinline__ void hsap_lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N of this wave's vector-memory operations are in flight (they complete in
// issue order) and all its LDS operations are done, then the workgroup barrier.  Used by the
// direct-to-LDS rings: the transfers a step may leave in flight are its own, the youngest.
template <int N>
__device__ __forceinline__ void vm_wait_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt is a six-bit count");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// Unpadded LDS tiles of CPR 16-byte chunks per row (CPR = 16: 128 bf16 per
// row; CPR = 8: 64 bf16) store chunk c of row r at chunk c ^ f(r).  f is
// chosen so that both access patterns of the attention kernels hit 16
// distinct 16-byte bank slots:
//   row reads (ds_read_b128): 16 consecutive rows, one chunk;
//   transpose reads (ds_read_b64_tr_b16, 32 lanes): 4 aligned rows x an
//   aligned group of 4 chunks;
// and a row's chunks remain a permutation of themselves.
template <int CPR>
__device__ __forceinline__ int swz_chunk(int r, int c) {
  static_assert(CPR == 16 || CPR == 8, "swizzle defined for 64- and 128-wide rows");
  if constexpr (CPR == 16) return c ^ (4 * (r & 3) + ((r >> 2) & 3));
  else return c ^ (4 * ((r >> 1) & 1) + ((r >> 2) & 3));
}
// element offset of (row r, column e) in such a tile; e % 8 is kept within the chunk
template <int CPR>
__device__ __forceinline__ int swz(int r, int e) {
  return r * (CPR * 8) + swz_chunk<CPR>(r, e >> 3) * 8 + (e & 7);
}

}  // namespace hsap
