// Device helpers shared by the attention kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ut {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// D = A(32x16) * B(16x32) + C. Lane l holds A[l%32][8(l/32)+e], B[8(l/32)+e][l%32]
// (e = 0..7) and C[8(i/4) + 4(l/32) + i%4][l%32] (i = 0..15).
__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// D = A(16x32) * B(32x16) + C. Lane l holds A[l%16][8(l/16)+e],
// B[8(l/16)+e][l%16] (e = 0..7) and C[4(l/16) + i][l%16] (i = 0..3).
// At equal FLOPs this shape draws less power than the 32x32x16 one: under the
// board's power limit it sustains a higher clock on random operands.
__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Transposing LDS read: in each 16-lane group, lanes 4r..4r+3 address row r
// (four consecutive 16-bit elements each); lane j receives element j of the
// 16-element rows r = 0..3.
__device__ inline s16x4 lds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
}

// Value of lane l ^ 32 combined with this lane's (both halves get the result).
__device__ inline float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Combined over the four 16-lane groups (lanes l, l^16, l^32, l^48).
__device__ inline float quad_max(float x) {
  x = pair_max(x);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float quad_sum(float x) {
  x = pair_sum(x);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Two floats rounded to bf16 (nearest even) and packed, a in the low half.
__device__ inline unsigned pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(unsigned, v);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS byte offset of logical 16-byte chunk c of row r in a tile of CPR chunks
// per row. The XOR swizzle makes both access patterns conflict-free: 32-row
// b128 reads of one chunk (the swizzle is injective over 16 consecutive rows)
// and transposing 8-byte reads of 4 consecutive rows x 4 chunks (those rows
// differ in the swizzle's upper two bits).
template <int CPR>
__device__ inline int lds_off(int r, int c) {
  static_assert(CPR == 16 || CPR == 8, "rows of 128 or 64 bf16");
  const int sw = CPR == 16 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((r >> 1) & 7);
  return r * CPR * 16 + ((c ^ sw) << 4);
}

// LDS byte offset of logical 16-byte chunk c of row r for the 16x16x32
// kernels. Their two access patterns are b128 reads of one chunk over 16
// consecutive rows (one per 16-lane group) and transposing 8-byte reads of
// rows 4g..4g+3 (lane group g) over two adjacent chunks, where a half-wave
// covers 8 rows. The swizzle is a permutation over any 16 consecutive rows
// (first pattern) whose value >> 1 differs between the 8 rows of either half
// (second pattern), so neither pattern has bank conflicts.
template <int CPR>
__device__ inline int swz_off(int r, int c) {
  static_assert(CPR == 16 || CPR == 8, "rows of 128 or 64 bf16");
  const int sw = CPR == 16 ? (((r & 7) << 1) | ((r >> 3) & 1))
                           : ((((r >> 1) & 3) << 1) | ((r >> 3) & 1));
  return r * CPR * 16 + ((c ^ sw) << 4);
}

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor, 32-bit data format

// A raw buffer descriptor over `bytes` bytes from `base`; loads past the range
// read zeros.
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kRsrcWord3);
}

// One 16-byte-per-lane buffer load straight into LDS: lane L writes at
// lds + 16 L (lds must be wave-uniform).
__device__ inline void buffer_load_lds16(__amdgpu_buffer_rsrc_t rs, char* lds, int voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16,
                                           voffset, 0, 0, 0);
}

// Where sample b's rows live. Uniform batch (cu == nullptr): tokens
// [b N, b N + N) of the packed [B N, H, D] tensors, per-row statistics (LSE
// and its relatives) laid out [B, H, N]. Variable lengths: tokens
// [cu[b], cu[b + 1]) and statistics laid out [H, T] over all T tokens.
struct SampleRows {
  int64_t tok0;    // first token of the sample
  int n;           // its length
  int64_t stat0;   // index of (head h, the sample's first token) in the statistics
};
// Offsets are clamped to [0, T] and lengths to N_all (the block grid's
// extent), so no offsets can send an access outside the tensors.
__device__ inline SampleRows sample_rows(const int32_t* __restrict__ cu, int64_t T, int b, int h,
                                         int H, int N_all) {
  if (cu) {
    const int64_t t0 = min(max((int64_t)cu[b], (int64_t)0), T);
    const int64_t t1 = min(max((int64_t)cu[b + 1], t0), T);
    return SampleRows{t0, (int)min(t1 - t0, (int64_t)N_all), (int64_t)h * T + t0};
  }
  return SampleRows{(int64_t)b * N_all, N_all, ((int64_t)b * H + h) * N_all};
}

}  // namespace ut
