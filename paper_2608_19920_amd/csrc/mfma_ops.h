// Operand types and LDS helpers of the bf16 matrix-core kernels (gfx950).
//
// v_mfma_f32_16x16x32_bf16, C = A B + C with A 16x32, B 32x16, C 16x16:
//   A: lane l holds row l%16, k = 8*(l/16) .. +7   (8 bf16)
//   B: lane l holds column l%16, the same k        (8 bf16)
//   C: lane l holds rows 4*(l/16) .. +3 of column l%16 (4 float)
// Two 16-row C blocks (rows 4g..4g+3 and 16+4g..16+4g+3 in lane group g)
// therefore form one B (or A) operand of a following product over those 32
// indices, with k-index 8g+u <-> index 4g+u (u < 4) and 16+4g+u-4 (u >= 4).
#pragma once

#include "internal.h"

namespace h2o {
namespace mfma {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ s16x4 lds_read_tr16(const bf16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)((__attribute__((address_space(3))) bf16_t*)(p)));
}

// Operand with k running down the 32 rows of a row-major [32][pitch] LDS
// tile: lane i of group g receives tile[4g + u][16*cb + i] (u = 0..3) and
// tile[16 + 4g + u][16*cb + i], i.e. column 16*cb + i of the tile as the
// A (or B) operand's row, in the k order of a C-block pair (header comment).
// ds_read_b64_tr_b16 hands lane i of a 16-lane group element i%4 of the
// 8-byte chunks addressed by lanes 4u + i/4, u = 0..3; lane 4u + c therefore
// addresses row 4g + u, columns 16*cb + 4c .. +3.
__device__ __forceinline__ bf16x8 tr_operand(const bf16_t* tile, int pitch, int cb, int lane) {
  const int g = lane >> 4, i = lane & 15;
  const bf16_t* base = tile + (4 * g + (i >> 2)) * pitch + 16 * cb + 4 * (i & 3);
  const s16x4 lo = lds_read_tr16(base);
  const s16x4 hi = lds_read_tr16(base + 16 * pitch);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Operand with k along a row: row `row` of a row-major LDS tile, elements
// k0 + 8*(lane/16) .. +7 (one 16-byte read).
__device__ __forceinline__ bf16x8 row_operand(const bf16_t* tile, int pitch, int row, int k0,
                                              int lane) {
  return *reinterpret_cast<const bf16x8*>(tile + row * pitch + k0 + 8 * (lane >> 4));
}

// The pair of C blocks (c0: indices 4g.., c1: 16+4g..) as one bf16 operand.
__device__ __forceinline__ bf16x8 pack_pair(const f32x4& c0, const f32x4& c1) {
  bf16x8 r;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    r[u] = (__bf16)c0[u];
    r[4 + u] = (__bf16)c1[u];
  }
  return r;
}

}  // namespace mfma
}  // namespace h2o
