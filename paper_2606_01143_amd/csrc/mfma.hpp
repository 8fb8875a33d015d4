// gfx950 matrix-core and LDS-transpose primitives used by the bf16 kernels.
//
// v_mfma_f32_16x16x32_bf16 operand layout (lane l, c = l % 16, g = l / 16):
//   A (16 x 32): element j of lane l is A[c][8g + j]
//   B (32 x 16): element j of lane l is B[8g + j][c]
//   C (16 x 16): element i of lane l is C[4g + i][c]
// The contraction only needs A and B to agree on which k each (g, j) slot
// holds, so the kernels may assign any permutation of k to the slots as long
// as both operands use it.
//
// ds_read_b64_tr_b16 (LDS transpose read), per group of 16 lanes: if lane
// i of the group points at M[r0 + i / 4][c0 + 4 * (i % 4)] of a row-major
// 16-bit matrix M, lane c of the group receives M[r0 + 0..3][c0 + c].  That
// is the column access an MFMA operand needs when the contraction index runs
// along M's rows, so every LDS tile can stay in its natural row-major layout.
#pragma once

#include "common.hpp"

namespace spr {

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Four 16-bit values of column (c0 + lane%16) from rows r0 .. r0+3 of the
// row-major LDS tile `tile` (row stride `stride` elements).  r0 and c0 may
// differ between the four 16-lane groups.
__device__ __forceinline__ bf16x4 lds_col4(const bf16* tile, int stride, int r0, int c0, int c) {
  const bf16* p = tile + (r0 + (c >> 2)) * stride + c0 + 4 * (c & 3);
  s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
  return __builtin_bit_cast(bf16x4, v);
}

__device__ __forceinline__ bf16x8 join(const bf16x4& lo, const bf16x4& hi) {
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

__device__ __forceinline__ bf16x8 pack8(const f32x4& lo, const f32x4& hi) {
  return bf16x8{f2bf(lo[0]), f2bf(lo[1]), f2bf(lo[2]), f2bf(lo[3]),
                f2bf(hi[0]), f2bf(hi[1]), f2bf(hi[2]), f2bf(hi[3])};
}

__device__ __forceinline__ bf16x8 zero8() {
  const bf16 z = f2bf(0.f);
  return bf16x8{z, z, z, z, z, z, z, z};
}

}  // namespace spr
