// LDS tile layouts and gfx950 matrix-core fragments shared by the bf16
// kernels.
//
// v_mfma_f32_32x32x16_bf16 operand layout (lane l, r = l % 32, h = l / 32):
//   A (32 x 16): element j of lane l is A[r][8 h + j]
//   B (16 x 32): element j of lane l is B[8 h + j][r]
//   C (32 x 32): element i of lane l is C[8 (i / 4) + 4 h + i % 4][r]
// The contraction only needs A and B to agree on which k each (h, j) slot
// holds.  When the k index of a product is the row index of a C result
// (P^T dO, dS^T Q, V^T P^T, K^T dS^T), the kernels take a 16-row k-step u of
// a 32-row block straight from C elements 8 u .. 8 u + 7, so slot (h, j)
// holds row 16 u + 4 h + j (j < 4) or 16 u + 8 + 4 h + j - 4 (j >= 4).
//
// A row tile of 64 rows x d columns is staged through LDS twice:
//   natural    [64][d + 8]: the 16-byte row reads of A operands hit distinct
//              banks thanks to the 8-element pad;
//   transposed [d][64]: column access for the products that contract over
//              rows.  Rows are kept in 8-byte chunks of 4; chunk c of column
//              d is stored at chunk position c ^ sw(d), sw(d) = (d % 16) ^
//              (d / 16).  Both the staging writes (16 lanes = 16 columns
//              8 apart, one chunk) and the fragment reads (16 consecutive
//              columns, one chunk) then hit 16 distinct chunk slots, i.e.
//              every bank once.
// Each staging thread holds 4 consecutive rows x 8 columns (four 16-byte
// global loads, one full row per 16 lanes), writes them to the natural tile
// as-is and to the transposed tile as eight 4-row columns.
#pragma once

#include "common.hpp"

namespace spr {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kTileRows = 64;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  return f32x16{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
}

__device__ __forceinline__ bf16x8 zero_bf8() {
  const bf16 z = (bf16)0.f;
  return bf16x8{z, z, z, z, z, z, z, z};
}

__device__ __forceinline__ int tr_swz(int d) { return (d & 15) ^ ((d >> 4) & 15); }

template <int D>
struct TileGeom {
  static constexpr int NST = D + 8;                      // natural row stride (elements)
  static constexpr int NAT = kTileRows * NST;            // natural tile elements
  static constexpr int TRN = D * kTileRows;              // transposed tile elements
  static constexpr int CPR = D / 8;                      // 16-byte chunks per row
  static constexpr int STAGERS = kTileRows * CPR / 4;    // threads that stage a tile
};

// C elements 8u .. 8u+7 of a 32x32 result, rounded to bf16: the (h, j) slots
// of k-step u when the result's row index is contracted next.
__device__ __forceinline__ bf16x8 c_to_kfrag(const f32x16& c, int u) {
  return bf16x8{(bf16)c[8 * u + 0], (bf16)c[8 * u + 1], (bf16)c[8 * u + 2], (bf16)c[8 * u + 3],
                (bf16)c[8 * u + 4], (bf16)c[8 * u + 5], (bf16)c[8 * u + 6], (bf16)c[8 * u + 7]};
}

// 16 contiguous bytes of a natural-tile row: A operand slot (h, j) = column
// col0 + 8 h + j of row `row`.
template <int D>
__device__ __forceinline__ bf16x8 nat_frag(const bf16* nat, int row, int col0, int h) {
  return *(const bf16x8*)(nat + row * TileGeom<D>::NST + col0 + 8 * h);
}

// Column d of the transposed tile, rows 4 c_lo .. +3 then 4 c_hi .. +3.
__device__ __forceinline__ bf16x8 trn_frag(const bf16* trn, int d, int c_lo, int c_hi) {
  const int s = tr_swz(d);
  const bf16x4 lo = *(const bf16x4*)(trn + d * kTileRows + ((c_lo ^ s) << 2));
  const bf16x4 hi = *(const bf16x4*)(trn + d * kTileRows + ((c_hi ^ s) << 2));
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// Staging of one 64-row tile: rows row0 .. row0 + 63 of a token-major
// [rows, H, D] tensor, head hh; rows >= nvalid are zero.
template <int D>
struct Stager {
  bf16x8 v[4];

  __device__ __forceinline__ void load(const bf16* base, int row0, int nvalid, int H, int hh,
                                       int tid) {
    constexpr int CPR = TileGeom<D>::CPR;
    if (tid < TileGeom<D>::STAGERS) {
      const int c16 = tid % CPR, rg = tid / CPR;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * rg + i;
        v[i] = r < nvalid ? *(const bf16x8*)(base + ((size_t)(row0 + r) * H + hh) * D + 8 * c16)
                          : zero_bf8();
      }
    }
  }

  __device__ __forceinline__ void store_nat(bf16* nat, int tid) const {
    constexpr int CPR = TileGeom<D>::CPR;
    if (tid < TileGeom<D>::STAGERS) {
      const int c16 = tid % CPR, rg = tid / CPR;
#pragma unroll
      for (int i = 0; i < 4; ++i) *(bf16x8*)(nat + (4 * rg + i) * TileGeom<D>::NST + 8 * c16) = v[i];
    }
  }

  __device__ __forceinline__ void store_trn(bf16* trn, int tid) const {
    constexpr int CPR = TileGeom<D>::CPR;
    if (tid < TileGeom<D>::STAGERS) {
      const int c16 = tid % CPR, rg = tid / CPR;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int d = 8 * c16 + j;
        const bf16x4 col = {v[0][j], v[1][j], v[2][j], v[3][j]};
        *(bf16x4*)(trn + d * kTileRows + ((rg ^ tr_swz(d)) << 2)) = col;
      }
    }
  }
};

}  // namespace spr
