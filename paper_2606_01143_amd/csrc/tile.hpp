// LDS tile layouts and gfx950 matrix-core fragments shared by the bf16
// kernels.
//
// v_mfma_f32_32x32x16_bf16 operand layout (lane l, r = l % 32, h = l / 32):
//   A (32 x 16): element j of lane l is A[r][8 h + j]
//   B (16 x 32): element j of lane l is B[8 h + j][r]
//   C (32 x 32): element i of lane l is C[8 (i / 4) + 4 h + i % 4][r]
// The contraction only needs A and B to agree on which k each (h, j) slot
// holds.
//
// Tiles are 64 rows x d columns and live in LDS in two forms:
//
// natural [64][d + 8], rows PERMUTED: LDS row m holds tile row perm16(m),
//   which swaps bits 2 and 3 of the row index (an involution inside every
//   16-row block).  Used as the A operand of products that contract over d
//   (S = Q K^T, S^T = K Q^T, ...).  With the permutation, element i of a C
//   result in lane (r, h) belongs to tile row 16 (i / 8) + 8 h + i % 8, so
//   C elements 8 u .. 8 u + 7 of a 32-row block are eight CONSECUTIVE rows
//   16 u + 8 h + 0..7: exactly the B/A slots (h, j) = row 16 u + 8 h + j of
//   a 16-row k-step when those rows are contracted next (P^T dO, dS^T Q,
//   V^T P^T, K^T dS^T).  The 8-element pad keeps the 16-byte row reads of
//   eight lanes on distinct banks.
// transposed [d][64] in 16-byte chunks of 8 rows: chunk c of column d sits
//   at chunk position c ^ trn_swz(d), trn_swz(d) = (d % 8) ^ (d / 8 % 8).
//   A k-step fragment (8 consecutive rows of one column) is one 16-byte
//   read; eight lanes reading eight consecutive columns hit eight distinct
//   positions, and the staging writes (columns 8 apart) spread likewise.
//
// Each staging thread holds 4 consecutive rows x 8 columns (four 16-byte
// global loads; 16 lanes cover a row of d = 128), writes them to the natural
// tile at the permuted rows and to the transposed tile as eight 4-row
// half-chunks.
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

// v_exp_f32: 2^x without the denormal-range fix-up of exp2f; softmax weights
// below 2^-126 are flushed to zero, far below bf16 resolution.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// tile row held by LDS row m of a natural tile (and vice versa)
__device__ __forceinline__ int perm16(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

// tile row of C element i in lane half h, within a 32-row block whose A
// operand came from a natural (permuted) tile
__device__ __forceinline__ int c_row(int i, int h) { return 16 * (i >> 3) + 8 * h + (i & 7); }

__device__ __forceinline__ int trn_swz(int d) { return (d & 7) ^ ((d >> 3) & 7); }

template <int D>
struct TileGeom {
  static constexpr int NST = D + 8;                      // natural row stride (elements)
  static constexpr int NAT = kTileRows * NST;            // natural tile elements
  static constexpr int TRN = D * kTileRows;              // transposed tile elements
  static constexpr int CPR = D / 8;                      // 16-byte chunks per row
  static constexpr int STAGERS = kTileRows * CPR / 4;    // threads that stage a tile
};

// C elements 8u .. 8u+7 of a 32x32 result, rounded to bf16: rows 16 u + 8 h
// + 0..7 of the block as the (h, j) slots of the next product's k-step.
__device__ __forceinline__ bf16x8 c_to_kfrag(const f32x16& c, int u) {
  return bf16x8{(bf16)c[8 * u + 0], (bf16)c[8 * u + 1], (bf16)c[8 * u + 2], (bf16)c[8 * u + 3],
                (bf16)c[8 * u + 4], (bf16)c[8 * u + 5], (bf16)c[8 * u + 6], (bf16)c[8 * u + 7]};
}

// Element offset of the A-operand read of LDS row `row`, columns
// col0 + 8 h .. + 7 of a natural tile.
template <int D>
__device__ __forceinline__ int nat_off(int row, int col0, int h) {
  return row * TileGeom<D>::NST + col0 + 8 * h;
}

// Element offset of rows 16 u + 8 h .. + 7 of column d of a transposed tile.
__device__ __forceinline__ int trn_off(int d, int u, int h) {
  return d * kTileRows + 8 * ((2 * u + h) ^ trn_swz(d));
}

__device__ __forceinline__ bf16x8 lds8(const bf16* base, int off) {
  return *(const bf16x8*)(base + off);
}

// Keeps the compiler from moving memory operations across this point: the
// next tile's LDS stores must stay after the current tile's products so the
// wait on their global loads does not precede the matrix work.
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Staging of one 64-row tile: rows row0 .. row0 + 63 of a token-major
// [rows, H, D] tensor, head hh; rows >= nvalid are zero.  A thread's four
// rows are four named registers of 32-bit words (two bf16 per word): the
// transposed store builds its 4-row columns with byte selects (v_perm_b32)
// instead of element extraction, which keeps everything in VGPRs.
template <int D>
struct Stager {
  u32x4 v0, v1, v2, v3;

  __device__ __forceinline__ void load(const bf16* base, int row0, int nvalid, int H, int hh,
                                       int tid) {
    constexpr int CPR = TileGeom<D>::CPR;
    if (tid < TileGeom<D>::STAGERS) {
      const int c16 = tid % CPR, rg = tid / CPR;
      const bf16* p = base + ((size_t)(row0 + 4 * rg) * H + hh) * D + 8 * c16;
      const size_t rs = (size_t)H * D;
      const u32x4 z = {0u, 0u, 0u, 0u};
      if (nvalid >= kTileRows) {  // full tile: no per-row checks
        v0 = *(const u32x4*)(p);
        v1 = *(const u32x4*)(p + rs);
        v2 = *(const u32x4*)(p + 2 * rs);
        v3 = *(const u32x4*)(p + 3 * rs);
      } else {
        const int rr = 4 * rg;
        v0 = rr + 0 < nvalid ? *(const u32x4*)(p) : z;
        v1 = rr + 1 < nvalid ? *(const u32x4*)(p + rs) : z;
        v2 = rr + 2 < nvalid ? *(const u32x4*)(p + 2 * rs) : z;
        v3 = rr + 3 < nvalid ? *(const u32x4*)(p + 3 * rs) : z;
      }
    }
  }

  __device__ __forceinline__ void store_nat(bf16* nat, int tid) const {
    constexpr int CPR = TileGeom<D>::CPR, NST = TileGeom<D>::NST;
    if (tid < TileGeom<D>::STAGERS) {
      const int c16 = tid % CPR, rg = tid / CPR;
      // rows 4 rg + i live at LDS rows perm16(4 rg + i) = perm16(4 rg) + i
      bf16* p = nat + perm16(4 * rg) * NST + 8 * c16;
      *(u32x4*)(p) = v0;
      *(u32x4*)(p + NST) = v1;
      *(u32x4*)(p + 2 * NST) = v2;
      *(u32x4*)(p + 3 * NST) = v3;
    }
  }

  __device__ __forceinline__ void store_trn(bf16* trn, int tid) const {
    constexpr int CPR = TileGeom<D>::CPR;
    if (tid < TileGeom<D>::STAGERS) {
      const int c16 = tid % CPR, rg = tid / CPR;
      // rows 4 rg .. 4 rg + 3 are half (rg & 1) of the 8-row chunk rg / 2;
      // word w of a row holds columns 2 w (low half) and 2 w + 1 (high half)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const unsigned lo01 = __builtin_amdgcn_perm(v1[w], v0[w], 0x05040100u);
        const unsigned lo23 = __builtin_amdgcn_perm(v3[w], v2[w], 0x05040100u);
        const unsigned hi01 = __builtin_amdgcn_perm(v1[w], v0[w], 0x07060302u);
        const unsigned hi23 = __builtin_amdgcn_perm(v3[w], v2[w], 0x07060302u);
        const int d0 = 8 * c16 + 2 * w, d1 = d0 + 1;
        *(u32x2*)(trn + d0 * kTileRows + 8 * ((rg >> 1) ^ trn_swz(d0)) + 4 * (rg & 1)) =
            u32x2{lo01, lo23};
        *(u32x2*)(trn + d1 * kTileRows + 8 * ((rg >> 1) ^ trn_swz(d1)) + 4 * (rg & 1)) =
            u32x2{hi01, hi23};
      }
    }
  }
};

}  // namespace spr
