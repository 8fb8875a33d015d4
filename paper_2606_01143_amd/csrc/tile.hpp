// LDS tiles and gfx950 matrix-core fragments shared by the bf16 kernels.
//
// v_mfma_f32_32x32x16_bf16 operand layout (lane l, r = l % 32, h = l / 32):
//   A (32 x 16): slot j of lane l holds A[r][k(h, j)]
//   B (16 x 32): slot j of lane l holds B[k(h, j)][r]
//   C (32 x 32): element i of lane l holds C[8 (i / 4) + 4 h + i % 4][r]
// A and B only have to agree on which k each slot (h, j) stands for.  Two
// k orders are used:
//   natural    k(h, j) = 8 h + j, for products that contract over the head
//              dimension d: the operand is 16 contiguous bytes of one tile
//              row (one ds_read_b128) or of a register-resident row;
//   C-order    k(h, j) = 4 h + j (j < 4), 8 + 4 h + j - 4 (j >= 4), for
//              products that contract over rows of a previous C result
//              (P V, dS K, P^T dO, dS^T Q): then the slots of a 16-row
//              k-step v are exactly C elements 8 v .. 8 v + 7, so the
//              probabilities never leave the registers; the other operand
//              is read transposed from its row-major tile with two
//              ds_read_b64_tr_b16 (rows 4 h .. 4 h + 3 and 8 + 4 h ..).
//
// Tiles: 64 rows x D bf16, row-major, filled straight from global memory by
// global_load_lds_dwordx4 (no VGPR staging).  One load instruction writes
// 1 KB contiguously (lane l -> bytes 16 l), so the layout is chosen on the
// global side: 16-byte chunk c of row m is stored at chunk position
// c ^ swz(m).  swz makes both access kinds conflict-free on the 64 banks:
//   ds_read_b128 of an A/B row operand: 16 lanes read 16 rows at one chunk;
//   ds_read_b64_tr_b16: 16 lanes read 4 consecutive rows x 32 bytes.
// Rows of a partial tile repeat the last valid row: the values stay finite
// and the kernels mask what they must.
#pragma once

#include "common.hpp"

namespace spr {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4_t;

constexpr int kTileRows = 64;
constexpr int kThreads = 256;  // 4 waves per workgroup in every bf16 kernel

template <int D>
struct Tile {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int ELEMS = kTileRows * D;      // bf16 elements per tile
  static constexpr int RPI = 64 / CH;              // rows per 1 KB load instruction
};

template <int D>
__device__ __forceinline__ int swz(int row);
template <>
__device__ __forceinline__ int swz<128>(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }
template <>
__device__ __forceinline__ int swz<64>(int row) { return (((row >> 1) & 1) << 2) | ((row >> 2) & 3); }

// element offset of (row, col) in a swizzled tile
template <int D>
__device__ __forceinline__ int toff(int row, int col) {
  return row * D + ((((col >> 3) ^ swz<D>(row))) << 3) + (col & 7);
}

// wave index inside the workgroup, in a scalar register (wave-uniform)
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  return f32x16{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
}

// v_exp_f32: 2^x without the denormal fix-up of exp2f; softmax weights below
// 2^-126 flush to zero, far below bf16 resolution.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Scheduling templates for a run of n products fed by LDS reads (r reads
// per product): the first `ahead` reads are issued before any product, then
// each product is followed by the reads of a later one, so the read latency
// hides behind the matrix work instead of stalling every product.
template <int N, int R, int AHEAD>
__device__ __forceinline__ void sched_reads_ahead() {
  __builtin_amdgcn_sched_group_barrier(0x100, AHEAD * R, 0);
#pragma unroll
  for (int k = 0; k < N - AHEAD; ++k) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, AHEAD, 0);
}

// Keeps the compiler from moving memory operations across this point (the
// next tile's loads must be issued before the current tile's products).
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// Waits for this wave's direct-to-LDS loads, then for every wave.
__device__ __forceinline__ void tile_barrier() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
}

// Registers loaded from global memory before a tile loop pass through here
// once the loads are issued.  The compiler then waits for those loads at
// this point, before the loop.  Otherwise its waits stay at their first use
// inside the loop, and since it does not count the untracked direct-to-LDS
// loads, they would also wait, every iteration, for the next tile's loads.
template <typename T>
__device__ __forceinline__ void settle(T& x) {
  asm volatile("" : "+v"(x));
}

// A kernel-argument pointer held in scalar registers from here on.  Without
// it the compiler turns "c ? a.x : a.y" inside a loop into a load of the
// selected argument slot on every iteration, each a scalar-memory round
// trip the wave waits for.
template <typename T>
__device__ __forceinline__ T* in_sgpr(T* p) {
  asm volatile("" : "+s"(p));
  return p;
}
// c ? x : y on two uniform pointers, as a register select (the same folding
// would otherwise select between the addresses the two values live at)
template <typename T>
__device__ __forceinline__ T* pick(bool c, T* x, T* y) {
  asm volatile("" : "+s"(x), "+s"(y));
  return c ? x : y;
}

// Direct-to-LDS loads: lane l's 16 (or 4) bytes at gptr land at LDS byte
// address lds + 16 l (4 l).  They are issued through inline assembly so that
// the compiler does not track them: it would otherwise wait for every such
// load before any later LDS read it cannot prove disjoint from the
// destination, including reads of the other buffer of a multi-buffered
// tile, which defeats loading one tile ahead.  Every caller waits for its
// own loads (vmcnt) and then for the workgroup before reading the data
// (tile_barrier).  M0 takes the LDS address one wait state before the load.
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const lds_void_t*)p;
}
__device__ __forceinline__ void dma_lds16(const void* gptr, unsigned lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void dma_lds4(const void* gptr, unsigned lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(gptr), "s"(lds)
               : "memory", "m0");
}
// The same with a scalar base address and a 32-bit per-lane byte offset:
// no per-lane 64-bit address arithmetic at the call site.
__device__ __forceinline__ void dma_lds16_s(unsigned voff, const void* sbase, unsigned lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void dma_lds4_s(unsigned voff, const void* sbase, unsigned lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

// Loads ROWS-row tiles of token-major [rows, H, D] tensors (one head) into
// swizzled LDS tiles, this wave's share of the 1 KB instructions out of NW
// loading waves.  The per-lane byte offsets within a tile depend only on
// the lane, the wave and H, so they are computed once; a tile then costs a
// scalar base address and one instruction per KB.  Rows at or past nvalid
// (ragged end, nvalid >= 1) repeat the last valid row.
template <int D, int NW, int ROWS>
struct TileLoader {
  static constexpr int CH = D / 8;      // 16-byte chunks per row
  static constexpr int RPI = 64 / CH;   // rows per instruction
  static constexpr int IPW = ROWS / RPI / NW;
  static_assert(IPW * RPI * NW == ROWS, "loading waves must split the tile evenly");
  unsigned off[IPW];
  int lrow0, lane_row;  // first tile row of this wave's share, lane's row within an instruction
  __device__ __forceinline__ void init(int H, int w, int lane) {
    lrow0 = w * IPW * RPI;
    lane_row = lane / CH;
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int lrow = lrow0 + i * RPI + lane_row;
      const int c = (lane % CH) ^ swz<D>(lrow);
      off[i] = ((unsigned)lrow * H * D + 8 * c) * 2;
    }
  }
  __device__ __forceinline__ void load(bf16* tile, const bf16* base, int row0, int nvalid, int H,
                                       int hh) const {
    const bf16* sb = base + ((size_t)row0 * H + hh) * D;
    if (nvalid >= ROWS) {
#pragma unroll
      for (int i = 0; i < IPW; ++i) dma_lds16_s(off[i], sb, lds_addr(tile + (lrow0 + i * RPI) * D));
    } else {
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const int lrow = lrow0 + i * RPI + lane_row;
        const unsigned back = (unsigned)(lrow - min(lrow, nvalid - 1)) * H * D * 2;
        dma_lds16_s(off[i] - back, sb, lds_addr(tile + (lrow0 + i * RPI) * D));
      }
    }
  }
};

// 64 fp32 values v[(row0 + i) * stride] (i < 64; rows at or past nvalid
// repeat the last valid one) into LDS, by one wave, offsets precomputed.
struct RowVecLoader {
  unsigned off;
  int lane;
  __device__ __forceinline__ void init(int stride, int lane_) {
    lane = lane_;
    off = (unsigned)lane * stride * 4;
  }
  __device__ __forceinline__ void load(float* dst, const float* src, int row0, int nvalid, int stride) const {
    const float* sb = src + (size_t)row0 * stride;
    const unsigned o = nvalid >= 64 ? off : (unsigned)min(lane, nvalid - 1) * stride * 4;
    dma_lds4_s(o, sb, lds_addr(dst));
  }
};

// Rows row0 .. row0 + ROWS - 1 of a token-major [rows, H, D] tensor, head
// hh, into a swizzled LDS tile; rows at or past row0 + nvalid (nvalid >= 1)
// repeat row row0 + nvalid - 1.  Called by NW waves (w = index among them,
// < NW), each issuing an equal share of the 1 KB load instructions.
template <int D, int NW = 4, int ROWS = kTileRows>
__device__ __forceinline__ void load_tile(bf16* tile, const bf16* base, int row0, int nvalid,
                                          int H, int hh, int w, int lane) {
  constexpr int CH = Tile<D>::CH, RPI = Tile<D>::RPI;
  constexpr int IPW = ROWS / RPI / NW;
  static_assert(IPW * RPI * NW == ROWS, "loading waves must split the tile evenly");
  const int last = row0 + nvalid - 1;
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int lrow0 = (w * IPW + i) * RPI;
    const int lrow = lrow0 + lane / CH;
    const int c = (lane % CH) ^ swz<D>(lrow);
    const int grow = min(row0 + lrow, last);
    dma_lds16(base + ((size_t)grow * H + hh) * D + 8 * c, lds_addr(tile + lrow0 * D));
  }
}

// 64 fp32 row values v[(row0 + i) * stride] (i < 64; rows past nvalid repeat
// the last valid one) into LDS, by one wave.
__device__ __forceinline__ void load_row_vec(float* dst, const float* src, int row0, int nvalid,
                                             int stride, int lane) {
  const int row = min(row0 + lane, row0 + nvalid - 1);
  dma_lds4(src + (size_t)row * stride, lds_addr(dst));
}

// Per-lane LDS offsets of the operand reads.  swz depends only on the low
// four bits of the row, so moving a read by a multiple of 16 rows adds
// 16 m D to its offset: the kernels precompute the lane-dependent part once
// and add row offsets as compile-time constants, which the hardware takes as
// the instruction's immediate offset.
template <int D>
struct FragOffsets {
  int row[D / 16];    // natural-k read of row r, cols 16 k + 8 h .. + 7
  int trlo[D / 32];   // transposed read, rows 4 h .. 4 h + 3, col 32 db + r
  int trhi[D / 32];   // rows 8 + 4 h .. 8 + 4 h + 3
  __device__ __forceinline__ void init(int lane) {
    const int r = lane & 31, h = lane >> 5, i16 = lane & 15;
#pragma unroll
    for (int k = 0; k < D / 16; ++k) row[k] = toff<D>(r, 16 * k + 8 * h);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int col = 32 * db + (lane & 16) + 4 * (i16 & 3);
      trlo[db] = toff<D>(4 * h + (i16 >> 2), col);
      trhi[db] = toff<D>(8 + 4 * h + (i16 >> 2), col);
    }
  }
};

// natural-k operand: tile row row0 + r (row0 a multiple of 16), columns
// 16 k + 8 h .. + 7
template <int D>
__device__ __forceinline__ bf16x8 row_frag(const bf16* tile, const FragOffsets<D>& fo, int row0, int k) {
  return *(const bf16x8*)(tile + row0 * D + fo.row[k]);
}

// C-order operand read transposed from a row-major tile: slot (h, j) of lane
// (r, h) holds tile[base + k(h, j)][32 db + r] (base a multiple of 16).
template <int D>
__device__ __forceinline__ bf16x8 tr_frag(const bf16* tile, const FragOffsets<D>& fo, int base, int db) {
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(tile + base * D + fo.trlo[db]));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(tile + base * D + fo.trhi[db]));
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// C-order operand from registers: elements 8 v .. 8 v + 7 of a C result,
// i.e. its rows 16 v + k(h, j), rounded to bf16.
__device__ __forceinline__ bf16x8 c_kfrag(const f32x16& c, int v) {
  return bf16x8{(bf16)c[8 * v + 0], (bf16)c[8 * v + 1], (bf16)c[8 * v + 2], (bf16)c[8 * v + 3],
                (bf16)c[8 * v + 4], (bf16)c[8 * v + 5], (bf16)c[8 * v + 6], (bf16)c[8 * v + 7]};
}

// row of C element i in lane half h (within a 32-row block) is c_row0(i) + 4 h
__device__ __forceinline__ constexpr int c_row0(int i) { return 8 * (i >> 2) + (i & 3); }

}  // namespace spr
