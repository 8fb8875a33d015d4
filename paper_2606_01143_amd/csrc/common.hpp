// Shared definitions for the gfx950 kernels of libspr.
//
// Every kernel works on one "virtual sequence" [P || S(s)] per suffix s: the
// prefix segment (rows/keys 0..P-1 of the *_p buffers) followed by suffix s
// (rows cu[s]..cu[s+1]-1 of the packed *_s buffers).  Keys are never copied
// into a concatenated buffer; each tile reads from whichever segment it
// belongs to.  Tiles never straddle the two segments: the tile grid of the
// prefix covers [0, P) and the tile grid of each suffix restarts at its first
// token, so every tile is either all-prefix or all-one-suffix.
//
// Visibility (causal, inclusive): prefix row r sees prefix keys j <= r;
// suffix row t of s sees every prefix key and suffix keys j <= t of s.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spr {

typedef __bf16 bf16;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// All arguments of one attention launch.  Unused fields are null/zero.
struct AttnArgs {
  // prefix segment: rows and keys 0..P-1
  const void* q_p;
  const void* k_p;
  const void* v_p;
  void* o_p;
  float* lse_p;        // [P, Hq]
  const void* do_p;    // upstream adjoint of the prefix rows (bwd)
  float* dd_p;         // rowsum(dO * O) [P, Hq] (bwd)
  float* lse2_p;       // LSE * log2(e) [P, Hq] (bf16 bwd)
  float* dq_acc_p;     // fp32 dQ accumulator [P, Hq, d] (bwd)
  // suffix segment: packed rows, suffix s = rows cu[s] .. cu[s+1]-1
  const void* q_s;
  const void* k_s;
  const void* v_s;
  void* o_s;
  float* lse_s;        // [total_len, Hq]
  const void* do_s;
  float* dd_s;         // [total_len, Hq]
  float* lse2_s;       // [total_len, Hq]
  float* dq_acc_s;     // [total_len, Hq, d]
  // bf16 backward: dQ is written once, scaled, in the storage dtype; the
  // dense baseline accumulates the prefix rows' dQ over the trajectories in
  // dq_acc_p (unscaled) instead
  void* dq_p;
  void* dq_s;
  int32_t dq_p_accumulate;
  // bf16 backward, atomic dQ: the key-outer blocks add the unscaled dS K of
  // their keys into dq_acc_p (prefix rows) / dq_acc_s (suffix rows), fp32
  // accumulators the caller zeroes first and converts afterwards; the launch
  // then has no query-outer role
  int32_t dq_atomic;
  const int32_t* cu;   // device cu_seqlens
  int32_t P;
  int32_t total_len;
  int32_t hq;
  int32_t hkv;
  float scale;         // softmax scale
  float scale_log2;    // softmax scale * log2(e)
  int32_t seq_base;    // first suffix of this launch
  int32_t n_seq;       // suffixes in this launch
  // query-outer launches (forward, fp32 dQ): grid.x = prefix row tiles then
  // suffix row tiles of suffix seq_base + blockIdx.z
  int32_t n_prefix_q_tiles;
  // bf16 forward and backward over suffix rows only may split each row
  // tile's keys into n_split contiguous ranges.  Forward: split j writes its
  // normalized partial output part_o[j][row][h][:] (fp32) and partial
  // log2-domain LSE part_lse[j][row][h]; backward: split j writes its
  // unscaled partial dQ part_dq[j][row][h][:] (fp32).  A combine kernel
  // merges the splits in index order afterwards.
  int32_t n_split;
  float* part_o;
  float* part_lse;
  float* part_dq;
  int32_t n_suffix_q_tiles;
  // key-outer launches (backward): grid.x = prefix key tiles, then
  // n_seq * n_suffix_k_tiles suffix key tiles
  int32_t n_prefix_k_tiles;
  int32_t n_suffix_k_tiles;
  int32_t prefix_rows;   // prefix-key tiles also take the prefix rows (causal)
  int32_t suffix_rows;   // prefix-key tiles take the suffix rows of suffixes
                         // seq_base .. seq_base+n_seq-1 (all visible)
  int32_t pk_mode;       // prefix-key epilogue: 0 => gk/gv += fp32 gradient;
                         // 1 => dk_p/dv_p = gradient + gk/gv in storage dtype
  // bf16 backward launches with few key tiles may cut each key tile's row
  // sweep into kv_rsplit contiguous shares.  Share j writes its scaled fp32
  // partial dK/dV to part_dk/part_dv[j][key row][Hkv][d], where the key row
  // is the prefix key, or P + the packed row of a suffix key; a combine
  // kernel then sums the shares in index order and applies the epilogue.
  int32_t kv_rsplit;
  float* part_dk;
  float* part_dv;
  float* gk;             // [P, Hkv, d] fp32
  float* gv;
  void* dk_p;
  void* dv_p;
  void* dk_s;
  void* dv_s;
};

enum PkMode { kPkAccumulate = 0, kPkInject = 1 };

__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }

template <typename T>
__device__ __forceinline__ float to_f32(T x);
template <>
__device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f32<bf16>(bf16 x) { return (float)x; }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// First row and row count of packed suffix s: cu[s] .. cu[s+1]-1, clamped
// into [0, total_len] with a non-negative count.  Offsets that break the
// documented contract then give wrong rows but never an access outside the
// caller's buffers.
struct SegRows {
  int base, len;
};
__device__ __forceinline__ SegRows suffix_rows(const int32_t* cu, int s, int total_len) {
  const int lo = min(max(cu[s], 0), total_len);
  const int hi = min(max(cu[s + 1], lo), total_len);
  return {lo, hi - lo};
}
// The rows of suffixes s0 .. s1-1 together, clamped the same way.
__device__ __forceinline__ SegRows suffix_span(const int32_t* cu, int s0, int s1, int total_len) {
  const int lo = min(max(cu[s0], 0), total_len);
  const int hi = min(max(cu[s1], lo), total_len);
  return {lo, hi - lo};
}

}  // namespace spr
