// Host-side launchers of the gfx950 kernels and the per-kernel event timer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.hpp"

namespace spr {

// --- per-kernel timing (enabled through spr_profile_enable) -------------
bool profile_enabled(const char* kernel);
void profile_record(const char* kernel, hipEvent_t begin, hipEvent_t end);
hipEvent_t profile_event();  // from a pool owned by the profiler

// Brackets one kernel launch with two events on `stream` while profiling
// is enabled; a no-op otherwise.
class ProfileScope {
 public:
  ProfileScope(const char* kernel, hipStream_t stream) : kernel_(kernel), stream_(stream) {
    if (profile_enabled(kernel)) {
      begin_ = profile_event();
      end_ = profile_event();
      if (begin_ && end_) hipEventRecord(begin_, stream_);
    }
  }
  ~ProfileScope() {
    if (begin_ && end_) {
      hipEventRecord(end_, stream_);
      profile_record(kernel_, begin_, end_);
    }
  }
  ProfileScope(const ProfileScope&) = delete;
  ProfileScope& operator=(const ProfileScope&) = delete;

 private:
  const char* kernel_;
  hipStream_t stream_;
  hipEvent_t begin_ = nullptr;
  hipEvent_t end_ = nullptr;
};

// --- fp32 storage path (kernels_f32.hip) --------------------------------
hipError_t launch_fwd_f32(const AttnArgs& a, int head_dim, int n_z, hipStream_t st);
hipError_t launch_bwd_f32(const AttnArgs& a, int head_dim, int n_qz, hipStream_t st);

// --- bf16 storage path, MFMA (kernels_bf16_fwd.hip, kernels_bf16_bwd.hip) --
hipError_t launch_fwd_bf16(const AttnArgs& a, int head_dim, int n_z, hipStream_t st);
hipError_t launch_fwd_bf16_wide(const AttnArgs& a, int head_dim, int n_z, hipStream_t st);
int fwd_bf16_wide_block_q();
hipError_t launch_bwd_bf16(const AttnArgs& a, int head_dim, int n_qz, bool deterministic,
                           hipStream_t st);
// Row-tile sizes the launchers expect in AttnArgs (q tiles / k tiles).
int fwd_bf16_block_q();
// key splits of the bf16 suffix forward for n_row_blocks (row tile, q head,
// suffix) blocks and a prefix of prefix_len keys
int fwd_bf16_split(int n_row_blocks, int prefix_len);
int bwd_bf16_block_k();
// key-outer role alone with six wave pairs (192 keys) per workgroup, one
// workgroup per CU, for the prefix backward of long prefixes (default mode)
hipError_t launch_bwd_bf16_kv_wide(const AttnArgs& a, int head_dim, hipStream_t st);
int bwd_bf16_kv_wide_block_k();
int bwd_bf16_kv_wide_slots();
// key splits of the bf16 suffix backward's query-outer role for
// n_row_blocks (row tile, q head, suffix) blocks that each sweep
// n_key_tiles key tiles
int bwd_bf16_qsplit(int n_row_blocks, int n_key_tiles);
int bwd_bf16_kvsplit(long kv_tiles, long max_tiles, bool kv_alone, int slots = 512);
int bwd_bf16_block_q();
int f32_block_q();
int f32_block_k();

// --- auxiliary kernels (kernels_aux.hip) ----------------------------------
// dd[row * hq + h] = sum_d dO[row,h,d] * O[row,h,d] and
// lse2[row * hq + h] = lse[row * hq + h] * log2(e) for rows [0, rows), or,
// when cu != nullptr, for the rows cu[seq] .. cu[seq+1]-1 of one packed
// suffix (rows then bounds their count, total_rows is the buffers' row
// count the offsets are clamped to); dO == nullptr gives dd = 0.
hipError_t launch_row_dot(int dtype, const void* dO, const void* O, int rows, int total_rows,
                          const int32_t* cu, int seq, int hq, int head_dim, float* dd,
                          const float* lse, float* lse2, hipStream_t st);
hipError_t launch_fill_zero(float* p, size_t n, hipStream_t st);
// out = acc * scale (+ add when add != nullptr), converted to `dtype`
hipError_t launch_convert(int dtype, const float* acc, float scale, const float* add,
                          void* out, size_t n, hipStream_t st);
// dst += src
hipError_t launch_accumulate(float* dst, const float* src, size_t n, hipStream_t st);
// padded suffix layout: cu/lens_c from device lengths, and row gather
// (padded -> packed) or scatter (packed -> padded, padding rows zeroed)
hipError_t launch_seq_offsets(const int32_t* lens, int n, int s_max, int32_t* cu, int32_t* lens_c,
                              hipStream_t st);
constexpr int kMaxRowMoves = 6;
struct RowMove {
  const void* src;
  void* dst;
  size_t row_bytes;  // a multiple of 4
};
// few suffixes: the move kernels derive the offsets from `lens` themselves;
// many: cu / lens_c must come from launch_seq_offsets first
bool rows_move_needs_offsets(int n);
hipError_t launch_rows_move(bool gather, const RowMove* moves, int count, const int32_t* lens,
                            const int32_t* cu, const int32_t* lens_c, int n, int s_max, hipStream_t st);

// decoder-layer token-wise operations (kernels_layer.hip)
hipError_t launch_rmsnorm_fwd(int rows, int width, float eps, const void* x, void* y, float* rstd,
                              hipStream_t st);
hipError_t launch_rmsnorm_bwd(int rows, int width, const void* x, const float* rstd, const void* dy,
                              const void* add, void* dx, hipStream_t st);
hipError_t launch_rope(int tokens, int heads, int d, int pos0, double theta, const void* x, void* y,
                       bool inverse, hipStream_t st);
hipError_t launch_swiglu_fwd(long n, const void* g, const void* u, void* m, hipStream_t st);
hipError_t launch_swiglu_bwd(long n, const void* g, const void* u, const void* dm, void* dg, void* du,
                             hipStream_t st);

// MoE router aux-loss accounting (kernels_moe.hip).  Statistics layout:
// int64 count[E], double mass[E], int64 total, int64 invalid.
int moe_blocks(int n_tokens);
size_t moe_workspace_bytes(int E, int n_tokens);
hipError_t launch_moe_accumulate(const float* p, const int* r, int n, int E, int k, int mult,
                                 const int* mu, void* stats, void* ws, hipStream_t st);
hipError_t launch_moe_loss(const void* stats, int E, int k, double coef, double* f, double* pe,
                           double* loss, hipStream_t st);
hipError_t launch_moe_grad(const void* stats, int E, int k, double scale, int n, int mult,
                           const int* mu, float* dp, hipStream_t st);

}  // namespace spr
