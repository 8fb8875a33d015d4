// C ABI of libspr: argument validation, workspace layout and dispatch of the
// three-phase schedule (paper Sec. 3.2) and the dense-recompute baseline.
//
// Nothing is launched unless every check passes.  The library keeps no state
// between calls except the optional event profiler.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/spr.h"
#include "../../include/spr_moe.h"
#include "../../include/spr_layer.h"
#include "common.hpp"
#include "launch.hpp"

namespace spr {

namespace {

thread_local std::string g_last_error;

spr_status fail(spr_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

spr_status ok() {
  g_last_error.clear();
  return SPR_OK;
}

size_t dtype_bytes(int dtype) { return dtype == SPR_F32 ? 4 : 2; }

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int tiles(int n, int b) { return n <= 0 ? 0 : (n + b - 1) / b; }

// ------------------------------------------------------------ validation
spr_status check_dims(const spr_dims* d) {
  if (d == nullptr) return fail(SPR_ERR_INVALID_ARG, "dims is null");
  if (d->num_q_heads < 1 || d->num_kv_heads < 1)
    return fail(SPR_ERR_INVALID_ARG, "num_q_heads and num_kv_heads must be >= 1");
  if (d->num_q_heads % d->num_kv_heads != 0)
    return fail(SPR_ERR_INVALID_ARG, "num_q_heads must be a multiple of num_kv_heads");
  if (d->prefix_len < 0) return fail(SPR_ERR_INVALID_ARG, "prefix_len must be >= 0");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SPR_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (d->dtype != SPR_F32 && d->dtype != SPR_BF16)
    return fail(SPR_ERR_UNSUPPORTED, "dtype must be SPR_F32 or SPR_BF16");
  if ((d->flags & ~(uint32_t)(SPR_DETERMINISTIC | SPR_ATOMIC_DQ)) != 0)
    return fail(SPR_ERR_UNSUPPORTED, "unknown flag bits");
  if ((d->flags & SPR_DETERMINISTIC) && (d->flags & SPR_ATOMIC_DQ))
    return fail(SPR_ERR_INVALID_ARG, "SPR_ATOMIC_DQ contradicts SPR_DETERMINISTIC");
  if (!(d->softmax_scale >= 0.f) || isinf(d->softmax_scale))
    return fail(SPR_ERR_INVALID_ARG, "softmax_scale must be finite and >= 0");
  return SPR_OK;
}

spr_status check_padded_sizes(int32_t n, int32_t s_max) {
  if (n < 1) return fail(SPR_ERR_INVALID_ARG, "number of suffixes must be >= 1");
  if (s_max < 1) return fail(SPR_ERR_INVALID_ARG, "s_max must be >= 1");
  if ((int64_t)n * s_max > INT32_MAX) return fail(SPR_ERR_INVALID_ARG, "n * s_max exceeds 2^31 - 1");
  return SPR_OK;
}

spr_status check_suffix_sizes(int32_t n, int32_t max_len, int32_t total_len) {
  if (n < 1) return fail(SPR_ERR_INVALID_ARG, "number of suffixes must be >= 1");
  if (max_len < 1) return fail(SPR_ERR_INVALID_ARG, "max_len must be >= 1");
  if (total_len < n || total_len < max_len)
    return fail(SPR_ERR_INVALID_ARG, "total_len must be >= n and >= max_len");
  if ((int64_t)n * max_len < total_len)
    return fail(SPR_ERR_INVALID_ARG, "total_len exceeds n * max_len");
  return SPR_OK;
}

struct Buf {
  const void* p;
  size_t bytes;
  const char* name;
  bool required;
  uintptr_t align = 16;  // LSE and cu_seqlens are read as 4-byte scalars
};

spr_status check_bufs(const std::vector<Buf>& bufs) {
  for (const Buf& b : bufs) {
    if (b.bytes == 0) continue;
    if (b.p == nullptr) {
      if (b.required) return fail(SPR_ERR_INVALID_ARG, std::string(b.name) + " is null");
      continue;
    }
    if (((uintptr_t)b.p & (b.align - 1)) != 0)
      return fail(SPR_ERR_MISALIGNED,
                  std::string(b.name) + " is not " + std::to_string(b.align) + "-byte aligned");
  }
  return SPR_OK;
}

bool overlaps(const Buf& a, const Buf& b) {
  if (a.p == nullptr || b.p == nullptr || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.bytes;
  const uintptr_t b0 = (uintptr_t)b.p, b1 = b0 + b.bytes;
  return a0 < b1 && b0 < a1;
}

// every buffer in `inout` must overlap nothing else in `all`
spr_status check_aliasing(const std::vector<Buf>& inout, const std::vector<Buf>& all) {
  for (const Buf& x : inout)
    for (const Buf& y : all) {
      if (x.p == y.p && x.name == y.name) continue;
      if (overlaps(x, y))
        return fail(SPR_ERR_ALIASING, std::string(x.name) + " overlaps " + y.name);
    }
  return SPR_OK;
}

spr_status hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess)
    return fail(SPR_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return SPR_OK;
}

float eff_scale(const spr_dims* d) {
  return d->softmax_scale > 0.f ? d->softmax_scale : 1.0f / sqrtf((float)d->head_dim);
}

AttnArgs base_args(const spr_dims* d) {
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.P = d->prefix_len;
  a.hq = d->num_q_heads;
  a.hkv = d->num_kv_heads;
  a.scale = eff_scale(d);
  a.scale_log2 = a.scale * kLog2e;
  a.n_split = 1;
  a.kv_rsplit = 1;
  return a;
}

// key splits of the suffix forward (bf16 path only), see fwd_bf16_split
int suffix_fwd_splits(const spr_dims* d, int32_t n_mb, int32_t max_len) {
  if (d->dtype != SPR_BF16) return 1;
  const int nrb = tiles(max_len, fwd_bf16_block_q()) * d->num_q_heads * n_mb;
  return fwd_bf16_split(nrb, d->prefix_len);
}

bool atomic_dq(const spr_dims* d);

// key splits of the suffix backward's query-outer role (bf16 path only),
// see bwd_bf16_qsplit
int suffix_bwd_splits(const spr_dims* d, int32_t n_mb, int32_t max_len) {
  if (d->dtype != SPR_BF16 || atomic_dq(d)) return 1;
  const int nrb = tiles(max_len, bwd_bf16_block_q()) * d->num_q_heads * n_mb;
  const int nkt = tiles(d->prefix_len, bwd_bf16_block_k()) + tiles(max_len, bwd_bf16_block_k());
  return bwd_bf16_qsplit(nrb, nkt);
}

// row shares of the backward's key-outer role (bf16 path only), see
// bwd_bf16_kvsplit.  Work is counted in (32-row tile, q head) steps of the
// 64-key tiles, from the sizes alone (so that packed and padded calls of
// the same sizes agree): a causal key range of len keys costs
// g * ceil((len - k0) / 32) steps for the tile at k0.
long causal_steps(long len, long g, long bk = 64) {
  long s = 0;
  for (long k0 = 0; k0 < len; k0 += bk) s += g * ((len - k0 + 31) / 32);
  return s;
}
// dQ of the bf16 backward: by default a query-outer role recomputes S and
// dP for it (7 products per visible pair, no atomics, bitwise
// reproducible); with SPR_ATOMIC_DQ the key-outer blocks add it with fp32
// atomics (5 products per pair, one launch role).
bool atomic_dq(const spr_dims* d) {
  return d->dtype == SPR_BF16 && (d->flags & SPR_ATOMIC_DQ) != 0;
}

int bwd_kv_splits(const spr_dims* d, long kv_steps, long max_steps) {
  if (d->dtype != SPR_BF16) return 1;
  return bwd_bf16_kvsplit(kv_steps * d->num_kv_heads, max_steps, atomic_dq(d));
}
// The forward in its twelve-wave form (96 rows of four q heads per
// workgroup, three waves on every SIMD) for bf16 groups of four q heads per
// kv head (or a multiple), when the launch needs no key splits and its
// workgroups (wide_tiles 96-row tiles over all sequences, per kv head and
// group of four q heads) fill the GPU at least four times.  Measured on the
// prefix forward: from 1368 workgroups (P = 16384, Hkv = 8) 3-5% faster,
// at 688 (P = 8192) 3% slower.
constexpr long kFwdWideMinBlocks = 1024;
bool fwd_wide(const spr_dims* d, long wide_tiles) {
  if (d->dtype != SPR_BF16 || d->num_q_heads % (4 * d->num_kv_heads) != 0) return false;
  const long g4 = d->num_q_heads / d->num_kv_heads / 4;
  return wide_tiles * d->num_kv_heads * g4 >= kFwdWideMinBlocks;
}

// The key-outer-only launch (bf16, default mode): the key-outer role alone,
// six wave pairs (192 keys) per workgroup at three waves per SIMD, then the
// query-outer role in a launch of its own.  It pays when its own work fills
// the GPU several times over: at least kKvWideMinSteps (32-row tile, q head)
// steps of 192-key tiles over all kv heads, 128 per CU.  Below that the two
// roles share one launch, where together they fill it.  (Phase C measured:
// 175 steps per CU and more, 8-15% faster; 87 and fewer, 6-42% slower.)  The
// same rule serves Phase C, the dense baseline's per-trajectory backward and
// the suffix backward (the packed dense baseline's whole trajectories among
// them).
constexpr long kKvWideMinSteps = 32768;
bool kv_wide(const spr_dims* d, long wide_steps) {
  return d->dtype == SPR_BF16 && !atomic_dq(d) && wide_steps * d->num_kv_heads >= kKvWideMinSteps;
}
long wide_bk() { return bwd_bf16_kv_wide_block_k(); }
// Phase C: causal prefix rows
long prefix_wide_steps(const spr_dims* d) {
  return causal_steps(d->prefix_len, d->num_q_heads / d->num_kv_heads, wide_bk());
}
// the dense per-trajectory launch: prefix key tiles see the causal prefix
// rows and the suffix rows, suffix key tiles their own rows
long dense_wide_steps(const spr_dims* d, int32_t max_len) {
  const long g = d->num_q_heads / d->num_kv_heads, sr = g * ((max_len + 31) / 32);
  return causal_steps(d->prefix_len, g, wide_bk()) + (long)tiles(d->prefix_len, (int)wide_bk()) * sr +
         causal_steps(max_len, g, wide_bk());
}
// Phase B: prefix key tiles see every suffix row (at most n_mb * max_len),
// suffix key tiles their own causal rows
long suffix_wide_steps(const spr_dims* d, int32_t n_mb, int32_t max_len) {
  const long g = d->num_q_heads / d->num_kv_heads, rows = (long)n_mb * max_len;
  return (long)tiles(d->prefix_len, (int)wide_bk()) * g * ((rows + 31) / 32) +
         (long)n_mb * causal_steps(max_len, g, wide_bk());
}
bool prefix_kv_wide(const spr_dims* d) { return kv_wide(d, prefix_wide_steps(d)); }
bool dense_kv_wide(const spr_dims* d, int32_t max_len) { return kv_wide(d, dense_wide_steps(d, max_len)); }
// In Phase B the prefix key tiles all sweep every suffix row of the
// microbatch, so their workgroups are equally long; one per CU, they run in
// rounds of 256, and a last round mostly empty costs more than the launch
// gains.  With a prefix the key-outer-only launch is taken only when those
// rounds are at least 85% full (measured: 688 and 1200 tiles, 90% and 94%
// full, 2-11% faster; 88, 172 and 344 tiles, 34-67%, 4-10% slower).
bool suffix_kv_wide(const spr_dims* d, int32_t n_mb, int32_t max_len) {
  if (!kv_wide(d, suffix_wide_steps(d, n_mb, max_len))) return false;
  if (d->prefix_len == 0) return true;
  const long n = (long)tiles(d->prefix_len, (int)wide_bk()) * d->num_kv_heads;
  const long slots = bwd_bf16_kv_wide_slots();
  return n * 100 >= 85 * slots * ((n + slots - 1) / slots);
}
int suffix_bwd_kv_splits(const spr_dims* d, int32_t n_mb, int32_t max_len) {
  const long g = d->num_q_heads / d->num_kv_heads, rows = (long)n_mb * max_len;
  const long max_steps = d->prefix_len > 0 ? g * ((rows + 31) / 32) : g * ((max_len + 31) / 32);
  if (suffix_kv_wide(d, n_mb, max_len))  // wide key tiles, one slot per CU, no query-outer role
    return bwd_bf16_kvsplit(suffix_wide_steps(d, n_mb, max_len) * d->num_kv_heads, max_steps, true,
                            bwd_bf16_kv_wide_slots());
  const long pre = (long)tiles(d->prefix_len, bwd_bf16_block_k()) * g * ((rows + 31) / 32);
  const long kv = pre + (long)n_mb * causal_steps(max_len, g);
  return bwd_kv_splits(d, kv, max_steps);
}
// Phase C: causal prefix rows; key tile 0 sweeps all P
int prefix_bwd_kv_splits(const spr_dims* d) {
  const long g = d->num_q_heads / d->num_kv_heads;
  const long max_steps = g * ((d->prefix_len + 31) / 32);
  if (prefix_kv_wide(d))  // wide key tiles, one slot per CU, no query-outer role
    return bwd_bf16_kvsplit(prefix_wide_steps(d) * d->num_kv_heads, max_steps, true, bwd_bf16_kv_wide_slots());
  return bwd_kv_splits(d, causal_steps(d->prefix_len, g), max_steps);
}
// the dense baseline's per-trajectory launch: prefix key tiles see the
// causal prefix rows and the suffix rows, suffix key tiles their own rows
int dense_bwd_kv_splits(const spr_dims* d, int32_t max_len) {
  const long g = d->num_q_heads / d->num_kv_heads, P = d->prefix_len;
  const long sr = g * ((max_len + 31) / 32);
  if (dense_kv_wide(d, max_len))  // wide key tiles, one slot per CU, no query-outer role
    return bwd_bf16_kvsplit(dense_wide_steps(d, max_len) * d->num_kv_heads, g * ((P + 31) / 32) + sr, true,
                            bwd_bf16_kv_wide_slots());
  const long kv = causal_steps(P, g) + (long)tiles(d->prefix_len, bwd_bf16_block_k()) * sr +
                  causal_steps(max_len, g);
  return bwd_kv_splits(d, kv, g * ((P + 31) / 32) + sr);
}

int block_q(int dtype) { return dtype == SPR_BF16 ? fwd_bf16_block_q() : f32_block_q(); }
int block_k(int dtype) { return dtype == SPR_BF16 ? bwd_bf16_block_k() : f32_block_k(); }

hipError_t launch_fwd(const spr_dims* d, const AttnArgs& a, int n_z, hipStream_t st) {
  return d->dtype == SPR_BF16 ? launch_fwd_bf16(a, d->head_dim, n_z, st)
                              : launch_fwd_f32(a, d->head_dim, n_z, st);
}
// A forward over the prefix rows (prefix) and/or the suffix rows of n_z
// sequences of at most max_len rows: the row tile counts of a follow the
// form fwd_wide picks.
hipError_t launch_forward(const spr_dims* d, AttnArgs a, bool prefix, int32_t max_len, int n_z, hipStream_t st) {
  const int qw = fwd_bf16_wide_block_q();
  const long pw = prefix ? tiles(d->prefix_len, qw) : 0, sw = max_len > 0 ? tiles(max_len, qw) : 0;
  if (a.n_split <= 1 && fwd_wide(d, pw + (long)n_z * sw)) {
    a.n_prefix_q_tiles = (int)pw;
    a.n_suffix_q_tiles = (int)sw;
    return launch_fwd_bf16_wide(a, d->head_dim, n_z, st);
  }
  const int q = block_q(d->dtype);
  a.n_prefix_q_tiles = prefix ? tiles(d->prefix_len, q) : 0;
  a.n_suffix_q_tiles = max_len > 0 ? tiles(max_len, q) : 0;
  return launch_fwd(d, a, n_z, st);
}

hipError_t launch_bwd(const spr_dims* d, const AttnArgs& a, int n_qz, hipStream_t st) {
  return d->dtype == SPR_BF16
             ? launch_bwd_bf16(a, d->head_dim, n_qz, (d->flags & SPR_DETERMINISTIC) != 0, st)
             : launch_bwd_f32(a, d->head_dim, n_qz, st);
}

// ------------------------------------------------------------- workspace
struct WsLayout {
  size_t dd_p = 0, dq_acc_p = 0, dd_s = 0, dq_acc_s = 0, dk_acc_p = 0, dv_acc_p = 0;
  size_t lse2_p = 0, lse2_s = 0;
  size_t part_o = 0, part_lse = 0, part_dq = 0, part_dk = 0, part_dv = 0;
  // padded layout: offsets, clamped lengths, packed copies, inner workspace
  size_t cu = 0, lens_c = 0, pq = 0, pk = 0, pv = 0, po = 0, plse = 0, pdo = 0;
  size_t pdq = 0, pdk = 0, pdv = 0, inner = 0, inner_bytes = 0;
  size_t total = 0;
};

WsLayout ws_layout(int op, const spr_dims* d, int32_t n_mb, int32_t max_len, int32_t total_len) {
  WsLayout w;
  const size_t hq = d->num_q_heads, hkv = d->num_kv_heads, hd = d->head_dim;
  const size_t P = d->prefix_len, T = total_len > 0 ? total_len : 0;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  // the bf16 path writes dQ directly (query-outer kernel); the fp32 path
  // accumulates it in fp32 and converts
  const bool f32 = d->dtype == SPR_F32;
  switch (op) {
    case SPR_OP_PREFIX_FWD:
      break;
    case SPR_OP_SUFFIX_FWD: {
      const size_t ns = suffix_fwd_splits(d, n_mb, max_len);
      if (ns > 1) {
        w.part_o = take(ns * T * hq * hd * 4);
        w.part_lse = take(ns * T * hq * 4);
      }
      break;
    }
    case SPR_OP_SUFFIX_BWD: {
      w.dd_s = take(hq * T * 4);
      w.lse2_s = take(hq * T * 4);
      if (f32 || atomic_dq(d)) w.dq_acc_s = take(T * hq * hd * 4);
      const size_t ns = suffix_bwd_splits(d, n_mb, max_len);
      if (ns > 1) w.part_dq = take(ns * T * hq * hd * 4);
      const size_t rs = suffix_bwd_kv_splits(d, n_mb, max_len);
      if (rs > 1) {
        w.part_dk = take(rs * (P + T) * hkv * hd * 4);
        w.part_dv = take(rs * (P + T) * hkv * hd * 4);
      }
      break;
    }
    case SPR_OP_PREFIX_BWD: {
      w.dd_p = take(hq * P * 4);
      w.lse2_p = take(hq * P * 4);
      if (f32 || atomic_dq(d)) w.dq_acc_p = take(P * hq * hd * 4);
      const size_t rs = prefix_bwd_kv_splits(d);
      if (rs > 1) {
        w.part_dk = take(rs * P * hkv * hd * 4);
        w.part_dv = take(rs * P * hkv * hd * 4);
      }
      break;
    }
    case SPR_OP_SUFFIX_FWD_PADDED:
    case SPR_OP_SUFFIX_BWD_PADDED: {
      // packed copies for the worst case of n_mb full suffixes
      const size_t R = (size_t)(n_mb > 0 ? n_mb : 0) * (size_t)(max_len > 0 ? max_len : 0);
      const size_t eb = dtype_bytes(d->dtype);
      const bool bwd = op == SPR_OP_SUFFIX_BWD_PADDED;
      w.cu = take((size_t)(n_mb + 1) * 4);
      w.lens_c = take((size_t)(n_mb > 0 ? n_mb : 0) * 4);
      w.pq = take(R * hq * hd * eb);
      w.pk = take(R * hkv * hd * eb);
      w.pv = take(R * hkv * hd * eb);
      w.po = take(R * hq * hd * eb);
      w.plse = take(R * hq * 4);
      if (bwd) {
        w.pdo = take(R * hq * hd * eb);
        w.pdq = take(R * hq * hd * eb);
        w.pdk = take(R * hkv * hd * eb);
        w.pdv = take(R * hkv * hd * eb);
      }
      w.inner_bytes = ws_layout(bwd ? SPR_OP_SUFFIX_BWD : SPR_OP_SUFFIX_FWD, d, n_mb, max_len, (int32_t)R).total;
      w.inner = take(w.inner_bytes);
      break;
    }
    case SPR_OP_DENSE_BASELINE:
      w.dd_p = take(hq * P * 4);
      w.lse2_p = take(hq * P * 4);
      w.dq_acc_p = take(P * hq * hd * 4);
      w.dd_s = take(hq * T * 4);
      w.lse2_s = take(hq * T * 4);
      if (f32 || atomic_dq(d)) w.dq_acc_s = take(T * hq * hd * 4);
      w.dk_acc_p = take(P * hkv * hd * 4);
      w.dv_acc_p = take(P * hkv * hd * 4);
      {
        const size_t rs = dense_bwd_kv_splits(d, max_len);
        if (rs > 1) {
          w.part_dk = take(rs * (P + T) * hkv * hd * 4);
          w.part_dv = take(rs * (P + T) * hkv * hd * 4);
        }
      }
      break;
    default:
      break;
  }
  w.total = off;
  return w;
}

spr_status check_ws(const WsLayout& w, const void* ws, size_t ws_bytes) {
  if (w.total == 0) return SPR_OK;
  if (ws == nullptr) return fail(SPR_ERR_WORKSPACE, "workspace is null");
  if (ws_bytes < w.total)
    return fail(SPR_ERR_WORKSPACE, "workspace too small: need " + std::to_string(w.total) +
                                       " bytes, got " + std::to_string(ws_bytes));
  if (((uintptr_t)ws & 15u) != 0) return fail(SPR_ERR_MISALIGNED, "workspace is not 16-byte aligned");
  return SPR_OK;
}

template <typename T>
T* at(void* base, size_t off) {
  return (T*)((char*)base + off);
}

// ---------------------------------------------------------------- profiler
struct ProfRec {
  const char* name;
  hipEvent_t b, e;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::string g_prof_only;  // empty: every kernel
std::vector<ProfRec> g_prof_pending;
std::vector<hipEvent_t> g_prof_pool;
std::map<std::string, std::pair<double, int>> g_prof_totals;
std::vector<std::string> g_prof_names;

void prof_drain_locked() {
  for (const ProfRec& r : g_prof_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.e) == hipSuccess && hipEventElapsedTime(&ms, r.b, r.e) == hipSuccess) {
      auto& t = g_prof_totals[r.name];
      if (t.second == 0 && std::find(g_prof_names.begin(), g_prof_names.end(), r.name) == g_prof_names.end())
        g_prof_names.push_back(r.name);
      t.first += ms;
      t.second += 1;
    }
    g_prof_pool.push_back(r.b);
    g_prof_pool.push_back(r.e);
  }
  g_prof_pending.clear();
}

}  // namespace

bool profile_enabled(const char* kernel) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  return g_prof_on && (g_prof_only.empty() || g_prof_only == kernel);
}

hipEvent_t profile_event() {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void profile_record(const char* kernel, hipEvent_t begin, hipEvent_t end) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_pending.push_back({kernel, begin, end});
}

}  // namespace spr

using namespace spr;

extern "C" {

const char* spr_version(void) { return "spr 0.1.0 (gfx950)"; }

const char* spr_last_error(void) { return g_last_error.c_str(); }

const char* spr_status_string(int32_t s) {
  switch (s) {
    case SPR_OK: return "SPR_OK";
    case SPR_ERR_INVALID_ARG: return "SPR_ERR_INVALID_ARG";
    case SPR_ERR_UNSUPPORTED: return "SPR_ERR_UNSUPPORTED";
    case SPR_ERR_MISALIGNED: return "SPR_ERR_MISALIGNED";
    case SPR_ERR_ALIASING: return "SPR_ERR_ALIASING";
    case SPR_ERR_WORKSPACE: return "SPR_ERR_WORKSPACE";
    case SPR_ERR_HIP: return "SPR_ERR_HIP";
    default: return "SPR_ERR_UNKNOWN";
  }
}

spr_status spr_workspace_size(int32_t op, const spr_dims* dims, int32_t n_mb, int32_t max_len,
                              int32_t total_len, size_t* bytes) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if (bytes == nullptr) return fail(SPR_ERR_INVALID_ARG, "bytes is null");
  if (op < SPR_OP_PREFIX_FWD || op > SPR_OP_SUFFIX_BWD_PADDED)
    return fail(SPR_ERR_INVALID_ARG, "unknown op");
  if (op == SPR_OP_SUFFIX_FWD_PADDED || op == SPR_OP_SUFFIX_BWD_PADDED) {
    if ((st = check_padded_sizes(n_mb, max_len)) != SPR_OK) return st;
  } else if (op != SPR_OP_PREFIX_FWD && op != SPR_OP_PREFIX_BWD) {
    st = check_suffix_sizes(n_mb, max_len, total_len);
    if (st != SPR_OK) return st;
  }
  *bytes = ws_layout(op, dims, n_mb, max_len, total_len).total;
  return ok();
}

spr_status spr_prefix_fwd(const spr_dims* dims, const void* q_p, const void* k_p, const void* v_p,
                          void* o_p, float* lse_p, hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype);
  std::vector<Buf> bufs = {{q_p, P * hq * hd * eb, "q_p", true},
                           {k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {o_p, P * hq * hd * eb, "o_p", true},
                           {lse_p, hq * P * 4, "lse_p", true, 4}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if (P == 0) return ok();
  AttnArgs a = base_args(dims);
  a.q_p = q_p; a.k_p = k_p; a.v_p = v_p; a.o_p = o_p; a.lse_p = lse_p;
  if ((st = hip_check(launch_forward(dims, a, true, 0, 1, stream), "prefix forward")) != SPR_OK) return st;
  return ok();
}

spr_status spr_suffix_attn_fwd(const spr_dims* dims, const void* k_p, const void* v_p,
                               const void* q_s, const void* k_s, const void* v_s,
                               const int32_t* cu_seqlens, int32_t n_mb, int32_t max_len,
                               int32_t total_len, void* o_s, float* lse_s, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if ((st = check_suffix_sizes(n_mb, max_len, total_len)) != SPR_OK) return st;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype), T = total_len;
  std::vector<Buf> bufs = {{k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {q_s, T * hq * hd * eb, "q_s", true},
                           {k_s, T * hkv * hd * eb, "k_s", true},
                           {v_s, T * hkv * hd * eb, "v_s", true},
                           {cu_seqlens, (size_t)(n_mb + 1) * 4, "cu_seqlens", true, 4},
                           {o_s, T * hq * hd * eb, "o_s", true},
                           {lse_s, hq * T * 4, "lse_s", true, 4}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const WsLayout w = ws_layout(SPR_OP_SUFFIX_FWD, dims, n_mb, max_len, total_len);
  if ((st = check_ws(w, ws, ws_bytes)) != SPR_OK) return st;
  AttnArgs a = base_args(dims);
  a.k_p = k_p; a.v_p = v_p;
  a.q_s = q_s; a.k_s = k_s; a.v_s = v_s; a.o_s = o_s; a.lse_s = lse_s;
  a.cu = cu_seqlens;
  a.total_len = total_len;
  a.seq_base = 0;
  a.n_seq = n_mb;
  a.n_split = suffix_fwd_splits(dims, n_mb, max_len);
  if (a.n_split > 1) {
    a.part_o = at<float>(ws, w.part_o);
    a.part_lse = at<float>(ws, w.part_lse);
  }
  if ((st = hip_check(launch_forward(dims, a, false, max_len, n_mb, stream), "suffix forward")) != SPR_OK)
    return st;
  return ok();
}

// ------------------------------------------ static scratch, no allocation
// For callers that cannot allocate device memory (code under graph capture,
// tight serving loops): a file-scope device array serves as the workspace
// of spr_suffix_attn_fwd_noalloc.  Each GPU the library runs on holds its
// own copy for the life of the process.  In host code the array's name is
// not a device address: the address is looked up once per device with
// hipGetSymbolAddress and only that pointer is passed to kernels.
namespace {
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;
}  // namespace
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// the current device's scratch address, looked up on the device's first use
spr_status scratch_of_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPR_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SPR_ERR_UNSUPPORTED, "device index beyond the static scratch table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SPR_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SPR_OK;
}
}  // namespace

spr_status spr_suffix_attn_fwd_noalloc(const spr_dims* dims, const void* k_p, const void* v_p,
                                       const void* q_s, const void* k_s, const void* v_s,
                                       const int32_t* cu_seqlens, int32_t n_mb, int32_t max_len,
                                       int32_t total_len, void* o_s, float* lse_s,
                                       hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if ((st = check_suffix_sizes(n_mb, max_len, total_len)) != SPR_OK) return st;
  const size_t need = ws_layout(SPR_OP_SUFFIX_FWD, dims, n_mb, max_len, total_len).total;
  if (need > kStaticScratchBytes)
    return fail(SPR_ERR_WORKSPACE, "these sizes need " + std::to_string(need) +
                                       " bytes of scratch; the static scratch holds " +
                                       std::to_string(kStaticScratchBytes));
  void* ws = nullptr;
  if ((st = scratch_of_current_device(&ws)) != SPR_OK) return st;
  // every scratch byte the forward reads it first writes in the same call
  return spr_suffix_attn_fwd(dims, k_p, v_p, q_s, k_s, v_s, cu_seqlens, n_mb, max_len, total_len,
                             o_s, lse_s, ws, kStaticScratchBytes, stream);
}

spr_status spr_check_cu_seqlens(const int32_t* cu_host, int32_t n_mb, int32_t max_len,
                                int32_t total_len) {
  if (cu_host == nullptr) return fail(SPR_ERR_INVALID_ARG, "cu_seqlens (host copy) is null");
  spr_status st = check_suffix_sizes(n_mb, max_len, total_len);
  if (st != SPR_OK) return st;
  if (cu_host[0] != 0) return fail(SPR_ERR_INVALID_ARG, "cu_seqlens[0] must be 0");
  int32_t longest = 0;
  for (int32_t s = 0; s < n_mb; ++s) {
    const int64_t len = (int64_t)cu_host[s + 1] - cu_host[s];
    if (len < 1)
      return fail(SPR_ERR_INVALID_ARG, "suffix " + std::to_string(s) + " has length " +
                                           std::to_string(len) + " (every suffix needs >= 1 token)");
    if (len > max_len)
      return fail(SPR_ERR_INVALID_ARG, "suffix " + std::to_string(s) + " is longer than max_len");
    longest = std::max(longest, (int32_t)len);
  }
  if (cu_host[n_mb] != total_len)
    return fail(SPR_ERR_INVALID_ARG, "cu_seqlens[n_mb] must equal total_len");
  if (longest != max_len) return fail(SPR_ERR_INVALID_ARG, "max_len is not the longest suffix");
  return ok();
}

spr_status spr_suffix_attn_bwd_accum(const spr_dims* dims, const void* k_p, const void* v_p,
                                     const void* q_s, const void* k_s, const void* v_s,
                                     const void* o_s, const float* lse_s, const void* do_s,
                                     const int32_t* cu_seqlens, int32_t n_mb, int32_t max_len,
                                     int32_t total_len, void* dq_s, void* dk_s, void* dv_s,
                                     float* gk_cache, float* gv_cache, void* ws, size_t ws_bytes,
                                     hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if ((st = check_suffix_sizes(n_mb, max_len, total_len)) != SPR_OK) return st;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype), T = total_len;
  std::vector<Buf> bufs = {{k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {q_s, T * hq * hd * eb, "q_s", true},
                           {k_s, T * hkv * hd * eb, "k_s", true},
                           {v_s, T * hkv * hd * eb, "v_s", true},
                           {o_s, T * hq * hd * eb, "o_s", true},
                           {lse_s, hq * T * 4, "lse_s", true, 4},
                           {do_s, T * hq * hd * eb, "do_s", true},
                           {cu_seqlens, (size_t)(n_mb + 1) * 4, "cu_seqlens", true, 4},
                           {dq_s, T * hq * hd * eb, "dq_s", true},
                           {dk_s, T * hkv * hd * eb, "dk_s", true},
                           {dv_s, T * hkv * hd * eb, "dv_s", true},
                           {gk_cache, P * hkv * hd * 4, "gk_cache", true},
                           {gv_cache, P * hkv * hd * 4, "gv_cache", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const WsLayout w = ws_layout(SPR_OP_SUFFIX_BWD, dims, n_mb, max_len, total_len);
  if ((st = check_ws(w, ws, ws_bytes)) != SPR_OK) return st;
  std::vector<Buf> all = bufs;
  all.push_back({ws, w.total, "ws", false});
  if ((st = check_aliasing({bufs[12], bufs[13]}, all)) != SPR_OK) return st;

  const bool f32 = dims->dtype == SPR_F32;
  const bool aq = atomic_dq(dims);
  float* dd_s = at<float>(ws, w.dd_s);
  float* lse2_s = at<float>(ws, w.lse2_s);
  float* dq_acc = (f32 || aq) ? at<float>(ws, w.dq_acc_s) : nullptr;
  if ((st = hip_check(launch_row_dot(dims->dtype, do_s, o_s, total_len, total_len, nullptr, 0, (int)hq,
                                     (int)hd, dd_s, lse_s, lse2_s, stream), "row statistic")) != SPR_OK)
    return st;
  if (dq_acc && (st = hip_check(launch_fill_zero(dq_acc, T * hq * hd, stream), "dq clear")) != SPR_OK)
    return st;
  AttnArgs a = base_args(dims);
  a.dq_s = dq_s;
  a.k_p = k_p; a.v_p = v_p;
  a.q_s = q_s; a.k_s = k_s; a.v_s = v_s; a.do_s = do_s;
  a.lse_s = const_cast<float*>(lse_s);
  a.dd_s = dd_s; a.lse2_s = lse2_s; a.dq_acc_s = dq_acc;
  a.cu = cu_seqlens;
  a.total_len = total_len;
  a.seq_base = 0;
  a.n_seq = n_mb;
  a.n_prefix_k_tiles = tiles(dims->prefix_len, block_k(dims->dtype));
  a.n_suffix_k_tiles = tiles(max_len, block_k(dims->dtype));
  a.prefix_rows = 0;
  a.suffix_rows = 1;
  a.pk_mode = kPkAccumulate;
  a.gk = gk_cache; a.gv = gv_cache;
  a.dk_s = dk_s; a.dv_s = dv_s;
  if (aq) {
    a.dq_atomic = 1;  // the key-outer blocks add dQ; no query-outer role
  } else {
    a.n_suffix_q_tiles = tiles(max_len, block_q(dims->dtype));
    a.n_split = suffix_bwd_splits(dims, n_mb, max_len);
    if (a.n_split > 1) a.part_dq = at<float>(ws, w.part_dq);
  }
  a.kv_rsplit = suffix_bwd_kv_splits(dims, n_mb, max_len);
  if (a.kv_rsplit > 1) {
    a.part_dk = at<float>(ws, w.part_dk);
    a.part_dv = at<float>(ws, w.part_dv);
  }
  if (suffix_kv_wide(dims, n_mb, max_len)) {
    // the key-outer role alone on 192-key tiles, then the query-outer role
    // (as Phase C of a long prefix)
    AttnArgs kv = a;
    kv.n_prefix_k_tiles = tiles(dims->prefix_len, bwd_bf16_kv_wide_block_k());
    kv.n_suffix_k_tiles = tiles(max_len, bwd_bf16_kv_wide_block_k());
    kv.n_suffix_q_tiles = 0;
    kv.n_split = 1;
    kv.part_dq = nullptr;
    if ((st = hip_check(launch_bwd_bf16_kv_wide(kv, dims->head_dim, stream), "suffix backward, dK/dV")) != SPR_OK)
      return st;
    AttnArgs q = a;
    q.n_prefix_k_tiles = 0;
    q.n_suffix_k_tiles = 0;
    q.kv_rsplit = 1;
    q.part_dk = q.part_dv = nullptr;
    if ((st = hip_check(launch_bwd(dims, q, n_mb, stream), "suffix backward, dQ")) != SPR_OK) return st;
  } else if ((st = hip_check(launch_bwd(dims, a, n_mb, stream), "suffix backward")) != SPR_OK) {
    return st;
  }
  if (dq_acc && (st = hip_check(launch_convert(dims->dtype, dq_acc, a.scale, nullptr, dq_s,
                                               T * hq * hd, stream), "dq convert")) != SPR_OK)
    return st;
  return ok();
}

// ------------------------------------------------- padded suffix layout
spr_status spr_suffix_attn_fwd_padded(const spr_dims* dims, const void* k_p, const void* v_p,
                                      const void* q_s, const void* k_s, const void* v_s,
                                      const int32_t* seq_lens, int32_t n, int32_t s_max, void* o_s,
                                      float* lse_s, void* ws, size_t ws_bytes, hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if ((st = check_padded_sizes(n, s_max)) != SPR_OK) return st;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype), R = (size_t)n * s_max;
  std::vector<Buf> bufs = {{k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {q_s, R * hq * hd * eb, "q_s", true},
                           {k_s, R * hkv * hd * eb, "k_s", true},
                           {v_s, R * hkv * hd * eb, "v_s", true},
                           {seq_lens, (size_t)n * 4, "seq_lens", true, 4},
                           {o_s, R * hq * hd * eb, "o_s", true},
                           {lse_s, R * hq * 4, "lse_s", true, 4}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const WsLayout w = ws_layout(SPR_OP_SUFFIX_FWD_PADDED, dims, n, s_max, 0);
  if ((st = check_ws(w, ws, ws_bytes)) != SPR_OK) return st;
  std::vector<Buf> all = bufs;
  all.push_back({ws, w.total, "ws", false});
  if ((st = check_aliasing({bufs[6], bufs[7], all.back()}, all)) != SPR_OK) return st;
  int32_t* cu = at<int32_t>(ws, w.cu);
  int32_t* lens_c = at<int32_t>(ws, w.lens_c);
  void *pq = at<char>(ws, w.pq), *pk = at<char>(ws, w.pk), *pv = at<char>(ws, w.pv), *po = at<char>(ws, w.po);
  float* plse = at<float>(ws, w.plse);
  // the offsets in workspace, for the packed calls: written by the gather
  // itself unless there are too many suffixes for it
  if (rows_move_needs_offsets(n) &&
      (st = hip_check(launch_seq_offsets(seq_lens, n, s_max, cu, lens_c, stream), "offsets")) != SPR_OK)
    return st;
  const RowMove in[] = {{q_s, pq, hq * hd * eb}, {k_s, pk, hkv * hd * eb}, {v_s, pv, hkv * hd * eb}};
  if ((st = hip_check(launch_rows_move(true, in, 3, seq_lens, cu, lens_c, n, s_max, stream), "gather")) != SPR_OK) return st;
  if ((st = spr_suffix_attn_fwd(dims, k_p, v_p, pq, pk, pv, cu, n, s_max, (int32_t)R, po, plse,
                                at<char>(ws, w.inner), w.inner_bytes, stream)) != SPR_OK)
    return st;
  const RowMove out[] = {{po, o_s, hq * hd * eb}, {plse, lse_s, hq * 4}};
  if ((st = hip_check(launch_rows_move(false, out, 2, seq_lens, cu, lens_c, n, s_max, stream), "scatter")) != SPR_OK)
    return st;
  return ok();
}

spr_status spr_suffix_attn_bwd_accum_padded(const spr_dims* dims, const void* k_p, const void* v_p,
                                            const void* q_s, const void* k_s, const void* v_s,
                                            const void* o_s, const float* lse_s, const void* do_s,
                                            const int32_t* seq_lens, int32_t n, int32_t s_max,
                                            void* dq_s, void* dk_s, void* dv_s, float* gk_cache,
                                            float* gv_cache, void* ws, size_t ws_bytes,
                                            hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if ((st = check_padded_sizes(n, s_max)) != SPR_OK) return st;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype), R = (size_t)n * s_max;
  std::vector<Buf> bufs = {{k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {q_s, R * hq * hd * eb, "q_s", true},
                           {k_s, R * hkv * hd * eb, "k_s", true},
                           {v_s, R * hkv * hd * eb, "v_s", true},
                           {o_s, R * hq * hd * eb, "o_s", true},
                           {lse_s, R * hq * 4, "lse_s", true, 4},
                           {do_s, R * hq * hd * eb, "do_s", true},
                           {seq_lens, (size_t)n * 4, "seq_lens", true, 4},
                           {dq_s, R * hq * hd * eb, "dq_s", true},
                           {dk_s, R * hkv * hd * eb, "dk_s", true},
                           {dv_s, R * hkv * hd * eb, "dv_s", true},
                           {gk_cache, P * hkv * hd * 4, "gk_cache", true},
                           {gv_cache, P * hkv * hd * 4, "gv_cache", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const WsLayout w = ws_layout(SPR_OP_SUFFIX_BWD_PADDED, dims, n, s_max, 0);
  if ((st = check_ws(w, ws, ws_bytes)) != SPR_OK) return st;
  std::vector<Buf> all = bufs;
  all.push_back({ws, w.total, "ws", false});
  if ((st = check_aliasing({bufs[12], bufs[13], all.back()}, all)) != SPR_OK) return st;
  int32_t* cu = at<int32_t>(ws, w.cu);
  int32_t* lens_c = at<int32_t>(ws, w.lens_c);
  void *pq = at<char>(ws, w.pq), *pk = at<char>(ws, w.pk), *pv = at<char>(ws, w.pv), *po = at<char>(ws, w.po);
  void *pdo = at<char>(ws, w.pdo), *pdq = at<char>(ws, w.pdq), *pdk = at<char>(ws, w.pdk), *pdv = at<char>(ws, w.pdv);
  float* plse = at<float>(ws, w.plse);
  // the offsets in workspace, for the packed calls: written by the gather
  // itself unless there are too many suffixes for it
  if (rows_move_needs_offsets(n) &&
      (st = hip_check(launch_seq_offsets(seq_lens, n, s_max, cu, lens_c, stream), "offsets")) != SPR_OK)
    return st;
  const RowMove in[] = {{q_s, pq, hq * hd * eb}, {k_s, pk, hkv * hd * eb}, {v_s, pv, hkv * hd * eb},
                        {o_s, po, hq * hd * eb},  {lse_s, plse, hq * 4},      {do_s, pdo, hq * hd * eb}};
  if ((st = hip_check(launch_rows_move(true, in, 6, seq_lens, cu, lens_c, n, s_max, stream), "gather")) != SPR_OK) return st;
  if ((st = spr_suffix_attn_bwd_accum(dims, k_p, v_p, pq, pk, pv, po, plse, pdo, cu, n, s_max, (int32_t)R, pdq,
                                      pdk, pdv, gk_cache, gv_cache, at<char>(ws, w.inner), w.inner_bytes,
                                      stream)) != SPR_OK)
    return st;
  const RowMove out[] = {{pdq, dq_s, hq * hd * eb}, {pdk, dk_s, hkv * hd * eb}, {pdv, dv_s, hkv * hd * eb}};
  if ((st = hip_check(launch_rows_move(false, out, 3, seq_lens, cu, lens_c, n, s_max, stream), "scatter")) != SPR_OK)
    return st;
  return ok();
}

namespace {
constexpr int kPartDq = 1, kPartDkv = 2;

// Phase C (paper App. A.3-A.5); `parts` selects the prefix rows' dQ, the
// prefix keys' dK/dV with the injected cache, or both in one launch.
spr_status prefix_bwd_parts(const spr_dims* dims, const void* q_p, const void* k_p,
                            const void* v_p, const void* o_p, const float* lse_p,
                            const void* do_p, const float* gk_cache, const float* gv_cache,
                            void* dq_p, void* dk_p, void* dv_p, void* ws, size_t ws_bytes,
                            hipStream_t stream, int parts) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  const bool want_dq = parts & kPartDq, want_dkv = parts & kPartDkv;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype);
  std::vector<Buf> bufs = {{q_p, P * hq * hd * eb, "q_p", true},
                           {k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {o_p, P * hq * hd * eb, "o_p", true},
                           {lse_p, hq * P * 4, "lse_p", true, 4},
                           {do_p, P * hq * hd * eb, "do_p", false},
                           {gk_cache, P * hkv * hd * 4, "gk_cache", want_dkv},
                           {gv_cache, P * hkv * hd * 4, "gv_cache", want_dkv},
                           {dq_p, P * hq * hd * eb, "dq_p", want_dq},
                           {dk_p, P * hkv * hd * eb, "dk_p", want_dkv},
                           {dv_p, P * hkv * hd * eb, "dv_p", want_dkv}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const WsLayout w = ws_layout(SPR_OP_PREFIX_BWD, dims, 0, 0, 0);
  if (do_p != nullptr && (st = check_ws(w, ws, ws_bytes)) != SPR_OK) return st;
  std::vector<Buf> all = bufs;
  if (do_p != nullptr) all.push_back({ws, w.total, "ws", false});
  if (want_dkv && (st = check_aliasing({bufs[6], bufs[7]}, all)) != SPR_OK) return st;
  if (P == 0) return ok();
  const float scale = eff_scale(dims);
  if (do_p == nullptr) {
    // G_Y = 0: dQ_P = 0, dK_P = G_K, dV_P = G_V (paper App. A.5)
    if (want_dq &&
        (st = hip_check(launch_fill_zero((float*)dq_p, P * hq * hd * eb / 4, stream), "dq zero")) != SPR_OK)
      return st;
    if (want_dkv &&
        (st = hip_check(launch_convert(dims->dtype, gk_cache, 1.f, nullptr, dk_p, P * hkv * hd, stream),
                        "dk convert")) != SPR_OK)
      return st;
    if (want_dkv &&
        (st = hip_check(launch_convert(dims->dtype, gv_cache, 1.f, nullptr, dv_p, P * hkv * hd, stream),
                        "dv convert")) != SPR_OK)
      return st;
    return ok();
  }
  const bool f32 = dims->dtype == SPR_F32;
  // the whole Phase C adds dQ atomically from the key-outer blocks; the dQ
  // half alone keeps its query-outer role (fewer products without dK/dV)
  const bool aq = atomic_dq(dims) && want_dq && want_dkv;
  float* dd_p = at<float>(ws, w.dd_p);
  float* lse2_p = at<float>(ws, w.lse2_p);
  float* dq_acc = (f32 || aq) && want_dq ? at<float>(ws, w.dq_acc_p) : nullptr;
  if ((st = hip_check(launch_row_dot(dims->dtype, do_p, o_p, (int)P, (int)P, nullptr, 0, (int)hq, (int)hd,
                                     dd_p, lse_p, lse2_p, stream), "row statistic")) != SPR_OK)
    return st;
  if (dq_acc && (st = hip_check(launch_fill_zero(dq_acc, P * hq * hd, stream), "dq clear")) != SPR_OK)
    return st;
  AttnArgs a = base_args(dims);
  a.q_p = q_p; a.k_p = k_p; a.v_p = v_p; a.do_p = do_p;
  a.lse_p = const_cast<float*>(lse_p);
  a.dd_p = dd_p; a.lse2_p = lse2_p;
  a.prefix_rows = 1;
  a.suffix_rows = 0;
  if (want_dq) {
    a.dq_p = dq_p;
    a.dq_acc_p = dq_acc;
    if (aq)
      a.dq_atomic = 1;
    else
      a.n_prefix_q_tiles = tiles(dims->prefix_len, block_q(dims->dtype));
  }
  const bool wide = prefix_kv_wide(dims);
  if (want_dkv) {
    a.pk_mode = kPkInject;
    a.gk = const_cast<float*>(gk_cache); a.gv = const_cast<float*>(gv_cache);
    a.dk_p = dk_p; a.dv_p = dv_p;
    a.n_prefix_k_tiles = tiles(dims->prefix_len, wide ? bwd_bf16_kv_wide_block_k() : block_k(dims->dtype));
    a.kv_rsplit = prefix_bwd_kv_splits(dims);
    if (a.kv_rsplit > 1) {
      a.part_dk = at<float>(ws, w.part_dk);
      a.part_dv = at<float>(ws, w.part_dv);
    }
  }
  if (wide) {
    // the key-outer role alone, then the query-outer role
    if (want_dkv) {
      AttnArgs kv = a;
      kv.n_prefix_q_tiles = 0;
      if ((st = hip_check(launch_bwd_bf16_kv_wide(kv, dims->head_dim, stream), "prefix backward, dK/dV")) != SPR_OK)
        return st;
    }
    if (want_dq) {
      AttnArgs q = a;
      q.n_prefix_k_tiles = 0;
      q.kv_rsplit = 1;
      if ((st = hip_check(launch_bwd(dims, q, 1, stream), "prefix backward, dQ")) != SPR_OK) return st;
    }
  } else if ((st = hip_check(launch_bwd(dims, a, 1, stream), "prefix backward")) != SPR_OK) {
    return st;
  }
  if (dq_acc && (st = hip_check(launch_convert(dims->dtype, dq_acc, scale, nullptr, dq_p, P * hq * hd,
                                               stream), "dq convert")) != SPR_OK)
    return st;
  return ok();
}
}  // namespace

spr_status spr_prefix_bwd(const spr_dims* dims, const void* q_p, const void* k_p, const void* v_p,
                          const void* o_p, const float* lse_p, const void* do_p,
                          const float* gk_cache, const float* gv_cache, void* dq_p, void* dk_p,
                          void* dv_p, void* ws, size_t ws_bytes, hipStream_t stream) {
  return prefix_bwd_parts(dims, q_p, k_p, v_p, o_p, lse_p, do_p, gk_cache, gv_cache, dq_p, dk_p,
                          dv_p, ws, ws_bytes, stream, kPartDq | kPartDkv);
}

spr_status spr_prefix_bwd_dq(const spr_dims* dims, const void* q_p, const void* k_p,
                             const void* v_p, const void* o_p, const float* lse_p,
                             const void* do_p, void* dq_p, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  return prefix_bwd_parts(dims, q_p, k_p, v_p, o_p, lse_p, do_p, nullptr, nullptr, dq_p, nullptr,
                          nullptr, ws, ws_bytes, stream, kPartDq);
}

spr_status spr_prefix_bwd_dkv(const spr_dims* dims, const void* q_p, const void* k_p,
                              const void* v_p, const void* o_p, const float* lse_p,
                              const void* do_p, const float* gk_cache, const float* gv_cache,
                              void* dk_p, void* dv_p, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  return prefix_bwd_parts(dims, q_p, k_p, v_p, o_p, lse_p, do_p, gk_cache, gv_cache, nullptr, dk_p,
                          dv_p, ws, ws_bytes, stream, kPartDkv);
}

spr_status spr_dense_recompute_baseline(
    const spr_dims* dims, const void* q_p, const void* k_p, const void* v_p, const void* do_p_seq,
    const void* q_s, const void* k_s, const void* v_s, const void* do_s,
    const int32_t* cu_seqlens, int32_t n, int32_t max_len, int32_t total_len, void* o_p,
    float* lse_p, void* o_s, float* lse_s, void* dq_s, void* dk_s, void* dv_s, void* dq_p,
    void* dk_p, void* dv_p, void* ws, size_t ws_bytes, hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  if ((st = check_suffix_sizes(n, max_len, total_len)) != SPR_OK) return st;
  const size_t P = dims->prefix_len, hq = dims->num_q_heads, hkv = dims->num_kv_heads,
               hd = dims->head_dim, eb = dtype_bytes(dims->dtype), T = total_len;
  std::vector<Buf> bufs = {{q_p, P * hq * hd * eb, "q_p", true},
                           {k_p, P * hkv * hd * eb, "k_p", true},
                           {v_p, P * hkv * hd * eb, "v_p", true},
                           {do_p_seq, (size_t)n * P * hq * hd * eb, "do_p_seq", false},
                           {q_s, T * hq * hd * eb, "q_s", true},
                           {k_s, T * hkv * hd * eb, "k_s", true},
                           {v_s, T * hkv * hd * eb, "v_s", true},
                           {do_s, T * hq * hd * eb, "do_s", true},
                           {cu_seqlens, (size_t)(n + 1) * 4, "cu_seqlens", true, 4},
                           {o_p, P * hq * hd * eb, "o_p", true},
                           {lse_p, hq * P * 4, "lse_p", true, 4},
                           {o_s, T * hq * hd * eb, "o_s", true},
                           {lse_s, hq * T * 4, "lse_s", true, 4},
                           {dq_s, T * hq * hd * eb, "dq_s", true},
                           {dk_s, T * hkv * hd * eb, "dk_s", true},
                           {dv_s, T * hkv * hd * eb, "dv_s", true},
                           {dq_p, P * hq * hd * eb, "dq_p", true},
                           {dk_p, P * hkv * hd * eb, "dk_p", true},
                           {dv_p, P * hkv * hd * eb, "dv_p", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const WsLayout w = ws_layout(SPR_OP_DENSE_BASELINE, dims, n, max_len, total_len);
  if ((st = check_ws(w, ws, ws_bytes)) != SPR_OK) return st;
  float* dd_p = at<float>(ws, w.dd_p);
  float* dq_acc_p = at<float>(ws, w.dq_acc_p);
  const bool f32 = dims->dtype == SPR_F32;
  float* dd_s = at<float>(ws, w.dd_s);
  float* lse2_p = at<float>(ws, w.lse2_p);
  float* lse2_s = at<float>(ws, w.lse2_s);
  const bool aq = atomic_dq(dims);
  float* dq_acc_s = (f32 || aq) ? at<float>(ws, w.dq_acc_s) : nullptr;
  float* dk_acc = at<float>(ws, w.dk_acc_p);
  float* dv_acc = at<float>(ws, w.dv_acc_p);
  const float scale = eff_scale(dims);
  const bool have_dop = do_p_seq != nullptr;
#define SPR_TRY(expr, what) \
  if ((st = hip_check((expr), (what))) != SPR_OK) return st
  SPR_TRY(launch_fill_zero(dq_acc_p, P * hq * hd, stream), "clear");
  if (dq_acc_s) SPR_TRY(launch_fill_zero(dq_acc_s, T * hq * hd, stream), "clear");
  SPR_TRY(launch_fill_zero(dk_acc, P * hkv * hd, stream), "clear");
  SPR_TRY(launch_fill_zero(dv_acc, P * hkv * hd, stream), "clear");
  // one trajectory at a time, as a dense trainer runs them
  for (int32_t i = 0; i < n; ++i) {
    AttnArgs a = base_args(dims);
    a.q_p = q_p; a.k_p = k_p; a.v_p = v_p; a.o_p = o_p; a.lse_p = lse_p;
    a.q_s = q_s; a.k_s = k_s; a.v_s = v_s; a.o_s = o_s; a.lse_s = lse_s;
    a.cu = cu_seqlens;
    a.total_len = total_len;
    a.seq_base = i;
    a.n_seq = 1;
    SPR_TRY(launch_forward(dims, a, true, max_len, 1, stream), "dense forward");
    const void* dop_i = have_dop ? (const char*)do_p_seq + (size_t)i * P * hq * hd * eb : nullptr;
    if (have_dop && P > 0)
      SPR_TRY(launch_row_dot(dims->dtype, dop_i, o_p, (int)P, (int)P, nullptr, 0, (int)hq, (int)hd, dd_p,
                             lse_p, lse2_p, stream), "row statistic");
    SPR_TRY(launch_row_dot(dims->dtype, do_s, o_s, max_len, total_len, cu_seqlens, i, (int)hq, (int)hd, dd_s,
                           lse_s, lse2_s, stream), "row statistic");
    a.do_p = dop_i; a.dd_p = dd_p; a.lse2_p = lse2_p; a.dq_acc_p = dq_acc_p;
    a.do_s = do_s; a.dd_s = dd_s; a.lse2_s = lse2_s; a.dq_acc_s = dq_acc_s;
    a.dq_s = dq_s;
    a.dq_p_accumulate = 1;
    a.n_prefix_k_tiles = tiles(dims->prefix_len, block_k(dims->dtype));
    a.n_suffix_k_tiles = tiles(max_len, block_k(dims->dtype));
    a.prefix_rows = have_dop ? 1 : 0;
    a.suffix_rows = 1;
    a.pk_mode = kPkAccumulate;
    a.gk = dk_acc; a.gv = dv_acc;
    a.dk_s = dk_s; a.dv_s = dv_s;
    a.n_prefix_q_tiles = have_dop ? tiles(dims->prefix_len, block_q(dims->dtype)) : 0;
    a.n_suffix_q_tiles = tiles(max_len, block_q(dims->dtype));
    if (aq) {
      // dQ of the prefix rows sums over the trajectories in dq_acc_p and of
      // the suffix rows in dq_acc_s, both by the key-outer blocks' atomics
      a.dq_atomic = 1;
      a.n_prefix_q_tiles = 0;
      a.n_suffix_q_tiles = 0;
    }
    const bool wide = dense_kv_wide(dims, max_len);
    if (wide) {
      a.n_prefix_k_tiles = tiles(dims->prefix_len, bwd_bf16_kv_wide_block_k());
      a.n_suffix_k_tiles = tiles(max_len, bwd_bf16_kv_wide_block_k());
    }
    a.kv_rsplit = dense_bwd_kv_splits(dims, max_len);
    if (a.kv_rsplit > 1) {
      a.part_dk = at<float>(ws, w.part_dk);
      a.part_dv = at<float>(ws, w.part_dv);
    }
    if (wide) {
      // the key-outer role alone, then the query-outer role (as Phase C)
      AttnArgs kv = a;
      kv.n_prefix_q_tiles = 0;
      kv.n_suffix_q_tiles = 0;
      SPR_TRY(launch_bwd_bf16_kv_wide(kv, dims->head_dim, stream), "dense backward, dK/dV");
      AttnArgs q = a;
      q.n_prefix_k_tiles = 0;
      q.n_suffix_k_tiles = 0;
      q.kv_rsplit = 1;
      SPR_TRY(launch_bwd(dims, q, 1, stream), "dense backward, dQ");
    } else {
      SPR_TRY(launch_bwd(dims, a, 1, stream), "dense backward");
    }
  }
  SPR_TRY(launch_convert(dims->dtype, dq_acc_p, scale, nullptr, dq_p, P * hq * hd, stream), "convert");
  SPR_TRY(launch_convert(dims->dtype, dk_acc, 1.f, nullptr, dk_p, P * hkv * hd, stream), "convert");
  SPR_TRY(launch_convert(dims->dtype, dv_acc, 1.f, nullptr, dv_p, P * hkv * hd, stream), "convert");
  if (dq_acc_s) SPR_TRY(launch_convert(dims->dtype, dq_acc_s, scale, nullptr, dq_s, T * hq * hd, stream), "convert");
#undef SPR_TRY
  return ok();
}

spr_status spr_gkv_cache_zero(const spr_dims* dims, float* gk_cache, float* gv_cache,
                              hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  const size_t n = (size_t)dims->prefix_len * dims->num_kv_heads * dims->head_dim;
  if ((st = check_bufs({{gk_cache, n * 4, "gk_cache", true}, {gv_cache, n * 4, "gv_cache", true}})) != SPR_OK)
    return st;
  if (n == 0) return ok();
  if ((st = hip_check(launch_fill_zero(gk_cache, n, stream), "cache zero")) != SPR_OK) return st;
  if ((st = hip_check(launch_fill_zero(gv_cache, n, stream), "cache zero")) != SPR_OK) return st;
  return ok();
}

spr_status spr_gkv_accumulate(const spr_dims* dims, float* gk_cache, float* gv_cache,
                              const float* dgk, const float* dgv, hipStream_t stream) {
  spr_status st = check_dims(dims);
  if (st != SPR_OK) return st;
  const size_t n = (size_t)dims->prefix_len * dims->num_kv_heads * dims->head_dim;
  std::vector<Buf> bufs = {{gk_cache, n * 4, "gk_cache", true}, {gv_cache, n * 4, "gv_cache", true},
                           {dgk, n * 4, "dgk", true}, {dgv, n * 4, "dgv", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = check_aliasing({bufs[0], bufs[1]}, bufs)) != SPR_OK) return st;
  if (n == 0) return ok();
  if ((st = hip_check(launch_accumulate(gk_cache, dgk, n, stream), "cache accumulate")) != SPR_OK)
    return st;
  if ((st = hip_check(launch_accumulate(gv_cache, dgv, n, stream), "cache accumulate")) != SPR_OK)
    return st;
  return ok();
}

// ------------------------------------------------ decoder-layer token ops
namespace {
spr_status check_rows(int32_t rows, int32_t width) {
  if (rows < 0) return fail(SPR_ERR_INVALID_ARG, "rows must be >= 0");
  if (width < 8 || width % 8 != 0 || width > 16384)
    return fail(SPR_ERR_UNSUPPORTED, "width must be a multiple of 8 in [8, 16384]");
  return SPR_OK;
}
spr_status check_rope(int32_t tokens, int32_t heads, int32_t d, int32_t pos0, double theta) {
  if (tokens < 0 || heads < 1 || pos0 < 0) return fail(SPR_ERR_INVALID_ARG, "tokens/pos0 >= 0, heads >= 1");
  if (d < 2 || d % 2 != 0 || d > 256) return fail(SPR_ERR_UNSUPPORTED, "head_dim must be even, at most 256");
  if (!(theta > 1.0) || !isfinite(theta)) return fail(SPR_ERR_INVALID_ARG, "theta must be finite and > 1");
  return SPR_OK;
}
}  // namespace

spr_status spr_rmsnorm_fwd(int32_t rows, int32_t width, float eps, const void* x, void* y, float* rstd,
                           hipStream_t stream) {
  spr_status st = check_rows(rows, width);
  if (st != SPR_OK) return st;
  if (!(eps >= 0.f) || isinf(eps)) return fail(SPR_ERR_INVALID_ARG, "eps must be finite and >= 0");
  const size_t n = (size_t)rows * width * 2;
  std::vector<Buf> bufs = {{x, n, "x", true}, {y, n, "y", true}, {rstd, (size_t)rows * 4, "rstd", true, 4}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = check_aliasing({bufs[2]}, bufs)) != SPR_OK) return st;
  if ((st = hip_check(launch_rmsnorm_fwd(rows, width, eps, x, y, rstd, stream), "rmsnorm")) != SPR_OK) return st;
  return ok();
}

spr_status spr_rmsnorm_bwd(int32_t rows, int32_t width, const void* x, const float* rstd, const void* dy,
                           const void* add, void* dx, hipStream_t stream) {
  spr_status st = check_rows(rows, width);
  if (st != SPR_OK) return st;
  const size_t n = (size_t)rows * width * 2;
  std::vector<Buf> bufs = {{x, n, "x", true}, {rstd, (size_t)rows * 4, "rstd", true, 4}, {dy, n, "dy", true},
                           {add, n, "add", false}, {dx, n, "dx", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = check_aliasing({bufs[4]}, {bufs[0], bufs[1], bufs[2]})) != SPR_OK) return st;
  if ((st = hip_check(launch_rmsnorm_bwd(rows, width, x, rstd, dy, add, dx, stream), "rmsnorm bwd")) != SPR_OK)
    return st;
  return ok();
}

spr_status spr_rope_fwd(int32_t tokens, int32_t heads, int32_t head_dim, int32_t pos0, double theta,
                        const void* x, void* y, hipStream_t stream) {
  spr_status st = check_rope(tokens, heads, head_dim, pos0, theta);
  if (st != SPR_OK) return st;
  const size_t n = (size_t)tokens * heads * head_dim * 2;
  std::vector<Buf> bufs = {{x, n, "x", true}, {y, n, "y", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if (x != y && (st = check_aliasing({bufs[1]}, bufs)) != SPR_OK) return st;
  if ((st = hip_check(launch_rope(tokens, heads, head_dim, pos0, theta, x, y, false, stream), "rope")) != SPR_OK)
    return st;
  return ok();
}

spr_status spr_rope_bwd(int32_t tokens, int32_t heads, int32_t head_dim, int32_t pos0, double theta,
                        const void* dy, void* dx, hipStream_t stream) {
  spr_status st = check_rope(tokens, heads, head_dim, pos0, theta);
  if (st != SPR_OK) return st;
  const size_t n = (size_t)tokens * heads * head_dim * 2;
  std::vector<Buf> bufs = {{dy, n, "dy", true}, {dx, n, "dx", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if (dy != dx && (st = check_aliasing({bufs[1]}, bufs)) != SPR_OK) return st;
  if ((st = hip_check(launch_rope(tokens, heads, head_dim, pos0, theta, dy, dx, true, stream), "rope bwd")) !=
      SPR_OK)
    return st;
  return ok();
}

spr_status spr_swiglu_fwd(int64_t n, const void* g, const void* u, void* m, hipStream_t stream) {
  if (n < 0 || n % 8 != 0) return fail(SPR_ERR_INVALID_ARG, "n must be a non-negative multiple of 8");
  const size_t b = (size_t)n * 2;
  std::vector<Buf> bufs = {{g, b, "g", true}, {u, b, "u", true}, {m, b, "m", true}};
  spr_status st;
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = check_aliasing({bufs[2]}, bufs)) != SPR_OK) return st;
  if ((st = hip_check(launch_swiglu_fwd(n, g, u, m, stream), "swiglu")) != SPR_OK) return st;
  return ok();
}

spr_status spr_swiglu_bwd(int64_t n, const void* g, const void* u, const void* dm, void* dg, void* du,
                          hipStream_t stream) {
  if (n < 0 || n % 8 != 0) return fail(SPR_ERR_INVALID_ARG, "n must be a non-negative multiple of 8");
  const size_t b = (size_t)n * 2;
  std::vector<Buf> bufs = {{g, b, "g", true}, {u, b, "u", true}, {dm, b, "dm", true}, {dg, b, "dg", true},
                           {du, b, "du", true}};
  spr_status st;
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = check_aliasing({bufs[3], bufs[4]}, bufs)) != SPR_OK) return st;
  if ((st = hip_check(launch_swiglu_bwd(n, g, u, dm, dg, du, stream), "swiglu bwd")) != SPR_OK) return st;
  return ok();
}

// ------------------------------------------------------ MoE aux accounting
namespace {
spr_status check_moe(int32_t E, int32_t k) {
  if (E < 4 || E > 1024 || E % 4 != 0)
    return fail(SPR_ERR_UNSUPPORTED, "n_experts must be a multiple of 4 in [4, 1024]");
  if (k < 1 || k > E) return fail(SPR_ERR_INVALID_ARG, "top_k must be in [1, n_experts]");
  return SPR_OK;
}
size_t moe_stats_size(int32_t E) { return 16 * (size_t)E + 16; }
}  // namespace

spr_status spr_moe_stats_bytes(int32_t n_experts, size_t* bytes) {
  spr_status st = check_moe(n_experts, 1);
  if (st != SPR_OK) return st;
  if (bytes == nullptr) return fail(SPR_ERR_INVALID_ARG, "bytes is null");
  *bytes = moe_stats_size(n_experts);
  return ok();
}

spr_status spr_moe_stats_zero(int32_t n_experts, void* stats, hipStream_t stream) {
  spr_status st = check_moe(n_experts, 1);
  if (st != SPR_OK) return st;
  if ((st = check_bufs({{stats, moe_stats_size(n_experts), "stats", true}})) != SPR_OK) return st;
  if ((st = hip_check(launch_fill_zero((float*)stats, moe_stats_size(n_experts) / 4, stream), "stats zero")) !=
      SPR_OK)
    return st;
  return ok();
}

spr_status spr_moe_aux_workspace_size(int32_t n_experts, int32_t n_tokens, size_t* bytes) {
  spr_status st = check_moe(n_experts, 1);
  if (st != SPR_OK) return st;
  if (n_tokens < 0) return fail(SPR_ERR_INVALID_ARG, "n_tokens must be >= 0");
  if (bytes == nullptr) return fail(SPR_ERR_INVALID_ARG, "bytes is null");
  *bytes = moe_workspace_bytes(n_experts, n_tokens);
  return ok();
}

spr_status spr_moe_aux_accumulate(int32_t n_experts, int32_t top_k, int32_t n_tokens,
                                  const float* probs, const int32_t* experts,
                                  int32_t multiplicity, const int32_t* token_multiplicity,
                                  void* stats, void* ws, size_t ws_bytes, hipStream_t stream) {
  spr_status st = check_moe(n_experts, top_k);
  if (st != SPR_OK) return st;
  if (n_tokens < 0) return fail(SPR_ERR_INVALID_ARG, "n_tokens must be >= 0");
  if (token_multiplicity == nullptr && multiplicity < 0)
    return fail(SPR_ERR_INVALID_ARG, "multiplicity must be >= 0");
  const size_t n = (size_t)n_tokens, E = (size_t)n_experts, k = (size_t)top_k;
  std::vector<Buf> bufs = {{probs, n * E * 4, "probs", true},
                           {experts, n * k * 4, "experts", true, 4},
                           {token_multiplicity, n * 4, "token_multiplicity", false, 4},
                           {stats, moe_stats_size(n_experts), "stats", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  const size_t need = moe_workspace_bytes(n_experts, n_tokens);
  if (need > 0) {
    if (ws == nullptr) return fail(SPR_ERR_WORKSPACE, "workspace is null");
    if (ws_bytes < need)
      return fail(SPR_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes, got " +
                                         std::to_string(ws_bytes));
    if (((uintptr_t)ws & 15u) != 0) return fail(SPR_ERR_MISALIGNED, "workspace is not 16-byte aligned");
  }
  std::vector<Buf> all = bufs;
  all.push_back({ws, need, "ws", false});
  if ((st = check_aliasing({bufs[3]}, all)) != SPR_OK) return st;
  if (n_tokens == 0) return ok();
  if ((st = hip_check(launch_moe_accumulate(probs, experts, n_tokens, n_experts, top_k, multiplicity,
                                            token_multiplicity, stats, ws, stream),
                      "moe accumulate")) != SPR_OK)
    return st;
  return ok();
}

spr_status spr_moe_aux_loss(int32_t n_experts, int32_t top_k, double aux_coef, const void* stats,
                            double* f, double* p, double* loss, hipStream_t stream) {
  spr_status st = check_moe(n_experts, top_k);
  if (st != SPR_OK) return st;
  if (!isfinite(aux_coef)) return fail(SPR_ERR_INVALID_ARG, "aux_coef must be finite");
  const size_t E = (size_t)n_experts;
  std::vector<Buf> bufs = {{stats, moe_stats_size(n_experts), "stats", true},
                           {f, E * 8, "f", false, 8},
                           {p, E * 8, "p", false, 8},
                           {loss, 8, "loss", true, 8}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = hip_check(launch_moe_loss(stats, n_experts, top_k, aux_coef, f, p, loss, stream), "moe loss")) !=
      SPR_OK)
    return st;
  return ok();
}

spr_status spr_moe_aux_grad(int32_t n_experts, int32_t top_k, double aux_coef, double upstream,
                            const void* stats, int32_t n_tokens, int32_t multiplicity,
                            const int32_t* token_multiplicity, float* dprobs, hipStream_t stream) {
  spr_status st = check_moe(n_experts, top_k);
  if (st != SPR_OK) return st;
  if (!isfinite(aux_coef) || !isfinite(upstream))
    return fail(SPR_ERR_INVALID_ARG, "aux_coef and upstream must be finite");
  if (n_tokens < 0) return fail(SPR_ERR_INVALID_ARG, "n_tokens must be >= 0");
  if (token_multiplicity == nullptr && multiplicity < 0)
    return fail(SPR_ERR_INVALID_ARG, "multiplicity must be >= 0");
  const size_t n = (size_t)n_tokens, E = (size_t)n_experts;
  std::vector<Buf> bufs = {{stats, moe_stats_size(n_experts), "stats", true},
                           {token_multiplicity, n * 4, "token_multiplicity", false, 4},
                           {dprobs, n * E * 4, "dprobs", true}};
  if ((st = check_bufs(bufs)) != SPR_OK) return st;
  if ((st = check_aliasing({bufs[2]}, bufs)) != SPR_OK) return st;
  if (n_tokens == 0) return ok();
  if ((st = hip_check(launch_moe_grad(stats, n_experts, top_k, upstream * aux_coef, n_tokens, multiplicity,
                                      token_multiplicity, dprobs, stream),
                      "moe grad")) != SPR_OK)
    return st;
  return ok();
}

spr_status spr_profile_enable(int32_t enable, const char* only_kernel) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = enable != 0;
  g_prof_only = only_kernel != nullptr ? only_kernel : "";
  return SPR_OK;
}

spr_status spr_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  prof_drain_locked();
  g_prof_totals.clear();
  g_prof_names.clear();
  return SPR_OK;
}

spr_status spr_profile_query(const char* kernel, double* total_ms, int32_t* count) {
  if (kernel == nullptr || total_ms == nullptr || count == nullptr)
    return fail(SPR_ERR_INVALID_ARG, "null argument");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  prof_drain_locked();
  auto it = g_prof_totals.find(kernel);
  *total_ms = it == g_prof_totals.end() ? 0.0 : it->second.first;
  *count = it == g_prof_totals.end() ? 0 : it->second.second;
  return SPR_OK;
}

int32_t spr_profile_num_kernels(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  prof_drain_locked();
  return (int32_t)g_prof_names.size();
}

const char* spr_profile_kernel_name(int32_t index) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (index < 0 || index >= (int32_t)g_prof_names.size()) return "";
  return g_prof_names[index].c_str();
}

}  // extern "C"
