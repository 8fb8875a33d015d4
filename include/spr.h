/*
 * spr.h -- C ABI of libspr, schedule-level shared-prefix attention for one
 * GRPO prompt group [P||S(1)] ... [P||S(N)] on AMD Instinct MI355X (gfx950).
 *
 * The operation (paper Sec. 2.1, Sec. 3.1-3.2, App. A): causal attention
 * forward and backward for N sequences that share one prefix of P tokens,
 * computed as a three-phase schedule:
 *
 *   Phase A  spr_prefix_fwd            prefix forward once; K_P/V_P stay in
 *                                      HBM as the forward cache.
 *   Phase B  spr_suffix_attn_fwd       per suffix microbatch: queries attend
 *            spr_suffix_attn_bwd_accum to the prefix K/V (all visible) and to
 *                                      their own suffix causally; backward
 *                                      adds the prefix-side gK/gV into one
 *                                      fp32 gradient cache.
 *   Phase C  spr_prefix_bwd            prefix backward once on the
 *                                      accumulated cache.
 *
 * spr_dense_recompute_baseline is the comparison, not the method: it
 * recomputes full causal attention over every [P||S(i)] and sums the prefix
 * gradients, which is what a dense trainer does.
 *
 * Conventions shared by every call
 * --------------------------------
 * Layout   Token-major, contiguous: Q, O, dO, dQ are [T, Hq, d]; K, V, dK, dV
 *          are [T, Hkv, d]; d contiguous.  The G = Hq/Hkv query heads that
 *          share kv head g are heads g*G .. g*G+G-1 (q head h reads kv head
 *          h / G).  LSE is [T, Hq] fp32, token-major like every other
 *          tensor (a microbatch slice of a packed group stays contiguous):
 *          the natural log of the row sum of exp of the scaled scores.  The
 *          gradient cache G_K, G_V is [P, Hkv, d] fp32.
 * Suffixes Packed with no padding: suffix i of a microbatch occupies rows
 *          cu_seqlens[i] .. cu_seqlens[i+1]-1 of the suffix tensors.
 *          cu_seqlens is a DEVICE int32 array of n+1 entries with
 *          cu_seqlens[0] = 0, strictly increasing (every suffix has >= 1
 *          token), cu_seqlens[n] = total_len; max_len (host) is the longest
 *          suffix.  The library does not read device memory on the host:
 *          callers that hold a host copy validate it with
 *          spr_check_cu_seqlens (the Python binding always does).  The
 *          kernels clamp every offset into [0, total_len] and every segment
 *          to a non-negative length, so inconsistent device values give
 *          wrong rows but no access outside the caller's buffers.
 * Mask     Causal, inclusive of the diagonal.  A prefix row r sees prefix
 *          keys 0..r.  A suffix row at local position t sees every prefix key
 *          and keys 0..t of its own suffix, never another suffix (paper
 *          Sec. 3.2 Phase B and Sec. 4.2).
 * Scale    softmax_scale, 0 meaning 1/sqrt(d) (paper Sec. 3.1).
 * Dtypes   SPR_F32 or SPR_BF16 storage for every input and output tensor;
 *          LSE, the cache and all accumulation are fp32.
 * Memory   Every pointer is device memory owned by the caller, 16-byte
 *          aligned (LSE and cu_seqlens: 4-byte aligned, so that microbatch
 *          slices of a packed group's LSE qualify).  The library never
 *          allocates, frees or keeps a pointer
 *          past the call.  Calls that take a workspace need at least the
 *          bytes spr_workspace_size reports (256-byte aligned).
 * Streams  Every call is asynchronous on `stream` and never synchronises the
 *          host.  The cache read-modify-write is not atomic across calls:
 *          every spr_suffix_attn_bwd_accum into one cache, and the
 *          spr_prefix_bwd that reads it, must be ordered (one stream, or
 *          explicit events).  Calls on different caches may run concurrently.
 * Errors   Each call returns an spr_status.  On any error nothing is
 *          launched and spr_last_error() describes the cause (thread-local).
 *          SPR_ERR_INVALID_ARG: null required pointer, negative or
 *          inconsistent sizes, Hq % Hkv != 0, n < 1.  SPR_ERR_UNSUPPORTED:
 *          head_dim not 64 or 128, unknown dtype or flag.
 *          SPR_ERR_MISALIGNED: a pointer not 16-byte aligned.
 *          SPR_ERR_ALIASING: an in-out cache overlaps another argument.
 *          SPR_ERR_WORKSPACE: workspace missing or too small.
 *          SPR_ERR_HIP: a HIP launch failed (detail in spr_last_error()).
 */
#ifndef SPR_H
#define SPR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum spr_dtype { SPR_F32 = 0, SPR_BF16 = 1 } spr_dtype;

/* flags */
enum {
  /* Every output bitwise reproducible run to run: dQ of the bf16 backward
   * from a query-outer role with no floating-point atomics.  This is the
   * default; the bit is accepted for callers that state it. */
  SPR_DETERMINISTIC = 1u << 0,
  /* bf16 backward: the key-outer blocks add dQ = dS K / sqrt(d) into an fp32
   * accumulator with fp32 atomics (5 matrix products per visible pair
   * instead of 7, no query-outer role); dQ is then reproducible only to
   * rounding, dK/dV/G_K/G_V stay bitwise.  Measured about 3x slower on
   * MI355X (the atomic traffic, P/64 adds of every dQ element, exceeds what
   * the L2 sustains), so it is opt-in.  Not with SPR_DETERMINISTIC. */
  SPR_ATOMIC_DQ = 1u << 1
};

typedef struct spr_dims {
  int32_t num_q_heads;  /* Hq >= 1 */
  int32_t num_kv_heads; /* Hkv >= 1, Hq % Hkv == 0 */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t prefix_len;   /* P >= 0; P == 0 makes the prefix calls no-ops */
  float softmax_scale;  /* 0 => 1/sqrt(d) */
  int32_t dtype;        /* spr_dtype */
  uint32_t flags;       /* 0, SPR_DETERMINISTIC or SPR_ATOMIC_DQ */
} spr_dims;

typedef enum spr_status {
  SPR_OK = 0,
  SPR_ERR_INVALID_ARG = 1,
  SPR_ERR_UNSUPPORTED = 2,
  SPR_ERR_MISALIGNED = 3,
  SPR_ERR_ALIASING = 4,
  SPR_ERR_WORKSPACE = 5,
  SPR_ERR_HIP = 6
} spr_status;

typedef enum spr_op {
  SPR_OP_PREFIX_FWD = 0,
  SPR_OP_SUFFIX_FWD = 1,
  SPR_OP_SUFFIX_BWD = 2,
  SPR_OP_PREFIX_BWD = 3,
  SPR_OP_DENSE_BASELINE = 4,
  SPR_OP_SUFFIX_FWD_PADDED = 5,
  SPR_OP_SUFFIX_BWD_PADDED = 6
} spr_op;

/*
 * Phase A (paper Sec. 3.2 "Phase A: prefix forward"; App. A.1 H_1 = P_11 V_1).
 * Causal attention of the prefix rows over the prefix keys.
 *   q_p [P,Hq,d], k_p/v_p [P,Hkv,d] in; o_p [P,Hq,d], lse_p [P,Hq] out.
 * K_P/V_P are read in place by every later call: they are the forward cache.
 */
spr_status spr_prefix_fwd(const spr_dims* dims, const void* q_p, const void* k_p,
                          const void* v_p, void* o_p, float* lse_p, hipStream_t stream);

/*
 * Phase B forward (paper Sec. 3.1 H_2 = Attn(Q_2, [K_1;K_2], [V_1;V_2]);
 * App. A.1 H_2 = P_21 V_1 + P_22 V_2 with one joint row softmax).
 * One packed microbatch of n_mb suffixes.  The prefix K/V are read directly,
 * never concatenated with the suffix K/V.
 *   k_p/v_p [P,Hkv,d]; q_s [total_len,Hq,d]; k_s/v_s [total_len,Hkv,d] in;
 *   o_s [total_len,Hq,d], lse_s [total_len,Hq] out.
 */
spr_status spr_suffix_attn_fwd(const spr_dims* dims, const void* k_p, const void* v_p,
                               const void* q_s, const void* k_s, const void* v_s,
                               const int32_t* cu_seqlens, int32_t n_mb, int32_t max_len,
                               int32_t total_len, void* o_s, float* lse_s, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/*
 * spr_suffix_attn_fwd without a workspace argument and without any device
 * allocation, for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, semantics and outputs as spr_suffix_attn_fwd (bitwise: the
 * same kernels with the same launch shapes).  Its workspace is a static
 * device array of 64 MiB (67108864 bytes) that every GPU the library runs
 * on holds until the process ends; its address is looked
 * up on the first call on each device, which must be the calling thread's
 * current device.  Sizes whose workspace (spr_workspace_size of
 * SPR_OP_SUFFIX_FWD) exceeds the scratch are rejected with
 * SPR_ERR_WORKSPACE and nothing is launched.  All calls on one GPU share
 * that GPU's scratch: two calls that overlap in time on one GPU (different
 * streams, or host threads) race and give undefined results; calls ordered
 * on one stream are safe.
 */
spr_status spr_suffix_attn_fwd_noalloc(const spr_dims* dims, const void* k_p, const void* v_p,
                                       const void* q_s, const void* k_s, const void* v_s,
                                       const int32_t* cu_seqlens, int32_t n_mb, int32_t max_len,
                                       int32_t total_len, void* o_s, float* lse_s,
                                       hipStream_t stream);

/*
 * Host-side check of a packed microbatch's suffix offsets, for callers that
 * hold a host copy of the cu_seqlens they upload (the library never reads
 * device memory on the host).  SPR_OK iff cu_host[0] == 0, every suffix
 * length cu_host[s+1] - cu_host[s] is in [1, max_len], the longest equals
 * max_len and cu_host[n_mb] == total_len; otherwise SPR_ERR_INVALID_ARG
 * naming the first violation (a zero-length suffix included).  Launches
 * nothing.
 */
spr_status spr_check_cu_seqlens(const int32_t* cu_host, int32_t n_mb, int32_t max_len,
                                int32_t total_len);

/*
 * Phase B backward with gradient-cache accumulation (paper App. A.2-A.3):
 *   dV_2 = P_22^T dO, dP = dO [V_1;V_2]^T, [dS_21, dS_22] = joint softmax
 *   backward, dQ_2 = (dS_21 K_1 + dS_22 K_2)/sqrt(d), dK_2 = dS_22^T Q_2/sqrt(d),
 *   and the prefix coupling gradients gV_1 = P_21^T dO, gK_1 = dS_21^T Q_2/sqrt(d),
 *   which are ADDED to gk_cache/gv_cache (fp32, [P,Hkv,d], in-out, +=).
 * Inputs o_s, lse_s are this microbatch's spr_suffix_attn_fwd outputs and
 * do_s [total_len,Hq,d] its upstream adjoint (any trajectory weight alpha(i)
 * is folded into do_s, paper App. A.1).  Outputs dq_s [total_len,Hq,d],
 * dk_s/dv_s [total_len,Hkv,d].  Each (prefix tile, kv head) of the cache is
 * updated by exactly one workgroup, so the cache result is bitwise
 * reproducible for a fixed sequence of calls.  The caches must not overlap
 * any other argument.
 */
spr_status spr_suffix_attn_bwd_accum(const spr_dims* dims, const void* k_p, const void* v_p,
                                     const void* q_s, const void* k_s, const void* v_s,
                                     const void* o_s, const float* lse_s, const void* do_s,
                                     const int32_t* cu_seqlens, int32_t n_mb, int32_t max_len,
                                     int32_t total_len, void* dq_s, void* dk_s, void* dv_s,
                                     float* gk_cache, float* gv_cache, void* ws, size_t ws_bytes,
                                     hipStream_t stream);

/*
 * Phase B with batch-plus-padding suffixes (paper Sec. 2.1, Sec. 4.2: the
 * schedule is transparent to the suffix organisation).  Suffix tensors are
 * [n, s_max, H, d] (LSE [n, s_max, Hq]); suffix i holds seq_lens[i] valid
 * rows (a DEVICE int32 array of n entries, each in [1, s_max]; the library
 * clamps values into [0, s_max] so that no access leaves the buffers) and
 * rows t >= seq_lens[i] are padding: they attend to nothing, nothing attends
 * to them, and every output row of padding is set to zero.  The valid rows
 * are gathered into the packed layout inside the workspace, run through the
 * packed calls above, and scattered back, so the results (and the cache
 * update) are bitwise those of the packed calls on the same suffixes.
 * Workspace: spr_workspace_size(SPR_OP_SUFFIX_{FWD,BWD}_PADDED, dims, n,
 * s_max, 0).  Other arguments as in the packed calls.
 */
spr_status spr_suffix_attn_fwd_padded(const spr_dims* dims, const void* k_p, const void* v_p,
                                      const void* q_s, const void* k_s, const void* v_s,
                                      const int32_t* seq_lens, int32_t n, int32_t s_max, void* o_s,
                                      float* lse_s, void* ws, size_t ws_bytes, hipStream_t stream);
spr_status spr_suffix_attn_bwd_accum_padded(const spr_dims* dims, const void* k_p, const void* v_p,
                                            const void* q_s, const void* k_s, const void* v_s,
                                            const void* o_s, const float* lse_s, const void* do_s,
                                            const int32_t* seq_lens, int32_t n, int32_t s_max,
                                            void* dq_s, void* dk_s, void* dv_s, float* gk_cache,
                                            float* gv_cache, void* ws, size_t ws_bytes,
                                            hipStream_t stream);

/*
 * Phase C (paper App. A.3-A.5): one prefix backward with the injected cache,
 *   dQ_1 = dS_11 K_1/sqrt(d), dK_1 = dS_11^T Q_1/sqrt(d) + G_K,
 *   dV_1 = P_11^T G_Y + G_V, dS_11 = P_11 * (dP_11 - rowsum(dP_11 * P_11)),
 *   dP_11 = G_Y V_1^T.
 * do_p [P,Hq,d] is the accumulated direct prefix-row adjoint G_Y; NULL means
 * zero (the common suffix-only loss, App. A.5), in which case dq_p = 0,
 * dk_p = G_K and dv_p = G_V exactly (rounded to the storage dtype).
 * o_p, lse_p are spr_prefix_fwd's outputs.  Outputs dq_p [P,Hq,d],
 * dk_p/dv_p [P,Hkv,d].
 */
spr_status spr_prefix_bwd(const spr_dims* dims, const void* q_p, const void* k_p,
                          const void* v_p, const void* o_p, const float* lse_p,
                          const void* do_p, const float* gk_cache, const float* gv_cache,
                          void* dq_p, void* dk_p, void* dv_p, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/*
 * Phase C in two independent halves (same equations as spr_prefix_bwd).
 * The prefix rows' dQ_1 = dS_11 K_1/sqrt(d) involves only prefix attention
 * (App. A.3): it reads no cache and no Phase B output, so it may run as
 * soon as spr_prefix_fwd is done, e.g. on another stream while Phase B
 * runs.  spr_prefix_bwd_dkv computes dK_1 and dV_1 with the injected cache
 * and must be ordered after every spr_suffix_attn_bwd_accum into that cache.
 * Arguments mean what they mean in spr_prefix_bwd; each half takes a
 * workspace of spr_workspace_size(SPR_OP_PREFIX_BWD) bytes, and two calls
 * that may run concurrently need separate workspaces.  Together the two
 * calls give exactly spr_prefix_bwd's outputs.
 */
spr_status spr_prefix_bwd_dq(const spr_dims* dims, const void* q_p, const void* k_p,
                             const void* v_p, const void* o_p, const float* lse_p,
                             const void* do_p, void* dq_p, void* ws, size_t ws_bytes,
                             hipStream_t stream);
spr_status spr_prefix_bwd_dkv(const spr_dims* dims, const void* q_p, const void* k_p,
                              const void* v_p, const void* o_p, const float* lse_p,
                              const void* do_p, const float* gk_cache, const float* gv_cache,
                              void* dk_p, void* dv_p, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/*
 * Dense recompute baseline (paper Sec. 2.1 and Sec. 3.2 cost model
 * T_base = N C_full): for i = 0..n-1, full causal forward and backward over
 * the sequence [P||S(i)], one sequence at a time, with upstream adjoint
 * [do_p_seq[i]; dO_S(i)].  The prefix is recomputed n times.
 *   do_p_seq [n,P,Hq,d] per-trajectory prefix-row adjoints (NULL => zero).
 * Outputs: o_p/lse_p (the prefix forward, identical for every i), o_s/lse_s,
 * dq_s/dk_s/dv_s per suffix row, and dq_p/dk_p/dv_p = the sum over i of each
 * sequence's prefix-row gradients (accumulated in fp32 in the workspace).
 */
spr_status spr_dense_recompute_baseline(
    const spr_dims* dims, const void* q_p, const void* k_p, const void* v_p,
    const void* do_p_seq, const void* q_s, const void* k_s, const void* v_s, const void* do_s,
    const int32_t* cu_seqlens, int32_t n, int32_t max_len, int32_t total_len, void* o_p,
    float* lse_p, void* o_s, float* lse_s, void* dq_s, void* dk_s, void* dv_s, void* dq_p,
    void* dk_p, void* dv_p, void* ws, size_t ws_bytes, hipStream_t stream);

/* Workspace bytes that `op` needs for these sizes (0 is a valid answer).
 * n_mb/max_len/total_len are ignored by the prefix ops. */
spr_status spr_workspace_size(int32_t op, const spr_dims* dims, int32_t n_mb, int32_t max_len,
                              int32_t total_len, size_t* bytes);

/* G_K = G_V = 0 for a new prompt group (paper Sec. 4.1: the cache lives for
 * one prompt group).  Uses a fill kernel, no memset node. */
spr_status spr_gkv_cache_zero(const spr_dims* dims, float* gk_cache, float* gv_cache,
                              hipStream_t stream);

/* G_K += dgk, G_V += dgv elementwise over [P,Hkv,d] fp32 (paper App. A.8:
 * the N lightweight element-wise accumulations).  The fused accumulation
 * inside spr_suffix_attn_bwd_accum does not need it; it serves callers that
 * hold a separate per-microbatch gK/gV and measures the HBM-bound cache
 * update on its own. */
spr_status spr_gkv_accumulate(const spr_dims* dims, float* gk_cache, float* gv_cache,
                              const float* dgk, const float* dgv, hipStream_t stream);

/* Per-kernel GPU timing with HIP events, off by default.  While enabled,
 * every kernel the library launches (or, when only_kernel is not NULL, every
 * launch of that kernel only) is bracketed by two events on its stream.
 * spr_profile_query waits for the recorded events and returns the summed
 * milliseconds and launch count of the kernels whose name equals `kernel`
 * (names as listed by spr_profile_kernel_name).  Not thread-safe against
 * concurrent enable/reset; recording itself is. */
spr_status spr_profile_enable(int32_t enable, const char* only_kernel);
spr_status spr_profile_reset(void);
spr_status spr_profile_query(const char* kernel, double* total_ms, int32_t* count);
int32_t spr_profile_num_kernels(void);
const char* spr_profile_kernel_name(int32_t index);

const char* spr_status_string(int32_t status);
const char* spr_last_error(void);
const char* spr_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPR_H */
