/*
 * spr_moe.h -- MoE router auxiliary-loss accounting under prefix reuse
 * (paper Sec. 3.5, Sec. 4.6, App. B), part of libspr.
 *
 * With prefix reuse the P shared prefix tokens of a prompt group exist once
 * physically but stand for N logical copies (one per trajectory in the
 * baseline's reduction scope).  For a token-local Top-k router with an
 * auxiliary load-balancing loss, every physical token u carries a
 * multiplicity m_u (N for a shared prefix token, 1 for a suffix token) and
 * the statistics of App. B are
 *   C_e = sum_u m_u sum_j 1[r[u,j] = e]   (hard count, no gradient)
 *   R_e = sum_u m_u p[u,e],   M = sum_u m_u,
 *   f_e = C_e / (k M),  P_e = R_e / M,  L_aux = lambda E sum_e f_e P_e,
 * which equal those of the batch with every prefix copy materialized.  The
 * router-probability gradient (C_e constant) is
 *   dL_aux/dp[u,e] = lambda E f_e m_u / M.
 *
 * Use: spr_moe_stats_zero once per reduction scope; spr_moe_aux_accumulate
 * for the prefix tokens (Phase A, multiplicity N) and for each suffix
 * microbatch (Phase B, multiplicity 1), in any order; then
 * spr_moe_aux_loss and spr_moe_aux_grad for each token set (the prefix's
 * in Phase C).
 *
 * Conventions: n_experts E with 4 <= E <= 1024 and E % 4 == 0; 1 <= top_k
 * <= E; every pointer is device memory owned by the caller (probs and the
 * statistics 16-byte aligned, int32 arrays 4-byte aligned); calls are
 * asynchronous on `stream`; on a validation error nothing is launched and
 * spr_last_error() says why.  Accumulations into one statistics buffer must
 * be ordered (one stream or events).  Every reduction runs in a fixed order:
 * results are bitwise reproducible.
 */
#ifndef SPR_MOE_H
#define SPR_MOE_H

#include "spr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Statistics buffer of one reduction scope: int64 count[E] at byte 0,
 * double mass[E] at 8E, int64 total at 16E, int64 invalid at 16E + 8 (the
 * selected-expert ids outside [0, E) that were skipped).  bytes = 16E + 16. */
spr_status spr_moe_stats_bytes(int32_t n_experts, size_t* bytes);

/* Clears a statistics buffer. */
spr_status spr_moe_stats_zero(int32_t n_experts, void* stats, hipStream_t stream);

/* Workspace bytes spr_moe_aux_accumulate needs for n_tokens tokens. */
spr_status spr_moe_aux_workspace_size(int32_t n_experts, int32_t n_tokens, size_t* bytes);

/* Adds n_tokens tokens to the statistics (App. B C_e, R_e, M):
 *   probs [n_tokens, E] fp32 router probabilities; experts [n_tokens, top_k]
 *   int32 selected experts; token_multiplicity [n_tokens] int32 (>= 0) or
 *   NULL, in which case every token has `multiplicity` (>= 0).
 * Expert ids outside [0, E) are skipped and counted in `invalid`. */
spr_status spr_moe_aux_accumulate(int32_t n_experts, int32_t top_k, int32_t n_tokens,
                                  const float* probs, const int32_t* experts,
                                  int32_t multiplicity, const int32_t* token_multiplicity,
                                  void* stats, void* ws, size_t ws_bytes, hipStream_t stream);

/* f_e, P_e and L_aux from the statistics: f and p [E] fp64 (either may be
 * NULL), loss [1] fp64.  M = 0 gives zeros. */
spr_status spr_moe_aux_loss(int32_t n_experts, int32_t top_k, double aux_coef,
                            const void* stats, double* f, double* p, double* loss,
                            hipStream_t stream);

/* dprobs[u,e] = upstream * aux_coef * E * f_e * m_u / M (fp32, written, not
 * added) for n_tokens tokens with multiplicities as in
 * spr_moe_aux_accumulate.  M = 0 gives zeros. */
spr_status spr_moe_aux_grad(int32_t n_experts, int32_t top_k, double aux_coef, double upstream,
                            const void* stats, int32_t n_tokens, int32_t multiplicity,
                            const int32_t* token_multiplicity, float* dprobs,
                            hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPR_MOE_H */
