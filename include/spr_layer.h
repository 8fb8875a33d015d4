/*
 * spr_layer.h -- token-wise operations of a Llama3-style decoder layer, so
 * that a whole layer can run through the three-phase schedule (paper
 * Sec. 3.1: everything outside attention acts on each token on its own;
 * App. A.6: the weight gradients are the prefix part once plus the suffix
 * parts).  The projection GEMMs are left to the BLAS library.
 *
 * All tensors are bf16, row-major, device memory owned by the caller,
 * 16-byte aligned; statistics are fp32.  Rows are tokens.  Calls are
 * asynchronous on `stream`; on a validation error nothing is launched and
 * spr_last_error() says why.
 */
#ifndef SPR_LAYER_H
#define SPR_LAYER_H

#include "spr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* RMSNorm with unit gain: y = x * r, r = 1 / sqrt(mean(x^2) + eps) per row.
 * x, y [rows, width] (width a multiple of 8, at most 16384); rstd [rows]
 * fp32 out (kept for the backward). */
spr_status spr_rmsnorm_fwd(int32_t rows, int32_t width, float eps, const void* x, void* y,
                           float* rstd, hipStream_t stream);

/* dx = r (dy - x r^2 mean(dy * x)) + add, with r from the forward; `add`
 * [rows, width] (the residual branch's gradient) may be NULL. */
spr_status spr_rmsnorm_bwd(int32_t rows, int32_t width, const void* x, const float* rstd,
                           const void* dy, const void* add, void* dx, hipStream_t stream);

/* Rotary position embedding, rotate-half pairing (j, j + d/2) at angle
 * (pos0 + t) * theta^(-2j/d) for token t: x, y [tokens, heads, head_dim]
 * (head_dim even, at most 256).  The backward is the rotation by the
 * negative angle (inverse = transpose).  Angles are reduced in fp64. */
spr_status spr_rope_fwd(int32_t tokens, int32_t heads, int32_t head_dim, int32_t pos0, double theta,
                        const void* x, void* y, hipStream_t stream);
spr_status spr_rope_bwd(int32_t tokens, int32_t heads, int32_t head_dim, int32_t pos0, double theta,
                        const void* dy, void* dx, hipStream_t stream);

/* SwiGLU: m = silu(g) * u; backward dg = dm u silu'(g), du = dm silu(g).
 * All [n] with n a multiple of 8. */
spr_status spr_swiglu_fwd(int64_t n, const void* g, const void* u, void* m, hipStream_t stream);
spr_status spr_swiglu_bwd(int64_t n, const void* g, const void* u, const void* dm, void* dg, void* du,
                          hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPR_LAYER_H */
