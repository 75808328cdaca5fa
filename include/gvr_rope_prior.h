/*
 * gvr_rope_prior.h -- the static RoPE/YaRN prior of the indexer scores, for
 * use as the guessed index set of gvr_topk when no previous Top-K exists
 * (the first decode step, or a row whose history was dropped).
 *
 * Sec. 3.2 ("Theoretical Basis: Toeplitz Structure and RoPE Frequency
 * Analysis"): with all-ones query and key vectors, the positional part of a
 * RoPE dot product at relative position Delta is
 *     g(Delta) = 2 * sum_{i=0}^{d/2-1} cos(Delta * theta'_i),
 * a function of Delta alone (the score matrix is Toeplitz). Sec. 3.3
 * ("Pre-Computed Candidate Indices") takes the K relative positions with the
 * largest g as a static index set, P_static = argtopk_{Delta >= 0} g(Delta).
 * A query scoring the keys j = 0 .. n-1 at distance Delta = j (the layout of
 * the paper's synthetic benchmark, Sec. 6.3.1) can hand P_static straight to
 * gvr_topk as prev_topk; the result stays exact whatever the guess.
 *
 * Angles (Sec. 3.2, "YaRN extension"; the values of the synthetic-data
 * appendix are the defaults):
 *   theta_i  = base^(-2i/d),  i = 0 .. d/2 - 1
 *   x(beta)  = d * ln(L / (2 pi beta)) / (2 ln base)
 *   lo = max(floor(x(beta_fast)), 0),  hi = min(ceil(x(beta_slow)), d - 1)
 *   gamma_i  = clamp((i - lo) / max(hi - lo, 1e-3), 0, 1)
 *   theta'_i = theta_i * (1 - gamma_i) + (theta_i / s) * gamma_i
 * so pairs turning more than beta_fast times over the original context L
 * keep their angle and pairs turning less than beta_slow times are slowed
 * by the scale s. s = 1 gives plain RoPE. All of it, g and the selection
 * are computed in float64 on the device.
 *
 * Memory and ownership: array arguments are DEVICE pointers on the current
 * HIP device, owned by the caller; `params` is a HOST pointer (NULL = the
 * defaults) read during the call only. Work is enqueued on `stream` (a
 * hipStream_t as void*, NULL = the null stream); the call does not
 * synchronise. Argument errors are reported before anything is enqueued.
 * The library allocates nothing.
 */
#ifndef GVR_ROPE_PRIOR_H
#define GVR_ROPE_PRIOR_H

#include <stdint.h>

#include "gvr_topk.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gvr_rope_params {
    int32_t d_rope;     /* rotary dimensions d: even, 2 .. 512 (64 for DeepSeek-V3.2) */
    int32_t orig_ctx;   /* YaRN original context length L, >= 1 (4096) */
    double base;        /* RoPE base, finite and > 1 (10000) */
    double scale;       /* YaRN scaling factor s, finite and > 0 (40; 1 = plain RoPE) */
    double beta_fast;   /* ramp start, in rotations over L, finite and > 0 (32) */
    double beta_slow;   /* ramp end, in rotations over L, finite and > 0 (1) */
} gvr_rope_params;

/* Fill *params with the DeepSeek-V3.2 indexer values listed above. */
void gvr_rope_params_default(gvr_rope_params* params);

/* g(Delta) of Sec. 3.2 for Delta = 0 .. n-1.
 *   g:     [n] float64, written in full (may be NULL when n == 0).
 *   theta: [d/2] float64 receiving theta'_i, or NULL.
 * Errors: GVR_ERR_INVALID_ARG (n < 0, bad params, g NULL with n > 0),
 *         GVR_ERR_TOO_LONG (n > 2^31 - 16), GVR_ERR_HIP (launch failed). */
gvr_status gvr_rope_g(int64_t n, const gvr_rope_params* params, double* g, double* theta,
                      void* stream);

/* P_static of Sec. 3.3 over Delta = 0 .. n-1: g is computed into `g` (as by
 * gvr_rope_g, so the caller can read it afterwards) and the K largest values
 * are selected -- the lower Delta first among equal values (-0.0 counts as
 * +0.0) -- and written to out_delta[0 .. K) in ascending order; when n <= K
 * out_delta receives 0 .. n-1 followed by -1.
 *   g:         [n] float64 (may be NULL when n == 0).
 *   out_delta: [K] int32, written in full.
 * Errors: as gvr_rope_g, plus GVR_ERR_UNSUPPORTED_K (K < 1 or K > GVR_MAX_K)
 *         and GVR_ERR_INVALID_ARG for a NULL out_delta. */
gvr_status gvr_rope_prior(int64_t n, int32_t K, const gvr_rope_params* params, double* g,
                          int32_t* out_delta, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GVR_ROPE_PRIOR_H */
