/*
 * gvr_indexer.h -- decode-time indexer scores of DeepSeek Sparse Attention in
 * FP8 on MI355X (gfx950), and the indexer followed by gvr_topk.
 *
 * Sec. 2.1 (Eq. indexer): the index score of past token s for the current
 * query token is a weighted sum over the h indexer heads of the ReLU'd
 * query-key dot products,
 *     I[b][s] = sum_{j<H} w[b][j] * ReLU( q[b][j] . k'[g][s] ),
 *     k'[g][s] = k_scale[g][s] * k[g][s],   g = b / group,
 * with one key vector per token shared by all heads (MQA). Rows b of one
 * request share its key cache g: `group` consecutive rows per cache (the
 * speculative draft rows of one request, next_n of them). The K-th largest
 * I[b][s] over s < n_b are what the sparse attention keeps (K = 2048).
 *
 * Number formats:
 *   - q, k: FP8 E4M3 bytes in the OCP format (bias 7, no infinities,
 *     0x7F / 0xFF are NaN, largest finite 448), the format gfx950's matrix
 *     cores read. A query's own dequantisation scale is folded into w.
 *   - w, k_scale, I: float32. Products of two FP8 values are exact in
 *     float32; the dot products accumulate in float32 on the matrix cores,
 *     the head sum in float32, so I differs from the exact value by rounding
 *     only: |I - I_exact| <= (D + H + 4) 2^-24 sum_j |w_j| sum_d |q_jd k'_d|
 *     (D - 1 additions per dot product in any order, one rounding each for
 *     the key scale and the head weight, H - 1 head additions, and slack
 *     for second-order terms).
 *
 * Layouts (all DEVICE pointers, owned by the caller; row stride ld):
 *   q       [B][H][D] bytes        w       [B][H] f32
 *   k       [B/group][ld][D] bytes k_scale [B/group][ld] f32
 *   row_len [B] i32 or NULL (= ld; values clamped to [0, ld])
 *   scores  [B][ld] f32: I[b][s] written for s < n_b only
 * Supported shapes: H in {32, 64, 128}, D in {64, 128}, group in 1..4,
 * B a multiple of group, ld <= 2^31 - 16.
 *
 * Errors (reported before anything is enqueued): GVR_ERR_INVALID_ARG for a
 * NULL pointer, a negative size or an unsupported H, D or group;
 * GVR_ERR_TOO_LONG for ld > 2^31 - 16; GVR_ERR_HIP if a launch fails.
 * B == 0 is a no-op. Work is enqueued on `stream` (hipStream_t as void*);
 * the calls do not synchronise. gvr_indexer_scores allocates nothing and may
 * be captured into a HIP graph: the first call on a device sizes its grid
 * from the device's resident workgroup count (queried once, not during a
 * capture; a captured first call uses a fixed chunk size, same result).
 */
#ifndef GVR_INDEXER_H
#define GVR_INDEXER_H

#include <stdint.h>

#include "gvr_topk.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Index scores I (Sec. 2.1, Eq. indexer) for every row and every s < n_b:
 * one kernel on the matrix cores (gfx950's 16x16x128 FP8 matrix op), bound by
 * HBM on the key cache (D + 4 bytes per key and cache, 4 bytes written per
 * score). */
gvr_status gvr_indexer_scores(const uint8_t* q, const float* w, const uint8_t* k, const float* k_scale,
                              int64_t B, int32_t H, int32_t D, int32_t group, int64_t ld,
                              const int32_t* row_len, float* scores, void* stream);

/* The indexer, then gvr_topk_ex on its scores (same stream, back to back):
 * out_idx [B][K] receives the exact Top-K of every row of I (see
 * gvr_topk.h for the result definition, prev_topk, options and stats).
 * `scores` [B][ld] f32 is the caller's buffer for I and keeps it.
 *
 * Fused guess (Sec. 4.2.1, Phase 1): with a prev_topk, K >= 8 and the
 * default schedule (not option flag 4, not flag 1), the indexer kernel also
 * scores the keys at each row's strided sample of prev_topk (every
 * ceil(K / 256)-th entry) with the same matrix steps as the row's scores, so
 * the sampled scores equal the ones written, and reduces them to the row's
 * guess statistics (T_spec, valid samples, pmin, pmax, sample sum). It
 * leaves them in the last 8 words of the row's out_idx, where the Top-K
 * reads them instead of gathering the sample's scores after the indexer;
 * the Top-K then overwrites out_idx with the result. The answer, the row
 * stats and the path are those of gvr_topk_ex on the same scores and guess
 * (prev_topk may alias out_idx: each row's sample is read before its
 * statistics are written). */
gvr_status gvr_indexer_topk(const uint8_t* q, const float* w, const uint8_t* k, const float* k_scale,
                            int64_t B, int32_t H, int32_t D, int32_t group, int64_t ld,
                            const int32_t* row_len, float* scores, const int32_t* prev_topk, int32_t K,
                            int32_t* out_idx, void* stream, const gvr_options* options,
                            gvr_row_stats* stats);

#ifdef __cplusplus
}
#endif

#endif /* GVR_INDEXER_H */
