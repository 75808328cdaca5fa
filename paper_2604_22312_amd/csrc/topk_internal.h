// topk_internal.h -- library-internal entry of the Top-K for the fused
// indexer path (gvr_indexer_topk); not part of the C ABI.
#ifndef GVR_TOPK_INTERNAL_H
#define GVR_TOPK_INTERNAL_H

#include <stdint.h>

#include "gvr_topk.h"

namespace gvr_internal {

// gvr_topk_ex whose rows take their guess statistics (T_spec, valid sample
// count, pmin, pmax and the sample sum as gvr_dev::GuessStats words) from
// the last gvr_dev::kGuessWords words of each out_idx row, where the
// indexer wrote them, instead of gathering the scores at prev_topk's
// sample; out_idx is then overwritten by the result. Needs K >= kGuessWords.
gvr_status topk_with_guess_stats(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                                 const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                                 const gvr_options* options, gvr_row_stats* stats);

}  // namespace gvr_internal

#endif  // GVR_TOPK_INTERNAL_H
