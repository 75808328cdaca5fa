// guess.h -- Phase 1 of Guess-Verify-Refine (Sec. 4.2.1) over the scores at
// a strided sample of the previous step's Top-K, as one wave computes it.
// Shared by the Top-K kernel (which gathers the sampled scores itself) and
// the indexer kernel (which scores the sampled keys while it computes the
// row, for gvr_indexer_topk), so both give the same T_spec bit for bit.
#ifndef GVR_GUESS_H
#define GVR_GUESS_H

#include "wave_ops.h"

namespace gvr_dev {

constexpr int kGuessSamples = 256;   // guessed indices used: every st-th entry of prev_topk, st = ceil(K / 256)
constexpr int kGuessBins = 1024;     // bins of the sampled-key histogram (16 per lane of one wave)
constexpr int kSpecQuantile = 65;    // T_spec: sampled key of rank ceil(65 / 2048 * samples) from the bottom
constexpr int kGuessMaxK = 2048;     // the quantile's denominator (the largest K)

// Sample stride and sample count for a Top-K of size K.
DEV int guess_stride(int K) { return (K + kGuessSamples - 1) / kGuessSamples; }
DEV int guess_count(int K) {
    const int st = guess_stride(K);
    return (K + st - 1) / st;
}

// The statistics of one row's sample: T_spec (0xFFFFFFFF without a valid
// sample), the number of valid samples, their smallest and largest key, and
// the sum of their values (for pmean; summed in a fixed order).
struct GuessStats {
    uint32_t ts;
    int cnt;
    uint32_t mn, mx;
    float sum;
};

// Words of a row's GuessStats as gvr_indexer_topk hands them to the Top-K.
constexpr int kGuessWords = 8;

// One wave: lane l holds samples l + 64 c (c < 4), value gv[c], valid ok[c].
// T_spec is the lower edge of the histogram bin (kGuessBins bins over
// [pmin, pmax]) holding the valid sample of rank ceil(65 m / 2048) from the
// bottom (m valid samples), at least key 1. gh: kGuessBins ints of LDS this
// wave owns (cleared here; a wave's LDS accesses complete in order).
DEV GuessStats guess_from_samples(const float (&gv)[4], const bool (&ok)[4], int* gh) {
    uint32_t gk[4];
    int cnt = 0;
    uint32_t mn = 0xFFFFFFFFu, mx = 0u;
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        gk[c] = key_of(gv[c]);
        if (ok[c]) {
            mn = min(mn, gk[c]);
            mx = max(mx, gk[c]);
            sum += gv[c];
            ++cnt;
        }
    }
    cnt = wave_sum(cnt);
    mn = wave_min_u(mn);
    mx = wave_max_u(mx);
    sum = wave_sum_f(sum);
    uint32_t ts = 0xFFFFFFFFu;
    if (cnt > 0) {
        const int lane = (int)__lane_id();
        const uint64_t width = (uint64_t)mx - mn + 1;
        const uint32_t sh = bin_shift(width, log2i(kGuessBins));
        int4* h4 = reinterpret_cast<int4*>(gh) + lane * 4;   // lane owns 16 bins
#pragma unroll
        for (int j = 0; j < 4; ++j) h4[j] = make_int4(0, 0, 0, 0);
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (ok[c]) __hip_atomic_fetch_add(&gh[(gk[c] - mn) >> sh], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        int h[16];
        int s16 = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int4 v = h4[j];
            h[4 * j] = v.x;
            h[4 * j + 1] = v.y;
            h[4 * j + 2] = v.z;
            h[4 * j + 3] = v.w;
            s16 += v.x + v.y + v.z + v.w;
        }
        const int target = max(1, (kSpecQuantile * cnt + kGuessMaxK - 1) / kGuessMaxK);
        const int incl = wave_incl_scan(s16, lane);
        const int excl = incl - s16;
        const uint64_t hit = __ballot(excl < target && incl >= target);
        const int L = hit ? (int)__builtin_ctzll(hit) : 0;
        int jsel = 0, run = excl;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if (run < target && run + h[j] >= target) jsel = j;
            run += h[j];
        }
        jsel = __builtin_amdgcn_readlane(jsel, L);
        ts = mn + ((uint32_t)(L * 16 + jsel) << sh);
    }
    return GuessStats{ts, cnt, mn, mx, sum};
}

}  // namespace gvr_dev

#endif  // GVR_GUESS_H
