// wave_ops.h -- wave64 building blocks shared by the Top-K and the indexer
// kernels (gfx950): sortable keys of fp32 values, lane masks, DPP wave
// reductions and scans, histogram bin shifts.
#ifndef GVR_WAVE_OPS_H
#define GVR_WAVE_OPS_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#ifndef DEV
#define DEV __device__ __forceinline__
#endif

namespace gvr_dev {

constexpr int kWave = 64;

// Sortable key of an fp32 bit pattern: flip every bit of a negative value,
// the sign bit of the rest (unsigned key order = value order, -0 < +0, NaNs
// at the ends by sign).
DEV uint32_t key_of_bits(uint32_t u) { return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u); }
DEV uint32_t key_of(float v) { return key_of_bits(__float_as_uint(v)); }
DEV float float_of_key(uint32_t k) { return __uint_as_float((k & 0x80000000u) ? (k ^ 0x80000000u) : ~k); }

// Mask of lanes [0, r) for any r (wave-uniform): scalar instructions only.
DEV uint64_t first_lanes(int r) { return r >= kWave ? ~0ull : (r <= 0 ? 0ull : (1ull << r) - 1ull); }

// Number of set bits of m below this lane, plus acc.
DEV uint32_t lanes_below(uint64_t m, uint32_t acc) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, acc));
}

// Wave-wide reductions and scans with DPP (VALU lane moves, no LDS round
// trip): quad_perm / row_half_mirror / row_mirror combine the 16 lanes of a
// row, readlane combines the four rows; every lane gets the result.
template <int CTRL, int ROW_MASK = 0xF>
DEV int dpp_i(int old, int x) {
    return __builtin_amdgcn_update_dpp(old, x, CTRL, ROW_MASK, 0xF, false);
}
constexpr int kQuadSwap1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kQuadSwap2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;
constexpr int kRowShr1 = 0x111;
constexpr int kRowBcast15 = 0x142;
constexpr int kRowBcast31 = 0x143;

DEV int wave_sum(int v) {
    v += dpp_i<kQuadSwap1>(0, v);
    v += dpp_i<kQuadSwap2>(0, v);
    v += dpp_i<kRowHalfMirror>(0, v);
    v += dpp_i<kRowMirror>(0, v);
    return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) + __builtin_amdgcn_readlane(v, 32) +
           __builtin_amdgcn_readlane(v, 48);
}
DEV float wave_sum_f(float v) {
    // fixed combination order: pairs, quads, halves, rows, then rows 0..3
    v += __int_as_float(dpp_i<kQuadSwap1>(0, __float_as_int(v)));
    v += __int_as_float(dpp_i<kQuadSwap2>(0, __float_as_int(v)));
    v += __int_as_float(dpp_i<kRowHalfMirror>(0, __float_as_int(v)));
    v += __int_as_float(dpp_i<kRowMirror>(0, __float_as_int(v)));
    return ((__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)) +
             __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16))) +
            __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32))) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
}
DEV uint32_t wave_min_u(uint32_t v) {
    v = min(v, (uint32_t)dpp_i<kQuadSwap1>(0, (int)v));
    v = min(v, (uint32_t)dpp_i<kQuadSwap2>(0, (int)v));
    v = min(v, (uint32_t)dpp_i<kRowHalfMirror>(0, (int)v));
    v = min(v, (uint32_t)dpp_i<kRowMirror>(0, (int)v));
    return min(min((uint32_t)__builtin_amdgcn_readlane((int)v, 0), (uint32_t)__builtin_amdgcn_readlane((int)v, 16)),
               min((uint32_t)__builtin_amdgcn_readlane((int)v, 32), (uint32_t)__builtin_amdgcn_readlane((int)v, 48)));
}
DEV uint32_t wave_max_u(uint32_t v) {
    v = max(v, (uint32_t)dpp_i<kQuadSwap1>(0, (int)v));
    v = max(v, (uint32_t)dpp_i<kQuadSwap2>(0, (int)v));
    v = max(v, (uint32_t)dpp_i<kRowHalfMirror>(0, (int)v));
    v = max(v, (uint32_t)dpp_i<kRowMirror>(0, (int)v));
    return max(max((uint32_t)__builtin_amdgcn_readlane((int)v, 0), (uint32_t)__builtin_amdgcn_readlane((int)v, 16)),
               max((uint32_t)__builtin_amdgcn_readlane((int)v, 32), (uint32_t)__builtin_amdgcn_readlane((int)v, 48)));
}
// Inclusive prefix sum over the 64 lanes: Hillis-Steele shifts inside each
// 16-lane row (lanes without a source add 0), then row_bcast:15 / :31 carry
// the row totals into the rows above.
DEV int wave_incl_scan(int v, int /*lane*/) {
    v += dpp_i<kRowShr1>(0, v);
    v += dpp_i<kRowShr1 + 1>(0, v);
    v += dpp_i<kRowShr1 + 3>(0, v);
    v += dpp_i<kRowShr1 + 7>(0, v);
    v += dpp_i<kRowBcast15, 0xA>(0, v);
    v += dpp_i<kRowBcast31, 0xC>(0, v);
    return v;
}
// Smallest s with (2^lg_bins << s) >= width, for 1 <= width <= 2^32: bins of
// 2^s keys from the window's low edge cover `width` keys.
DEV uint32_t bin_shift(uint64_t width, int lg_bins) {
    const int bits = 64 - __builtin_clzll(width - 1 | 1);   // bit length of width - 1 (>= 1)
    return (uint32_t)max(0, (width <= 1 ? 0 : bits) - lg_bins);
}
constexpr int log2i(int v) { return v <= 1 ? 0 : 1 + log2i(v / 2); }

}  // namespace gvr_dev

#endif  // GVR_WAVE_OPS_H
