// gvr_topk.hip -- Guess-Verify-Refine exact Top-K and radix-select Top-K for
// MI355X (gfx950), behind the C ABI declared in include/gvr_topk.h.
//
// One workgroup (1024 threads, 16 wave64s) owns one row; rows never talk to
// each other, so a call is a single ordinary launch with one workgroup per
// row and no device workspace. Each wave streams a contiguous sub-range of
// the row with a rolling window of dwordx4 loads (8 slabs of 1 KB in flight
// per wave), so the candidates it keeps are in ascending index order.
//
//   Guess (Sec. 4.2.1, Phase 1). While the first slabs of the row are in
//   flight, the workgroup gathers the row's scores at prev_topk and reduces
//   them to pmin / pmax (and pmean, reported in the stats). A small LDS
//   histogram of the gathered keys gives T_spec, the 65th-smallest gathered
//   key: a threshold that the previous step's Top-K makes likely to hold a
//   few thousand elements of the current row, i.e. inside [K, C].
//
//   Threshold search (Sec. 4.2.2, Phase 2). The first full-row pass counts
//   f(T) = #{key >= T} (Sec. 4.1) at every edge of a 256-bin window over
//   [pmin, pmax] of key space (wave-private LDS histograms: the count cache),
//   and so evaluates 257 thresholds in one sweep instead of one.
//
//   Collect (Sec. 4.2.3, Phase 3). In the same sweep every element with
//   key >= T_spec is appended to its wave's LDS list (ballot + mbcnt ranks,
//   no atomics). If K <= f(T_spec) <= C, Lemma 1 (Sec. 4.1) says the lists
//   hold the exact answer and the row is never read again.
//
//   Refine (Sec. 4.2.4, Phase 4). The window histogram names the bin that
//   holds the K-th key; a 2048-bin LDS histogram over the listed keys in that
//   bin narrows it to the exact K-th key T* (two levels for a ~3-binade
//   window). Every key > T* and the first K - #{key > T*} keys equal to T*
//   (lower index first) are written out in ascending index order.
//
//   When the guess does not deliver (no valid prev_topk, f(T_spec) < K, or a
//   wave's list overflows) the row is streamed again: count passes narrow a
//   256-bin window around the K-th key (8 bits of key per pass), then one
//   collect pass gathers the <= C candidates at the accepted threshold with
//   exact per-wave offsets from the count cache, or, when ties straddle
//   [K, C], an emit pass writes the selection directly. radix_topk runs only
//   this path, starting from the whole key range: a distribution-agnostic
//   radix select (Sec. 2.2).

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>

#include "gvr_topk.h"

#define DEV __device__ __forceinline__

namespace {

constexpr int kBlock = 1024;
constexpr int kWave = 64;
constexpr int kNW = kBlock / kWave;            // 16 waves
constexpr int kU = 8;                          // slabs in flight per wave
constexpr int kBins = 256;                     // bins of a counting window
constexpr int kBinsX = kBins + 1;              // + "at or above the window"
constexpr int kCap = GVR_MAX_CANDIDATES;       // list capacity (LDS)
constexpr int kCapW = kCap / kNW;              // per-wave list capacity, first pass
constexpr int kRefBins = 4096;                 // bins of a refine level (12 bits of key)
constexpr int kGuessBins = kBlock;             // bins of the gathered-key histogram (1 per thread)
constexpr int kGuessPerThread = (GVR_MAX_K + kBlock - 1) / kBlock;
constexpr int kSpecRank = 64;                  // T_spec = gathered key of this rank from the bottom
constexpr int kMaxPasses = 8;                  // 2 + at most 4 narrowing passes + 1 final pass suffice

static_assert(GVR_MAX_CANDIDATES % kNW == 0, "per-wave capacity");

struct Params {
    const float* scores;
    int64_t ld;
    const int32_t* row_len;
    const int32_t* prev;
    int32_t* out;
    gvr_row_stats* stats;
    int32_t K;
    int32_t capacity;    // C
    int32_t use_guess;   // 0: radix schedule
};

// ------------------------------------------------------------------ helpers

DEV uint32_t key_of_bits(uint32_t u) { return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u); }
DEV uint32_t key_of(float v) { return key_of_bits(__float_as_uint(v)); }

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
// Lane v of every wave reads wave v's value: one LDS read + one wave
// reduction per cross-wave sum.
DEV int sum_over_waves(const int* vals, int lane) { return wave_sum(lane < kNW ? vals[lane] : 0); }
DEV int sum_over_waves_below(const int* vals, int lane, int wave) { return wave_sum(lane < wave ? vals[lane] : 0); }

DEV int64_t stamp() { return (int64_t)__builtin_amdgcn_s_memtime(); }

// A window of key space: bins j < kBins cover [lo + j<<shift, lo + (j+1)<<shift);
// bin kBins holds every key >= lo + kBins<<shift; keys below lo are not counted.
struct Window {
    uint32_t lo;
    uint32_t shift;
};
DEV Window make_window(uint32_t a, uint32_t b) {   // covers [a, b], b >= a
    const uint64_t width = (uint64_t)b - a + 1;
    uint32_t s = 0;
    while (((uint64_t)kBins << s) < width) ++s;
    return Window{a, s};
}
DEV uint64_t edge_of(const Window& w, int j) { return (uint64_t)w.lo + ((uint64_t)j << w.shift); }

// ------------------------------------------------------------------ LDS
struct Smem {
    uint2 list[kCap];                   // candidates (key, index), per-wave segments
    union {
        int hist[kNW][kBinsX];          // wave-private counting histograms
        int rhist[kRefBins];            // refine / guess histogram
    } u;
    int F[kBinsX + 1];                  // F[j] = f(edge j) over the row
    uint2 dummy[kBlock];                // sink of the unconditional list stores
    int seg_off[kNW];                   // list segment of each wave
    int seg_cnt[kNW];
    int wa[kNW];
    int wb[kNW];
    int red[4][kNW];
    float redf[kNW];
    int scal[8];
};

// Block-wide exclusive scan of one int (all kBlock threads). Returns the total.
DEV int block_excl_scan(int& a, Smem& sm, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    const int ia = wave_incl_scan(a, lane);
    if (lane == kWave - 1) sm.wa[wave] = ia;
    __syncthreads();
    const int before = sum_over_waves_below(sm.wa, lane, wave);
    const int tot = sum_over_waves(sm.wa, lane);
    __syncthreads();
    a = before + ia - a;
    return tot;
}

// ------------------------------------------------------------------ streaming
// One wave streams float4 blocks [qb, qe) of the row in slabs of 64 blocks
// with kU slabs in flight; `body(v, q, qs)` gets each lane's block q, its data
// and the slab's first block qs. Every block index is clamped to qlast, so no
// load leaves the 16-byte blocks that hold the row (refills past the wave's
// last slab re-read the row's last block and are never used); bodies mask
// elements outside [0, n) themselves. `prologue()` runs once after the first
// loads are issued. The refill of a buffer slot is issued after its slab is
// consumed and unconditionally, so each slot keeps one register set and a
// slab waits only for its own load (vmcnt(kU - 1)), not for all of them.
template <typename Pro, typename Body>
DEV void stream_wave(const float4* __restrict__ xa, int qb, int qe, int qlast, int lane, Pro&& prologue,
                     Body&& body) {
    const int nslab = qe > qb ? (qe - qb + 63) >> 6 : 0;
    float4 buf[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) buf[u] = xa[min(qb + u * 64 + lane, qlast)];
    prologue();
    int s0 = 0;
    for (; s0 + kU <= nslab; s0 += kU) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int s = s0 + u;
            body(buf[u], qb + s * 64 + lane, qb + s * 64);
            buf[u] = xa[min(qb + (s + kU) * 64 + lane, qlast)];
        }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u)
        if (s0 + u < nslab) body(buf[u], qb + (s0 + u) * 64 + lane, qb + (s0 + u) * 64);
}

// Count key k (if `in`) into bin min((k - lo) >> sh, kBins) of a wave-private
// histogram. With AGG, lanes sharing the first active lane's bin add in one
// atomic: wide (radix) windows map most keys of a wave to a few bins, and
// same-address LDS atomics serialise.
template <bool AGG>
DEV void hist_add(int* hw, uint32_t k, bool in, uint32_t lo, uint32_t sh) {
    const uint32_t b = min((k - lo) >> sh, (uint32_t)kBins);
    if (!AGG) {
        if (in) __hip_atomic_fetch_add(&hw[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        return;
    }
    const uint64_t act = __ballot(in);
    if (!act) return;
    const uint32_t lead = __builtin_amdgcn_readlane(b, (int)__builtin_ctzll(act));
    const uint64_t same = __ballot(in && b == lead);
    if (in && b == lead) {
        if (lanes_below(same, 0) == 0)
            __hip_atomic_fetch_add(&hw[lead], (int)__popcll(same), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    } else if (in) {
        __hip_atomic_fetch_add(&hw[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
}

DEV void block_keys(const float4& v, uint32_t (&k)[4]) {
    k[0] = key_of(v.x);
    k[1] = key_of(v.y);
    k[2] = key_of(v.z);
    k[3] = key_of(v.w);
}

// ------------------------------------------------------------------ refine
// Exact K-th key among the listed candidates. The K-th key lies in
// [wlo, whi]; `above` listed candidates lie above whi. Wave w's list segment
// is list[seg_off[w] .. + seg_cnt[w]).
DEV uint32_t refine_kth(Smem& sm, uint32_t wlo, uint32_t whi, int above, int K, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    int need = K - above;   // >= 1
    for (int level = 0; level < 4 && wlo != whi; ++level) {
        const uint64_t width = (uint64_t)whi - wlo + 1;
        uint32_t s = 0;
        while (((uint64_t)kRefBins << s) < width) ++s;
        for (int i = tid; i < kRefBins; i += kBlock) sm.u.rhist[i] = 0;
        __syncthreads();
        {
            const uint2* seg = sm.list + sm.seg_off[wave];
            const int cnt = sm.seg_cnt[wave];
            for (int i = lane; i < cnt; i += kWave) {
                const uint32_t kk = seg[i].x;
                if (kk >= wlo && kk <= whi)
                    __hip_atomic_fetch_add(&sm.u.rhist[(kk - wlo) >> s], 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
        __syncthreads();
        constexpr int PER = kRefBins / kBlock;   // 4 bins per thread
        int loc[PER];
        int mine = 0;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            loc[q] = sm.u.rhist[tid * PER + q];
            mine += loc[q];
        }
        int a = mine;
        const int tot = block_excl_scan(a, sm, tid);
        int run = tot - a - mine;   // bins above this thread's range
        if (tid == 0) sm.scal[0] = -1;
        __syncthreads();
#pragma unroll
        for (int q = PER - 1; q >= 0; --q) {
            const int nr = run + loc[q];
            if (run < need && nr >= need) {
                sm.scal[0] = tid * PER + q;
                sm.scal[1] = run;
            }
            run = nr;
        }
        __syncthreads();
        const int b = sm.scal[0];
        const int ab = sm.scal[1];
        __syncthreads();
        if (b < 0) break;   // cannot happen for consistent counts; keeps every path finite
        need -= ab;
        const uint64_t nlo = (uint64_t)wlo + ((uint64_t)b << s);
        uint64_t nhi = nlo + ((uint64_t)1 << s) - 1;
        if (nhi > whi) nhi = whi;
        wlo = (uint32_t)nlo;
        whi = (uint32_t)nhi;
    }
    return wlo;
}

// Write the selection from the lists: every key > T, then the first `take`
// keys == T in list (= index) order; output in ascending index order.
DEV void emit_from_lists(Smem& sm, uint32_t T, int K, int32_t* out, int tid, int* n_gt_out) {
    const int lane = tid & 63, wave = tid >> 6;
    const uint2* seg = sm.list + sm.seg_off[wave];
    const int cnt = sm.seg_cnt[wave];
    int gt = 0, eq = 0;
    for (int i = lane; i < cnt; i += kWave) {
        const uint32_t kk = seg[i].x;
        gt += kk > T;
        eq += kk == T;
    }
    gt = wave_sum(gt);
    eq = wave_sum(eq);
    if (lane == 0) {
        sm.wa[wave] = gt;
        sm.wb[wave] = eq;
    }
    __syncthreads();
    int gb = sum_over_waves_below(sm.wa, lane, wave);
    int eb = sum_over_waves_below(sm.wb, lane, wave);
    const int gtot = sum_over_waves(sm.wa, lane);
    const int take = K - gtot;
    for (int i0 = 0; i0 < cnt; i0 += kWave) {
        const int i = i0 + lane;
        uint32_t kk = 0;
        int idx = 0;
        if (i < cnt) {
            kk = seg[i].x;
            idx = (int)seg[i].y;
        }
        const bool fg = i < cnt && kk > T;
        const bool fe = i < cnt && kk == T;
        const uint64_t mg = __ballot(fg), me = __ballot(fe);
        const int g = gb + (int)lanes_below(mg, 0), e = eb + (int)lanes_below(me, 0);
        if (fg) {
            const int o = g + min(e, take);
            if (o >= 0 && o < K) out[o] = idx;
        } else if (fe && e < take) {
            const int o = g + e;
            if (o >= 0 && o < K) out[o] = idx;
        }
        gb += __popcll(mg);
        eb += __popcll(me);
    }
    *n_gt_out = gtot;
}

// ------------------------------------------------------------------ kernel
__global__ __launch_bounds__(kBlock) void topk_row_kernel(Params p) {
    __shared__ Smem sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const int64_t t0 = stamp();

    int64_t n64 = p.row_len ? (int64_t)p.row_len[row] : p.ld;
    n64 = n64 < 0 ? 0 : (n64 > p.ld ? p.ld : n64);
    const int n = (int)n64;
    const int K = p.K;
    const float* x = p.scores + row * p.ld;
    int32_t* out = p.out + row * (int64_t)K;
    gvr_row_stats* st = p.stats ? p.stats + row : nullptr;

    // (a1) row classify: n <= K -> 0..n-1 then -1 padding.
    if (n <= K) {
        for (int i = tid; i < K; i += kBlock) out[i] = (i < n) ? i : -1;
        if (st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = GVR_PATH_TRIVIAL;
            s.t_start = t0;
            s.t_refine = stamp();
            *st = s;
        }
        return;
    }

    // Float4 blocks of the row (virtual index = element index + aoff, so a
    // block is one aligned 16-byte load) and this wave's contiguous share.
    const int aoff = (int)(((uintptr_t)x >> 2) & 3);
    const float4* xa = reinterpret_cast<const float4*>(x - aoff);
    const int nq = (n + aoff + 3) >> 2;
    const int qlast = nq - 1;
    const int per = ((nq + kNW - 1) / kNW + 63) & ~63;   // whole slabs per wave
    const int qb = min(wave * per, nq), qe = min(qb + per, nq);
    const int cap = p.capacity;
    const bool all_mode = (n <= cap) && (per * 4 <= kCapW);   // every element is a candidate

    // ---------------- pass 1 parameters and state
    bool have_prev = p.use_guess && p.prev && !all_mode;
    int gvalid = 0;
    uint32_t gmin = 0xFFFFFFFFu, gmax = 0u, tspec = 0xFFFFFFFFu;
    float gsum = 0.f;
    Window win = make_window(0u, 0xFFFFFFFFu);
    bool spec = all_mode || have_prev;   // pass 1 collects key >= tspec (else: counts)
    int cnt_w = 0;              // this wave's elements >= tspec (counted past capacity)
    int64_t t1 = t0;

    // The guess indices are loaded before the first slabs (8 KB per row), so
    // they return first; the gathers x[prev] go out right behind the slabs.
    int pq[kGuessPerThread];
    if (have_prev) {
        const int32_t* pv = p.prev + row * (int64_t)K;
#pragma unroll
        for (int m = 0; m < kGuessPerThread; ++m) {
            const int j = tid + m * kBlock;
            pq[m] = (j < K) ? pv[j] : -1;
        }
    }
    if (!spec)
        for (int i = tid; i < kNW * kBinsX; i += kBlock) (&sm.u.hist[0][0])[i] = 0;
    if (tid < kNW) sm.seg_off[tid] = tid * kCapW;
    // Guess statistics (Phase 1), run while the first slabs are in flight.
    auto prologue = [&]() {
        if (all_mode) {
            tspec = 0u;
        } else if (have_prev) {
            float gv[kGuessPerThread];
            uint32_t gk[kGuessPerThread];
            bool ok[kGuessPerThread];
#pragma unroll
            for (int m = 0; m < kGuessPerThread; ++m) {
                ok[m] = pq[m] >= 0 && pq[m] < n;
                gv[m] = ok[m] ? x[pq[m]] : 0.f;
            }
#pragma unroll
            for (int m = 0; m < kGuessPerThread; ++m) {
                gk[m] = key_of(gv[m]);
                if (ok[m]) {
                    gmin = min(gmin, gk[m]);
                    gmax = max(gmax, gk[m]);
                    gsum += gv[m];
                    ++gvalid;
                }
            }
            gvalid = wave_sum(gvalid);
            gmin = wave_min_u(gmin);
            gmax = wave_max_u(gmax);
            gsum = wave_sum_f(gsum);
            if (lane == 0) {
                sm.red[0][wave] = gvalid;
                sm.red[1][wave] = (int)gmin;
                sm.red[2][wave] = (int)gmax;
                sm.redf[wave] = gsum;
            }
            for (int i = tid; i < kGuessBins; i += kBlock) sm.u.rhist[i] = 0;
            if (tid == 0) sm.scal[0] = 0;
            __syncthreads();
            gvalid = sum_over_waves(sm.red[0], lane);
            gmin = wave_min_u(lane < kNW ? (uint32_t)sm.red[1][lane] : 0xFFFFFFFFu);
            gmax = wave_max_u(lane < kNW ? (uint32_t)sm.red[2][lane] : 0u);
            gsum = 0.f;
            for (int v = 0; v < kNW; ++v) gsum += sm.redf[v];   // pmean: fixed order
            if (gvalid > 0) {
                // T_spec: lower edge of the histogram bin (over [pmin, pmax])
                // holding the (kSpecRank + 1)-th smallest gathered key.
                const uint64_t width = (uint64_t)gmax - gmin + 1;
                uint32_t sh = 0;
                while (((uint64_t)kGuessBins << sh) < width) ++sh;
#pragma unroll
                for (int m = 0; m < kGuessPerThread; ++m)
                    if (ok[m])
                        __hip_atomic_fetch_add(&sm.u.rhist[(gk[m] - gmin) >> sh], 1, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_WORKGROUP);
                __syncthreads();
                // thread t owns bin t; a block scan finds the bin holding the target
                const int cnt = sm.u.rhist[tid];
                int below = cnt;
                block_excl_scan(below, sm, tid);
                const int target = min(kSpecRank + 1, gvalid);
                if (below < target && below + cnt >= target) sm.scal[0] = tid;
                __syncthreads();
                tspec = gmin + ((uint32_t)sm.scal[0] << sh);
            } else {
                tspec = 0xFFFFFFFFu;   // no usable guess: pass 1 keeps nothing useful
                have_prev = false;
            }
        }
        __syncthreads();
        t1 = stamp();
    };

    // ---------------- pass 1: speculative collect (or the first count pass)
    int* hw = sm.u.hist[wave];
    uint2* lw = sm.list + wave * kCapW;
    // Append the listed elements of one lane's block (keys k, first index e0)
    // whose key is >= tspec (and, in edge slabs, lies in [0, n)).
    // Lanes whose element is not kept write to a private dummy slot, so the
    // four stores of a slab need no exec-mask juggling; one capacity check per
    // slab (wave-uniform) replaces per-element checks.
    uint2* const dummy = sm.dummy + tid;
    auto collect = [&](const uint32_t (&k)[4], int e0, bool edge) {
        const bool v0 = !edge || (e0 >= 0 && e0 < n), v1 = !edge || (e0 + 1 >= 0 && e0 + 1 < n);
        const bool v2 = !edge || (e0 + 2 >= 0 && e0 + 2 < n), v3 = !edge || (e0 + 3 >= 0 && e0 + 3 < n);
        const bool f0 = v0 && k[0] >= tspec, f1 = v1 && k[1] >= tspec;
        const bool f2 = v2 && k[2] >= tspec, f3 = v3 && k[3] >= tspec;
        const uint64_t m0 = __ballot(f0), m1 = __ballot(f1), m2 = __ballot(f2), m3 = __ballot(f3);
        const int total = __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
        cnt_w = __builtin_amdgcn_readfirstlane(cnt_w);   // wave-uniform: keep it scalar
        if (cnt_w + total <= kCapW) {
            int p = cnt_w + (int)lanes_below(m3, lanes_below(m2, lanes_below(m1, lanes_below(m0, 0))));
            *(f0 ? lw + p : dummy) = make_uint2(k[0], (uint32_t)e0);
            p += f0;
            *(f1 ? lw + p : dummy) = make_uint2(k[1], (uint32_t)(e0 + 1));
            p += f1;
            *(f2 ? lw + p : dummy) = make_uint2(k[2], (uint32_t)(e0 + 2));
            p += f2;
            *(f3 ? lw + p : dummy) = make_uint2(k[3], (uint32_t)(e0 + 3));
        }
        cnt_w += total;   // counted past capacity: the overflow is detected later
    };
    stream_wave(xa, qb, qe, qlast, lane, prologue, [&](const float4& v, int q, int qs) {
        uint32_t k[4];
        block_keys(v, k);
        const int e0 = 4 * q - aoff;
        const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);   // wave-uniform
        if (spec) {
            if (edge) collect(k, e0, true);
            else collect(k, e0, false);
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                hist_add<true>(hw, k[c], !edge || (e0 + c >= 0 && e0 + c < n), 0u, win.shift);
        }
    });
    int passes = 1;
    int f_spec = 0;
    bool overflow = false;
    if (spec) {
        if (lane == 0) {
            sm.seg_cnt[wave] = min(cnt_w, kCapW);
            sm.wa[wave] = cnt_w;
        }
        __syncthreads();
        f_spec = sum_over_waves(sm.wa, lane);
        overflow = wave_max_u(lane < kNW ? (uint32_t)sm.wa[lane] : 0u) > (uint32_t)kCapW;
        __syncthreads();
    }

    // Row totals per bin and F[j] = f(edge j) = sum_{b >= j} G[b].
    auto compute_F = [&]() {
        __syncthreads();   // every wave's histogram updates are done
        int g = 0;
        const int b = kBins - tid;   // thread t owns bin kBins - t (t < kBinsX)
        if (b >= 0)
            for (int v = 0; v < kNW; ++v) g += sm.u.hist[v][b];
        int a = g;
        block_excl_scan(a, sm, tid);
        if (b >= 0) sm.F[b] = a + g;
        if (tid == 0) sm.F[kBinsX] = 0;
        __syncthreads();
    };
    // Largest bin j with F[j] >= K (-1 if F[0] < K).
    auto crossing = [&]() {
        if (tid == 0) sm.scal[2] = -1;
        __syncthreads();
        if (tid < kBinsX && sm.F[tid] >= K && sm.F[tid + 1] < K) sm.scal[2] = tid;
        __syncthreads();
        const int j = sm.scal[2];
        __syncthreads();
        return j;
    };
    // Count pass over window `win` (wave-private histograms, then F).
    auto count_pass = [&]() {
        __syncthreads();
        for (int i = tid; i < kNW * kBinsX; i += kBlock) (&sm.u.hist[0][0])[i] = 0;
        __syncthreads();
        const uint32_t lo = win.lo, sh = win.shift;
        stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
            uint32_t k[4];
            block_keys(v, k);
            const int e0 = 4 * q - aoff;
            const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const bool ok = !edge || (e0 + c >= 0 && e0 + c < n);
                hist_add<true>(hw, k[c], ok && k[c] >= lo, lo, sh);
            }
        });
        ++passes;
        __syncthreads();
        compute_F();
    };

    int path = all_mode ? GVR_PATH_ALL : (have_prev ? GVR_PATH_GUESS : GVR_PATH_NO_GUESS);
    uint32_t T = 0, rlo = 0, rhi = 0xFFFFFFFFu;
    int above = 0, cands = 0;
    bool done_lists = false;   // lists hold every key >= T
    bool ties = false;
    uint32_t tstar = 0;
    int n_gt_row = 0;
    int64_t t2 = t1, t3 = t1;

    if (spec && !overflow && f_spec >= K && f_spec <= cap) {
        // The speculative lists hold every key >= T_spec, hence the answer
        // (Lemma 1); the refine window is the range of the listed keys.
        T = tspec;
        cands = f_spec;
        done_lists = true;
        uint32_t mn = 0xFFFFFFFFu, mx = 0u;
        {
            const uint2* seg = sm.list + sm.seg_off[wave];
            const int cnt = sm.seg_cnt[wave];
            for (int i = lane; i < cnt; i += kWave) {
                mn = min(mn, seg[i].x);
                mx = max(mx, seg[i].x);
            }
            mn = wave_min_u(mn);
            mx = wave_max_u(mx);
            if (lane == 0) {
                sm.red[1][wave] = (int)mn;
                sm.red[2][wave] = (int)mx;
            }
            __syncthreads();
            mn = wave_min_u(lane < kNW ? (uint32_t)sm.red[1][lane] : 0xFFFFFFFFu);
            mx = wave_max_u(lane < kNW ? (uint32_t)sm.red[2][lane] : 0u);
        }
        rlo = mn;
        rhi = mx;
        above = 0;
    } else {
        if (spec) {
            // The guess fell short (or a wave's list overflowed): count passes
            // around T_spec, whose f is known, then collect or emit.
            if (path == GVR_PATH_GUESS) path = GVR_PATH_NARROWED;
            win = (f_spec < K) ? make_window(0u, tspec - 1u) : make_window(tspec, 0xFFFFFFFFu);
            count_pass();
        } else {
            compute_F();   // pass 1 was the first count pass (whole key range)
        }
        for (;;) {
            const int j = crossing();
            int decision = 2;   // 0 collect, 1 ties, 2 narrow
            Window nw = win;
            if (j < 0) {
                nw = make_window(0u, win.lo - 1u);   // K-th key below the window
            } else if (sm.F[j] <= cap) {
                decision = 0;
            } else if (j == kBins) {
                nw = make_window((uint32_t)edge_of(win, kBins), 0xFFFFFFFFu);
            } else if (win.shift == 0) {
                decision = 1;
            } else {
                const uint64_t e = edge_of(win, j);
                nw = make_window((uint32_t)e,
                                 (uint32_t)std::min<uint64_t>(e + ((uint64_t)1 << win.shift) - 1, 0xFFFFFFFFu));
            }
            if (decision == 2 && passes >= kMaxPasses) decision = -1;
            if (decision == 0) {
                // Collect pass at T = edge j with exact per-wave offsets.
                const uint64_t e = edge_of(win, j);
                T = (uint32_t)e;
                cands = sm.F[j];
                rlo = T;
                rhi = (j < kBins) ? (uint32_t)std::min<uint64_t>(e + ((uint64_t)1 << win.shift) - 1, 0xFFFFFFFFu)
                                  : 0xFFFFFFFFu;
                above = (j < kBins) ? sm.F[j + 1] : 0;
                int mine = 0;
                for (int b = j + lane; b < kBinsX; b += kWave) mine += sm.u.hist[wave][b];
                mine = wave_sum(mine);
                if (lane == 0) sm.wa[wave] = mine;
                __syncthreads();
                const int off = sum_over_waves_below(sm.wa, lane, wave);
                __syncthreads();
                if (lane == 0) {
                    sm.seg_off[wave] = off;
                    sm.seg_cnt[wave] = mine;
                }
                __syncthreads();
                uint2* lc = sm.list + off;
                int run = 0;
                stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
                    uint32_t k[4];
                    block_keys(v, k);
                    const int e0 = 4 * q - aoff;
                    bool f[4];
                    uint64_t m[4];
                    const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        f[c] = k[c] >= T && (!edge || (e0 + c >= 0 && e0 + c < n));
                        m[c] = __ballot(f[c]);
                    }
                    int pos = run + (int)lanes_below(m[3], lanes_below(m[2], lanes_below(m[1], lanes_below(m[0], 0))));
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if (f[c]) {
                            if (pos < mine) lc[pos] = make_uint2(k[c], (uint32_t)(e0 + c));
                            ++pos;
                        }
                    }
                    run += __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
                });
                ++passes;
                done_lists = true;
                break;
            }
            if (decision == 1) {
                // The K-th key T* is isolated and f(T*) > C: emit directly.
                ties = true;
                tstar = (uint32_t)edge_of(win, j);
                n_gt_row = sm.F[j + 1];
                const int take = K - n_gt_row;
                int g_mine = 0;
                const int e_mine = sm.u.hist[wave][j];
                for (int b = j + 1 + lane; b < kBinsX; b += kWave) g_mine += sm.u.hist[wave][b];
                g_mine = wave_sum(g_mine);
                if (lane == 0) {
                    sm.wa[wave] = g_mine;
                    sm.wb[wave] = e_mine;
                }
                __syncthreads();
                int gb = sum_over_waves_below(sm.wa, lane, wave);
                int eb = sum_over_waves_below(sm.wb, lane, wave);
                stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
                    uint32_t k[4];
                    block_keys(v, k);
                    const int e0 = 4 * q - aoff;
                    const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
                    bool fg[4], fe[4];
                    uint64_t mg[4], me[4];
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const bool ok = !edge || (e0 + c >= 0 && e0 + c < n);
                        fg[c] = ok && k[c] > tstar;
                        fe[c] = ok && k[c] == tstar;
                        mg[c] = __ballot(fg[c]);
                        me[c] = __ballot(fe[c]);
                    }
                    int g = gb + (int)lanes_below(mg[3], lanes_below(mg[2], lanes_below(mg[1], lanes_below(mg[0], 0))));
                    int ee = eb + (int)lanes_below(me[3], lanes_below(me[2], lanes_below(me[1], lanes_below(me[0], 0))));
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if (fg[c]) {
                            const int o = g + min(ee, take);
                            if (o >= 0 && o < K) out[o] = e0 + c;
                            ++g;
                        } else if (fe[c]) {
                            const int o = g + ee;
                            if (ee < take && o >= 0 && o < K) out[o] = e0 + c;
                            ++ee;
                        }
                    }
                    gb += __popcll(mg[0]) + __popcll(mg[1]) + __popcll(mg[2]) + __popcll(mg[3]);
                    eb += __popcll(me[0]) + __popcll(me[1]) + __popcll(me[2]) + __popcll(me[3]);
                });
                ++passes;
                break;
            }
            if (decision < 0) break;   // unreachable for 32-bit keys; keeps the loop finite
            win = nw;
            count_pass();
        }
    }
    t2 = stamp();

    if (ties) {
        if (st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = GVR_PATH_TIES;
            s.passes = passes;
            s.candidates = 0;
            s.threshold = tstar;
            s.kth_key = tstar;
            s.n_gt = n_gt_row;
            s.guess_valid = gvalid;
            s.spec_threshold = tspec;
            s.spec_count = f_spec;
            s.pmean = gvalid ? gsum / (float)gvalid : 0.f;
            s.t_start = t0;
            s.t_guess = t1;
            s.t_search = t2;
            s.t_collect = t2;
            s.t_refine = stamp();
            *st = s;
        }
        return;
    }
    if (!done_lists) {
        for (int i = tid; i < K; i += kBlock) out[i] = -1;
        if (st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = -1;
            s.passes = passes;
            *st = s;
        }
        return;
    }
    __syncthreads();
    t3 = stamp();
    // ---------------- (a5) refine the listed candidates and emit
    const uint32_t kth = refine_kth(sm, rlo, rhi, above, K, tid);
    int ngt = 0;
    emit_from_lists(sm, kth, K, out, tid, &ngt);
    if (st && tid == 0) {
        gvr_row_stats s = {};
        s.n = n;
        s.path = path;
        s.passes = passes;
        s.candidates = cands;
        s.threshold = T;
        s.kth_key = kth;
        s.n_gt = ngt;
        s.guess_valid = gvalid;
        s.spec_threshold = tspec;
        s.spec_count = f_spec;
        s.pmean = gvalid ? gsum / (float)gvalid : 0.f;
        s.t_start = t0;
        s.t_guess = t1;
        s.t_search = t2;
        s.t_collect = t3;
        s.t_refine = stamp();
        *st = s;
    }
}

// ------------------------------------------------------------------ host side

gvr_status validate(const float* scores, int64_t B, int64_t ld, int32_t K, const int32_t* out,
                    const gvr_options* opt, int* capacity, int* use_guess) {
    if (K < 1 || K > GVR_MAX_K) return GVR_ERR_UNSUPPORTED_K;
    if (B < 0 || ld < 0) return GVR_ERR_INVALID_ARG;
    if (B > 0 && (!scores || !out)) return GVR_ERR_INVALID_ARG;
    if (ld > (int64_t)0x7FFFFFF0) return GVR_ERR_TOO_LONG;
    int cap = GVR_MAX_CANDIDATES;
    if (opt) {
        if (opt->capacity != 0) {
            if (opt->capacity < K || opt->capacity > GVR_MAX_CANDIDATES) return GVR_ERR_INVALID_ARG;
            cap = opt->capacity;
        }
        if ((opt->flags & ~1) || opt->reserved0 || opt->reserved1) return GVR_ERR_INVALID_ARG;
        if (opt->flags & 1) *use_guess = 0;
    }
    *capacity = cap;
    return GVR_OK;
}

gvr_status run(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev,
               int32_t K, int32_t* out, void* stream, const gvr_options* opt, gvr_row_stats* stats,
               int use_guess) {
    int cap = 0;
    gvr_status st = validate(scores, B, ld, K, out, opt, &cap, &use_guess);
    if (st != GVR_OK) return st;
    if (B == 0) return GVR_OK;
    // One workgroup per row; the grid is split only past 2^31 - 1 rows.
    for (int64_t r0 = 0; r0 < B; r0 += 0x7FFFFFFF) {
        const int64_t rows = std::min<int64_t>(B - r0, 0x7FFFFFFF);
        Params q;
        q.scores = scores + r0 * ld;
        q.ld = ld;
        q.row_len = row_len ? row_len + r0 : nullptr;
        q.prev = prev ? prev + r0 * K : nullptr;
        q.out = out + r0 * K;
        q.stats = stats ? stats + r0 : nullptr;
        q.K = K;
        q.capacity = cap;
        q.use_guess = use_guess;
        hipLaunchKernelGGL(topk_row_kernel, dim3((unsigned)rows), dim3(kBlock), 0, (hipStream_t)stream, q);
        if (hipGetLastError() != hipSuccess) return GVR_ERR_HIP;
    }
    return GVR_OK;
}

}  // namespace

extern "C" {

gvr_status gvr_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                    int32_t K, int32_t* out_idx, void* stream) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, nullptr, nullptr, 1);
}

gvr_status radix_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                      int32_t K, int32_t* out_idx, void* stream) {
    (void)prev_topk;
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, nullptr, nullptr, 0);
}

gvr_status gvr_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                       int32_t K, int32_t* out_idx, void* stream, const gvr_options* options,
                       gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats, 1);
}

gvr_status radix_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                         int32_t* out_idx, void* stream, const gvr_options* options, gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, options, stats, 0);
}

const char* gvr_status_string(gvr_status s) {
    switch (s) {
        case GVR_OK: return "ok";
        case GVR_ERR_INVALID_ARG: return "invalid argument";
        case GVR_ERR_UNSUPPORTED_K: return "unsupported K (1 <= K <= 2048)";
        case GVR_ERR_HIP: return "HIP runtime error";
        case GVR_ERR_TOO_LONG: return "row stride too long";
    }
    return "unknown status";
}

const char* gvr_version(void) { return "gvr_topk 0.2 (gfx950, one workgroup per row)"; }

}  // extern "C"
