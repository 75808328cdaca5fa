// gvr_topk.hip -- Guess-Verify-Refine exact Top-K and radix-select Top-K for
// MI355X (gfx950), behind the C ABI declared in include/gvr_topk.h.
//
// Workgroups of 1024 threads (16 wave64s). A row is handled by one
// workgroup, or split over S of them ("parts", up to 16) when few long rows
// would leave compute units idle and the streaming time saved outweighs the
// merge; the parts of one row are placed on one XCD so they share its L2.
// The same code, instantiated for 8 waves (6144-entry lists, two workgroups
// per compute unit) and 4 waves (4096-entry lists, three per compute unit),
// serves calls with more rows than compute units.
//
//   Guess (Sec. 4.2.1, Phase 1). Wave 0 of every part gathers the scores at a
//   strided sample of prev_topk (every 8th entry for K = 2048, 256 in all)
//   and reduces them to pmin / pmax / pmean and T_spec, the lower edge of the
//   histogram bin (over [pmin, pmax]) holding the sampled key of rank
//   ceil(65 / 2048 * samples): a threshold the previous step's Top-K makes
//   likely to leave a few thousand elements of the current row above it, so
//   that K <= f(T_spec) <= C. Waves 1..15 have their first slabs (1 KB per
//   wave: 64 lanes x one 16-byte load) in flight meanwhile and wait on an LDS
//   flag, not a barrier, so a stalled load issue never delays T_spec.
//
//   Verify / collect (Sec. 4.2.2-4.2.3, Phases 2-3). One pass over the
//   part's slabs counts f(T_spec) and appends every element at or above it
//   to per-wave LDS lists (ballot + mbcnt ranks, no atomics; each wave
//   streams a contiguous range, so its list is in index order). The test
//   runs on raw fp32 bits (one compare, see SpecTest), and every lane stores
//   each element, kept ones at their rank and the others to a dummy slot, so
//   a slab costs a few scalar instructions. With S > 1 each part
//   publishes its list and count to a workspace and the last part of the row
//   to arrive (one agent-scope atomic per part) merges them. If
//   K <= f(T_spec) <= C, Lemma 1 (Sec. 4.1) says the list holds the exact
//   answer: the row was read once.
//
//   Refine (Sec. 4.2.4, Phase 4). One LDS histogram level over the listed
//   keys (built while the lists are turned into keys), a two-scan bin search
//   by one wave, then that wave ranks the few keys of the K-th key's bin to
//   get T* and the per-segment emission offsets (a crowded bin is resolved
//   from its min / max or narrowed); every key > T* and the first
//   K - #{key > T*} keys equal to T* (lower index first) are written out in
//   ascending index order.
//
//   When the guess does not deliver, what the speculative pass counted is
//   used first: its histogram level counts every key >= T_spec even where a
//   list overflowed, so if f(T_spec) > C the bin holding the K-th key gives
//   a threshold T' with K <= f(T') <= C, and one collect pass over the row
//   lists the keys >= T' (if K <= f(T_spec) <= C but a list overflowed, the
//   collect is at T_spec). Otherwise (f(T_spec) < K, no valid prev_topk, or
//   a crowded bin) count passes narrow a 256-bin window of key space around
//   the K-th key (each pass evaluates f at 257 thresholds: the count cache
//   of Phase 2 generalised), then one collect pass gathers the <= C
//   candidates at the accepted threshold with exact per-wave offsets, or,
//   when ties straddle [K, C], an emit pass writes the selection directly.
//   radix_topk (one workgroup per row) is a distribution-agnostic radix
//   select (Sec. 2.2): a digit pass counts the top 11 key bits of the row,
//   the bin holding the K-th key is collected in one more pass (or narrowed
//   by count passes when it holds more than C keys).
//
//   On request (option flag 4) the paper's own Phase 2 schedule runs instead
//   of the speculative pass: T0 = pmean of all guessed scores, one threshold
//   counted per full-row pass, damped secant steps with a bisection fallback,
//   then one collect pass at the accepted threshold. Option flag 8 runs the
//   paper's own Phase 4 (min / max, histogram, snap iterations) instead of
//   the refine above.

#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "gvr_topk.h"
#include "host_plan.h"
#include "wave_ops.h"
#include "guess.h"
#include "topk_internal.h"

#define DEV __device__ __forceinline__

namespace {

using gvr_host::kMaxParts;
using gvr_host::kMaxSpecLd;
using gvr_host::kNWLong;
using gvr_host::kNWMid;
using gvr_host::kNWShort;
using gvr_host::kPartCap;
using gvr_host::kXcds;
using namespace gvr_dev;

constexpr int kU = 8;                          // slabs in flight per wave (count / collect passes)
constexpr int kSU = 8;                         // slabs in flight per wave (speculative pass)
constexpr int kBins = 256;                     // bins of a counting window
constexpr int kBinsX = kBins + 1;              // + "at or above the window"
constexpr int kCapWLong = 1024;                // per-wave list capacity of the 16- and 4-wave shapes
constexpr int kCapWMid = 768;                  // per-wave list capacity of the 8-wave shape

// Workgroup shape: NW wave64s. The 16-wave shape (1024 list entries per wave,
// 128 KB of lists, one workgroup per compute unit) streams a long row as fast
// as one compute unit can and is the only one that splits rows. The 8-wave
// shape (768 entries per wave, 48 KB, two workgroups per compute unit) and
// the 4-wave shape (1024 per wave, 32 KB, three per compute unit) serve
// batches with more rows than compute units, whose time goes into per-row
// latency that several resident rows overlap.
template <int NW>
struct Shape {
    static constexpr int kNW = NW;
    static constexpr int kBlock = NW * kWave;
    static constexpr int kSW = NW - 1;          // streaming waves of the speculative pass (wave 0: guess)
    static constexpr int kCapW = NW == 8 ? kCapWMid : kCapWLong;   // per-wave list capacity, speculative pass
    static constexpr int kCap = NW * kCapW;     // list capacity C (LDS)
};
static_assert(Shape<kNWLong>::kCap == gvr_host::kCapLong && Shape<kNWMid>::kCap == gvr_host::kCapMid &&
                  Shape<kNWShort>::kCap == gvr_host::kCapShort,
              "shape capacities as the host plans them");
static_assert(Shape<kNWLong>::kCap == GVR_MAX_CANDIDATES, "the long-row shape holds the largest capacity");
static_assert(kPartCap == Shape<kNWLong>::kCap, "a workspace slot holds one part's lists");
constexpr int kRefBins = 4096;                 // bins of a narrowing refine level (12 bits of key)
constexpr int kRefBins1 = 2048;                // bins of the first refine level (32 per lane of one wave)
constexpr int kDigitShift = 21;                // radix digit: the top 11 key bits, one first-level bin each
static_assert(kRefBins1 + kGuessBins <= kRefBins, "guess histogram above the first refine level");
static_assert(kGuessMaxK == GVR_MAX_K, "the T_spec quantile is taken over the largest K");
static_assert(kRefBins1 == gvr_host::kSlotHistBins, "a workspace slot holds one part's first refine level");
constexpr int kSmall = 64;                     // refine: K-th key's bin resolved by one wave up to this size
constexpr int kMaxPasses = 8;                  // 2 + at most 4 narrowing passes + 1 final pass suffice
constexpr int kMaxSecant = 8;                  // probes of the secant search after T0 (I_max)

static_assert((kBins & (kBins - 1)) == 0 && (kRefBins & (kRefBins - 1)) == 0 && (kRefBins1 & (kRefBins1 - 1)) == 0 &&
                  (kGuessBins & (kGuessBins - 1)) == 0, "bin counts are powers of two");
static_assert(kSmall * 4 <= kRefBins, "refine candidates over the histogram");

struct Params {
    const float* scores;
    int64_t ld;
    const int32_t* row_len;
    const int32_t* prev;
    int32_t* out;
    gvr_row_stats* stats;
    int32_t K;
    int32_t capacity;    // C
    int32_t rows;        // rows of this launch
    int32_t parts;       // S: workgroups per row
    int32_t chunk;       // gridDim.x / 8: consecutive (row, part) slots per XCD
    int32_t scatter;     // 1: slot = blockIdx.x (parts of a row on different XCDs)
    int32_t secant;      // 1: the paper's Phase 2 (secant counting passes) instead of the speculative pass
    int32_t paper_refine; // 1: the paper's Phase 4 (min/max, histogram, snap iterations) instead of refine_emit
    uint64_t* arrivals;  // [rows] parts that finished the speculative pass (S > 1), per XCD above
                         // bit 16; 0 between calls
    int32_t* part_count; // [rows][S] f(threshold) of each part, bit 31 = a wave list overflowed
    uint32_t* part_thresh; // [rows][S] threshold of each part's list (T_spec, the same in every part)
    int32_t* part_hist;  // [rows][S][kRefBins1] each part's first refine level over [T_spec, pmax]
    const int32_t* gstats; // or NULL: GuessStats words of every row (row stride K), from the indexer
    int32_t ordered_merge; // arrival counter updated with agent-scope release / acquire
    uint64_t* part_list; // [rows][S][kPartCap] (fp32 bits | index << 32) of each part
};

// ------------------------------------------------------------------ helpers

// Lane v of every wave reads wave v's value: one LDS read + one wave
// reduction per cross-wave sum.
template <int NW>
DEV int sum_over_waves(const int* vals, int lane) { return wave_sum(lane < NW ? vals[lane] : 0); }
DEV int sum_over_waves_below(const int* vals, int lane, int wave) { return wave_sum(lane < wave ? vals[lane] : 0); }

// Time stamps of the row stats: the GPU's constant-rate clock (100 MHz on
// MI355X), so phase times do not depend on the shader clock.
DEV int64_t stamp() { return (int64_t)__builtin_amdgcn_s_memrealtime(); }

// Workgroup barrier that orders LDS accesses only: unlike __syncthreads()
// it does not wait for the wave's outstanding global loads, so prefetched
// slabs stay in flight across it.
DEV void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}


// A window of key space: bins j < kBins cover [lo + j<<shift, lo + (j+1)<<shift);
// bin kBins holds every key >= lo + kBins<<shift; keys below lo are not counted.
struct Window {
    uint32_t lo;
    uint32_t shift;
};
DEV Window make_window(uint32_t a, uint32_t b) {   // covers [a, b], b >= a
    const uint64_t width = (uint64_t)b - a + 1;
    const uint32_t s = bin_shift(width, log2i(kBins));
    return Window{a, s};
}
DEV uint64_t edge_of(const Window& w, int j) { return (uint64_t)w.lo + ((uint64_t)j << w.shift); }

// Raw buffer resource over [base, base + bytes): 32-bit per-lane offsets.
typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
constexpr int kBufWord3 = 0x00020000;   // 32-bit data format, no swizzle
DEV __amdgpu_buffer_rsrc_t row_rsrc(const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kBufWord3);
}
// 16-byte buffer load (the speculative pass: rows within its 32-bit offsets);
// NT: with the non-temporal hint (a streamed row is read once).
template <bool NT>
DEV float4 buf_load16(__amdgpu_buffer_rsrc_t r, int off) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, NT ? 2 : 0);
    return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
}
// Device-scope loads of what other workgroups published (they skip the
// vector L1).
DEV int ld_agent(const int32_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
DEV uint64_t ld_agent(const uint64_t* p) { return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
// Byte offset of an LDS object (its address in the LDS aperture).
DEV uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}
// Two dwords to LDS at a byte address: the pair's registers need not be
// adjacent (no copies into a register pair).
DEV void lds_store_pair(uint32_t addr, uint32_t a, uint32_t b) {
    asm volatile("ds_write2_b32 %0, %1, %2 offset1:1" : : "v"(addr), "v"(a), "v"(b) : "memory");
}
// q + (this lane's bit of m): one add-with-carry taking the lane mask as carry-in.
DEV int add_lane_bit(int q, uint64_t m) {
    int r;
    uint64_t carry_out;
    asm volatile("v_addc_co_u32_e64 %0, %1, 0, %2, %3" : "=v"(r), "=&s"(carry_out) : "v"(q), "s"(m));
    return r;
}

// ------------------------------------------------------------------ LDS
// List segments: the candidate list is a sequence of NW segments in index
// order, segment w held at list[seg_off[w] .. + seg_cnt[w]) and handled by
// wave w (its own list after a pass, or its even share of a split row's
// merged list).
template <int NW>
struct Smem {
    uint2 list[Shape<NW>::kCap];                   // candidates (key, index), in segments
    union alignas(16) {
        int hist[NW][kBinsX];          // wave-private counting histograms
        int rhist[kRefBins];            // refine / guess histogram
    } u;
    int F[kBinsX + 1];                  // F[j] = f(edge j) over the row
    int seg_off[NW];
    int seg_cnt[NW];
    int sga[NW];                        // per-segment counts (keys > T, keys == T), then exclusive offsets
    int sgb[NW];
    int wa[NW];
    int wb[NW];
    int red[4][NW];
    float redf[NW];
    int scal[8];
    int guess_ready;                    // set by wave 0 once T_spec is in scal[4..7]
};
// Passes over the lists read four 64-entry chunks at a time, up to 255
// entries past a segment's count (masked afterwards): the list must be
// followed by that much LDS.
template <int NW>
constexpr bool lds_slack_ok() {
    return offsetof(Smem<NW>, u) == sizeof(uint2) * Shape<NW>::kCap && sizeof(Smem<NW>::u) >= 4 * kWave * sizeof(uint2);
}
static_assert(lds_slack_ok<kNWLong>() && lds_slack_ok<kNWShort>() && lds_slack_ok<kNWMid>(),
              "LDS slack after the candidate list");

// Block-wide exclusive scan of one int (all threads of the workgroup). Returns the total.
template <int NW>
DEV int block_excl_scan(int& a, Smem<NW>& sm, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    const int ia = wave_incl_scan(a, lane);
    if (lane == kWave - 1) sm.wa[wave] = ia;
    __syncthreads();
    const int before = sum_over_waves_below(sm.wa, lane, wave);
    const int tot = sum_over_waves<NW>(sm.wa, lane);
    __syncthreads();
    a = before + ia - a;
    return tot;
}

// ------------------------------------------------------------------ streaming
// One wave streams float4 blocks [qb, qe) of the row (64-bit addresses: a
// full-row pass serves rows of any length) in slabs of 64 blocks with kU
// slabs in flight;
// `body(v, q, qs)` gets each lane's block q, its data
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
// histogram.
DEV void hist_add(int* hw, uint32_t k, bool in, uint32_t lo, uint32_t sh) {
    const uint32_t b = min((k - lo) >> sh, (uint32_t)kBins);
    if (in) __hip_atomic_fetch_add(&hw[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

DEV void block_keys(const float4& v, uint32_t (&k)[4]) {
    k[0] = key_of(v.x);
    k[1] = key_of(v.y);
    k[2] = key_of(v.z);
    k[3] = key_of(v.w);
}

// ------------------------------------------------------------------ refine
// Exclusive offsets of the per-segment counts sga[] and sgb[] over the nseg
// segments (in place), by wave 0; the totals go to scal[5] and scal[6].
template <int NW>
DEV void seg_scan(Smem<NW>& sm, int nseg, int lane) {
    static_assert(NW <= kWave, "one segment per lane");
    const int a = lane < nseg ? sm.sga[lane] : 0, b = lane < nseg ? sm.sgb[lane] : 0;
    const int ia = wave_incl_scan(a, lane), ib = wave_incl_scan(b, lane);
    if (lane < nseg) {
        sm.sga[lane] = ia - a;
        sm.sgb[lane] = ib - b;
    }
    if (lane == kWave - 1) {
        sm.scal[5] = ia;
        sm.scal[6] = ib;
    }
}

// Exact K-th key among the listed candidates. The K-th key lies in
// [wlo, whi]; `above` listed candidates lie above whi. Histogram levels of
// kRefBins bins narrow the window; the first also finds the window's
// smallest and largest listed key, and if they are one key it is the K-th.
template <int NW>
DEV uint32_t refine_kth(Smem<NW>& sm, uint32_t wlo, uint32_t whi, int above, int K, int tid) {
    using W = Shape<NW>;
    const int lane = tid & 63, wave = tid >> 6;
    int need = K - above;   // >= 1
    for (int level = 0; level < 4 && wlo != whi; ++level) {
        const uint64_t width = (uint64_t)whi - wlo + 1;
        const uint32_t s = bin_shift(width, log2i(kRefBins));
        for (int i = tid; i < kRefBins; i += W::kBlock) sm.u.rhist[i] = 0;
        lds_barrier();
        uint32_t kmn = 0xFFFFFFFFu, kmx = 0u;   // the first level also finds the window's smallest and largest key
        {
            const int j = wave;
            const uint2* seg = sm.list + sm.seg_off[j];
            const int cnt = sm.seg_cnt[j];
            for (int i = lane; i < cnt; i += kWave) {
                const uint32_t kk = seg[i].x;
                if (kk >= wlo && kk <= whi) {
                    __hip_atomic_fetch_add(&sm.u.rhist[(kk - wlo) >> s], 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
                    kmn = min(kmn, kk);
                    kmx = max(kmx, kk);
                }
            }
        }
        if (level == 0) {
            kmn = wave_min_u(kmn);
            kmx = wave_max_u(kmx);
            if (lane == 0) {
                sm.red[2][wave] = (int)kmn;
                sm.red[3][wave] = (int)kmx;
            }
        }
        lds_barrier();
        if (level == 0) {
            // one key in the window (ties, as in rounded scores): it is T*
            const uint32_t mn = wave_min_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0xFFFFFFFFu);
            const uint32_t mx = wave_max_u(lane < NW ? (uint32_t)sm.red[3][lane] : 0u);
            if (mn == mx) return mn;
        }
        constexpr int PER = kRefBins / W::kBlock;   // 4 bins per thread
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
        lds_barrier();
#pragma unroll
        for (int q = PER - 1; q >= 0; --q) {
            const int nr = run + loc[q];
            if (run < need && nr >= need) {
                sm.scal[0] = tid * PER + q;
                sm.scal[1] = run;
                sm.scal[2] = loc[q];
            }
            run = nr;
        }
        lds_barrier();
        const int b = sm.scal[0];
        const int ab = sm.scal[1];
        const int cb = sm.scal[2];
        lds_barrier();
        if (b < 0) break;   // cannot happen for consistent counts; keeps every path finite
        need -= ab;
        const uint64_t nlo = (uint64_t)wlo + ((uint64_t)b << s);
        uint64_t nhi = nlo + ((uint64_t)1 << s) - 1;
        if (nhi > whi) nhi = whi;
        wlo = (uint32_t)nlo;
        whi = (uint32_t)nhi;
        if (wlo != whi && cb <= kSmall) {
            // A few candidates left in the window: copy their keys to a
            // small LDS array (over the histogram, no longer needed) and let
            // wave 0 rank them, one candidate per lane, against LDS-broadcast
            // keys: T* is the need-th largest of them.
            uint32_t* const skey = reinterpret_cast<uint32_t*>(sm.u.rhist);
            if (tid == 0) sm.scal[3] = 0;
            lds_barrier();
            {
                const uint2* seg = sm.list + sm.seg_off[wave];
                const int cnt = sm.seg_cnt[wave];
                for (int i0 = 0; i0 < cnt; i0 += kWave) {   // wave-uniform bound: every lane runs each step
                    const int i = i0 + lane;
                    const uint32_t kk = i < cnt ? seg[i].x : 0u;
                    const bool in = i < cnt && kk >= wlo && kk <= whi;
                    const uint64_t m = __ballot(in);
                    if (m) {   // wave-uniform
                        int base = 0;
                        if (lane == 0)
                            base = __hip_atomic_fetch_add(&sm.scal[3], (int)__popcll(m), __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_WORKGROUP);
                        base = __builtin_amdgcn_readfirstlane(base);
                        const int pos = base + (int)lanes_below(m, 0);
                        if (in && pos < kSmall) skey[pos] = kk;
                    }
                }
            }
            lds_barrier();
            if (wave == 0) {
                const int c = min(cb, kSmall);
                const bool v = lane < c;
                const uint32_t mine = v ? skey[lane] : 0u;
                int gt = 0, ge = 0;
                for (int j = 0; j < c; ++j) {
                    const uint32_t o = skey[j];   // one address for the wave: a broadcast
                    gt += o > mine;
                    ge += o >= mine;
                }
                const uint64_t hit = __ballot(v && gt < need && ge >= need);
                const uint32_t kth = hit ? __builtin_amdgcn_readlane(mine, (int)__builtin_ctzll(hit)) : wlo;
                if (lane == 0) sm.scal[0] = (int)kth;
            }
            lds_barrier();
            const uint32_t kth = (uint32_t)sm.scal[0];
            lds_barrier();   // scal[0] is read before it is written again
            return kth;
        }
    }
    return wlo;
}

// Emission of segment j: the segments before it hold `gb` keys > T and `eb`
// keys == T; write every key > T and the first `take` keys == T (list order =
// index order) at their ranks: ascending index output.
template <int NW>
DEV void emit_segment(const Smem<NW>& sm, int j, uint32_t T, int K, int take, int gb, int eb, int32_t* out,
                      int lane) {
    const uint2* seg = sm.list + sm.seg_off[j];
    const int cnt = sm.seg_cnt[j];
    for (int i0 = 0; i0 < cnt; i0 += 4 * kWave) {
        const int rem = cnt - i0;
        uint2 en[4];   // four entries per lane read before any is written out
#pragma unroll
        for (int c = 0; c < 4; ++c) en[c] = seg[i0 + c * kWave + lane];   // past the count: masked below
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint64_t vm = first_lanes(rem - c * kWave);   // valid lanes
            const uint32_t kk = en[c].x;
            const uint64_t mg = __ballot(kk > T) & vm, me = __ballot(kk == T) & vm;
            const bool fg = (mg >> lane) & 1, fe = (me >> lane) & 1;
            const int g = gb + (int)lanes_below(mg, 0);
            if (me == 0) {   // no key == T here (wave-uniform): keys > T go after min(eb, take) ties
                const int o = g + min(eb, take);
                if (fg && o < K) out[o] = (int)en[c].y;
            } else {
                // a key > T goes after the first min(ties before it, take)
                // ties; a tie is taken while fewer than `take` precede it, at
                // the same position formula (one predicated store)
                const int e = eb + (int)lanes_below(me, 0);
                const int o = g + min(e, take);
                if ((fg || (fe && e < take)) && o < K) out[o] = (int)en[c].y;
            }
            gb += __popcll(mg);
            eb += __popcll(me);
        }
    }
}

// Every wave emits its segments at the offsets in sga / sgb (after seg_scan).
template <int NW>
DEV void emit_segments(const Smem<NW>& sm, uint32_t T, int K, int take, int32_t* out, int lane, int wave) {
    {
        const int j = wave;
        emit_segment(sm, j, T, K, take, sm.sga[j], sm.sgb[j], out, lane);
    }
}

// Write the selection from the lists: every key > T, then the first `take`
// keys == T in list (= index) order; output in ascending index order.
template <int NW>
DEV void emit_from_lists(Smem<NW>& sm, uint32_t T, int K, int32_t* out, int tid, int* n_gt_out) {
    const int lane = tid & 63, wave = tid >> 6;
    {
        const int j = wave;
        const uint2* seg = sm.list + sm.seg_off[j];
        const int cnt = sm.seg_cnt[j];
        int gt = 0, eq = 0;
        for (int i = lane; i < cnt; i += kWave) {
            const uint32_t kk = seg[i].x;
            gt += kk > T;
            eq += kk == T;
        }
        gt = wave_sum(gt);
        eq = wave_sum(eq);
        if (lane == 0) {
            sm.sga[j] = gt;
            sm.sgb[j] = eq;
        }
    }
    lds_barrier();
    if (wave == 0) seg_scan(sm, NW, lane);
    lds_barrier();
    const int gtot = sm.scal[5];
    emit_segments(sm, T, K, K - gtot, out, lane, wave);
    *n_gt_out = gtot;
}

// f(key) for every listed entry of this wave's segments (lane-strided).
template <int NW, typename F>
DEV void for_my_keys(const Smem<NW>& sm, int wave, int lane, F&& f) {
    {
        const int j = wave;
        const uint2* seg = sm.list + sm.seg_off[j];
        const int cnt = sm.seg_cnt[j];
        for (int i = lane; i < cnt; i += kWave) f(seg[i].x);
    }
}

// The paper's Phase 4 (Sec. 4.2.4), kept as an option for comparison with
// refine_emit. (4a) min / max of the listed keys; (4b) a histogram of
// kPaperBins bins over [min, max] and the wave-parallel K-th bin search: every
// wave sums its kPaperBins / 16 bins (wave 0 holds the top ones), one thread
// scans the 16 wave totals from the top, and one lane of the wave found scans
// that wave's bins, 160 serial steps in all; (4d) snap iterations: T starts
// inside the K-th bin where the bin's count places the K-th key (linear
// interpolation over the bin's key range) and each iteration counts
// #{key >= T} and #{key > T} and finds the nearest listed keys above and
// below T in one pass over the lists, moving T to one of them until
// #{key > T} < K <= #{key >= T}; (4e) every key > T and the first K - #{key > T}
// keys == T (lower index first) are written out. T only visits listed keys
// between its start and the K-th key, all inside one bin, so the iterations
// end; after kMaxSnap of them the K-th key is isolated by refine_kth inside
// the bin instead (not reached on the workloads measured).
constexpr int kPaperBins = 2048;
constexpr int kMaxSnap = 64;
template <int NW>
DEV uint32_t paper_refine_emit(Smem<NW>& sm, int K, int32_t* out, int tid, int* n_gt_out, int* snaps_out) {
    using W = Shape<NW>;
    const int lane = tid & 63, wave = tid >> 6;
    // (4a) min / max
    uint32_t mn = 0xFFFFFFFFu, mx = 0u;
    for_my_keys(sm, wave, lane, [&](uint32_t kk) {
        mn = min(mn, kk);
        mx = max(mx, kk);
    });
    mn = wave_min_u(mn);
    mx = wave_max_u(mx);
    if (lane == 0) {
        sm.red[2][wave] = (int)mn;
        sm.red[3][wave] = (int)mx;
    }
    for (int i = tid; i < kPaperBins; i += W::kBlock) sm.u.rhist[i] = 0;
    lds_barrier();
    const uint32_t kmin = wave_min_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0xFFFFFFFFu);
    const uint32_t kmax = wave_max_u(lane < NW ? (uint32_t)sm.red[3][lane] : 0u);
    // (4b) histogram over [kmin, kmax]
    const uint32_t sh = bin_shift((uint64_t)kmax - kmin + 1, log2i(kPaperBins));
    for_my_keys(sm, wave, lane, [&](uint32_t kk) {
        __hip_atomic_fetch_add(&sm.u.rhist[(kk - kmin) >> sh], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    });
    lds_barrier();
    constexpr int kPerWave = kPaperBins / NW;   // wave w holds bins [top - kPerWave (w + 1), top - kPerWave w)
    {
        const int b0 = kPaperBins - kPerWave * (wave + 1);
        int t = 0;
#pragma unroll
        for (int j = 0; j < kPerWave / kWave; ++j) t += sm.u.rhist[b0 + j * kWave + lane];
        t = wave_sum(t);
        if (lane == 0) sm.wa[wave] = t;
    }
    lds_barrier();
    if (tid == 0) {   // target wave: one serial step per wave from the top
        int run = 0, w = 0;
        for (; w < NW - 1 && run + sm.wa[w] < K; ++w) run += sm.wa[w];
        sm.scal[0] = w;
        sm.scal[1] = run;
    }
    lds_barrier();
    if (wave == sm.scal[0] && lane == 0) {   // exact bin: up to kPerWave serial steps from the top of the wave's bins
        int run = sm.scal[1];
        int b = kPaperBins - kPerWave * wave - 1;
        const int bend = kPaperBins - kPerWave * (wave + 1);
        for (; b > bend && run + sm.u.rhist[b] < K; --b) run += sm.u.rhist[b];
        sm.scal[2] = b;
        sm.scal[3] = run;
    }
    lds_barrier();
    const int kb = sm.scal[2];
    const int above = sm.scal[3];
    const int h = max(sm.u.rhist[kb], 1);
    const uint64_t blo = (uint64_t)kmin + ((uint64_t)kb << sh);
    const uint64_t bhi = std::min<uint64_t>(blo + ((uint64_t)1 << sh) - 1, kmax);
    // (4d) snap iterations from the interpolated start
    const int r = max(K - above, 1);   // rank of the K-th key inside the bin, from the top
    uint32_t T = (uint32_t)(bhi - ((uint64_t)(2 * r - 1) * (bhi - blo + 1)) / (uint64_t)(2 * h));
    T = (uint32_t)std::max<uint64_t>(T, blo);
    int snaps = 0, ngt = 0;
    bool found = false;
    while (snaps < kMaxSnap) {
        ++snaps;
        int ge = 0, gt = 0;
        uint32_t up = 0xFFFFFFFFu, down = 0u;
        for_my_keys(sm, wave, lane, [&](uint32_t kk) {
            ge += kk >= T;
            gt += kk > T;
            if (kk > T) up = min(up, kk);
            if (kk < T) down = max(down, kk);
        });
        ge = wave_sum(ge);
        gt = wave_sum(gt);
        up = wave_min_u(up);
        down = wave_max_u(down);
        lds_barrier();   // the previous iteration's totals are read
        if (lane == 0) {
            sm.wa[wave] = ge;
            sm.wb[wave] = gt;
            sm.red[2][wave] = (int)up;
            sm.red[3][wave] = (int)down;
        }
        lds_barrier();
        const int GE = sum_over_waves<NW>(sm.wa, lane);
        const int GT = sum_over_waves<NW>(sm.wb, lane);
        if (GT < K && K <= GE) {
            found = true;
            ngt = GT;
            break;
        }
        // fewer than K at or above T: step down; K or more above T: step up
        T = (GE < K) ? wave_max_u(lane < NW ? (uint32_t)sm.red[3][lane] : 0u)
                     : wave_min_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0xFFFFFFFFu);
    }
    lds_barrier();
    if (!found) T = refine_kth(sm, (uint32_t)blo, (uint32_t)bhi, above, K, tid);
    (void)ngt;
    // (4e) partition
    emit_from_lists(sm, T, K, out, tid, n_gt_out);
    *snaps_out = snaps;
    return T;
}

// First refine level: kRefBins1 bins of 2^sh keys from rlo; keys at or above
// rlo + (kRefBins1 - 1) << sh share the top bin.
DEV uint32_t ref_shift(uint32_t rlo, uint32_t bin_hi) {
    const uint64_t width = (uint64_t)bin_hi - rlo + 1;
    const uint32_t sh = bin_shift(width, log2i(kRefBins1));
    return sh;
}
DEV int ref_bin(uint32_t kk, uint32_t rlo, uint32_t sh) { return (int)min((kk - rlo) >> sh, (uint32_t)kRefBins1 - 1); }
template <int NW>
DEV void ref_hist_add(Smem<NW>& sm, uint32_t kk, uint32_t rlo, uint32_t sh) {
    __hip_atomic_fetch_add(&sm.u.rhist[ref_bin(kk, rlo, sh)], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// One wave: turn the fp32 bit patterns of its list segment seg[0, cnt) into
// keys in place and, if `hist`, add them to the first refine level from rlo.
// Four entries per lane are read before any is written back.
template <int NW>
DEV void keys_in_place(Smem<NW>& sm, uint2* seg, int cnt, bool hist, uint32_t rlo, uint32_t sh, int lane) {
    for (int i0 = 0; i0 < cnt; i0 += 4 * kWave) {
        uint32_t b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = i0 + j * kWave + lane;
            b[j] = seg[i].x;   // past the count: not written back
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = i0 + j * kWave + lane;
            if (i < cnt) {
                const uint32_t kk = key_of_bits(b[j]);
                seg[i].x = kk;
                if (hist) ref_hist_add(sm, kk, rlo, sh);
            }
        }
    }
}

// Wave 0: the bin b of a first refine level hb[0, kRefBins1) holding the
// need0-th key from the top (need0 >= 1, at most the histogram's total), with
// two wave scans; scal[0] = b, scal[2] = base + the keys in the bins above b,
// scal[3] = b's count.
template <int NW>
DEV void kth_bin_wave0(Smem<NW>& sm, const int* hb, int need0, int base, int lane) {
    // lane l owns bins [32 l, 32 l + 32)
    const int4* h4 = reinterpret_cast<const int4*>(hb) + lane * 8;
    int s = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int4 v = h4[j];
        s += v.x + v.y + v.z + v.w;
    }
    const int incl = wave_incl_scan(s, lane);
    const int total = __builtin_amdgcn_readlane(incl, 63);
    const int abv = total - incl;   // keys in the bins of higher lanes
    const uint64_t hit = __ballot(abv < need0 && abv + s >= need0);
    const int L = hit ? (int)__builtin_ctzll(hit) : 0;
    const int abv_l = __builtin_amdgcn_readlane(abv, L);
    const int hj = lane < 32 ? hb[L * 32 + lane] : 0;
    const int ij = wave_incl_scan(hj, lane);
    const int s_l = __builtin_amdgcn_readlane(ij, 63);
    const int abj = abv_l + s_l - ij;
    const uint64_t hit2 = __ballot(lane < 32 && abj < need0 && abj + hj >= need0);
    const int J = hit2 ? (int)__builtin_ctzll(hit2) : 0;
    if (lane == 0) {
        sm.scal[0] = L * 32 + J;
        sm.scal[2] = base + __builtin_amdgcn_readlane(abj, J);
        sm.scal[3] = __builtin_amdgcn_readlane(hj, J);
    }
}

// Exact K-th key T* among the listed candidates and the emission. The K-th
// key lies in [rlo, rhi]; `above` listed keys lie above rhi. One histogram
// level of kRefBins1 bins over [rlo, bin_hi] (keys in (bin_hi, rhi] count in
// the top bin; built here unless `hist_ready`), then wave 0 finds the
// bin b holding the K-th key with two wave scans. If b holds at most kSmall
// candidates, one pass over the lists copies them (with their segment) to a
// small LDS array and counts each segment's keys above b; wave 0 takes one
// candidate per lane, selects T* among them and the per-segment emission
// offsets, and every wave emits its segments. Otherwise histogram narrowing
// (refine_kth) continues inside b; a bin whose keys are all one value (ties)
// is resolved by its first level.
template <int NW>
DEV uint32_t refine_emit(Smem<NW>& sm, uint32_t rlo, uint32_t rhi, uint32_t bin_hi, int above, int K, int32_t* out,
                         int tid, int* n_gt_out, bool hist_ready) {
    using W = Shape<NW>;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t sh = ref_shift(rlo, bin_hi);
    int* hb = sm.u.rhist;
    if (tid == 0) sm.scal[1] = 0;   // ordered before its atomics by the barrier after the bin search
    if (!hist_ready) {
        for (int i = tid; i < kRefBins1; i += W::kBlock) hb[i] = 0;
        lds_barrier();
        for_my_keys(sm, wave, lane, [&](uint32_t kk) {
            if (kk >= rlo && kk <= rhi) ref_hist_add(sm, kk, rlo, sh);
        });
        lds_barrier();
    }
    // (a ready histogram is complete behind the caller's last barrier)
    const int need0 = K - above;   // >= 1: rank of T* among the keys in [rlo, rhi], from the top
    if (wave == 0) kth_bin_wave0(sm, hb, need0, above, lane);
    lds_barrier();
    const int b = sm.scal[0];
    const int above_b = sm.scal[2];   // listed keys above bin b
    const int cnt_b = sm.scal[3];
    const uint64_t lo64 = (uint64_t)rlo + ((uint64_t)b << sh);
    const uint32_t lo_b = (uint32_t)lo64;
    const uint32_t hi_b =
        b == kRefBins1 - 1 ? rhi : (uint32_t)std::min<uint64_t>(lo64 + ((uint64_t)1 << sh) - 1, rhi);
    if (lo_b == hi_b) {   // the bin is one key: T* = lo_b
        emit_from_lists(sm, lo_b, K, out, tid, n_gt_out);
        return lo_b;
    }
    if (cnt_b > kSmall) {   // narrowing inside the bin (a bin of one key ends after its first level)
        lds_barrier();
        const uint32_t kth = refine_kth(sm, lo_b, hi_b, above_b, K, tid);
        emit_from_lists(sm, kth, K, out, tid, n_gt_out);
        return kth;
    }
    // Copy bin b's candidates, with their segment, to one small LDS array over
    // the histogram (no longer needed; at most kSmall of them): a chunk that
    // holds some (rare) reserves room with one LDS atomic. Each wave counts
    // its segments' keys above the bin.
    uint4* const small = reinterpret_cast<uint4*>(sm.u.rhist);
    uint32_t* const skey = reinterpret_cast<uint32_t*>(small + kSmall);   // their keys alone, for the rank
    const uint32_t wid = hi_b - lo_b;
    {
        const int j = wave;
        const uint2* seg = sm.list + sm.seg_off[j];
        const int cnt = sm.seg_cnt[j];
        int gtl = 0;
        for (int i0 = 0; i0 < cnt; i0 += 4 * kWave) {
            uint2 en[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) en[c] = seg[i0 + c * kWave + lane];   // past the count: masked below
            // per lane: keys above the bin counted, bin members flagged (one
            // ballot for the four entries: members are rare)
            bool hit[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const bool valid = i0 + c * kWave + lane < cnt;
                gtl += (valid && en[c].x > hi_b) ? 1 : 0;
                hit[c] = valid && en[c].x - lo_b <= wid;
            }
            if (!__ballot(hit[0] || hit[1] || hit[2] || hit[3])) continue;   // (wave-uniform)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint64_t m = __ballot(hit[c]);
                if (m) {   // (wave-uniform)
                    int base = 0;
                    if (lane == 0)
                        base = __hip_atomic_fetch_add(&sm.scal[1], (int)__popcll(m), __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_WORKGROUP);
                    base = __builtin_amdgcn_readfirstlane(base);
                    const int pos = base + (int)lanes_below(m, 0);
                    if (((m >> lane) & 1) && pos < kSmall) {
                        small[pos] = make_uint4(en[c].x, en[c].y, (uint32_t)j, 0u);
                        skey[pos] = en[c].x;
                    }
                }
            }
        }
        const int gt_hi = wave_sum(gtl);
        if (lane == 0) {
            sm.sga[j] = gt_hi;
            sm.sgb[j] = 0;
        }
    }
    lds_barrier();
    if (wave == 0) {
        // Lane l takes the l-th copied candidate (any order).
        const bool v = lane < cnt_b;
        const uint4 mine = v ? small[lane] : make_uint4(0u, 0u, 0u, 0u);
        // T* is the need-th largest of them: the key of a lane with fewer
        // than `need` keys above it and at least `need` at or above it. Every
        // lane compares its key with each candidate's, four keys per LDS
        // read (one address for the whole wave: a broadcast).
        const int need = K - above_b;   // rank of T* inside the bin, from the top
        const uint4* sk4 = reinterpret_cast<const uint4*>(skey);
        int gt = 0, ge = 0;
#pragma unroll 4
        for (int j0 = 0; j0 < cnt_b; j0 += 4) {
            const uint4 kk = sk4[j0 >> 2];   // past cnt_b: masked below
            const uint32_t a[4] = {kk.x, kk.y, kk.z, kk.w};
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const bool in = j0 + jj < cnt_b;
                gt += in && a[jj] > mine.x;
                ge += in && a[jj] >= mine.x;
            }
        }
        const uint64_t hitk = __ballot(v && gt < need && ge >= need);
        const uint32_t kth = __builtin_amdgcn_readlane(mine.x, hitk ? (int)__builtin_ctzll(hitk) : 0);
        // Per segment: keys > T* (above the bin, plus the bin's) and == T*;
        // each candidate adds itself to its segment's counts.
        if (v && mine.x > kth) __hip_atomic_fetch_add(&sm.sga[mine.z], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (v && mine.x == kth) __hip_atomic_fetch_add(&sm.sgb[mine.z], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        seg_scan(sm, NW, lane);
        if (lane == 0) sm.scal[0] = (int)kth;
    }
    lds_barrier();
    const uint32_t kth = (uint32_t)sm.scal[0];
    const int gtot = sm.scal[5];
    emit_segments(sm, kth, K, K - gtot, out, lane, wave);
    *n_gt_out = gtot;
    return kth;
}

// ------------------------------------------------------------------ kernel

// Threshold test of the speculative pass on raw fp32 bits u: key(u) >= tkey.
// For tkey in the upper half (T >= +0) that is the signed compare
// (int)u >= (int)(tkey ^ 0x80000000) (negative patterns are negative ints);
// for tkey in the lower half (T <= -0) it is u <= ~tkey as unsigned (every
// non-negative pattern passes; a negative one passes iff ~u >= tkey), which
// is (int)(u ^ 0x7FFFFFFF) >= (int)(tkey ^ 0x80000000). Both cases: one xor
// with a wave-uniform mask and one signed compare, no key transform.
struct SpecTest {
    uint32_t flip;   // 0 or 0x7FFFFFFF
    int32_t bound;   // tkey ^ 0x80000000
};
DEV SpecTest make_spec_test(uint32_t tkey) {
    return SpecTest{tkey >= 0x80000000u ? 0u : 0x7FFFFFFFu, (int32_t)(tkey ^ 0x80000000u)};
}
// The fp32 pattern whose key is 0 (a NaN): it never passes a test with
// tkey >= 1, so it stands in for elements outside the row.
constexpr uint32_t kKeyZeroBits = 0xFFFFFFFFu;

DEV uint64_t pack_entry(uint32_t bits, uint32_t idx) { return (uint64_t)bits | ((uint64_t)idx << 32); }

template <bool GUESS, int NW, bool NT>
DEV void topk_body(const Params& p) {
    __shared__ Smem<NW> sm;
    using W = Shape<NW>;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int S = p.parts;
    // Slot (row, part) of this workgroup: consecutive slots on one XCD, so the
    // parts of a row share an L2 (scatter: the plain order, for tests of the
    // cross-XCD path).
    const int slot = p.scatter ? (int)blockIdx.x : (int)(blockIdx.x % kXcds) * p.chunk + (int)(blockIdx.x / kXcds);
    const int row_i = slot / S;
    const int part = slot - row_i * S;
    if (row_i >= p.rows) return;   // padding slot of the XCD-aligned grid
    const int64_t row = row_i;
    // Phase stamps are taken only when row stats are asked for: a clock read
    // is a scalar memory operation, and the next LDS wait would wait for it.
    const bool timed = p.stats != nullptr;
    auto tstamp = [&]() -> int64_t { return timed ? stamp() : (int64_t)0; };
    const int64_t t0 = tstamp();

    // Wave 0 samples the guess: every st_g-th entry of prev_topk (at most
    // kGuessSamples of them). The sample indices go out with the row length;
    // the gathers that depend on them are the only serial memory latency
    // before T_spec, and the part's first slabs are in flight meanwhile.
    const int st_g = guess_stride(p.K);
    const int m_g = guess_count(p.K);
    int pq[4] = {-1, -1, -1, -1};
    int gw[5] = {-1, 0, -1, 0, 0};   // the indexer's GuessStats words of this row (gvr_indexer_topk)
    if (GUESS && p.prev && wave == 0) {
        if (p.gstats) {
            const int32_t* g = p.gstats + row * (int64_t)p.K;
#pragma unroll
            for (int c = 0; c < 5; ++c) gw[c] = g[c];
        } else {
            const int32_t* pv = p.prev + row * (int64_t)p.K;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int i = lane + 64 * c;
                if (i < m_g) pq[c] = pv[i * st_g];
            }
        }
    }
    // Row length through the scalar cache (row is wave-uniform): it does not
    // wait behind the vector loads above.
    int64_t n64 = p.row_len ? (int64_t)__builtin_amdgcn_readfirstlane(
                                  *(const __attribute__((address_space(4))) int32_t*)(p.row_len + row))
                            : p.ld;
    n64 = n64 < 0 ? 0 : (n64 > p.ld ? p.ld : n64);
    const int n = (int)n64;
    const int K = p.K;
    const int cap = p.capacity;
    const float* x = p.scores + row * p.ld;
    int32_t* out = p.out + row * (int64_t)K;
    gvr_row_stats* st = p.stats ? p.stats + row : nullptr;

    // (a1) row classify: n <= K -> 0..n-1 then -1 padding (part 0 writes).
    if (n <= K) {
        if (part != 0) return;
        for (int i = tid; i < K; i += W::kBlock) out[i] = (i < n) ? i : -1;
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
    // block is one aligned 16-byte load and a slab of 64 blocks is eight
    // whole 128-byte lines: the first block starts the row's first line,
    // which never leaves the page holding the row's first element). Full-row
    // share of each wave (count / collect passes): [qb, qe).
    const int aoff = (int)(((uintptr_t)x >> 2) & 31);   // slabs start on 128-byte lines
    const float4* xa = reinterpret_cast<const float4*>(x - aoff);
    const int nq = (n + aoff + 3) >> 2;
    const int qlast = nq - 1;
    const int nslab_row = (nq + 63) >> 6;
    const int per = ((nslab_row + NW - 1) / NW) * 64;   // whole slabs per wave
    const int qb = min(wave * per, nq), qe = min(qb + per, nq);
    // This part's slabs [ps0, ps1); waves 1..15 stream them in the
    // speculative pass, wave 0 computes the guess meanwhile and streams
    // nothing: this wave's float4 blocks [sqb, sqe).
    const int ps = (nslab_row + S - 1) / S;
    const int ps0 = min(part * ps, nslab_row), ps1 = min(ps0 + ps, nslab_row);
    const int ws = (ps1 - ps0 + W::kSW - 1) / W::kSW;
    const int sw = wave - 1;
    const int sqb = wave == 0 ? 0 : min((ps0 + sw * ws) * 64, min(ps1 * 64, nq));
    const int sqe = wave == 0 ? 0 : min((ps0 + min((sw + 1) * ws, ps1 - ps0)) * 64, nq);
    const int nsl = sqe > sqb ? (sqe - sqb + 63) >> 6 : 0;

    // Every element is a candidate when the row fits the lists and there is
    // no guess, or the row is at most 2K long: there a guess cuts few
    // candidates and often leaves f(T_spec) < K (a guess also cuts the
    // candidates of longer short rows).
    const bool all_mode = (!(GUESS && p.prev) || n <= 2 * K) && (n <= cap) && (ws * 256 <= W::kCapW);
    bool have_prev = GUESS && p.prev && !all_mode;
    // The paper's Phase 2 schedule (secant counting passes), when asked for.
    const bool secant = GUESS && p.secant && have_prev;
    const bool spec = (all_mode || have_prev) && !secant;
    int gvalid = 0;
    uint32_t gmax = 0u, tspec = 0xFFFFFFFFu;
    float gsum = 0.f;
    int64_t t1 = t0, t2 = t0;
    int passes = 0;
    int f_spec = 0;          // f(tthr), or -1 if unknown
    bool hist_ready = false; // the refine's first histogram level is built (lists at tthr)
    bool hist_full = false;  // rhist counts every key >= tthr of the row (first-level bins)
    uint32_t tthr = 0u;      // threshold of the speculative lists
    bool overflow = false;
    // A part of a split row arrives once its published stores have
    // completed (reached the XCD's L2): one device-scope atomic on the row's
    // arrival word, which also counts the parts per XCD (5 bits per XCD above
    // 16 bits of arrivals; option flag 128: an agent-scope release /
    // acquire). True for the row's last part; *same_xcd: every part ran on
    // this part's XCD.
    auto arrive_last = [&](bool* same_xcd) -> bool {
        __builtin_amdgcn_s_waitcnt(0);   // this wave's stores have completed (reached L2)
        __syncthreads();
        if (tid == 0) {
            const uint32_t xcc = (uint32_t)__builtin_amdgcn_s_getreg((31 << 11) | 20) & 7u;   // HW_REG_XCC_ID
            const uint64_t add = 1ull + (1ull << (16 + 5 * xcc));
            const uint64_t old =
                p.ordered_merge
                    ? __hip_atomic_fetch_add(p.arrivals + row, add, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT)
                    : __hip_atomic_fetch_add(p.arrivals + row, add, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const uint64_t now = old + add;
            sm.scal[3] = (int)(old & 0xFFFFu);
            sm.scal[2] = (int)((now >> (16 + 5 * xcc)) & 31u) == S;   // all parts on this XCD
        }
        __syncthreads();
        *same_xcd = sm.scal[2] != 0;
        return sm.scal[3] == S - 1;
    };
    if (tid < NW) sm.seg_off[tid] = tid * W::kCapW;

    if (spec) {
        if (!all_mode) {
            if (tid == 0) sm.guess_ready = 0;
            lds_barrier();
        }
        // The part's first slabs, by buffer loads over the row's float4
        // blocks (lane offset clamped to the last block; refills past the
        // wave's share re-read its last slab, just fetched). Issuing them can
        // stall on a full memory pipeline, so the streaming waves do not meet
        // wave 0 at a barrier afterwards: they poll the guess_ready flag right
        // before their first slab.
        const __amdgpu_buffer_rsrc_t rrow = row_rsrc(xa, nq * 16);
        const int lane16 = lane * 16, qlast16 = qlast * 16;
        const int off_last = (sqb + max(nsl - 1, 0) * 64) * 16;   // the wave's last slab
        auto slab_load = [&](int s) {
            return buf_load16<NT>(rrow, min(lane16 + min((sqb + s * 64) * 16, off_last), qlast16));
        };
        float4 buf[kSU];
        if (nsl > 0) {
#pragma unroll
            for (int u = 0; u < kSU; ++u) buf[u] = slab_load(u);
        }

        if (all_mode) {
            tspec = 0u;
        } else {
            if (wave == 0) {
                // ---------------- (a2) guess statistics (Sec. 4.2.1) over the
                // sampled guessed scores: pmin, pmax, pmean, and T_spec = lower
                // edge of the histogram bin (over [pmin, pmax]) holding the
                // gathered key of rank ceil(65 * m / 2048) from the bottom.
                // From the indexer, when it scored the sample (one load).
                GuessStats gs;
                if (p.gstats) {
                    gs = GuessStats{(uint32_t)gw[0], gw[1], (uint32_t)gw[2], (uint32_t)gw[3], __int_as_float(gw[4])};
                } else {
                    bool ok[4];
                    float gv[4];
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        ok[c] = pq[c] >= 0 && pq[c] < n;
                        gv[c] = ok[c] ? x[pq[c]] : 0.f;
                    }
                    // (above the refine's first level, which stays free)
                    gs = guess_from_samples(gv, ok, sm.u.rhist + kRefBins1);
                }
                const uint32_t ts = gs.ts, mn = gs.mn, mx = gs.mx;
                const int cnt = gs.cnt;
                const float sum = gs.sum;
                {   // the refine's first level, filled after the pass
                    int4* r4 = reinterpret_cast<int4*>(sm.u.rhist) + lane * (kRefBins1 / 4 / kWave);
#pragma unroll
                    for (int j = 0; j < kRefBins1 / 4 / kWave; ++j) r4[j] = make_int4(0, 0, 0, 0);
                }
                if (lane == 0) {
                    sm.scal[4] = (int)ts;
                    sm.scal[5] = cnt;
                    sm.scal[6] = (int)mn;
                    sm.scal[7] = (int)mx;
                    sm.redf[0] = sum;
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
                    __hip_atomic_store(&sm.guess_ready, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                }
            }
        }

        // ---------------- (a3)+(a4) speculative pass over the part's slabs:
        // count and append every (fp32 bits, index) at or above T_spec.
        //
        // The test runs on the raw bits (SpecTest): one signed compare, plus
        // one xor for thresholds <= -0; the two forms are two copies of the
        // loop, chosen once. Thresholds are >= key 1, so the key-0 pattern
        // never passes: elements outside [0, n) in the row's two edge slabs
        // are replaced by it (a wave-uniform branch; interior slabs carry no
        // range test). A slab whose elements all fail costs the compares and
        // one branch. Otherwise each lane appends its kept elements at its
        // rank (kept elements of the lanes below, then its own in order), so
        // every list stays in index order; one capacity check per slab
        // (wave-uniform), and a wave whose list would overflow keeps counting.
        int cnt_w = 0;
        int stored_w = 0;   // entries listed when the list filled up
        uint2* lw = sm.list + wave * W::kCapW;
        // The streaming waves wait for T_spec here, with their first slabs in
        // flight (polling an LDS flag, not a barrier: issuing those loads may
        // stall a wave, which must not hold up wave 0).
        if (!all_mode) {
            while (__hip_atomic_load(&sm.guess_ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == 0)
                __builtin_amdgcn_s_sleep(1);
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
            tspec = (uint32_t)sm.scal[4];
            gvalid = sm.scal[5];
            gmax = (uint32_t)sm.scal[7];
            gsum = sm.redf[0];
            if (gvalid == 0) have_prev = false;   // no usable guess: the pass keeps (almost) nothing
        }
        t1 = tstamp();
        tspec = max(tspec, 1u);
        const SpecTest test = make_spec_test(tspec);
        // the refine's first level over [T_spec, max(pmax, T_spec)]
        const bool own_hist = !all_mode;
        const uint32_t hsh = ref_shift(tspec, max(gmax, tspec));
        // Slab s of this wave is the row's slab sg = sqb / 64 + s; slabs
        // [in_lo, in_hi) hold no element outside [0, n).
        const int in_lo = aoff > 0 ? 1 : 0, in_hi = (n + aoff) >> 8;
        const uint32_t lw_addr = lds_addr(lw);
        const uint32_t dummy = lds_addr(sm.list) + 8 * lane;   // wave 0's segment: never streamed into
        auto spec_pass = [&](auto flip_tag) {
            constexpr uint32_t kFlip = decltype(flip_tag)::value ? 0x7FFFFFFFu : 0u;
            // One slab. `room`: the list has room for a whole slab, so every
            // lane stores each element (kept ones at their rank, the others
            // to a private dummy slot) and the new count comes from the rank
            // of lane 63; otherwise the exact count decides (the overflow is
            // detected after the pass).
            auto slab = [&](const float4& v, int s, bool room) {
                const int sg = (sqb >> 6) + s;
                const int e0 = 4 * lane - aoff + 256 * sg;
                uint32_t k[4] = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)};
                if ((unsigned)(sg - in_lo) >= (unsigned)(in_hi - in_lo)) {   // edge slab (wave-uniform)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        if ((uint32_t)(e0 + c) >= (uint32_t)n) k[c] = kKeyZeroBits;
                }
                bool f[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) f[c] = (int32_t)(k[c] ^ kFlip) >= test.bound;
                const uint64_t m[4] = {__ballot(f[0]), __ballot(f[1]), __ballot(f[2]), __ballot(f[3])};
                const int below = (int)lanes_below(m[3], lanes_below(m[2], lanes_below(m[1], lanes_below(m[0], (uint32_t)cnt_w))));
                if (room) {
                    int q = below;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        lds_store_pair(f[c] ? lw_addr + 8 * q : dummy, k[c], (uint32_t)(e0 + c));
                        q = add_lane_bit(q, m[c]);
                    }
                    cnt_w = __builtin_amdgcn_readlane(q, kWave - 1);
                } else {
                    const int total = __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
                    if (cnt_w + total <= W::kCapW) {
                        int q = below;
#pragma unroll
                        for (int c = 0; c < 4; ++c) {
                            if (f[c]) lds_store_pair(lw_addr + 8 * q, k[c], (uint32_t)(e0 + c));
                            q = add_lane_bit(q, m[c]);
                        }
                    } else {
                        // The list is full: the kept keys go to the refine's
                        // first level only, so that it still counts every key
                        // >= T_spec (the entries already listed join it below).
                        if (cnt_w <= W::kCapW) stored_w = cnt_w;
                        if (own_hist) {
#pragma unroll
                            for (int c = 0; c < 4; ++c)
                                if (f[c]) ref_hist_add(sm, key_of_bits(k[c]), tspec, hsh);
                        }
                    }
                    cnt_w += total;   // counted past capacity: the overflow is detected below
                }
            };
            // Whole windows with their refills (no per-slab bounds), the last
            // whole window refilling only what remains, then the rest: no
            // load is left in flight after the pass.
            int s0 = 0;
            for (; s0 + 2 * kSU <= nsl; s0 += kSU) {
#pragma unroll
                for (int u = 0; u < kSU; ++u) {
                    slab(buf[u], s0 + u, cnt_w <= W::kCapW - 256);
                    buf[u] = slab_load(s0 + u + kSU);
                }
            }
            if (s0 + kSU <= nsl) {
#pragma unroll
                for (int u = 0; u < kSU; ++u) {
                    slab(buf[u], s0 + u, cnt_w <= W::kCapW - 256);
                    if (s0 + u + kSU < nsl) buf[u] = slab_load(s0 + u + kSU);
                }
                s0 += kSU;
            }
#pragma unroll
            for (int u = 0; u < kSU; ++u)
                if (s0 + u < nsl) slab(buf[u], s0 + u, false);
        };
        if (test.flip)
            spec_pass(std::true_type{});
        else
            spec_pass(std::false_type{});

        // Every wave turns its list into keys in place and adds them to the
        // refine's first histogram level over [T_spec, max(pmax, T_spec)]
        // (cleared by wave 0 before its flag): waves done with their slabs
        // do this while the others still stream.
        keys_in_place(sm, lw, cnt_w <= W::kCapW ? cnt_w : stored_w, own_hist, tspec, hsh, lane);
        if (lane == 0) {
            sm.wa[wave] = cnt_w;
            sm.seg_cnt[wave] = min(cnt_w, W::kCapW);
        }
        passes = 1;
        lds_barrier();
        t2 = tstamp();   // every wave of the part has streamed its slabs
        overflow = wave_max_u(lane < NW ? (uint32_t)sm.wa[lane] : 0u) > (uint32_t)W::kCapW;
        f_spec = overflow ? -1 : sum_over_waves<NW>(sm.wa, lane);
        hist_ready = own_hist && !overflow;
        hist_full = own_hist && S == 1;   // full lists or not, every kept key is in it
        tthr = tspec;

        if (overflow && S == 1) {
            // A wave's list overflowed, but every wave counted past its
            // capacity, so f(T_spec) is still exact. Candidates bunched in a
            // few waves' ranges (positional structure: recent tokens, RoPE
            // peaks) do this. If K <= f(T_spec) <= C a second pass over the
            // part's slabs (just read, so L2-resident) collects them again at
            // exact per-wave offsets instead of narrowing from scratch.
            const int f_all = sum_over_waves<NW>(sm.wa, lane);
            if (f_all < K || f_all > cap) f_spec = f_all;   // exact: the narrowing starts on the right side of T_spec
            if (f_all >= K && f_all <= cap) {
                const int off = sum_over_waves_below(sm.wa, lane, wave);
                const int mine = sm.wa[wave];
                lds_barrier();   // every count is read; the old lists are dead
                if (nsl > 0) {
#pragma unroll
                    for (int u = 0; u < kSU; ++u) buf[u] = slab_load(u);
                    const uint32_t base = lds_addr(sm.list + off);
                    auto repack = [&](auto flip_tag) {
                        constexpr uint32_t kFlip = decltype(flip_tag)::value ? 0x7FFFFFFFu : 0u;
                        int run = 0;
                        auto slab = [&](const float4& v, int s) {
                            const int sg = (sqb >> 6) + s;
                            const int e0 = 4 * lane - aoff + 256 * sg;
                            uint32_t k[4] = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                                             __float_as_uint(v.w)};
                            if ((unsigned)(sg - in_lo) >= (unsigned)(in_hi - in_lo)) {
#pragma unroll
                                for (int c = 0; c < 4; ++c)
                                    if ((uint32_t)(e0 + c) >= (uint32_t)n) k[c] = kKeyZeroBits;
                            }
                            bool f[4];
#pragma unroll
                            for (int c = 0; c < 4; ++c) f[c] = (int32_t)(k[c] ^ kFlip) >= test.bound;
                            const uint64_t m[4] = {__ballot(f[0]), __ballot(f[1]), __ballot(f[2]), __ballot(f[3])};
                            int q = (int)lanes_below(m[3], lanes_below(m[2], lanes_below(m[1], lanes_below(m[0], (uint32_t)run))));
#pragma unroll
                            for (int c = 0; c < 4; ++c) {
                                if (f[c] && q < mine) lds_store_pair(base + 8 * q, k[c], (uint32_t)(e0 + c));
                                q = add_lane_bit(q, m[c]);
                            }
                            run += __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
                        };
                        int s0 = 0;
                        for (; s0 + 2 * kSU <= nsl; s0 += kSU) {
#pragma unroll
                            for (int u = 0; u < kSU; ++u) {
                                slab(buf[u], s0 + u);
                                buf[u] = slab_load(s0 + u + kSU);
                            }
                        }
                        if (s0 + kSU <= nsl) {
#pragma unroll
                            for (int u = 0; u < kSU; ++u) {
                                slab(buf[u], s0 + u);
                                if (s0 + u + kSU < nsl) buf[u] = slab_load(s0 + u + kSU);
                            }
                            s0 += kSU;
                        }
#pragma unroll
                        for (int u = 0; u < kSU; ++u)
                            if (s0 + u < nsl) slab(buf[u], s0 + u);
                    };
                    if (test.flip)
                        repack(std::true_type{});
                    else
                        repack(std::false_type{});
                }
                keys_in_place(sm, sm.list + off, mine, false, 0u, 0u, lane);
                if (lane == 0) {
                    sm.seg_off[wave] = off;
                    sm.seg_cnt[wave] = mine;
                }
                ++passes;
                lds_barrier();
                overflow = false;
                f_spec = f_all;
                hist_ready = own_hist;
            }
        }

        if (S > 1) {
            // ---------------- publish the part; the last part of the row goes on.
            // Each wave writes its list at its offset in the part's packed,
            // index-ordered list. The parts of a row are launched on one XCD (the grid
            // mapping), so they share its L2: a part's plain stores have
            // reached that L2 once they complete (the vector L1 writes
            // through), and the last part reads them back from it with
            // device-scope loads, which do not use its L1. The arrival word,
            // updated by a device-scope atomic after the stores completed,
            // also counts the parts per XCD (5 bits per XCD above 16 bits of
            // arrivals): the last part uses the lists only if every part ran
            // on its XCD, and otherwise reads the whole row itself. On request
            // the atomic is an agent-scope release / acquire instead, the
            // memory model's form of this handoff (it writes back and
            // invalidates the XCD's L2 around the atomic).
            const int64_t slot0 = row * S;
            // The part's exact f(T_spec): every wave counted past its list's
            // capacity, so the sum is exact even after an overflow (bit 31).
            const int f_part = sum_over_waves<NW>(sm.wa, lane);
            if (!overflow) {
                const int off_w = sum_over_waves_below(sm.wa, lane, wave);
                uint64_t* pl = p.part_list + (slot0 + part) * kPartCap + off_w;
                const uint2* lw = sm.list + wave * W::kCapW;
                const int cnt = sm.wa[wave];
                for (int i = lane; i < cnt; i += kWave) pl[i] = pack_entry(lw[i].x, lw[i].y);
            }
            if (tid == 0) {
                p.part_count[slot0 + part] = (int32_t)((uint32_t)f_part | (overflow ? 0x80000000u : 0u));
                p.part_thresh[slot0 + part] = tthr;
            }
            if (own_hist && overflow) {   // this part's first refine level, as bin pairs (its list is incomplete)
                uint64_t* ph = reinterpret_cast<uint64_t*>(p.part_hist + (slot0 + part) * kRefBins1);
                for (int i = tid; i < kRefBins1 / 2; i += W::kBlock) ph[i] = reinterpret_cast<const uint64_t*>(sm.u.rhist)[i];
            }
            bool same_xcd = false;
            if (!arrive_last(&same_xcd)) return;   // another part of this row finishes it
            if (!same_xcd) {
                overflow = true;   // lists unusable: the fallback reads the whole row
                f_spec = -1;
            } else {
                // One round trip: every part's count and threshold (lane q:
                // part q) and, with at most four parts, the first entries of
                // every part's packed list (thread t: entries t + j * block),
                // loaded before it is known how many exist.
                const int c_tot = lane < S ? ld_agent(p.part_count + slot0 + lane) : 0;
                const uint32_t tp = lane < S ? (uint32_t)ld_agent((const int32_t*)p.part_thresh + slot0 + lane) : 0u;
                const bool spec_ld = S <= 4;
                const int spec_j = S <= 2 ? 2 : 1;   // chunks of one block per part
                uint64_t ev[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int q = spec_j == 2 ? k >> 1 : k, j = spec_j == 2 ? k & 1 : 0;
                    ev[k] = (spec_ld && q < S) ? ld_agent(p.part_list + (slot0 + q) * kPartCap + tid + j * W::kBlock)
                                               : 0ull;
                }
                // Totals of the row. Every part computes the same T_spec from
                // the same data; a part that kept another threshold (or
                // overflowed) sends the row to the fallback.
                const bool ovf = wave_max_u(lane < S && c_tot < 0 ? 1u : 0u) != 0u;
                const uint32_t trow = wave_max_u(tp);
                const bool mixed = wave_min_u(lane < S ? tp : 0xFFFFFFFFu) != trow;
                const int cc = c_tot & 0x7FFFFFFF;
                f_spec = mixed ? -1 : wave_sum(cc);
                overflow = ovf || mixed;
                tthr = trow;
                const int coff = wave_incl_scan(cc, lane) - cc;   // lane q: part q's offset in the merged list
                if (!mixed && own_hist && f_spec > cap) {
                    // The row's first refine level, which counts every key
                    // >= T_spec of the row: this part's own, plus the
                    // published level of every other part whose list
                    // overflowed (bin pair tid of each in one round trip),
                    // then the keys of the other parts' complete lists.
                    const uint32_t ovf_parts = (uint32_t)__ballot(lane < S && lane != part && c_tot < 0);
                    for (int i = tid; i < kRefBins1 / 2; i += W::kBlock) {
                        uint64_t hv[kMaxParts];
#pragma unroll
                        for (int k = 0; k < kMaxParts; ++k)
                            hv[k] = ((ovf_parts >> k) & 1u)
                                        ? ld_agent(reinterpret_cast<const uint64_t*>(p.part_hist + (slot0 + k) * kRefBins1) + i)
                                        : 0ull;
                        int2 h = reinterpret_cast<const int2*>(sm.u.rhist)[i];
#pragma unroll
                        for (int k = 0; k < kMaxParts; ++k) {
                            h.x += (int)(uint32_t)hv[k];
                            h.y += (int)(uint32_t)(hv[k] >> 32);
                        }
                        reinterpret_cast<int2*>(sm.u.rhist)[i] = h;
                    }
                    lds_barrier();   // the sums are in before the list keys are added
                    const uint32_t hsh2 = ref_shift(trow, max(gmax, trow));
                    for (int q = 0; q < S; ++q) {
                        const int cq = __builtin_amdgcn_readlane(c_tot, q);
                        if (q == part || cq < 0) continue;   // (wave-uniform)
                        const uint64_t* src = p.part_list + (slot0 + q) * kPartCap;
                        for (int i0 = 0; i0 < cq; i0 += 4 * W::kBlock) {
                            uint64_t e[4];
#pragma unroll
                            for (int u = 0; u < 4; ++u) {
                                const int i = i0 + u * W::kBlock + tid;
                                e[u] = i < cq ? ld_agent(src + i) : 0ull;
                            }
#pragma unroll
                            for (int u = 0; u < 4; ++u)
                                if (i0 + u * W::kBlock + tid < cq) ref_hist_add(sm, (uint32_t)e[u], trow, hsh2);
                        }
                    }
                    hist_full = true;   // complete behind the fallback's first barrier
                }
                if (!overflow && f_spec >= K && f_spec <= cap) {
                    // The merged list: the parts' packed lists one after the
                    // other (index order), split evenly over the waves. The
                    // other parts' keys join the refine's first level, which
                    // holds the own part's already.
                    const uint32_t msh = ref_shift(trow, max(gmax, trow));
                    auto put = [&](int P, uint64_t e, int q) {
                        sm.list[P] = make_uint2((uint32_t)e, (uint32_t)(e >> 32));
                        if (q != part && !all_mode) ref_hist_add(sm, (uint32_t)e, trow, msh);
                    };
                    if (spec_ld) {
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int q = spec_j == 2 ? k >> 1 : k, j = spec_j == 2 ? k & 1 : 0;
                            const int qq = min(q, S - 1);
                            const int cq = __builtin_amdgcn_readlane(cc, qq), oq = __builtin_amdgcn_readlane(coff, qq);
                            const int i = tid + j * W::kBlock;
                            if (q < S && i < cq) put(oq + i, ev[k], q);
                        }
                        // entries past the first spec_j blocks of a part (long lists)
                        for (int q = 0; q < S; ++q) {
                            const int cq = __builtin_amdgcn_readlane(cc, q), oq = __builtin_amdgcn_readlane(coff, q);
                            const uint64_t* src = p.part_list + (slot0 + q) * kPartCap;
                            for (int i0 = spec_j * W::kBlock; i0 < cq; i0 += 4 * W::kBlock) {
                                uint64_t e[4];
#pragma unroll
                                for (int u = 0; u < 4; ++u) {
                                    const int i = i0 + u * W::kBlock + tid;
                                    e[u] = i < cq ? ld_agent(src + i) : 0ull;
                                }
#pragma unroll
                                for (int u = 0; u < 4; ++u) {
                                    const int i = i0 + u * W::kBlock + tid;
                                    if (i < cq) put(oq + i, e[u], q);
                                }
                            }
                        }
                    } else {
                        // Thread t owns merged positions t + j * block and
                        // loads four of them (from their parts' lists) before
                        // it stores any.
                        for (int j0 = 0; j0 * W::kBlock < f_spec; j0 += 4) {
                            int qj[4] = {0, 0, 0, 0}, oj[4] = {0, 0, 0, 0};
                            for (int q = 1; q < S; ++q) {
                                const int bq = __builtin_amdgcn_readlane(coff, q);
#pragma unroll
                                for (int u = 0; u < 4; ++u) {
                                    const bool past = tid + (j0 + u) * W::kBlock >= bq;
                                    qj[u] += past;
                                    oj[u] = past ? bq : oj[u];
                                }
                            }
                            uint64_t e[4];
#pragma unroll
                            for (int u = 0; u < 4; ++u) {
                                const int P = tid + (j0 + u) * W::kBlock;
                                e[u] = P < f_spec ? ld_agent(p.part_list + (slot0 + qj[u]) * kPartCap + (P - oj[u])) : 0ull;
                            }
#pragma unroll
                            for (int u = 0; u < 4; ++u) {
                                const int P = tid + (j0 + u) * W::kBlock;
                                if (P < f_spec) put(P, e[u], qj[u]);
                            }
                        }
                    }
                    hist_ready = !all_mode;
                    const int chunk = (f_spec + NW - 1) / NW;
                    if (tid < NW) {
                        const int o = min(tid * chunk, f_spec);
                        sm.seg_off[tid] = o;
                        sm.seg_cnt[tid] = min(chunk, f_spec - o);
                    }
                                    lds_barrier();   // every wave reads the merged list, its segment table and histogram after this
                }
            }
            // Ready for the next call (issued after the loads above).
            if (tid == 0) __hip_atomic_store(p.arrivals + row, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }

    // The guess delivered (the usual case): refine the lists right away (the
    // lists, their segment table and the histogram are complete behind the
    // last barrier).
    if (spec && !all_mode && !overflow && f_spec >= K && f_spec <= cap) {
        const int64_t t3f = tstamp();
        int ngt = 0;
        int snaps = 0;
        const uint32_t kth = p.paper_refine
                                 ? paper_refine_emit(sm, K, out, tid, &ngt, &snaps)
                                 : refine_emit(sm, tthr, 0xFFFFFFFFu, max(gmax, tthr), 0, K, out, tid, &ngt, hist_ready);
        if (st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = GVR_PATH_GUESS;
            s.passes = passes;
            s.candidates = f_spec;
            s.threshold = tthr;
            s.kth_key = kth;
            s.n_gt = ngt;
            s.guess_valid = gvalid;
            s.spec_threshold = tspec;
            s.spec_count = f_spec;
            s.pmean = gvalid ? gsum / (float)gvalid : 0.f;
            s.refine_iters = snaps;
            s.t_start = t0;
            s.t_guess = t1;
            s.t_search = t2;
            s.t_collect = t3f;
            s.t_refine = stamp();
            *st = s;
        }
        return;
    }

    // Row-level decision (the single part, or the last part of the row).
    // Thread t owns the kBinsX bins from the top in groups of kFper:
    // bins kBins - kFper t - r, r < kFper (one bin each with 16 waves).
    constexpr int kFper = (kBinsX + W::kBlock - 1) / W::kBlock;
    auto compute_F = [&]() {
        __syncthreads();   // every wave's histogram updates are done
        int g[kFper];
        int mine = 0;
#pragma unroll
        for (int r = 0; r < kFper; ++r) {
            const int b = kBins - (kFper * tid + r);
            g[r] = 0;
            if (b >= 0)
                for (int v = 0; v < NW; ++v) g[r] += sm.u.hist[v][b];
            mine += g[r];
        }
        int a = mine;
        block_excl_scan(a, sm, tid);   // keys in the bins above this thread's
#pragma unroll
        for (int r = 0; r < kFper; ++r) {
            const int b = kBins - (kFper * tid + r);
            a += g[r];
            if (b >= 0) sm.F[b] = a;
        }
        if (tid == 0) sm.F[kBinsX] = 0;
        __syncthreads();
    };
    // Largest bin j with F[j] >= K (-1 if F[0] < K).
    auto crossing = [&]() {
        if (tid == 0) sm.scal[2] = -1;
        __syncthreads();
        for (int j = tid; j < kBinsX; j += W::kBlock)
            if (sm.F[j] >= K && sm.F[j + 1] < K) sm.scal[2] = j;
        __syncthreads();
        const int j = sm.scal[2];
        __syncthreads();
        return j;
    };
    int* hw = sm.u.hist[wave];
    Window win = make_window(0u, 0xFFFFFFFFu);
    // Count pass over window `win` (wave-private histograms, then F).
    auto count_pass = [&]() {
        __syncthreads();
        for (int i = tid; i < NW * kBinsX; i += W::kBlock) (&sm.u.hist[0][0])[i] = 0;
        __syncthreads();
        const uint32_t lo = win.lo, sh = win.shift;
        stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
            uint32_t k[4];
            block_keys(v, k);
            const int e0 = 4 * q - aoff;
            const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const bool okc = !edge || (e0 + c >= 0 && e0 + c < n);
                hist_add(hw, k[c], okc && k[c] >= lo, lo, sh);
            }
        });
        ++passes;
        __syncthreads();
        compute_F();
    };
    // The smallest and largest key of the row, in one pass: a count window
    // over the whole key range would crowd typical rows (values of a few
    // binades) into two or three of its bins and need an extra pass; the
    // first window spans [min, max] instead.
    auto minmax_pass = [&]() {
        uint32_t mn = 0xFFFFFFFFu, mx = 0u;
        stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
            uint32_t k[4];
            block_keys(v, k);
            const int e0 = 4 * q - aoff;
            const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const bool okc = !edge || (e0 + c >= 0 && e0 + c < n);
                mn = okc ? min(mn, k[c]) : mn;
                mx = okc ? max(mx, k[c]) : mx;
            }
        });
        ++passes;
        mn = wave_min_u(mn);
        mx = wave_max_u(mx);
        __syncthreads();
        if (lane == 0) {
            sm.red[2][wave] = (int)mn;
            sm.red[3][wave] = (int)mx;
        }
        __syncthreads();
        const uint32_t kmin = wave_min_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0xFFFFFFFFu);
        const uint32_t kmax = wave_max_u(lane < NW ? (uint32_t)sm.red[3][lane] : 0u);
        win = make_window(kmin, max(kmin, kmax));
    };
    // Radix digit pass: a histogram of the top 11 key bits (sign, exponent
    // and two mantissa bits: quarter-binade bins) of every element of the
    // row, in the first refine level's 2048 bins. Most elements of a row
    // fall in a few such bins, and same-address LDS atomics of one
    // instruction serialise, so the pass counts into kDigitCopies copies
    // (lane l adds to copy l % kDigitCopies; bin-major, so the copies of a
    // bin sit in different banks) in the lists' space, summed afterwards.
    constexpr int kDigitCopies = W::kCap * 2 >= kRefBins1 * 8 ? 8 : 4;
    static_assert(W::kCap * 2 >= kRefBins1 * kDigitCopies, "the digit histogram copies fit the lists' space");
    auto digit_pass = [&](int dqb, int dqe) {   // this wave's float4 blocks [dqb, dqe)
        int* dh = reinterpret_cast<int*>(sm.list);   // [kRefBins1][kDigitCopies]
        __syncthreads();
        for (int i = tid; i < kRefBins1 * kDigitCopies / 4; i += W::kBlock)
            reinterpret_cast<int4*>(dh)[i] = make_int4(0, 0, 0, 0);
        __syncthreads();
        int* dl = dh + (lane & (kDigitCopies - 1));
        stream_wave(xa, dqb, dqe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
            uint32_t k[4];
            block_keys(v, k);
            const int e0 = 4 * q - aoff;
            const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (!edge || (e0 + c >= 0 && e0 + c < n))
                    __hip_atomic_fetch_add(&dl[(k[c] >> kDigitShift) * kDigitCopies], 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
        });
        ++passes;
        __syncthreads();
        for (int i = tid; i < kRefBins1; i += W::kBlock) {
            const int4* c4 = reinterpret_cast<const int4*>(dh + i * kDigitCopies);
            int t = 0;
#pragma unroll
            for (int j = 0; j < kDigitCopies / 4; ++j) {
                const int4 v = c4[j];
                t += v.x + v.y + v.z + v.w;
            }
            sm.u.rhist[i] = t;
        }
        __syncthreads();
    };
    // Collect pass at threshold tc: every wave lists the keys >= tc of its
    // full-row share in its own list (up to kCapW entries, counted past
    // capacity: a share holds a few of them when f(tc) <= C is spread over
    // the row). A wave that overflowed sends the row through one more pass
    // at exact per-wave offsets. Returns f(tc); the lists hold every key >=
    // tc if it is at most C.
    auto collect_lists = [&](uint32_t tc) -> int {
        __syncthreads();   // the previous lists and histogram are dead
        // As in the speculative pass: the test on raw fp32 bits, every lane
        // stores each element (kept ones at their rank, the others to a
        // dummy slot in the histogram's space) while the slab fits the list.
        const uint32_t lc_addr = lds_addr(sm.list + wave * W::kCapW);
        const uint32_t dummy = lds_addr(sm.u.rhist) + 8 * lane;
        const bool every = tc == 0u;   // key 0 passes too: no compare
        const SpecTest test = make_spec_test(max(tc, 1u));
        int c = 0;
        stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
            const uint32_t k[4] = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)};
            const int e0 = 4 * q - aoff;
            bool f[4];
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) f[cc] = every || (int32_t)(k[cc] ^ test.flip) >= test.bound;
            if (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n) {   // an edge slab (wave-uniform)
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) f[cc] = f[cc] && e0 + cc >= 0 && e0 + cc < n;
            }
            const uint64_t m[4] = {__ballot(f[0]), __ballot(f[1]), __ballot(f[2]), __ballot(f[3])};
            const int total = __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
            if (c + total <= W::kCapW) {
                int qq = (int)lanes_below(m[3], lanes_below(m[2], lanes_below(m[1], lanes_below(m[0], (uint32_t)c))));
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    lds_store_pair(f[cc] ? lc_addr + 8 * qq : dummy, key_of_bits(k[cc]), (uint32_t)(e0 + cc));
                    qq = add_lane_bit(qq, m[cc]);
                }
            }
            c += total;   // counted past capacity
        });
        ++passes;
        if (lane == 0) sm.wa[wave] = c;
        __syncthreads();
        const int f = sum_over_waves<NW>(sm.wa, lane);
        const bool full = wave_max_u(lane < NW ? (uint32_t)sm.wa[lane] : 0u) > (uint32_t)W::kCapW;
        if (!full) {
            if (lane == 0) {
                sm.seg_off[wave] = wave * W::kCapW;
                sm.seg_cnt[wave] = c;
            }
        } else if (f <= cap) {
            const int off = sum_over_waves_below(sm.wa, lane, wave);
            __syncthreads();
            if (lane == 0) {
                sm.seg_off[wave] = off;
                sm.seg_cnt[wave] = c;
            }
            uint2* lp = sm.list + off;
            int run = 0;
            stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
                uint32_t k[4];
                block_keys(v, k);
                const int e0 = 4 * q - aoff;
                const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
                bool ff[4];
                uint64_t m[4];
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    ff[cc] = k[cc] >= tc && (!edge || (e0 + cc >= 0 && e0 + cc < n));
                    m[cc] = __ballot(ff[cc]);
                }
                int pos = run + (int)lanes_below(m[3], lanes_below(m[2], lanes_below(m[1], lanes_below(m[0], 0))));
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    if (ff[cc]) {
                        if (pos < c) lp[pos] = make_uint2(k[cc], (uint32_t)(e0 + cc));
                        ++pos;
                    }
                }
                run += __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
            });
            ++passes;
        }
            __syncthreads();
        return f;
    };

    int path = all_mode ? GVR_PATH_ALL : (have_prev ? GVR_PATH_GUESS : GVR_PATH_NO_GUESS);
    uint32_t T = 0, rlo = 0, rhi = 0xFFFFFFFFu, bin_hi = 0xFFFFFFFFu;
    bool use_hist = false;   // the refine's first level is already counted
    int above = 0, cands = 0;
    bool done_lists = false;   // lists hold every key >= T
    bool ties = false;
    uint32_t tstar = 0;
    int n_gt_row = 0;
    int64_t t3 = t1;

    // ---------------- the paper's schedule (Sec. 4.2.1-4.2.3), as an option:
    // Phase 1 over every valid guessed score, Phase 2 probes one threshold per
    // full-row counting pass (T0 = pmean, then secant steps toward f_target
    // inside the counted bracket, the first step damped to half the bracket,
    // bisection in key space when a step leaves it, at most kMaxSecant probes),
    // Phase 3 one collect pass at the accepted threshold.
    bool sec_ok = false;
    uint32_t sec_lo = 0u, sec_hi = 0xFFFFFFFFu;   // f(sec_lo) > C, f(sec_hi) < K (bracket, keys)
    uint32_t row_max = 0xFFFFFFFFu;
    if (secant) {
        if (tid < NW) sm.seg_off[tid] = 0;
        // Phase 1: all K guessed scores, 2 per thread.
        const int32_t* pv = p.prev + row * (int64_t)K;
        uint32_t mn = 0xFFFFFFFFu, mx = 0u;
        float sum = 0.f;
        int cnt = 0;
#pragma unroll
        for (int m = 0; m < (GVR_MAX_K + W::kBlock - 1) / W::kBlock; ++m) {
            const int j = tid + m * W::kBlock;
            const int idx = j < K ? pv[j] : -1;
            if (idx >= 0 && idx < n) {
                const float v = x[idx];
                const uint32_t kk = key_of(v);
                mn = min(mn, kk);
                mx = max(mx, kk);
                sum += v;
                ++cnt;
            }
        }
        cnt = wave_sum(cnt);
        mn = wave_min_u(mn);
        mx = wave_max_u(mx);
        sum = wave_sum_f(sum);
        if (lane == 0) {
            sm.red[0][wave] = cnt;
            sm.red[1][wave] = (int)mn;
            sm.red[2][wave] = (int)mx;
            sm.redf[wave] = sum;
        }
        __syncthreads();
        gvalid = sum_over_waves<NW>(sm.red[0], lane);
        gmax = wave_max_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0u);
        gsum = 0.f;
        for (int v = 0; v < NW; ++v) gsum += sm.redf[v];   // fixed order
        __syncthreads();
        t1 = tstamp();
        // f(T) over the row (per-wave counts kept in sm.wa for the collect);
        // the first pass also finds the row's smallest and largest key.
        auto count_ge = [&](uint32_t tk, bool minmax) {
            int c = 0;
            uint32_t lo = 0xFFFFFFFFu, hi = 0u;
            stream_wave(xa, qb, qe, qlast, lane, [] {}, [&](const float4& v, int q, int qs) {
                uint32_t k[4];
                block_keys(v, k);
                const int e0 = 4 * q - aoff;
                const bool edge = (4 * qs - aoff < 0 || 4 * qs + 255 - aoff >= n);
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    const bool okc = !edge || (e0 + cc >= 0 && e0 + cc < n);
                    c += (int)__popcll(__ballot(okc && k[cc] >= tk));
                    if (minmax && okc) {
                        lo = min(lo, k[cc]);
                        hi = max(hi, k[cc]);
                    }
                }
            });
            ++passes;
            if (minmax) {
                lo = wave_min_u(lo);
                hi = wave_max_u(hi);
            }
            if (lane == 0) {
                sm.wa[wave] = c;
                sm.red[1][wave] = (int)lo;
                sm.red[2][wave] = (int)hi;
            }
            __syncthreads();
            const int f = sum_over_waves<NW>(sm.wa, lane);
            if (minmax) {
                sec_lo = wave_min_u(lane < NW ? (uint32_t)sm.red[1][lane] : 0xFFFFFFFFu);
                row_max = wave_max_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0u);
            }
            __syncthreads();
            return f;
        };
        const int f_target = min(K + K / 2, (K + cap) / 2);
        uint32_t ka = gvalid > 0 ? key_of(gvalid > 0 ? gsum / (float)gvalid : 0.f) : 0x80000000u;   // T0 = pmean
        tspec = ka;
        int fa = count_ge(ka, true);
        f_spec = fa;
        // Bracket from the first pass: f(row min) = n > C, f(above row max) = 0 < K.
        int fl = n, fh = 0;
        sec_hi = row_max == 0xFFFFFFFFu ? 0xFFFFFFFFu : row_max + 1u;
        uint32_t kb = sec_hi;   // the other interpolation point
        int fb = 0;
        if (fa >= K && fa <= cap) {
            sec_ok = true;
        } else {
            if (fa > cap) {
                sec_lo = ka;
                fl = fa;
            } else {
                sec_hi = ka;
                fh = fa;
                kb = sec_lo;
                fb = fl;
            }
            for (int it = 0; it < kMaxSecant && !sec_ok; ++it) {
                if (sec_hi - sec_lo <= 1u) break;   // no admissible threshold: ties straddle [K, C]
                const float ta = float_of_key(ka), tb = float_of_key(kb);
                float t = ta + (float)(fa - f_target) * (tb - ta) / (float)(fa - fb);
                if (it == 0) {   // damping: at most half the bracket away from the last probe
                    const float half = 0.5f * (float_of_key(sec_hi) - float_of_key(sec_lo));
                    t = fminf(fmaxf(t, ta - half), ta + half);
                }
                uint32_t kn = key_of(t);
                if (!(t == t) || kn <= sec_lo || kn >= sec_hi) kn = sec_lo + (sec_hi - sec_lo) / 2u;   // bisect
                const int fn = count_ge(kn, false);
                kb = ka;
                fb = fa;
                ka = kn;
                fa = fn;
                if (fn >= K && fn <= cap) {
                    sec_ok = true;
                } else if (fn > cap) {
                    sec_lo = kn;
                    fl = fn;
                } else {
                    sec_hi = kn;
                    fh = fn;
                }
            }
        }
        (void)fl;
        (void)fh;
        t2 = tstamp();   // Phase 2 done (threshold accepted, or the search gave up)
        if (sec_ok) {
            // Phase 3: collect every key >= T at per-wave offsets from the
            // last pass's per-wave counts (sm.wa), in index order.
            T = ka;
            cands = fa;
            const int off = sum_over_waves_below(sm.wa, lane, wave);
            const int mine = sm.wa[wave];
            __syncthreads();
            if (lane == 0) {
                sm.seg_off[wave] = off;
                sm.seg_cnt[wave] = mine;
            }
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
            __syncthreads();
        }
    }

    if (secant && sec_ok) {
        // The collected lists hold every key >= T with K <= f(T) <= C (Lemma 1).
        path = GVR_PATH_SECANT;
        done_lists = true;
        rlo = T;
        rhi = 0xFFFFFFFFu;
        bin_hi = max(row_max, T);
        above = 0;
    } else if (spec && !overflow && f_spec >= K && f_spec <= cap) {
        // The speculative lists hold every key >= T_spec, hence the answer
        // (Lemma 1). The refine bins [T_spec, pmax] and puts the (few) keys
        // above pmax into its top bin.
        T = tthr;
        cands = f_spec;
        done_lists = true;
        use_hist = hist_ready && !all_mode;
        rlo = tthr;
        rhi = 0xFFFFFFFFu;
        bin_hi = max(gmax, tthr);
        above = 0;
        if (all_mode) {
            // No guess range: bin [min, max] of the (few) listed keys. When
            // they hold both signs the range is cut at the sign: the keys of
            // one sign lie binades away from the other's, so a range over
            // both would crowd each side into a few bins. With at least K
            // keys >= +0 the K-th key is one of them (range [min, max] of
            // those); otherwise it is negative, below all of them (range of
            // the negative keys, the others counted above it).
            constexpr uint32_t kPos = 0x80000000u;   // key of +0.0
            uint32_t mn = 0xFFFFFFFFu, mx = 0u;
            for_my_keys(sm, wave, lane, [&](uint32_t kk) {
                mn = min(mn, kk);
                mx = max(mx, kk);
            });
            mn = wave_min_u(mn);
            mx = wave_max_u(mx);
            if (lane == 0) {
                sm.red[2][wave] = (int)mn;
                sm.red[3][wave] = (int)mx;
            }
            __syncthreads();
            rlo = wave_min_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0xFFFFFFFFu);
            rhi = bin_hi = wave_max_u(lane < NW ? (uint32_t)sm.red[3][lane] : 0u);
            if (rlo < kPos && rhi >= kPos) {   // both signs (workgroup-uniform): one more pass
                uint32_t mn_p = 0xFFFFFFFFu, mx_n = 0u;
                int npos = 0;
                for_my_keys(sm, wave, lane, [&](uint32_t kk) {
                    const bool pos = kk >= kPos;
                    mn_p = pos ? min(mn_p, kk) : mn_p;
                    mx_n = pos ? mx_n : max(mx_n, kk);
                    npos += pos;
                });
                mn_p = wave_min_u(mn_p);
                mx_n = wave_max_u(mx_n);
                npos = wave_sum(npos);
                if (lane == 0) {
                    sm.red[0][wave] = (int)mn_p;
                    sm.red[1][wave] = (int)mx_n;
                    sm.wb[wave] = npos;
                }
                __syncthreads();
                const int np = sum_over_waves<NW>(sm.wb, lane);
                if (np >= K) {
                    rlo = wave_min_u(lane < NW ? (uint32_t)sm.red[0][lane] : 0xFFFFFFFFu);
                } else {
                    rhi = bin_hi = wave_max_u(lane < NW ? (uint32_t)sm.red[1][lane] : 0u);
                    above = np;
                }
            }
        }
    } else {
        bool whole_range = true;   // nothing bounds the K-th key yet
        bool digits_counted = false;   // rhist holds the row's digit histogram (split radix rows)
        if (!GUESS && S > 1) {
            // ---------------- a split radix row: each part counts the digits
            // of its share of the row (its waves split the part's slabs),
            // publishes the histogram, and the last part to arrive sums them
            // and goes on with the whole row (the handoff of the speculative
            // pass's merge). Parts that did not all run on one XCD leave the
            // last part to count the whole row itself.
            const int pw = (ps1 - ps0 + NW - 1) / NW;
            digit_pass(min((ps0 + min(wave * pw, ps1 - ps0)) * 64, nq), min((ps0 + min((wave + 1) * pw, ps1 - ps0)) * 64, nq));
            const int64_t slot0 = row * S;
            {
                uint64_t* ph = reinterpret_cast<uint64_t*>(p.part_hist + (slot0 + part) * kRefBins1);
                for (int i = tid; i < kRefBins1 / 2; i += W::kBlock) ph[i] = reinterpret_cast<const uint64_t*>(sm.u.rhist)[i];
            }
            bool same_xcd = false;
            if (!arrive_last(&same_xcd)) return;   // another part of this row finishes it
            if (same_xcd) {
                for (int i = tid; i < kRefBins1 / 2; i += W::kBlock) {
                    uint64_t hv[kMaxParts];
#pragma unroll
                    for (int k = 0; k < kMaxParts; ++k)
                        hv[k] = k < S ? ld_agent(reinterpret_cast<const uint64_t*>(p.part_hist + (slot0 + k) * kRefBins1) + i)
                                      : 0ull;
                    int sx = 0, sy = 0;
#pragma unroll
                    for (int k = 0; k < kMaxParts; ++k) {
                        sx += (int)(uint32_t)hv[k];
                        sy += (int)(uint32_t)(hv[k] >> 32);
                    }
                    reinterpret_cast<int2*>(sm.u.rhist)[i] = make_int2(sx, sy);
                }
                digits_counted = true;
            }
            // Ready for the next call (issued after the loads above).
            if (tid == 0) __hip_atomic_store(p.arrivals + row, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __syncthreads();   // the summed histogram is complete
        }
        if (secant) {
            // The secant search gave up: narrow inside its counted bracket.
            path = GVR_PATH_NARROWED;
            win = make_window(sec_lo, sec_hi - 1u);
            whole_range = false;
        }
        if (spec) {
            // The guess fell short (or a wave's list overflowed): count passes
            // over the whole row around T_spec, whose f is known.
            if (path == GVR_PATH_GUESS) path = GVR_PATH_NARROWED;
            if (f_spec >= 0) {   // else: unknown (lists unusable or overflowed), count the whole key range
                win = (f_spec < K) ? make_window(0u, tthr - 1u) : make_window(tthr, 0xFFFFFFFFu);
                whole_range = false;
            }
        }
        // What the speculative pass counted may name a threshold with
        // K <= f <= C right away: T_spec itself when its lists are
        // incomplete (a part's list overflowed), or, when f(T_spec) > C, the
        // lower edge of the first refine level's bin holding the K-th key
        // (the level counts every key >= T_spec). One collect pass then
        // lists the candidates; a crowded bin is narrowed by count passes.
        int coll = -1;   // f at the collect threshold tc (-1: none)
        uint32_t tc = 0u;
        if (spec && !secant && f_spec >= K && f_spec <= cap) {
            tc = tthr;
            coll = f_spec;
            rlo = tthr;
            rhi = 0xFFFFFFFFu;
            bin_hi = max(gmax, tthr);
            above = 0;
        } else if (spec && !secant && f_spec > cap && hist_full) {
            __syncthreads();   // the level is complete
            if (wave == 0) kth_bin_wave0(sm, sm.u.rhist, K, 0, lane);
            __syncthreads();
            const int b = sm.scal[0], above_b = sm.scal[2], cnt_b = sm.scal[3];
            __syncthreads();
            const uint32_t hsh = ref_shift(tthr, max(gmax, tthr));
            const uint64_t lo64 = (uint64_t)tthr + ((uint64_t)b << hsh);
            const uint64_t end64 = std::min<uint64_t>(lo64 + ((uint64_t)1 << hsh) - 1, 0xFFFFFFFFu);
            const uint32_t lo_b = (uint32_t)lo64;
            const uint32_t hi_b = b == kRefBins1 - 1 ? 0xFFFFFFFFu : (uint32_t)end64;   // the top bin is open
            if (above_b + cnt_b <= cap) {
                tc = lo_b;
                coll = above_b + cnt_b;
                rlo = lo_b;
                rhi = hi_b;
                bin_hi = (uint32_t)end64;
                above = b == kRefBins1 - 1 ? 0 : above_b;
            } else {
                win = make_window(lo_b, hi_b);
                whole_range = false;
            }
        }
        if (whole_range && coll < 0) {
            // Nothing bounds the K-th key: a digit pass, then the same choice
            // over its bins (a bin of more than C keys is narrowed).
            if (!digits_counted) digit_pass(qb, qe);
            if (wave == 0) kth_bin_wave0(sm, sm.u.rhist, K, 0, lane);
            __syncthreads();
            const int b = sm.scal[0], above_b = sm.scal[2], cnt_b = sm.scal[3];
            __syncthreads();
            const uint32_t lo_b = (uint32_t)b << kDigitShift;
            const uint32_t hi_b = lo_b + ((1u << kDigitShift) - 1u);
            if (above_b + cnt_b <= cap) {
                tc = lo_b;
                coll = above_b + cnt_b;
                rlo = lo_b;
                rhi = bin_hi = hi_b;
                above = above_b;
            } else {
                win = make_window(lo_b, hi_b);
            }
            whole_range = false;
        }
        if (coll >= 0) {
            const int f = collect_lists(tc);
            if (f == coll) {
                T = tc;
                cands = f;
                done_lists = true;
            } else {   // not what was counted (cannot happen): count from the row's [min, max]
                minmax_pass();
            }
        }
        if (!done_lists) {
        count_pass();
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
                bin_hi = rhi;
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
                        const bool okc = !edge || (e0 + c >= 0 && e0 + c < n);
                        fg[c] = okc && k[c] > tstar;
                        fe[c] = okc && k[c] == tstar;
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
        t2 = tstamp();
    }

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
        for (int i = tid; i < K; i += W::kBlock) out[i] = -1;
        if (st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = -1;
            s.passes = passes;
            *st = s;
        }
        return;
    }
    lds_barrier();
    t3 = tstamp();
    // ---------------- (a5) refine the listed candidates and emit
    int ngt = 0;
    int snaps = 0;
    const uint32_t kth = p.paper_refine ? paper_refine_emit(sm, K, out, tid, &ngt, &snaps)
                                        : refine_emit(sm, rlo, rhi, bin_hi, above, K, out, tid, &ngt, use_hist);
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
        s.refine_iters = snaps;
        s.t_start = t0;
        s.t_guess = t1;
        s.t_search = t2;
        s.t_collect = t3;
        s.t_refine = stamp();
        *st = s;
    }
}

template <int NW, bool NT>
__global__ __launch_bounds__(Shape<NW>::kBlock) void gvr_topk_kernel(Params p) { topk_body<true, NW, NT>(p); }
template <int NW>
__global__ __launch_bounds__(Shape<NW>::kBlock) void radix_topk_kernel(Params p) { topk_body<false, NW, false>(p); }

// ------------------------------------------------------------------ host side

int cu_count(int device) {
    static std::mutex m;
    static std::vector<int> cache;
    std::lock_guard<std::mutex> lk(m);
    if ((int)cache.size() <= device) cache.resize(device + 1, 0);
    if (cache[device] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || v <= 0) v = 256;
        cache[device] = v;
    }
    return cache[device];
}

// Device calls of the library-owned workspace cache.
struct HipDev {
    static int capturing(void* stream, bool* yes) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing((hipStream_t)stream, &cs) != hipSuccess) return 1;
        *yes = cs != hipStreamCaptureStatusNone;
        return 0;
    }
    static int alloc(void** p, size_t bytes) { return hipMalloc(p, bytes) == hipSuccess ? 0 : 1; }
    static int clear_async(void* p, size_t bytes, void* stream) {
        return hipMemsetAsync(p, 0, bytes, (hipStream_t)stream) == hipSuccess ? 0 : 1;
    }
};

gvr_host::WorkspaceCache<HipDev> g_workspaces;

// Scratch of the allocation-free entry point: the split-row workspace of up
// to kStaticSlots (row, part) slots (arrival words, counts, thresholds,
// per-wave counts, histograms, 128 KB of lists per slot: 34 MiB) as one device array.
// Each device that runs the library holds its own copy until the process
// ends. Its arrival words are zero when the library is loaded, and every
// launch leaves the words it used at zero again (the last part of a row
// resets its word), so they start at zero on every call.
constexpr size_t kScratchBytes = gvr_host::ws_layout(gvr_host::kStaticSlots).total;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The array's device address per device (hipGetSymbolAddress, once per
// device with that device current): host code uses it, never the array's
// name, which is a host-side stand-in.
gvr_status static_scratch(int device, void** out) {
    static std::mutex m;
    static std::vector<void*> ptrs;
    std::lock_guard<std::mutex> lk(m);
    if ((int)ptrs.size() <= device) ptrs.resize(device + 1, nullptr);
    if (!ptrs[device]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return GVR_ERR_HIP;
        ptrs[device] = ptr;
    }
    *out = ptrs[device];
    return GVR_OK;
}

// Where a split call's workspace comes from: the library's per-stream cache,
// the static array, or a buffer the caller passes in.
enum WsSource { kWsLibrary = 0, kWsStatic = 1, kWsCaller = 2 };

struct Workspace {
    WsSource source = kWsLibrary;
    void* base = nullptr;   // kWsCaller only
    size_t bytes = 0;
};

gvr_status run(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev,
               int32_t K, int32_t* out, void* stream, const gvr_options* opt, gvr_row_stats* stats,
               int use_guess, Workspace wsrc, const int32_t* gstats = nullptr) {
    gvr_host::CallOptions o;
    gvr_status st = gvr_host::validate(scores, B, ld, K, out, opt, use_guess, &o);
    if (st != GVR_OK) return st;
    int64_t caller_slots = 0;
    if (wsrc.source == kWsCaller) {
        if (wsrc.bytes > 0 && (!wsrc.base || (reinterpret_cast<uintptr_t>(wsrc.base) & 7))) return GVR_ERR_INVALID_ARG;
        caller_slots = gvr_host::ws_slots_fitting(wsrc.bytes);
    }
    if (B == 0) return GVR_OK;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return GVR_ERR_HIP;
    const int cus = cu_count(device);
    gvr_host::Plan plan;
    const int64_t max_slots = wsrc.source == kWsStatic   ? gvr_host::kStaticSlots
                              : wsrc.source == kWsCaller ? caller_slots
                                                         : gvr_host::kMaxSlots;
    st = gvr_host::plan_call(B, ld, K, prev != nullptr, o, cus, max_slots, wsrc.source != kWsLibrary, &plan);
    if (st != GVR_OK) return st;
    const bool guess = plan.guess;
    const int parts = plan.parts;
    gvr_host::WsPtrs ws;
    if (parts > 1) {
        if (wsrc.source == kWsStatic) {
            void* base = nullptr;
            st = static_scratch(device, &base);
            if (st != GVR_OK) return st;
            ws = gvr_host::ws_carve(base, gvr_host::kStaticSlots);
        } else if (wsrc.source == kWsCaller) {
            ws = gvr_host::ws_carve(wsrc.base, caller_slots);
        } else {
            st = g_workspaces.get(device, stream, B * (int64_t)parts, &ws);
            if (st != GVR_OK) return st;
        }
    }
    // Rows in launches of at most 2^24 (the grid holds 8 * chunk slots).
    const int64_t kRowsPerLaunch = (int64_t)1 << 24;
    for (int64_t r0 = 0; r0 < B; r0 += kRowsPerLaunch) {
        const int64_t rows = std::min<int64_t>(B - r0, kRowsPerLaunch);
        const int64_t rows_pad = (rows + kXcds - 1) / kXcds * kXcds;
        Params q;
        q.scores = scores + r0 * ld;
        q.ld = ld;
        q.row_len = row_len ? row_len + r0 : nullptr;
        q.prev = guess ? prev + r0 * K : nullptr;
        q.out = out + r0 * K;
        q.stats = stats ? stats + r0 : nullptr;
        q.K = K;
        q.capacity = plan.capacity;
        q.rows = (int32_t)rows;
        q.parts = parts;
        q.chunk = (int32_t)(rows_pad / kXcds * parts);
        q.scatter = o.scatter;
        q.secant = o.secant;
        q.paper_refine = o.paper_refine;
        q.arrivals = ws.arrivals;
        q.part_count = ws.part_count;
        q.part_thresh = ws.part_thresh;
        q.part_hist = ws.part_hist;
        q.part_list = ws.part_list;
        q.gstats = (guess && gstats) ? gstats + r0 * K : nullptr;
        q.ordered_merge = o.ordered_merge;
        const dim3 grid((unsigned)(rows_pad * parts));
        const hipStream_t hs = (hipStream_t)stream;
        if (plan.shape == kNWMid) {
            const dim3 block(Shape<kNWMid>::kBlock);
            if (guess)
                hipLaunchKernelGGL((gvr_topk_kernel<kNWMid, false>), grid, block, 0, hs, q);
            else
                hipLaunchKernelGGL(radix_topk_kernel<kNWMid>, grid, block, 0, hs, q);
        } else if (plan.shape == kNWShort) {
            const dim3 block(Shape<kNWShort>::kBlock);
            if (guess)
                hipLaunchKernelGGL((gvr_topk_kernel<kNWShort, false>), grid, block, 0, hs, q);
            else
                hipLaunchKernelGGL(radix_topk_kernel<kNWShort>, grid, block, 0, hs, q);
        } else {
            const dim3 block(Shape<kNWLong>::kBlock);
            if (guess && plan.stream_hint)
                hipLaunchKernelGGL((gvr_topk_kernel<kNWLong, true>), grid, block, 0, hs, q);
            else if (guess)
                hipLaunchKernelGGL((gvr_topk_kernel<kNWLong, false>), grid, block, 0, hs, q);
            else
                hipLaunchKernelGGL(radix_topk_kernel<kNWLong>, grid, block, 0, hs, q);
        }
        if (hipGetLastError() != hipSuccess) return GVR_ERR_HIP;
    }
    return GVR_OK;
}

}  // namespace

namespace gvr_internal {

gvr_status topk_with_guess_stats(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                                 const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                                 const gvr_options* options, gvr_row_stats* stats) {
    if (K < kGuessWords || !out_idx) return GVR_ERR_INVALID_ARG;
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats, 1, Workspace(),
               out_idx + (K - kGuessWords));
}

}  // namespace gvr_internal

extern "C" {

gvr_status gvr_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                    int32_t K, int32_t* out_idx, void* stream) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, nullptr, nullptr, 1, Workspace());
}

gvr_status radix_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                      int32_t K, int32_t* out_idx, void* stream) {
    (void)prev_topk;
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, nullptr, nullptr, 0, Workspace());
}

gvr_status gvr_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                       int32_t K, int32_t* out_idx, void* stream, const gvr_options* options,
                       gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats, 1, Workspace());
}

gvr_status gvr_topk_ex_noalloc(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                               const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                               const gvr_options* options, gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats, 1, Workspace{kWsStatic, nullptr, 0});
}

gvr_status radix_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                         int32_t* out_idx, void* stream, const gvr_options* options, gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, options, stats, 0, Workspace());
}

gvr_status gvr_workspace_size(int64_t B, int64_t ld, int32_t K, int use_guess, const gvr_options* options,
                              size_t* bytes) {
    if (!bytes) return GVR_ERR_INVALID_ARG;
    *bytes = 0;
    gvr_host::CallOptions o;
    gvr_status st = gvr_host::validate_sizes(B, ld, K, options, use_guess ? 1 : 0, &o);
    if (st != GVR_OK) return st;
    if (B == 0) return GVR_OK;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return GVR_ERR_HIP;
    gvr_host::Plan plan;
    st = gvr_host::plan_call(B, ld, K, use_guess != 0, o, cu_count(device), gvr_host::kMaxCallerSlots, true, &plan);
    if (st != GVR_OK) return st;
    if (plan.parts > 1) *bytes = gvr_host::ws_layout(B * (int64_t)plan.parts).total;
    return GVR_OK;
}

gvr_status gvr_topk_ex_ws(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                          const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                          const gvr_options* options, gvr_row_stats* stats, void* workspace, size_t ws_bytes) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats, 1,
               Workspace{kWsCaller, workspace, ws_bytes});
}

gvr_status radix_topk_ex_ws(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                            int32_t* out_idx, void* stream, const gvr_options* options, gvr_row_stats* stats,
                            void* workspace, size_t ws_bytes) {
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, options, stats, 0,
               Workspace{kWsCaller, workspace, ws_bytes});
}

const char* gvr_status_string(gvr_status s) {
    switch (s) {
        case GVR_OK: return "ok";
        case GVR_ERR_INVALID_ARG: return "invalid argument";
        case GVR_ERR_UNSUPPORTED_K: return "unsupported K (1 <= K <= 2048)";
        case GVR_ERR_WORKSPACE: return "a forced split needs more workspace than the call was given";
        case GVR_ERR_HIP: return "HIP runtime error";
        case GVR_ERR_TOO_LONG: return "row stride too long";
    }
    return "unknown status";
}

const char* gvr_version(void) { return "gvr_topk 0.3 (gfx950, split rows, last-part merge)"; }

}  // extern "C"
