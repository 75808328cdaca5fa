// host_plan.h -- host-side planning of a Top-K call: argument checks, the
// workgroup shape, the row split, and the split-row workspace (its layout and
// the per-stream cache). Plain C++ with no HIP dependency, so the library and
// a sanitizer build on the CPU compile the same code.
#ifndef GVR_HOST_PLAN_H
#define GVR_HOST_PLAN_H

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "gvr_topk.h"

namespace gvr_host {

// Workgroup shapes (waves per workgroup) and the candidate capacity C each
// holds in LDS.
constexpr int kNWLong = 16;    // 1024 entries per wave, one workgroup per compute unit
constexpr int kNWMid = 8;      // 768 entries per wave, two per compute unit
constexpr int kNWShort = 4;    // 1024 entries per wave, three per compute unit
constexpr int kCapLong = GVR_MAX_CANDIDATES;
constexpr int kCapMid = 8 * 768;
constexpr int kCapShort = 4 * 1024;

constexpr int kMaxParts = 16;          // workgroups per row
constexpr int kMinPartElems = 16384;   // a batch row is split only into parts at least this long
constexpr int kMaxSlots = 2048;        // (row, part) slots of one call, library-owned workspace
constexpr int kStaticSlots = GVR_NOALLOC_SLOTS;   // (row, part) slots of the allocation-free entry point
constexpr int kXcds = 8;               // gfx950 XCDs; workgroup i runs on XCD i % 8
// Longest row stride of the guess path: its speculative pass addresses a row
// through one buffer resource with 32-bit byte offsets (lane offset included),
// so 4 (ld + 3) + 1024 must stay below 2^31. Longer rows take the guess-free
// schedule, whose passes index the row with 64-bit addresses.
constexpr int64_t kMaxSpecLd = ((int64_t)1 << 29) - 4096;
constexpr int kPartCap = GVR_MAX_CANDIDATES;   // list entries of one (row, part) slot
constexpr int kSlotHistBins = 2048;            // bins of a part's first refine histogram level

// Options of one call after validation.
struct CallOptions {
    int capacity = GVR_MAX_CANDIDATES;
    int use_guess = 1;
    int parts = 0;          // 0: automatic
    int scatter = 0;
    int secant = 0;
    int paper_refine = 0;
    int shape = 0;          // 0: automatic
    int ordered_merge = 0;  // agent-scope release / acquire at a split row's merge
};

// Sizes and options of a call, without its pointers (the workspace query
// takes no arrays).
inline gvr_status validate_sizes(int64_t B, int64_t ld, int32_t K, const gvr_options* opt, int use_guess,
                                 CallOptions* o) {
    *o = CallOptions();
    o->use_guess = use_guess;
    if (K < 1 || K > GVR_MAX_K) return GVR_ERR_UNSUPPORTED_K;
    if (B < 0 || ld < 0) return GVR_ERR_INVALID_ARG;
    if (ld > (int64_t)0x7FFFFFF0) return GVR_ERR_TOO_LONG;
    if (opt) {
        if (opt->capacity != 0) {
            if (opt->capacity < K || opt->capacity > GVR_MAX_CANDIDATES) return GVR_ERR_INVALID_ARG;
            o->capacity = opt->capacity;
        }
        if ((opt->flags & ~255) || opt->reserved1) return GVR_ERR_INVALID_ARG;
        const int forced = (opt->flags >> 4) & 7;
        if (forced & (forced - 1)) return GVR_ERR_INVALID_ARG;   // two shapes forced
        if (opt->parts < 0 || opt->parts > kMaxParts) return GVR_ERR_INVALID_ARG;
        if (opt->flags & 1) o->use_guess = 0;
        o->scatter = (opt->flags >> 1) & 1;
        o->secant = (opt->flags >> 2) & 1;
        o->paper_refine = (opt->flags >> 3) & 1;
        o->ordered_merge = (opt->flags >> 7) & 1;
        o->shape = forced == 1 ? kNWShort : forced == 2 ? kNWLong : forced == 4 ? kNWMid : 0;
        o->parts = opt->parts;
    }
    return GVR_OK;
}

inline gvr_status validate(const void* scores, int64_t B, int64_t ld, int32_t K, const void* out,
                           const gvr_options* opt, int use_guess, CallOptions* o) {
    const gvr_status st = validate_sizes(B, ld, K, opt, use_guess, o);
    if (st != GVR_OK) return st;
    if (B > 0 && (!scores || !out)) return GVR_ERR_INVALID_ARG;
    return GVR_OK;
}

// Parts per row. Splitting a row over S workgroups divides its streaming
// time (one workgroup reads about 33 GB/s on MI355X) but costs the merge of
// the parts' candidate lists, about 8 us of memory round trips when many
// rows merge at once; split only when the time saved is larger, keep parts
// >= kMinPartElems long and stay within the compute units. A call of one or
// two rows leaves the chip nearly idle and its merges cost a few us: there
// 8 parts pay from 32K elements on and 16 from 192K (one row of 32K: 13.1 us
// in 8 parts, 13.7 in 4, 13.4 unsplit; 70K: 14.0 in 8, 14.8 in 4; 262K:
// 15.2 in 16, 16.0 in 8).
inline int choose_parts(int64_t rows, int64_t ld, int cus, bool radix = false) {
    if (rows <= 0 || rows >= cus) return 1;
    if (rows <= 2 && ld >= 32768 && cus >= 32 * rows) return ld < 196608 ? 8 : kMaxParts;
    // Up to a quarter as many rows as compute units, from 48K elements on:
    // four to eight parts per row (measured with a guess: 16 rows of 64K
    // 16.8 -> 14.9 us in 8 parts, 48 rows 17.0 -> 15.6 in 5, 32 rows of 57K
    // 16.2 -> 15.3 in 8; at 40K splitting gains nothing, and two parts never
    // pay for their merge).
    if (!radix && ld >= 49152 && cus / rows >= 4)
        return (int)std::min<int64_t>(std::min<int64_t>(cus / rows, kMaxParts), ld < 196608 ? 8 : kMaxParts);
    int64_t s = cus / rows;
    s = std::min<int64_t>(s, std::max<int64_t>(1, ld / kMinPartElems));
    s = std::min<int64_t>(s, kMaxParts);
    if (s <= 1) return 1;
    // One workgroup's time for the pass the parts share: the speculative
    // pass (~33 GB/s), or the radix digit pass (~25 GB/s, and the parts'
    // handoff is only the histograms).
    const double stream_us = (double)ld * 4.0 / (radix ? 25.0e3 : 33.0e3);
    const double saved_us = stream_us * (1.0 - 1.0 / (double)s);
    return saved_us > (radix ? 4.0 : 8.0) ? (int)s : 1;
}

// Workgroup shape of a call: waves per workgroup (16, 8 or 4). Up to one row
// per compute unit, 16 waves: one round of rows at the shortest per-row
// latency, and row splitting. With more rows, the rows run in rounds of one
// (16 waves), two (8) or three (4) workgroups per compute unit; the 8-wave
// shape has the best rate of rows per compute unit when the previous Top-K
// guides the rows (decode rows of 8K-64K elements: 1024 rows of 32K take
// 42 us against 55 with 16 waves and 73 with 4), except for rows longer
// than 40K in at most two rows per compute unit, where the 16-wave shape's
// shorter latency wins (512 rows of 64K: 40 us against 47); from 48K on
// the two are even at four rows per compute unit. Without a usable guess
// the radix schedule runs, where rows of at most 4K go to 4 waves (2048
// rows of 4K: 47 us against 73 with 8 waves) and longer ones to 8.
inline int choose_shape(int64_t rows, int64_t ld, int cus, bool guess) {
    if (rows <= cus) return kNWLong;
    if (!guess) return ld <= 4096 ? kNWShort : kNWMid;
    if (ld <= 40960 || rows > 2 * (int64_t)cus) return kNWMid;
    return kNWLong;
}

// The launch plan of one call.
struct Plan {
    bool guess = false;   // the guess kernel runs (else the guess-free one)
    int shape = kNWLong;  // waves per workgroup
    int capacity = GVR_MAX_CANDIDATES;
    int parts = 1;        // workgroups per row
    bool stream_hint = false;   // the speculative pass loads with the non-temporal hint
};

// Calls whose speculative pass loads its rows with the non-temporal hint:
// one round of 16-wave workgroups over at least 16 MiB of rows, whose rows
// stream from HBM and are read once. Measured per call: 128 rows of 100K
// 22.0 -> 21.2 us, 48 rows of 64K-256K 24.2 -> 23.7 us, and even after the
// indexer has just written the 128 rows; smaller calls (rows that a cache
// may still hold: 32 rows of 32K, 8 of 131K, single rows) and the batched
// 8-wave shape lose 0.1-3 us with it.
constexpr int64_t kStreamHintBytes = (int64_t)16 << 20;

// `max_slots` bounds rows * parts (the workspace's slots). An automatic split
// is lowered to fit; a split forced through the options is lowered too unless
// `reject_forced` is set, in which case a forced split that does not fit is
// GVR_ERR_WORKSPACE.
inline gvr_status plan_call(int64_t B, int64_t ld, int32_t K, bool have_prev, const CallOptions& o, int cus,
                            int64_t max_slots, bool reject_forced, Plan* out) {
    Plan p;
    // Rows of at most 2K elements list every element (the guess would cut
    // few candidates): when no row is longer, the guess-free kernel runs.
    p.guess = o.use_guess && have_prev && ld > 2 * (int64_t)K && ld <= kMaxSpecLd;
    p.shape = o.shape != 0 ? o.shape : choose_shape(B, ld, cus, p.guess);
    // A smaller C never changes the result.
    p.capacity = o.capacity;
    if (p.shape == kNWShort) p.capacity = std::min(p.capacity, kCapShort);
    if (p.shape == kNWMid) p.capacity = std::min(p.capacity, kCapMid);
    int parts = 1;
    const bool secant = p.guess && o.secant;   // the secant search reads whole rows
    if (p.shape == kNWLong && !secant) {
        if (o.parts > 0) {
            parts = o.parts;
            if (parts > 1 && (int64_t)parts * B > max_slots) {
                if (reject_forced) return GVR_ERR_WORKSPACE;
                parts = (int)std::max<int64_t>(1, max_slots / std::max<int64_t>(B, 1));
            }
        } else {
            parts = choose_parts(B, ld, cus, !p.guess);
            if (parts > 1 && (int64_t)parts * B > max_slots)
                parts = (int)std::max<int64_t>(1, max_slots / std::max<int64_t>(B, 1));
        }
    }
    p.parts = parts;
    p.stream_hint = p.guess && p.shape == kNWLong && B <= (int64_t)cus && B * ld * 4 >= kStreamHintBytes;
    *out = p;
    return GVR_OK;
}

// ------------------------------------------------------------ split-row workspace
// Layout for `slots` (row, part) slots: arrival words [rows <= slots] u64,
// part counts [slots] i32, part thresholds [slots] u32, part histograms
// [slots][kSlotHistBins] i32, part lists [slots][kPartCap] u64; each array
// starts on a 256-byte boundary.
constexpr size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct WsLayout {
    size_t arrivals, counts, thresh, hists, lists, total;
};

constexpr WsLayout ws_layout(int64_t slots) {
    const size_t s = (size_t)(slots < 0 ? 0 : slots);
    const size_t a = 0;
    const size_t c = a + align_up(s * sizeof(uint64_t), 256);
    const size_t t = c + align_up(s * sizeof(int32_t), 256);
    const size_t h = t + align_up(s * sizeof(uint32_t), 256);
    const size_t l = h + align_up(s * kSlotHistBins * sizeof(int32_t), 256);
    return WsLayout{a, c, t, h, l, l + s * (size_t)kPartCap * sizeof(uint64_t)};
}

struct WsPtrs {
    uint64_t* arrivals = nullptr;
    int32_t* part_count = nullptr;
    uint32_t* part_thresh = nullptr;
    int32_t* part_hist = nullptr;
    uint64_t* part_list = nullptr;
};

// Most (row, part) slots whose layout fits in `bytes` (0 if not even one),
// capped at kMaxCallerSlots.
constexpr int64_t kMaxCallerSlots = (int64_t)1 << 24;
inline int64_t ws_slots_fitting(size_t bytes) {
    const size_t per_slot = sizeof(uint64_t) + sizeof(int32_t) + sizeof(uint32_t) +
                            kSlotHistBins * sizeof(int32_t) + (size_t)kPartCap * sizeof(uint64_t);
    int64_t s = (int64_t)std::min<size_t>(bytes / per_slot, (size_t)kMaxCallerSlots);
    while (s > 0 && ws_layout(s).total > bytes) --s;
    return s;
}

inline WsPtrs ws_carve(void* base, int64_t slots) {
    const WsLayout L = ws_layout(slots);
    char* b = static_cast<char*>(base);
    WsPtrs w;
    w.arrivals = reinterpret_cast<uint64_t*>(b + L.arrivals);
    w.part_count = reinterpret_cast<int32_t*>(b + L.counts);
    w.part_thresh = reinterpret_cast<uint32_t*>(b + L.thresh);
    w.part_hist = reinterpret_cast<int32_t*>(b + L.hists);
    w.part_list = reinterpret_cast<uint64_t*>(b + L.lists);
    return w;
}

// Library-owned workspaces, one per (device, stream), grown on demand. `Dev`
// supplies the device calls (all return 0 on success):
//   int Dev::capturing(void* stream, bool* yes)    -- is the stream being captured
//   int Dev::alloc(void** p, size_t bytes)         -- device allocation
//   int Dev::clear_async(void* p, size_t bytes, void* stream)
// An outgrown buffer is retired, never freed: graphs captured earlier may
// still hold it in their kernel arguments, and launches queued on the stream
// may still use it. Every buffer lives until the process ends.
template <class Dev>
class WorkspaceCache {
public:
    struct Entry {
        int device;
        void* stream;
        int64_t slots;
        void* base;
    };

    gvr_status get(int device, void* stream, int64_t slots, WsPtrs* out) {
        std::lock_guard<std::mutex> lk(mu_);
        for (size_t i = 0; i < live_.size(); ++i) {
            Entry& e = live_[i];
            if (e.device == device && e.stream == stream) {
                if (e.slots >= slots) {
                    *out = ws_carve(e.base, e.slots);
                    return GVR_OK;
                }
                retired_.push_back(e.base);
                live_.erase(live_.begin() + (ptrdiff_t)i);
                break;
            }
        }
        bool cap = false;
        if (Dev::capturing(stream, &cap) != 0 || cap) return GVR_ERR_HIP;   // no allocation under capture
        const WsLayout L = ws_layout(slots);
        void* base = nullptr;
        if (Dev::alloc(&base, L.total) != 0 || !base) return GVR_ERR_HIP;
        // Arrival words start at zero; cleared on the call's own stream, ahead of its launch.
        if (Dev::clear_async(base, L.counts, stream) != 0) {
            retired_.push_back(base);
            return GVR_ERR_HIP;
        }
        live_.push_back(Entry{device, stream, slots, base});
        *out = ws_carve(base, slots);
        return GVR_OK;
    }

    size_t live_count() {
        std::lock_guard<std::mutex> lk(mu_);
        return live_.size();
    }
    size_t retired_count() {
        std::lock_guard<std::mutex> lk(mu_);
        return retired_.size();
    }

private:
    std::mutex mu_;
    std::vector<Entry> live_;
    std::vector<void*> retired_;
};

}  // namespace gvr_host

#endif  // GVR_HOST_PLAN_H
