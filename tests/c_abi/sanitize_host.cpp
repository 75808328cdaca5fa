// CPU-only driver built with AddressSanitizer and UndefinedBehaviorSanitizer
// (g++ / gcc, no GPU code): the host-side planning of a Top-K call
// (paper_2604_22312_amd/csrc/host_plan.h: argument checks, workgroup shape
// and row split, workspace layout, the per-stream workspace cache with its
// growth and keep-alive rule) and the C oracle (oracle/oracle_topk.c) against
// a brute-force full sort on tie-heavy rows with special values. Prints "ok".
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <limits>
#include <random>
#include <vector>

#include "host_plan.h"

extern "C" int oracle_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                           int32_t* out_idx, uint32_t* kth_key, int32_t* n_gt);

#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            exit(1);                                                      \
        }                                                                 \
    } while (0)

// A device stand-in: a static bump pool (nothing to leak), capture flag.
static unsigned char g_pool[64 << 20];
static size_t g_used = 0;
static bool g_capturing = false;
static int g_allocs = 0;
struct FakeDev {
    static int capturing(void*, bool* yes) {
        *yes = g_capturing;
        return 0;
    }
    static int alloc(void** p, size_t bytes) {
        const size_t a = (g_used + 255) / 256 * 256;
        if (a + bytes > sizeof(g_pool)) return 1;
        *p = g_pool + a;
        g_used = a + bytes;
        ++g_allocs;
        return 0;
    }
    static int clear_async(void* p, size_t bytes, void*) {
        memset(p, 0, bytes);
        return 0;
    }
};

static void check_validate() {
    using namespace gvr_host;
    CallOptions o;
    int dummy;
    CHECK(validate(&dummy, 4, 100, 0, &dummy, nullptr, 1, &o) == GVR_ERR_UNSUPPORTED_K);
    CHECK(validate(&dummy, 4, 100, 2049, &dummy, nullptr, 1, &o) == GVR_ERR_UNSUPPORTED_K);
    CHECK(validate(&dummy, -1, 100, 16, &dummy, nullptr, 1, &o) == GVR_ERR_INVALID_ARG);
    CHECK(validate(&dummy, 4, -1, 16, &dummy, nullptr, 1, &o) == GVR_ERR_INVALID_ARG);
    CHECK(validate(nullptr, 4, 100, 16, &dummy, nullptr, 1, &o) == GVR_ERR_INVALID_ARG);
    CHECK(validate(nullptr, 0, 100, 16, nullptr, nullptr, 1, &o) == GVR_OK);
    CHECK(validate(&dummy, 1, (int64_t)1 << 40, 16, &dummy, nullptr, 1, &o) == GVR_ERR_TOO_LONG);
    gvr_options bad[] = {{100, 0, 0, 0}, {0, 48, 0, 0}, {0, 256, 0, 0}, {0, 0, 17, 0}, {0, 0, -1, 0}, {0, 0, 0, 1},
                         {20000, 0, 0, 0}};
    for (const auto& b : bad) CHECK(validate(&dummy, 2, 100, 128, &dummy, &b, 1, &o) == GVR_ERR_INVALID_ARG);
    gvr_options good = {4096, 1 | 8 | 64 | 128, 3, 0};
    CHECK(validate(&dummy, 2, 100, 128, &dummy, &good, 1, &o) == GVR_OK);
    CHECK(o.capacity == 4096 && o.use_guess == 0 && o.paper_refine == 1 && o.shape == kNWMid && o.parts == 3 &&
          o.ordered_merge == 1);
}

static void check_plans() {
    using namespace gvr_host;
    CallOptions o;
    Plan p;
    // the benchmark's call: 128 rows of ~102K with a guess, 256 compute units
    CHECK(plan_call(128, 102463, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK);
    CHECK(p.guess && p.shape == kNWLong && p.parts == 1 && p.capacity == GVR_MAX_CANDIDATES && p.stream_hint);
    // the non-temporal hint: one round of 16-wave workgroups over >= 16 MiB of rows only
    CHECK(plan_call(48, 262144, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.stream_hint);
    CHECK(plan_call(32, 32831, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.stream_hint);
    CHECK(plan_call(8, 131079, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.stream_hint);
    CHECK(plan_call(512, 65537, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.shape == kNWLong &&
          !p.stream_hint);
    CHECK(plan_call(128, 102463, 2048, false, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.stream_hint);
    // 8 rows of 131K split into 8 parts; one row of 262K into 16
    CHECK(plan_call(8, 131079, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 8);
    CHECK(plan_call(1, 262144, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 16);
    CHECK(plan_call(1, 32768, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 8);
    CHECK(plan_call(2, 70690, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 8);
    CHECK(plan_call(1, 16384, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 1);
    // few rows from 48K elements: four to eight parts (with a guess)
    CHECK(plan_call(16, 65536, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 8);
    CHECK(plan_call(48, 65536, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 5);
    CHECK(plan_call(64, 102400, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 4);
    CHECK(plan_call(32, 40000, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 1);
    CHECK(plan_call(65, 65536, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 1);
    // no guess: the radix schedule splits few long rows too (8 parts of 131K),
    // not 100K rows at 128 per call and 32K rows at 32; short rows: 4 waves;
    // mid rows: 8 waves with their capacities
    CHECK(plan_call(8, 131079, 2048, false, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.guess && p.parts == 8);
    CHECK(plan_call(32, 32831, 2048, false, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.guess && p.parts == 1);
    // the secant search never splits; the radix schedule with the secant flag still may
    o.secant = 1;
    CHECK(plan_call(8, 131079, 2048, false, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.guess && p.parts == 8);
    o.secant = 0;
    CHECK(plan_call(2048, 4000, 2048, false, o, 256, kMaxSlots, false, &p) == GVR_OK && p.shape == kNWShort &&
          p.capacity == kCapShort);
    CHECK(plan_call(1024, 32768, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.shape == kNWMid &&
          p.capacity == kCapMid);
    // rows of at most 2K: the guess-free kernel
    CHECK(plan_call(4, 4096, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && !p.guess);
    // forced splits: lowered to the slots, or refused (allocation-free entry point)
    o.parts = 16;
    CHECK(plan_call(200, 50000, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == kMaxSlots / 200);
    CHECK(plan_call(17, 50000, 2048, true, o, 256, kStaticSlots, true, &p) == GVR_ERR_WORKSPACE);
    CHECK(plan_call(16, 50000, 2048, true, o, 256, kStaticSlots, true, &p) == GVR_OK && p.parts == 16);
    // the secant search never splits
    o.secant = 1;
    CHECK(plan_call(8, 131079, 2048, true, o, 256, kMaxSlots, false, &p) == GVR_OK && p.parts == 1);
    // choose_parts over many shapes stays within the compute units and the part limit
    for (int64_t rows = 1; rows <= 300; rows += 7)
        for (int64_t ld = 1000; ld <= 300000; ld = ld * 3 / 2) {
            const int s = choose_parts(rows, ld, 256);
            CHECK(s >= 1 && s <= kMaxParts && (s == 1 || rows * s <= 256 * 2));
        }
}

static void check_workspace() {
    using namespace gvr_host;
    // layout: every array 256-byte aligned, in order, sized for the slots
    for (int64_t slots : {1, 2, 7, 64, 256, 2048}) {
        const WsLayout L = ws_layout(slots);
        CHECK(L.arrivals == 0 && L.counts % 256 == 0 && L.thresh % 256 == 0 && L.hists % 256 == 0 &&
              L.lists % 256 == 0);
        CHECK(L.counts >= (size_t)slots * 8 && L.thresh - L.counts >= (size_t)slots * 4 &&
              L.hists - L.thresh >= (size_t)slots * 4 && L.lists - L.hists >= (size_t)slots * kSlotHistBins * 4);
        CHECK(L.total == L.lists + (size_t)slots * kPartCap * 8);
    }
    // a caller's buffer of ws_layout(n).total bytes holds n slots, and one byte fewer does not
    CHECK(ws_slots_fitting(0) == 0 && ws_slots_fitting(ws_layout(1).total - 1) == 0);
    for (int64_t slots : {1, 2, 7, 64, 255, 256, 2048, 5000}) {
        CHECK(ws_slots_fitting(ws_layout(slots).total) == slots);
        CHECK(ws_slots_fitting(ws_layout(slots).total - 1) == slots - 1);
        CHECK(ws_slots_fitting(ws_layout(slots + 1).total - 1) == slots);
    }
    CHECK(ws_slots_fitting((size_t)1 << 62) == kMaxCallerSlots);
    // a caller's workspace plans: automatic splits lowered to the slots that fit, forced ones refused
    {
        CallOptions o;
        Plan p;
        CHECK(plan_call(8, 131079, 2048, true, o, 256, 64, true, &p) == GVR_OK && p.parts == 8);
        CHECK(plan_call(8, 131079, 2048, true, o, 256, 40, true, &p) == GVR_OK && p.parts == 5);
        CHECK(plan_call(8, 131079, 2048, true, o, 256, 0, true, &p) == GVR_OK && p.parts == 1);
        o.parts = 4;
        CHECK(plan_call(8, 131079, 2048, true, o, 256, 31, true, &p) == GVR_ERR_WORKSPACE);
        CHECK(plan_call(8, 131079, 2048, true, o, 256, 32, true, &p) == GVR_OK && p.parts == 4);
        o.parts = 1;
        CHECK(plan_call(8, 131079, 2048, true, o, 256, 0, true, &p) == GVR_OK && p.parts == 1);
    }
    // the cache: reuse, growth with the outgrown buffer kept, refusal under capture
    WorkspaceCache<FakeDev> cache;
    int s1 = 0, s2 = 0;
    void* streamA = &s1;
    void* streamB = &s2;
    WsPtrs a, b, c, d;
    CHECK(cache.get(0, streamA, 8, &a) == GVR_OK && g_allocs == 1);
    a.arrivals[0] = 5;   // a kernel would leave it at zero; reuse must not clear it again
    CHECK(cache.get(0, streamA, 4, &b) == GVR_OK && g_allocs == 1 && b.arrivals == a.arrivals && b.arrivals[0] == 5);
    a.arrivals[0] = 0;
    CHECK(cache.get(0, streamA, 32, &c) == GVR_OK && g_allocs == 2 && c.arrivals != a.arrivals);
    CHECK(cache.retired_count() == 1 && cache.live_count() == 1);
    for (int i = 0; i < 32; ++i) CHECK(c.arrivals[i] == 0);
    c.part_list[32 * (int64_t)kPartCap - 1] = 7;   // the last entry of the last slot is inside the buffer
    CHECK(cache.get(1, streamA, 8, &d) == GVR_OK && g_allocs == 3 && cache.live_count() == 2);
    g_capturing = true;
    CHECK(cache.get(0, streamB, 8, &d) == GVR_ERR_HIP && g_allocs == 3);
    CHECK(cache.get(0, streamA, 16, &d) == GVR_OK && d.arrivals == c.arrivals);   // no allocation needed
    g_capturing = false;
}

static uint32_t key_of(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    return (u >> 31) ? ~u : (u | 0x80000000u);
}

static void check_oracle() {
    std::mt19937 rng(7);
    const float specials[] = {0.0f, -0.0f, std::numeric_limits<float>::infinity(), -std::numeric_limits<float>::infinity(),
                              std::numeric_limits<float>::quiet_NaN(), 1.0f, -1.0f, 1e-40f};
    for (int trial = 0; trial < 300; ++trial) {
        const int64_t ld = 1 + rng() % 300;
        const int64_t B = 1 + rng() % 4;
        const int32_t K = 1 + rng() % 64;
        std::vector<float> x(B * ld);
        std::vector<int32_t> rl(B);
        const int levels = 1 + rng() % 6;
        for (auto& v : x) v = (rng() % 10 == 0) ? specials[rng() % 8] : (float)(rng() % levels) - 2.0f;
        for (auto& r : rl) r = (int32_t)(rng() % (ld + 20)) - 10;
        std::vector<int32_t> out(B * K);
        std::vector<uint32_t> kth(B);
        std::vector<int32_t> ngt(B);
        CHECK(oracle_topk(x.data(), B, ld, rl.data(), K, out.data(), kth.data(), ngt.data()) == 0);
        for (int64_t b = 0; b < B; ++b) {
            const int64_t n = std::min<int64_t>(std::max<int32_t>(rl[b], 0), ld);
            std::vector<int32_t> idx(n);
            for (int64_t i = 0; i < n; ++i) idx[i] = (int32_t)i;
            std::stable_sort(idx.begin(), idx.end(),
                             [&](int32_t p, int32_t q) { return key_of(x[b * ld + p]) > key_of(x[b * ld + q]); });
            std::vector<int32_t> exp(K, -1);
            if (n <= K) {
                for (int64_t i = 0; i < n; ++i) exp[i] = (int32_t)i;
            } else {
                for (int32_t i = 0; i < K; ++i) exp[i] = idx[i];
                std::sort(exp.begin(), exp.end());
            }
            for (int32_t i = 0; i < K; ++i) CHECK(out[b * K + i] == exp[i]);
        }
    }
}

int main() {
    check_validate();
    check_plans();
    check_workspace();
    check_oracle();
    printf("ok\n");
    return 0;
}
