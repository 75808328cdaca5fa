// gvr_topk.hip -- Guess-Verify-Refine exact Top-K and radix-select Top-K for
// MI355X (gfx950), behind the C ABI declared in include/gvr_topk.h.
//
// Design (one cooperative launch per group of rows; all workgroups of a
// launch are co-resident):
//   * A row is split into S contiguous chunks, one workgroup (WG) each. Every
//     WG streams its chunk from HBM exactly once, converts it to sortable u32
//     keys and KEEPS IT IN VGPRs for the rest of the kernel: every later pass
//     over the row is on-chip ALU work, not HBM traffic.
//   * Guess (Sec. 4.2.1, Phase 1): each WG gathers the row's scores at
//     prev_topk and reduces them to pmin / pmax (and pmean for the stats).
//   * Threshold search (Sec. 4.2.2, Phase 2): a counting pass evaluates the
//     threshold count f(T) = #{key >= T} (Sec. 4.1) at every edge of a
//     512-bin window of key space in one sweep (wave-private LDS histograms;
//     the last bin holds everything at or above the window). The first window
//     is [key(pmin), key(pmax)] from the guess; a failed window is replaced by
//     the bin that brackets the K-th key (or by the key range below/above the
//     window), so a pass multiplies the resolution by 512. Per-WG histograms
//     are exchanged through the workspace with one per-row barrier per pass,
//     and every WG takes the same decision from the same sums.
//   * A threshold T is accepted when K <= f(T) <= C; by Lemma 1 (Sec. 4.1) the
//     candidate set {key >= T} then holds the exact answer.
//   * Collect (Sec. 4.2.3, Phase 3): each WG writes its candidates (key, index)
//     at offsets known in advance (per-WG prefix from the exchanged
//     histograms, per-wave counts from the wave-private histograms -- the
//     count cache -- and in-wave ballot/mbcnt ranks), so no atomic and no
//     second counting sweep is needed. Candidates land in ascending index
//     order.
//   * Refine (Sec. 4.2.4, Phase 4): the last WG of the row to finish its
//     collect (one global atomic per WG) loads the <= C candidates into LDS,
//     narrows a 2048-bin LDS histogram until the K-th key T* is isolated,
//     then emits every key > T* and the first K - #{key > T*} keys equal to
//     T* (lower index first) in ascending index order.
//   * If the K-th key is isolated by the counting passes themselves while
//     f(T*) > C (ties straddle [K, C]), the selection is emitted directly from
//     the registers, again in index order.
//   * radix_topk runs the same kernel without a guess: the first window is
//     the whole key range (9 bits of key per pass from the top), i.e. a
//     distribution-agnostic radix select (Sec. 2.2).

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "gvr_topk.h"

#define DEV __device__ __forceinline__

namespace {

constexpr int kWave = 64;
constexpr int kBinsLog2 = 9;
constexpr int kBins = 1 << kBinsLog2;         // bins of a counting pass
constexpr int kBinsX = kBins + 1;             // + "at or above the window"
constexpr int kXchStride = 528;               // ints per published histogram
constexpr int kRefBinsLog2 = 11;
constexpr int kRefBins = 1 << kRefBinsLog2;   // bins of a refine level
constexpr int kCmax = GVR_MAX_CANDIDATES;
constexpr int kMaxPasses = 12;                // safety cap; 5 always suffice
constexpr uint32_t kSpinLimit = 1u << 20;   // ~1 s of polling at most

// Per-row control block in the workspace (one 128-byte line per row).
struct RowCtl {
    unsigned arrive;   // barrier arrivals of the current generation
    unsigned gen;      // barrier generation
    unsigned ticket;   // collect completions (last one refines)
    unsigned err;      // set if a barrier wait gave up
    unsigned pad[28];
};

struct Params {
    const float* scores;
    int64_t ld;
    const int32_t* row_len;
    const int32_t* prev;
    int32_t* out;
    gvr_row_stats* stats;
    RowCtl* ctl;
    int* xch;
    uint32_t* cand_key;   // [rows][kCmax] candidate keys
    int32_t* cand_idx;    // [rows][kCmax] candidate indices
    int32_t K;
    int32_t rows;       // rows in this launch
    int32_t row0;       // first row of this launch
    int32_t S;          // workgroups per row in this launch
    int32_t capacity;   // C
    int32_t use_guess;  // 0: radix schedule
};

// ------------------------------------------------------------------ helpers

DEV uint32_t key_of_bits(uint32_t u) { return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u); }
DEV uint32_t key_of(float v) { return key_of_bits(__float_as_uint(v)); }

DEV uint32_t lanes_below(uint64_t m, uint32_t acc) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, acc));
}

DEV int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
DEV float wave_sum_f(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
DEV uint32_t wave_min_u(uint32_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, o, kWave));
    return v;
}
DEV uint32_t wave_max_u(uint32_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, kWave));
    return v;
}
// Inclusive prefix sum over the lanes of a wave.
DEV int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int t = __shfl_up(v, o, kWave);
        if (lane >= o) v += t;
    }
    return v;
}

// A window of key space: bins j < kBins cover [lo + j<<shift, lo + (j+1)<<shift);
// bin kBins holds every key >= lo + kBins<<shift. Keys below lo are not counted.
struct Window {
    uint32_t lo;
    uint32_t shift;
};

DEV Window make_window(uint32_t a, uint32_t b) {  // covers [a, b], b >= a
    uint64_t width = (uint64_t)b - a + 1;
    uint32_t s = 0;
    while (((uint64_t)kBins << s) < width) ++s;
    return Window{a, s};
}
DEV uint64_t edge_of(const Window& w, int j) { return (uint64_t)w.lo + ((uint64_t)j << w.shift); }

// Cross-workgroup communication. Data that another workgroup reads is written
// with device-coherent stores (agent-scope relaxed atomics: sc1, written
// through to the point of coherence) and read with device-coherent loads
// (sc1, never served by a stale cache line). Every wave waits for its own
// stores to complete (s_waitcnt) before the workgroup barrier that precedes
// the signalling atomic, so a workgroup that observes the signal reads
// complete data. No L2 write-back or invalidate is needed.
DEV void st_dev(int* p, int v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
DEV void st_dev(uint32_t* p, uint32_t v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
DEV int ld_dev(const int* p) { return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
DEV uint32_t ld_dev(const uint32_t* p) {
    return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
DEV void wait_mem() { __builtin_amdgcn_s_waitcnt(0); }

// Per-row barrier among the `parties` workgroups of a row. Called by one
// thread per WG after every wave of its WG has completed the stores being
// published. Gives up (flags err) after kSpinLimit polls so that every wave
// always terminates.
DEV void row_barrier(RowCtl* c, unsigned parties) {
    const unsigned g0 = ld_dev(&c->gen);
    wait_mem();   // read the generation before arriving
    const unsigned old = __hip_atomic_fetch_add(&c->arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == parties - 1) {
        st_dev(&c->arrive, 0u);
        wait_mem();
        __hip_atomic_fetch_add(&c->gen, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
        uint32_t spins = 0;
        while (ld_dev(&c->gen) == g0) {
            __builtin_amdgcn_s_sleep(1);
            if (++spins > kSpinLimit) {
                st_dev(&c->err, 1u);
                break;
            }
        }
    }
}

// ------------------------------------------------------------------ LDS
template <int NW>
struct SmemCount {
    int hist[NW][kBinsX];   // wave-private histograms (the per-wave count cache)
    int G[kBinsX];          // row totals per bin
    int pre[kBinsX];        // totals of the WGs before this one
    int F[kBinsX + 1];      // F[j] = f(edge j) (suffix sums of G)
};
struct SmemRefine {
    uint32_t key[kCmax];
    int32_t idx[kCmax];
    int hist[kRefBins];
};
template <int NW>
struct Smem {
    union {
        SmemCount<NW> c;
        SmemRefine r;
    } u;
    int red[4][NW];
    float redf[NW];
    int wtot[2][NW];
    int scal[16];
};

// Cross-wave helpers: lane v of every wave reads wave v's value, so a
// reduction over the NW waves costs one LDS read and one wave reduction
// (few VGPRs) instead of NW unrolled LDS reads.
template <int NW>
DEV int sum_over_waves(const int* vals, int lane) {
    return wave_sum(lane < NW ? vals[lane] : 0);
}
template <int NW>
DEV int sum_over_waves_below(const int* vals, int lane, int wave) {
    return wave_sum(lane < wave ? vals[lane] : 0);
}

// Block-wide exclusive scan of two ints (BLOCK threads). Returns totals.
template <int NW>
DEV void block_excl_scan2(int& a, int& b, int& tot_a, int& tot_b, int (&sa)[2][NW], int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    int ia = wave_incl_scan(a, lane), ib = wave_incl_scan(b, lane);
    if (lane == kWave - 1) {
        sa[0][wave] = ia;
        sa[1][wave] = ib;
    }
    __syncthreads();
    const int ba = sum_over_waves_below<NW>(sa[0], lane, wave);
    const int bb = sum_over_waves_below<NW>(sa[1], lane, wave);
    tot_a = sum_over_waves<NW>(sa[0], lane);
    tot_b = sum_over_waves<NW>(sa[1], lane);
    __syncthreads();
    a = ba + ia - a;
    b = bb + ib - b;
}

template <int NW>
DEV int block_sum(int v, Smem<NW>& sm, int tid) {
    v = wave_sum(v);
    if ((tid & 63) == 0) sm.red[0][tid >> 6] = v;
    __syncthreads();
    const int s = sum_over_waves<NW>(sm.red[0], tid & 63);
    __syncthreads();
    return s;
}

DEV int64_t stamp() { return (int64_t)__builtin_amdgcn_s_memtime(); }

// ------------------------------------------------------------------ refine
// Exact K-th selection among the c candidates (key, index) already staged in
// LDS in ascending index order. The K-th key is known to lie in [wlo, whi];
// `above` candidates lie above whi. Emits the K indices in ascending order.
template <int BLOCK, int NW>
DEV void refine_and_emit(Smem<NW>& sm, int c, uint32_t wlo, uint32_t whi, int above, int K,
                         int32_t* out, int tid, uint32_t* kth_out, int* ngt_out) {
    SmemRefine& r = sm.u.r;
    int need = K - above;   // >= 1
    for (int level = 0; level < 4; ++level) {
        if (wlo == whi) break;
        uint64_t width = (uint64_t)whi - wlo + 1;
        uint32_t s = 0;
        while (((uint64_t)kRefBins << s) < width) ++s;
        for (int i = tid; i < kRefBins; i += BLOCK) r.hist[i] = 0;
        __syncthreads();
        for (int i = tid; i < c; i += BLOCK) {
            uint32_t k = r.key[i];
            if (k >= wlo && k <= whi)
                __hip_atomic_fetch_add(&r.hist[(k - wlo) >> s], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        __syncthreads();
        // Suffix sums from the top bin: thread t owns bins [t*PER, (t+1)*PER).
        constexpr int PER = kRefBins / BLOCK;
        int loc[PER];
        int mysum = 0;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            loc[q] = r.hist[tid * PER + q];
            mysum += loc[q];
        }
        // exclusive "sum of bins above my range" = total - inclusive prefix
        int a = mysum, dummy = 0, tot = 0, tdummy = 0;
        block_excl_scan2<NW>(a, dummy, tot, tdummy, sm.wtot, tid);
        int above_me = tot - a - mysum;   // sum of bins with index > my range
        // find the bin where the count from the top reaches `need`
        int run = above_me;
        int found = -1, found_above = 0;
#pragma unroll
        for (int q = PER - 1; q >= 0; --q) {
            int nr = run + loc[q];
            if (found < 0 && run < need && nr >= need) {
                found = tid * PER + q;
                found_above = run;
            }
            run = nr;
        }
        if (found >= 0) {
            sm.scal[0] = found;
            sm.scal[1] = found_above;
        }
        __syncthreads();
        int b = sm.scal[0];
        int ab = sm.scal[1];
        __syncthreads();
        need -= ab;
        uint64_t nlo = (uint64_t)wlo + ((uint64_t)b << s);
        uint64_t nhi = nlo + ((uint64_t)1 << s) - 1;
        if (nhi > whi) nhi = whi;
        wlo = (uint32_t)nlo;
        whi = (uint32_t)nhi;
    }
    const uint32_t T = wlo;   // the K-th key
    // Ordered emission over the candidates in buffer (= index) order.
    const int seg = (c + BLOCK - 1) / BLOCK;
    const int i0 = min(tid * seg, c), i1 = min(i0 + seg, c);
    int gt = 0, eq = 0;
    for (int i = i0; i < i1; ++i) {
        uint32_t k = r.key[i];
        gt += (k > T);
        eq += (k == T);
    }
    int gtb = gt, eqb = eq, gtt = 0, eqt = 0;
    block_excl_scan2<NW>(gtb, eqb, gtt, eqt, sm.wtot, tid);
    const int take = K - gtt;   // ties to take, lower index first
    for (int i = i0; i < i1; ++i) {
        uint32_t k = r.key[i];
        if (k > T) {
            const int o = gtb + min(eqb, take);
            if (o >= 0 && o < K) out[o] = r.idx[i];
            ++gtb;
        } else if (k == T) {
            const int o = gtb + eqb;
            if (eqb < take && o >= 0 && o < K) out[o] = r.idx[i];
            ++eqb;
        }
    }
    *kth_out = T;
    *ngt_out = gtt;
}

// ------------------------------------------------------------------ kernel
template <int BLOCK, int R4, int MINW>
__global__ __launch_bounds__(BLOCK, MINW) void topk_rows_kernel(Params p) {
    constexpr int NW = BLOCK / kWave;
    constexpr int WSPAN = R4 * 256;   // elements of one wave's sub-chunk
    constexpr int CH = NW * WSPAN;    // elements of one WG's chunk
    __shared__ Smem<NW> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = blockIdx.x;
    const int rl = g / p.S, w = g % p.S;
    if (rl >= p.rows) return;
    const int64_t row = (int64_t)p.row0 + rl;
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
        if (w == 0) {
            for (int i = tid; i < K; i += BLOCK) out[i] = (i < n) ? i : -1;
            if (st && tid == 0) {
                gvr_row_stats s = {};
                s.n = n;
                s.path = GVR_PATH_TRIVIAL;
                s.t_start = t0;
                s.t_refine = stamp();
                *st = s;
            }
        }
        return;
    }
    const int aoff = (int)(((uintptr_t)x >> 2) & 3);   // x sits aoff floats into a 16-B block
    const int s_row = (n + aoff + CH - 1) / CH;
    if (w >= s_row) return;
    RowCtl* ctl = p.ctl + rl;
    int* xch = p.xch + (size_t)rl * 2 * p.S * kXchStride;
    uint32_t* ckey = p.cand_key + (size_t)rl * kCmax;
    int32_t* cidx = p.cand_idx + (size_t)rl * kCmax;
    const int cap = p.capacity;

    // ---------------- (a2) guess, overlapped with the chunk stream
    // The guess indices are loaded first (8 KB per row); the scattered
    // gathers x[prev] are issued right behind the chunk's loads, so both are
    // in flight together and the gathers mostly hit lines the row's
    // workgroups are streaming anyway.
    constexpr int KPT = (GVR_MAX_K + BLOCK - 1) / BLOCK;
    const bool have_prev = p.use_guess && p.prev;
    int pq[KPT];
    if (have_prev) {
        const int32_t* pv = p.prev + row * (int64_t)K;
#pragma unroll
        for (int m = 0; m < KPT; ++m) {
            const int j = tid + m * BLOCK;
            pq[m] = (j < K) ? pv[j] : -1;
        }
    }

    // ---------------- load the chunk once; keep it as keys in VGPRs
    // Virtual index v = element index + aoff, so that v % 4 == 0 is a 16-byte
    // boundary; the wave's sub-chunk starts at vb. Every slab issues one
    // unconditional dwordx4 load. Its block index is clamped to the last
    // block that holds an element of the row, so no load leaves the 16-byte
    // blocks that contain x[0..n); elements outside [0, n) are never used
    // (their key is set to 0 and they are excluded from every count).
    const int vb = w * CH + wave * WSPAN;
    const float4* xa = reinterpret_cast<const float4*>(x - aoff);
    const int qlast = (n - 1 + aoff) >> 2;
    uint32_t k[R4][4];
    float gv[KPT];
    {
        float4 raw[R4];
#pragma unroll
        for (int i = 0; i < R4; ++i) {
            const int q = min(((vb + i * 256) >> 2) + lane, qlast);
            raw[i] = xa[q];
        }
        if (have_prev) {
#pragma unroll
            for (int m = 0; m < KPT; ++m) gv[m] = (pq[m] >= 0 && pq[m] < n) ? x[pq[m]] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < R4; ++i) {
            k[i][0] = key_of(raw[i].x);
            k[i][1] = key_of(raw[i].y);
            k[i][2] = key_of(raw[i].z);
            k[i][3] = key_of(raw[i].w);
            const int s0 = vb + i * 256 - aoff;   // element index of the slab's first slot
            if (s0 < 0 || s0 + 255 >= n) {        // wave-uniform: an edge slab
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int e = s0 + lane * 4 + c;
                    if (e < 0 || e >= n) k[i][c] = 0u;
                }
            }
        }
    }

    // Guess statistics (Phase 1): pmin / pmax as keys, pmean for the stats.
    int gvalid = 0;
    uint32_t gmin = 0xFFFFFFFFu, gmax = 0u;
    float gsum = 0.f;
    if (have_prev) {
#pragma unroll
        for (int m = 0; m < KPT; ++m) {
            if (pq[m] >= 0 && pq[m] < n) {
                const uint32_t kk = key_of(gv[m]);
                gmin = min(gmin, kk);
                gmax = max(gmax, kk);
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
        __syncthreads();
        gvalid = sum_over_waves<NW>(sm.red[0], lane);
        gmin = wave_min_u(lane < NW ? (uint32_t)sm.red[1][lane] : 0xFFFFFFFFu);
        gmax = wave_max_u(lane < NW ? (uint32_t)sm.red[2][lane] : 0u);
        // pmean: fixed summation order (wave partials in wave order).
        gsum = 0.f;
        for (int v = 0; v < NW; ++v) gsum += sm.redf[v];
        __syncthreads();
    }
    const int64_t t1 = stamp();

    // Slots of this wave / WG that hold no element (their key is 0).
    auto valid_in = [&](int v0, int len) {   // #elements with virtual index in [v0, v0+len)
        int a = max(v0, aoff), b = min(v0 + len, n + aoff);
        return b > a ? b - a : 0;
    };
    const int inv_wave = WSPAN - valid_in(vb, WSPAN);

    // Candidate set parameters decided below.
    int path;
    int passes = 0;
    uint32_t T = 0;           // accepted threshold key
    int FT = 0;               // f(T) = candidates of the row
    int pre_ge = 0;           // candidates in the WGs before this one
    int wave_ge = 0;          // candidates of this wave
    uint32_t rlo = 0, rhi = 0xFFFFFFFFu;   // refine window for the K-th key
    int above = 0;            // candidates known to be above rhi
    bool ties = false;        // K-th key isolated by counting; emit directly
    int gt_pre = 0, eq_pre = 0, gt_wave = 0, eq_wave = 0, n_gt_row = 0;

    if (n <= cap) {
        // Every element is a candidate: counts are known without a pass.
        path = GVR_PATH_ALL;
        T = 0;
        FT = n;
        pre_ge = valid_in(0, w * CH);
        wave_ge = WSPAN - inv_wave;
    } else {
        const bool guess = p.use_guess && p.prev && gvalid > 0;
        path = guess ? GVR_PATH_GUESS : GVR_PATH_NO_GUESS;
        Window win = guess ? make_window(gmin, gmax) : make_window(0u, 0xFFFFFFFFu);
        int parity = 0;
        for (;;) {
            // Thread coordinates made opaque per iteration so that the many
            // thread-dependent addresses below are recomputed here rather than
            // hoisted out of the loop (where they would stay live next to the
            // register-resident keys).
            int tid_o = (int)threadIdx.x;
            asm volatile("" : "+v"(tid_o));
            const int tid = tid_o, lane = tid_o & 63, wave = tid_o >> 6;
            // ---- (a3) counting pass over the register-resident keys
            int* hw = sm.u.c.hist[wave];
            for (int b = lane; b < kBinsX; b += kWave) hw[b] = 0;
            // (LDS ops of one wave execute in order; no barrier needed here)
            const uint32_t lo = win.lo, sh = win.shift;
#pragma unroll
            for (int i = 0; i < R4; ++i) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t kk = k[i][c];
                    if (kk >= lo) {
                        const uint32_t b = min((kk - lo) >> sh, (uint32_t)kBins);
                        __hip_atomic_fetch_add(&hw[b], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    }
                }
            }
            if (lo == 0 && lane == 0 && inv_wave)
                __hip_atomic_fetch_add(&hw[0], -inv_wave, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            ++passes;
            __syncthreads();
            // WG totals, published for the other WGs of the row.
            int* mine = xch + ((size_t)parity * p.S + w) * kXchStride;
            for (int b = tid; b < kBinsX; b += BLOCK) {
                int t = 0;
#pragma unroll
                for (int v = 0; v < NW; ++v) t += sm.u.c.hist[v][b];
                st_dev(&mine[b], t);
            }
            wait_mem();
            __syncthreads();
            if (tid == 0) row_barrier(ctl, (unsigned)s_row);
            __syncthreads();
            const int* all = xch + (size_t)parity * p.S * kXchStride;
            for (int b = tid; b < kBinsX; b += BLOCK) {
                int tot = 0, pr = 0;
                for (int v = 0; v < s_row; ++v) {
                    int t = ld_dev(&all[(size_t)v * kXchStride + b]);
                    tot += t;
                    if (v < w) pr += t;
                }
                sm.u.c.G[b] = tot;
                sm.u.c.pre[b] = pr;
            }
            __syncthreads();
            // F[j] = sum_{b >= j} G[b]; block scan over bins in reverse order.
            {
                // thread t owns bin (kBins - t) and thread 0 also bin 0 at the end
                int b0 = kBins - tid;          // kBins .. kBins-BLOCK+1
                int v0 = (b0 >= 0) ? sm.u.c.G[b0] : 0;
                // bins below kBins-BLOCK+1 (if BLOCK < kBinsX) handled by a tail loop
                int a = v0, dz = 0, tot = 0, tz = 0;
                block_excl_scan2<NW>(a, dz, tot, tz, sm.wtot, tid);
                if (b0 >= 0) sm.u.c.F[b0] = a + v0;
                // remaining bins b < kBins - BLOCK + 1 (serial by thread 0; at most one)
                if (tid == 0) {
                    int run = tot;
                    for (int b = kBins - BLOCK; b >= 0; --b) {
                        run += sm.u.c.G[b];
                        sm.u.c.F[b] = run;
                    }
                    sm.u.c.F[kBinsX] = 0;
                    sm.scal[0] = -1;
                }
            }
            __syncthreads();
            for (int b = tid; b < kBinsX; b += BLOCK) {
                if (sm.u.c.F[b] >= K && sm.u.c.F[b + 1] < K) sm.scal[0] = b;
            }
            __syncthreads();
            const int j = sm.scal[0];
            const bool last_pass = passes >= kMaxPasses;
            int decision;   // 0 accept, 1 ties, 2 narrow
            Window nw = win;
            if (j < 0) {
                // f(lo) < K: the K-th key lies below the window.
                nw = make_window(0u, win.lo - 1u);
                decision = 2;
            } else {
                const uint64_t e = edge_of(win, j);
                const int fj = sm.u.c.F[j];
                if (fj <= cap) {
                    decision = 0;
                } else if (j == kBins) {
                    nw = make_window((uint32_t)e, 0xFFFFFFFFu);
                    decision = 2;
                } else if (win.shift == 0) {
                    decision = 1;
                } else {
                    uint64_t hi = e + ((uint64_t)1 << win.shift) - 1;
                    nw = make_window((uint32_t)e, (uint32_t)min(hi, (uint64_t)0xFFFFFFFFu));
                    decision = 2;
                }
            }
            if (decision == 2 && last_pass) decision = -1;
            if (decision == 0 || decision == 1) {
                const uint64_t e = edge_of(win, j);
                T = (uint32_t)e;
                FT = sm.u.c.F[j];
                if (decision == 0) {
                    // Candidate counts at T: row prefix and this wave's share.
                    int s1 = 0;
                    for (int b = j + tid; b < kBinsX; b += BLOCK) s1 += sm.u.c.pre[b];
                    int s2 = 0;
                    for (int b = j + lane; b < kBinsX; b += kWave) s2 += sm.u.c.hist[wave][b];
                    pre_ge = block_sum<NW>(s1, sm, tid);
                    wave_ge = wave_sum(s2);
                    if (j < kBins) {
                        rlo = T;
                        rhi = (uint32_t)min(e + ((uint64_t)1 << win.shift) - 1, (uint64_t)0xFFFFFFFFu);
                        above = sm.u.c.F[j + 1];
                    } else {
                        rlo = T;
                        rhi = 0xFFFFFFFFu;
                        above = 0;
                    }
                } else {
                    ties = true;
                    n_gt_row = sm.u.c.F[j + 1];
                    gt_pre = 0;
                    eq_pre = 0;
                    int a1 = 0, a2 = 0;
                    for (int b = j + 1 + tid; b < kBinsX; b += BLOCK) a1 += sm.u.c.pre[b];
                    gt_pre = block_sum<NW>(a1, sm, tid);
                    eq_pre = sm.u.c.pre[j];
                    for (int b = j + 1 + lane; b < kBinsX; b += kWave) a2 += sm.u.c.hist[wave][b];
                    gt_wave = wave_sum(a2);
                    eq_wave = sm.u.c.hist[wave][j];
                }
                break;
            }
            if (decision < 0) {
                if (tid == 0) st_dev(&ctl->err, 2u);
                T = 0xFFFFFFFFu;
                FT = 0;
                break;
            }
            if (path == GVR_PATH_GUESS) path = GVR_PATH_NARROWED;
            win = nw;
            parity ^= 1;
            __syncthreads();
        }
    }
    const int64_t t2 = stamp();

    if (ties) {
        // ---- K-th key T isolated with f(T) > C: emit the selection directly.
        const int take = K - n_gt_row;
        // wave prefixes of (gt, eq) inside the WG
        if (lane == 0) {
            sm.wtot[0][wave] = gt_wave;
            sm.wtot[1][wave] = eq_wave;
        }
        __syncthreads();
        int gb = gt_pre + sum_over_waves_below<NW>(sm.wtot[0], lane, wave);
        int eb = eq_pre + sum_over_waves_below<NW>(sm.wtot[1], lane, wave);
#pragma unroll
        for (int i = 0; i < R4; ++i) {
            bool fg[4], fe[4];
            uint64_t mg[4], me[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int e = vb + i * 256 + lane * 4 + c - aoff;
                const bool valid = (e >= 0 && e < n);
                fg[c] = valid && k[i][c] > T;
                fe[c] = valid && k[i][c] == T;
                mg[c] = __ballot(fg[c]);
                me[c] = __ballot(fe[c]);
            }
            uint32_t g_before = lanes_below(mg[3], lanes_below(mg[2], lanes_below(mg[1], lanes_below(mg[0], 0))));
            uint32_t e_before = lanes_below(me[3], lanes_below(me[2], lanes_below(me[1], lanes_below(me[0], 0))));
            int gpos = gb + (int)g_before, epos = eb + (int)e_before;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int e = vb + i * 256 + lane * 4 + c - aoff;
                if (fg[c]) {
                    const int o = gpos + min(epos, take);
                    if (o >= 0 && o < K) out[o] = e;
                    ++gpos;
                } else if (fe[c]) {
                    const int o = gpos + epos;
                    if (epos < take && o >= 0 && o < K) out[o] = e;
                    ++epos;
                }
            }
            gb += __popcll(mg[0]) + __popcll(mg[1]) + __popcll(mg[2]) + __popcll(mg[3]);
            eb += __popcll(me[0]) + __popcll(me[1]) + __popcll(me[2]) + __popcll(me[3]);
        }
        if (w == 0 && st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = GVR_PATH_TIES;
            s.passes = passes;
            s.candidates = 0;
            s.threshold = T;
            s.kth_key = T;
            s.n_gt = n_gt_row;
            s.guess_valid = gvalid;
            s.t_start = t0;
            s.t_guess = t1;
            s.t_search = t2;
            s.t_collect = t2;
            s.t_refine = stamp();
            *st = s;
        }
        return;
    }
    if (FT == 0) {
        // Search gave up (cannot happen for valid keys; kept so every path ends).
        if (w == 0)
            for (int i = tid; i < K; i += BLOCK) out[i] = -1;
        if (w == 0 && st && tid == 0) {
            gvr_row_stats s = {};
            s.n = n;
            s.path = -1;
            s.passes = passes;
            *st = s;
        }
        return;
    }

    // ---------------- (a4) collect: candidates key >= T at precomputed offsets
    if (lane == 0) sm.wtot[0][wave] = wave_ge;
    __syncthreads();
    int base = pre_ge + sum_over_waves_below<NW>(sm.wtot[0], lane, wave);
#pragma unroll
    for (int i = 0; i < R4; ++i) {
        bool f[4];
        uint64_t m[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            f[c] = (path == GVR_PATH_ALL) ? (vb + i * 256 + lane * 4 + c - aoff >= 0 &&
                                             vb + i * 256 + lane * 4 + c - aoff < n)
                                          : (k[i][c] >= T);
            m[c] = __ballot(f[c]);
        }
        int pos = base + (int)lanes_below(m[3], lanes_below(m[2], lanes_below(m[1], lanes_below(m[0], 0))));
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if (f[c]) {
                if (pos >= 0 && pos < cap) {
                    st_dev(&ckey[pos], k[i][c]);
                    st_dev(&cidx[pos], vb + i * 256 + lane * 4 + c - aoff);
                }
                ++pos;
            }
        }
        base += __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
    }
    // Publish, then one atomic per WG; the last WG of the row refines.
    wait_mem();
    __syncthreads();
    if (tid == 0) {
        const unsigned old = __hip_atomic_fetch_add(&ctl->ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const bool last = (old == (unsigned)s_row - 1);
        if (last) st_dev(&ctl->ticket, 0u);
        sm.scal[2] = last ? 1 : 0;
    }
    __syncthreads();
    if (!sm.scal[2]) return;
    const int64_t t3 = stamp();

    // ---------------- (a5) refine the <= C candidates in LDS
    const int c = min(FT, cap);
    for (int i = tid; i < c; i += BLOCK) {
        sm.u.r.key[i] = ld_dev(&ckey[i]);
        sm.u.r.idx[i] = ld_dev(&cidx[i]);
    }
    __syncthreads();
    uint32_t kth = 0;
    int ngt = 0;
    refine_and_emit<BLOCK, NW>(sm, c, rlo, rhi, above, K, out, tid, &kth, &ngt);
    if (st && tid == 0) {
        gvr_row_stats s = {};
        s.n = n;
        s.path = path;
        s.passes = passes;
        s.candidates = c;
        s.threshold = T;
        s.kth_key = kth;
        s.n_gt = ngt;
        s.guess_valid = gvalid;
        s.t_start = t0;
        s.t_guess = t1;
        s.t_search = t2;
        s.t_collect = t3;
        s.t_refine = stamp();
        *st = s;
    }
}

// ------------------------------------------------------------------ host side

struct Variant {
    const void* fn;
    int block;
    int r4;
    int occupancy;   // WGs per CU (filled per device)
};

template <int BLOCK, int R4, int MINW>
const void* fn_ptr() {
    return reinterpret_cast<const void*>(&topk_rows_kernel<BLOCK, R4, MINW>);
}

struct DeviceState {
    bool init = false;
    int cus = 0;
    int max_rows = 0;   // most rows one launch can hold (sizes the control area)
    std::vector<Variant> variants;
    void* ws = nullptr;
    size_t ws_bytes = 0;
};

std::mutex g_mu;
std::vector<DeviceState> g_dev;

// Workspace layout: [control blocks: max_rows x RowCtl][exchange: rows x 2 x S
// histograms][candidates: rows x C keys][candidates: rows x C indices]. The
// control area has a fixed size per device, so the self-cleaning barrier and
// ticket counters always sit on the same (zero) bytes whatever the shape of
// the call; the other areas are written before they are read.
size_t row_ws_bytes(int S) {
    return (size_t)2 * S * kXchStride * sizeof(int) + (size_t)kCmax * 2 * sizeof(uint32_t);
}

struct Plan {
    const Variant* v;
    int S;
    int rows_per_launch;
};

size_t ws_bytes_for(const DeviceState& ds, const Plan& pl) {
    return (size_t)ds.max_rows * sizeof(RowCtl) + (size_t)pl.rows_per_launch * row_ws_bytes(pl.S);
}

gvr_status init_device(int dev, DeviceState& ds) {
    if (ds.init) return GVR_OK;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return GVR_ERR_HIP;
    ds.cus = prop.multiProcessorCount;
    ds.variants = {
        {fn_ptr<512, 2, 4>(), 512, 2, 0},   {fn_ptr<512, 4, 4>(), 512, 4, 0},
        {fn_ptr<512, 8, 4>(), 512, 8, 0},   {fn_ptr<512, 16, 4>(), 512, 16, 0},
        {fn_ptr<512, 32, 2>(), 512, 32, 0},
    };
    for (auto& v : ds.variants) {
        int occ = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, v.fn, v.block, 0) != hipSuccess) return GVR_ERR_HIP;
        v.occupancy = occ;
        ds.max_rows = std::max(ds.max_rows, occ * ds.cus);
    }
    ds.init = true;
    return GVR_OK;
}

// Smallest register chunk whose grid fits on the chip at once, with at most
// kMaxS workgroups per row; else the largest chunk over several launches.
bool make_plan(const DeviceState& ds, int64_t B, int64_t ld, Plan& pl) {
    constexpr int kMaxS = 16;
    const Variant* best = nullptr;
    for (const auto& v : ds.variants) {
        if (v.occupancy < 1) continue;
        const int64_t ch = (int64_t)v.block * v.r4 * 4;
        const int64_t S = (ld + 3 + ch - 1) / ch;
        const int64_t cap = (int64_t)v.occupancy * ds.cus;
        if (S <= kMaxS && B * S <= cap) {
            pl.v = &v;
            pl.S = (int)S;
            pl.rows_per_launch = (int)B;
            return true;
        }
        best = &v;
    }
    if (!best) return false;
    const int64_t ch = (int64_t)best->block * best->r4 * 4;
    const int64_t S = (ld + 3 + ch - 1) / ch;
    const int64_t cap = (int64_t)best->occupancy * ds.cus;
    if (S > cap) return false;
    pl.v = best;
    pl.S = (int)S;
    pl.rows_per_launch = (int)std::min<int64_t>(B, cap / S);
    return true;
}

gvr_status validate(const float* scores, int64_t B, int64_t ld, int32_t K, const int32_t* out,
                    const gvr_options* opt, int* capacity, int* use_guess) {
    if (K < 1 || K > GVR_MAX_K) return GVR_ERR_UNSUPPORTED_K;
    if (B < 0 || ld < 0) return GVR_ERR_INVALID_ARG;
    if (B > 0 && (!scores || !out)) return GVR_ERR_INVALID_ARG;
    if (ld > (int64_t)0x7FFFFFF0) return GVR_ERR_TOO_LONG;
    if (B > (int64_t)0x7FFFFFFF) return GVR_ERR_INVALID_ARG;
    int cap = GVR_MAX_CANDIDATES;
    if (opt) {
        if (opt->capacity != 0) {
            if (opt->capacity < K || opt->capacity > GVR_MAX_CANDIDATES) return GVR_ERR_INVALID_ARG;
            cap = opt->capacity;
        }
        if (opt->flags & ~1) return GVR_ERR_INVALID_ARG;
        if (opt->flags & 1) *use_guess = 0;
        if (opt->max_passes < 0) *use_guess = 0;
    }
    *capacity = cap;
    return GVR_OK;
}

gvr_status run(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev,
               int32_t K, int32_t* out, void* stream, void* ws, size_t ws_bytes, const gvr_options* opt,
               gvr_row_stats* stats, int use_guess, bool own_ws) {
    int cap = 0;
    gvr_status st = validate(scores, B, ld, K, out, opt, &cap, &use_guess);
    if (st != GVR_OK) return st;
    if (B == 0) return GVR_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GVR_ERR_HIP;
    std::unique_lock<std::mutex> lk(g_mu);
    if ((int)g_dev.size() <= dev) g_dev.resize(dev + 1);
    DeviceState& ds = g_dev[dev];
    if ((st = init_device(dev, ds)) != GVR_OK) return st;
    Plan pl;
    if (!make_plan(ds, B, ld, pl)) return GVR_ERR_TOO_LONG;
    const size_t need = ws_bytes_for(ds, pl);
    if (own_ws) {
        if (ds.ws_bytes < need) {
            if (ds.ws) {
                if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return GVR_ERR_HIP;
                (void)hipFree(ds.ws);
                ds.ws = nullptr;
                ds.ws_bytes = 0;
            }
            if (hipMalloc(&ds.ws, need) != hipSuccess) return GVR_ERR_WORKSPACE;
            if (hipMemsetAsync(ds.ws, 0, need, (hipStream_t)stream) != hipSuccess) return GVR_ERR_HIP;
            ds.ws_bytes = need;
        }
        ws = ds.ws;
    } else {
        if (!ws || ws_bytes < need) return GVR_ERR_WORKSPACE;
        lk.unlock();
    }
    const int rpl = pl.rows_per_launch;
    char* base = (char*)ws;
    Params prm;
    prm.scores = scores;
    prm.ld = ld;
    prm.row_len = row_len;
    prm.prev = prev;
    prm.out = out;
    prm.stats = stats;
    prm.ctl = (RowCtl*)base;
    char* xbase = base + (size_t)ds.max_rows * sizeof(RowCtl);
    prm.xch = (int*)xbase;
    char* cbase = xbase + (size_t)rpl * (size_t)2 * pl.S * kXchStride * sizeof(int);
    prm.cand_key = (uint32_t*)cbase;
    prm.cand_idx = (int32_t*)(cbase + (size_t)rpl * kCmax * sizeof(uint32_t));
    prm.K = K;
    prm.S = pl.S;
    prm.capacity = cap;
    prm.use_guess = use_guess;
    for (int64_t r0 = 0; r0 < B; r0 += rpl) {
        const int rows = (int)std::min<int64_t>(rpl, B - r0);
        prm.rows = rows;
        prm.row0 = (int)r0;
        void* args[] = {&prm};
        hipError_t e = hipLaunchCooperativeKernel(pl.v->fn, dim3((unsigned)(rows * pl.S)), dim3(pl.v->block), args, 0,
                                                  (hipStream_t)stream);
        if (e != hipSuccess) return GVR_ERR_HIP;
    }
    return GVR_OK;
}

}  // namespace

extern "C" {

gvr_status gvr_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                    int32_t K, int32_t* out_idx, void* stream) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, nullptr, 0, nullptr, nullptr, 1, true);
}

gvr_status radix_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                      int32_t K, int32_t* out_idx, void* stream) {
    (void)prev_topk;
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, nullptr, 0, nullptr, nullptr, 0, true);
}

size_t gvr_workspace_size(int64_t B, int64_t ld, int32_t K) {
    if (K < 1 || K > GVR_MAX_K || B < 0 || ld < 0 || ld > (int64_t)0x7FFFFFF0) return 0;
    if (B == 0) return 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    std::lock_guard<std::mutex> lk(g_mu);
    if ((int)g_dev.size() <= dev) g_dev.resize(dev + 1);
    DeviceState& ds = g_dev[dev];
    if (init_device(dev, ds) != GVR_OK) return 0;
    Plan pl;
    if (!make_plan(ds, B, ld, pl)) return 0;
    return ws_bytes_for(ds, pl);
}

gvr_status gvr_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, const int32_t* prev_topk,
                       int32_t K, int32_t* out_idx, void* stream, void* workspace, size_t ws_bytes,
                       const gvr_options* options, gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, prev_topk, K, out_idx, stream, workspace, ws_bytes, options, stats, 1,
               false);
}

gvr_status radix_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                         int32_t* out_idx, void* stream, void* workspace, size_t ws_bytes,
                         const gvr_options* options, gvr_row_stats* stats) {
    return run(scores, B, ld, row_len, nullptr, K, out_idx, stream, workspace, ws_bytes, options, stats, 0, false);
}

const char* gvr_status_string(gvr_status s) {
    switch (s) {
        case GVR_OK: return "ok";
        case GVR_ERR_INVALID_ARG: return "invalid argument";
        case GVR_ERR_UNSUPPORTED_K: return "unsupported K (1 <= K <= 2048)";
        case GVR_ERR_WORKSPACE: return "workspace missing, too small or not allocatable";
        case GVR_ERR_HIP: return "HIP runtime error";
        case GVR_ERR_TOO_LONG: return "row stride too long for one launch";
    }
    return "unknown status";
}

const char* gvr_version(void) { return "gvr_topk 0.1 (gfx950)"; }

}  // extern "C"
