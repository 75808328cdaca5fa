// indexer.hip -- FP8 indexer scores of DeepSeek Sparse Attention (Sec. 2.1,
// Eq. indexer) on the MI355X matrix cores, behind include/gvr_indexer.h.
//
// One wave computes the scores of one row for a run of keys, 32 at a time
// (two 16-key tiles). Per tile the logits q[j] . k[s] of all H heads and 16
// keys are 16 x 16 blocks of gfx950's v_mfma_scale_f32_16x16x128_f8f6f4 with
// unit block scales (FP8 E4M3 operands, heads down the rows, keys across the
// columns, the whole head dimension in one step); the epilogue scales each
// key's column by its k_scale, applies ReLU, weights the heads and sums them.
// Lane l holds column l % 16 and, of the 128-byte reduction, the 32 bytes
// [32 (l / 16), + 32) of its head and of its key (a smaller D leaves the upper
// bytes of the query at zero); in the accumulators it holds heads
// 4 (l / 16) + i of its key, so the head sum is 4 fused multiply-adds per 16
// heads plus two exchanges across the four lanes of a key. With this layout a
// 16-byte load of 64 lanes touches 16 cache lines (4 lanes per key row), a
// quarter of what one key per lane pair would touch.
//
// Each lane keeps its 32 bytes of its query heads in registers for the whole
// run and the head weights sit in LDS (broadcast reads); the keys stream
// through a ring of kRing register buffers, kRing - 1 tiles in flight, with
// no branch in the steady state. When the rows of one cache (the draft rows
// of a request) pair up, one wave serves two of them: each key tile is loaded
// once and meets both rows' queries (reading it from two waves cost an
// eighth more time). Bound by HBM: D + 4 bytes per key and cache, 4 bytes
// written per score.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>

#include "gvr_indexer.h"
#include "guess.h"
#include "host_plan.h"
#include "topk_internal.h"

namespace {

using namespace gvr_dev;

constexpr int kWaves = 4;                // waves per workgroup
constexpr int kTile = 32;                // keys per ring slot (two 16-key matrix tiles)
constexpr int kTilesPerWave = 32;        // ring slots of one wave's run (1024 keys)
constexpr int kRing = 3;                 // key slots held per wave: kRing - 1 in flight while one is used
constexpr int kMinRun = 8 * kTile;       // shortest wave run the grid sizing picks (256 keys)
constexpr int64_t kMaxLd = ((int64_t)1 << 31) - 16;

typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
constexpr int kUnitScales = 0x7F7F7F7F;  // E8M0 block scales of 1.0 for the scaled matrix op

struct IdxParams {
    const uint8_t* q;
    const float* w;
    const uint8_t* k;
    const float* k_scale;
    const int32_t* row_len;
    float* scores;
    int64_t ld;
    int32_t rows;
    int32_t group;
    int32_t chunks;       // workgroups per cache (key chunks)
    int32_t chunk_keys;   // keys per workgroup chunk
    int32_t run_keys;     // keys per wave run (a multiple of kTile)
    // Fused guess (gvr_indexer_topk): workgroups [sample_base, + rows) score
    // the keys at row b's strided sample of prev [rows][K] and write the
    // sample's GuessStats words to gstats + b * K. prev NULL: none.
    const int32_t* prev;
    int32_t* gstats;
    int32_t K;
    int32_t sample_base;
};

// 32 bytes at p (16-byte aligned) as one matrix operand.
__device__ __forceinline__ v8i load32(const uint8_t* p) {
    const uint4* s = reinterpret_cast<const uint4*>(p);
    const uint4 a = s[0], b = s[1];
    return v8i{(int)a.x, (int)a.y, (int)a.z, (int)a.w, (int)b.x, (int)b.y, (int)b.z, (int)b.w};
}

// Score of the key in this lane's column of a 16-key tile for one row:
// the H / 16 matrix steps (16 heads x 16 keys, the whole head dimension per
// step), the key's scale, ReLU, the head weights wv (LDS, float4 per lane
// quarter) and the sum over heads; every lane of the key's column ends with
// it. The main loop and the fused guess both score keys here, so a sampled
// key's score equals the one written for it.
template <int H>
__device__ __forceinline__ float tile_score(const v8i (&qa)[H / 16], const v8i& kb, float ks, const float4* wv,
                                            int quarter) {
    constexpr int MT = H / 16;
    v4f acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        acc[mt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(qa[mt], kb, v4f{0.f, 0.f, 0.f, 0.f}, 0, 0, 0,
                                                                   kUnitScales, 0, kUnitScales);
    float sum = 0.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const float4 wq = wv[4 * mt + quarter];   // heads 16 mt + 4 quarter + (0..3)
        sum += wq.x * fmaxf(acc[mt][0] * ks, 0.f);
        sum += wq.y * fmaxf(acc[mt][1] * ks, 0.f);
        sum += wq.z * fmaxf(acc[mt][2] * ks, 0.f);
        sum += wq.w * fmaxf(acc[mt][3] * ks, 0.f);
    }
    sum += __shfl_xor(sum, 16, kWave);
    sum += __shfl_xor(sum, 32, kWave);   // the four lanes of the key now hold its score
    return sum;
}

// The fused guess of row b = blockIdx.x - sample_base: wave w scores samples
// [64 w, 64 w + 64) (four 16-key tiles; sample i is key prev[b][i * st],
// valid if inside [0, n_b)), then wave 0 reduces the 256 samples as the
// Top-K's Phase 1 does and writes the row's GuessStats words.
template <int H, int D>
__device__ void sample_guess(const IdxParams& p, int b, float* wl) {
    constexpr int MT = H / 16;
    __shared__ float sc[kGuessSamples];
    __shared__ int sv[kGuessSamples];
    __shared__ int gh[kGuessBins];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = b / p.group;
    int64_t n64 = p.row_len ? (int64_t)p.row_len[b] : p.ld;
    n64 = n64 < 0 ? 0 : (n64 > p.ld ? p.ld : n64);
    const int col = lane & 15, quarter = lane >> 4;
    const int qoff = 32 * (quarter % (D / 32));
    const bool qlive = 32 * quarter < D;
    for (int j = lane; j < H; j += kWave) wl[j] = p.w[(int64_t)b * H + j];
    v8i qa[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const v8i v = load32(p.q + (((int64_t)b * H + 16 * mt + col) * D + qoff));
        qa[mt] = qlive ? v : v8i{0, 0, 0, 0, 0, 0, 0, 0};
    }
    __builtin_amdgcn_wave_barrier();
    const float4* wv = reinterpret_cast<const float4*>(wl);
    const int st = guess_stride(p.K), m = guess_count(p.K);
    const int32_t* pv = p.prev + (int64_t)b * p.K;
    const uint8_t* kg = p.k + (int64_t)g * p.ld * D + qoff;
    const float* sg = p.k_scale + (int64_t)g * p.ld;
    int64_t key[4];
    bool ok[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int i = 64 * wave + 16 * t + col;
        const int64_t s = i < m ? (int64_t)pv[(int64_t)i * st] : -1;
        ok[t] = s >= 0 && s < n64;
        key[t] = ok[t] ? s : 0;   // an invalid sample scores key 0 (ld > 0), unused
    }
    v8i kb[4];
    float ks[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        kb[t] = load32(kg + key[t] * D);
        ks[t] = sg[key[t]];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const float v = tile_score<H>(qa, kb[t], ks[t], wv, quarter);
        if (quarter == 0) {
            sc[64 * wave + 16 * t + col] = v;
            sv[64 * wave + 16 * t + col] = ok[t];
        }
    }
    __syncthreads();
    if (wave == 0) {
        float gv[4];
        bool gok[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            gok[c] = sv[lane + 64 * c] != 0;
            gv[c] = gok[c] ? sc[lane + 64 * c] : 0.f;
        }
        const GuessStats gs = guess_from_samples(gv, gok, gh);
        if (lane == 0) {
            int32_t* o = p.gstats + (int64_t)b * p.K;
            o[0] = (int32_t)gs.ts;
            o[1] = gs.cnt;
            o[2] = (int32_t)gs.mn;
            o[3] = (int32_t)gs.mx;
            o[4] = __float_as_int(gs.sum);
        }
    }
}

template <int H, int D, int RG>
__global__ __launch_bounds__(kWaves * kWave) void indexer_kernel(IdxParams p) {
    constexpr int MT = H / 16;   // 16-head row tiles
    __shared__ float wl[kWaves][RG * H];
    if (p.prev && (int)blockIdx.x >= p.sample_base) {
        const int b = (int)blockIdx.x - p.sample_base;
        if (b < p.rows) sample_guess<H, D>(p, b, &wl[threadIdx.x >> 6][0]);
        return;
    }
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int G = p.group;
    // A wave serves RG rows of its cache (each key tile loaded once for them);
    // the cache's G / RG row slots share the workgroup's waves, wpr each.
    const int slots = G / RG;
    const int wpr = kWaves / slots;           // waves per row slot (one idle wave when G = 3)
    if (wave >= slots * wpr) return;
    const int g = blockIdx.x / p.chunks;      // cache
    const int c = blockIdx.x - g * p.chunks;  // key chunk
    const int slot_i = wave % slots, sub = wave / slots;
    const int64_t row0 = (int64_t)g * G + slot_i * RG;
    if (row0 >= p.rows) return;
    // Keys [s_begin, s_end) of this wave's run: up to the longest of its rows;
    // a row's scores are stored for its own keys only.
    int64_t nr[RG];
    int64_t n_max = 0;
#pragma unroll
    for (int rr = 0; rr < RG; ++rr) {
        int64_t n64 = p.row_len ? (int64_t)p.row_len[row0 + rr] : p.ld;
        n64 = n64 < 0 ? 0 : (n64 > p.ld ? p.ld : n64);
        nr[rr] = n64;
        n_max = max(n_max, n64);
    }
    const int64_t s_begin = (int64_t)c * p.chunk_keys + (int64_t)sub * p.run_keys;
    const int64_t s_end = min(s_begin + p.run_keys, n_max);
    if (s_begin >= s_end) return;
    const int col = lane & 15, quarter = lane >> 4;
    // Bytes [32 quarter, + 32) of the head dimension; with D = 64 the upper
    // two quarters re-read the lower two and the query there is zero.
    const int qoff = 32 * (quarter % (D / 32));
    const bool qlive = 32 * quarter < D;

    for (int j = lane; j < RG * H; j += kWave) wl[wave][j] = p.w[row0 * H + j];
    v8i qa[RG][MT];
#pragma unroll
    for (int rr = 0; rr < RG; ++rr) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const v8i v = load32(p.q + (((row0 + rr) * H + 16 * mt + col) * D + qoff));
            qa[rr][mt] = qlive ? v : v8i{0, 0, 0, 0, 0, 0, 0, 0};
        }
    }
    __builtin_amdgcn_wave_barrier();   // a wave's LDS accesses complete in order: its reads see its writes
    const float4* wv = reinterpret_cast<const float4*>(&wl[wave][0]);

    const uint8_t* kg = p.k + (int64_t)g * p.ld * D + qoff;
    const float* sg = p.k_scale + (int64_t)g * p.ld;
    float* out = p.scores + row0 * p.ld;
    // Column col of half t of slot u is key min(s_begin + 32 u + 16 t + col,
    // s_end - 1): lanes past the run recompute the run's last key and store
    // the same value there, so loads, matrix steps and stores run without
    // branches and the loads stay in flight across iterations.
    const int tiles = (int)((s_end - s_begin + kTile - 1) / kTile);
    auto key_at = [&](int u, int t) { return min(s_begin + (int64_t)u * kTile + 16 * t + col, s_end - 1); };
    struct Slot {
        v8i kb[2];
        float ks[2];
    };
    auto load_slot = [&](int u) {
        Slot r;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int64_t key = key_at(u, t);
            r.kb[t] = load32(kg + key * D);
            r.ks[t] = sg[key];
        }
        return r;
    };
    auto use_slot = [&](const Slot& r, int u) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int rr = 0; rr < RG; ++rr) {
                const float sum = tile_score<H>(qa[rr], r.kb[t], r.ks[t], wv + rr * (H / 4), quarter);
                // the run covers the longer row of the pair: store this row's own keys
                const int64_t key = key_at(u, t);
                if (key < nr[rr]) out[rr * p.ld + key] = sum;
            }
        }
    };
    Slot ring[kRing];
#pragma unroll
    for (int r = 0; r < kRing - 1; ++r) ring[r] = load_slot(r);
    constexpr int kAhead = kRing - 1;
    int u0 = 0;
    for (; u0 + kRing <= tiles; u0 += kRing) {
#pragma unroll
        for (int r = 0; r < kRing; ++r) {
            // the loads for slot u0 + r + kAhead go out before slot u0 + r is used
            ring[(r + kAhead) % kRing] = load_slot(u0 + r + kAhead);
            use_slot(ring[r], u0 + r);
        }
    }
#pragma unroll
    for (int r = 0; r < kRing - 1; ++r)   // the last slots (already loaded)
        if (u0 + r < tiles) use_slot(ring[r], u0 + r);
}

// Workgroups of one instance resident on the device at once (0 = unknown:
// the natural chunk size is used). Queried once per device, never while the
// stream is being captured into a graph.
template <int H, int D, int RG>
int resident_workgroups(void* stream) {
    static int cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    if (cached[dev] == 0) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing((hipStream_t)stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone)
            return 0;
        int per_cu = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, indexer_kernel<H, D, RG>, kWaves * kWave, 0) != hipSuccess)
            return 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cached[dev] = std::max(1, per_cu * cus);
    }
    return cached[dev];
}

template <int H, int D, int RG>
gvr_status launch(IdxParams q, int64_t caches, void* stream) {
    // Key chunks per cache. The natural size gives every wave a run of
    // kTilesPerWave tiles; the grid is then resized to whole rounds of the
    // workgroups the device holds at once: one round when the natural grid
    // fits (small batches get finer chunks that reach more compute units, runs
    // of at least kMinRun keys), else as many full rounds as it fills (no
    // partly filled last round).
    const int wpr = q.chunk_keys / (kTilesPerWave * kTile);
    int run = kTilesPerWave * kTile;
    const int slots = resident_workgroups<H, D, RG>(stream);
    if (slots > 0) {
        const int64_t nat = (q.ld + (int64_t)wpr * run - 1) / ((int64_t)wpr * run);
        const int64_t rounds = std::max<int64_t>(1, nat * caches / slots);
        const int64_t chunks = std::max<int64_t>(1, rounds * slots / caches);
        const int64_t per = (q.ld + chunks - 1) / chunks;                        // keys per chunk
        const int64_t r = ((per + wpr - 1) / wpr + kTile - 1) / kTile * kTile;   // per wave, whole tiles
        run = (int)std::max<int64_t>(std::min<int64_t>(r, 1 << 24), kMinRun);
    }
    q.run_keys = run;
    q.chunk_keys = wpr * run;
    const int64_t chunks = (q.ld + q.chunk_keys - 1) / q.chunk_keys;
    if (chunks * caches > 0x7FFFFFFF) return GVR_ERR_TOO_LONG;
    q.chunks = (int32_t)chunks;
    if (chunks * caches + (q.prev ? q.rows : 0) > 0x7FFFFFFF) return GVR_ERR_TOO_LONG;
    q.sample_base = (int32_t)(chunks * caches);   // the fused guess's workgroups follow the key chunks
    const unsigned grid = (unsigned)(chunks * caches + (q.prev ? q.rows : 0));
    hipLaunchKernelGGL((indexer_kernel<H, D, RG>), dim3(grid), dim3(kWaves * kWave), 0, (hipStream_t)stream, q);
    return hipGetLastError() == hipSuccess ? GVR_OK : GVR_ERR_HIP;
}

// Rows per wave: 2 when a cache's rows pair up and the two rows' query
// registers fit (H <= 64), else 1.
constexpr int rows_per_wave(int H, int group) { return (group % 2 == 0 && H <= 64) ? 2 : 1; }

template <int H, int D>
gvr_status launch_rg(const IdxParams& q, int64_t caches, void* stream) {
    if constexpr (H <= 64) {
        if (rows_per_wave(H, q.group) == 2) return launch<H, D, 2>(q, caches, stream);
    }
    return launch<H, D, 1>(q, caches, stream);
}

// The indexer launch; with prev (and gstats), also the fused guess.
gvr_status indexer_launch(const uint8_t* q, const float* w, const uint8_t* k, const float* k_scale, int64_t B,
                          int32_t H, int32_t D, int32_t group, int64_t ld, const int32_t* row_len, float* scores,
                          const int32_t* prev, int32_t K, int32_t* gstats, void* stream) {
    if (B < 0 || ld < 0) return GVR_ERR_INVALID_ARG;
    if (!(H == 32 || H == 64 || H == 128) || !(D == 64 || D == 128)) return GVR_ERR_INVALID_ARG;
    if (group < 1 || group > kWaves || B % group != 0) return GVR_ERR_INVALID_ARG;
    if (ld > kMaxLd) return GVR_ERR_TOO_LONG;
    if (B == 0 || ld == 0) return GVR_OK;
    if (!q || !w || !k || !k_scale || !scores) return GVR_ERR_INVALID_ARG;
    if (((uintptr_t)q | (uintptr_t)k) & 15) return GVR_ERR_INVALID_ARG;   // 16-byte loads
    if (B > 0x7FFFFFFF) return GVR_ERR_TOO_LONG;
    IdxParams p;
    p.q = q;
    p.w = w;
    p.k = k;
    p.k_scale = k_scale;
    p.row_len = row_len;
    p.scores = scores;
    p.ld = ld;
    p.rows = (int32_t)B;
    p.group = group;
    p.prev = gstats ? prev : nullptr;
    p.gstats = gstats;
    p.K = K;
    p.sample_base = 0;
    const int rg = rows_per_wave(H, group);
    const int wpr = kWaves / (group / rg);
    p.chunk_keys = wpr * kTilesPerWave * kTile;
    p.run_keys = kTilesPerWave * kTile;
    p.chunks = 0;
    const int64_t caches = B / group;
    if (H == 32) return D == 64 ? launch_rg<32, 64>(p, caches, stream) : launch_rg<32, 128>(p, caches, stream);
    if (H == 64) return D == 64 ? launch_rg<64, 64>(p, caches, stream) : launch_rg<64, 128>(p, caches, stream);
    return D == 64 ? launch_rg<128, 64>(p, caches, stream) : launch_rg<128, 128>(p, caches, stream);
}

}  // namespace

extern "C" {

gvr_status gvr_indexer_scores(const uint8_t* q, const float* w, const uint8_t* k, const float* k_scale,
                              int64_t B, int32_t H, int32_t D, int32_t group, int64_t ld,
                              const int32_t* row_len, float* scores, void* stream) {
    return indexer_launch(q, w, k, k_scale, B, H, D, group, ld, row_len, scores, nullptr, 0, nullptr, stream);
}

gvr_status gvr_indexer_topk(const uint8_t* q, const float* w, const uint8_t* k, const float* k_scale,
                            int64_t B, int32_t H, int32_t D, int32_t group, int64_t ld,
                            const int32_t* row_len, float* scores, const int32_t* prev_topk, int32_t K,
                            int32_t* out_idx, void* stream, const gvr_options* options,
                            gvr_row_stats* stats) {
    // The Top-K's own checks (K, options) with nothing enqueued: B = 0.
    gvr_status st = gvr_topk_ex(scores, 0, ld, row_len, prev_topk, K, out_idx, stream, options, stats);
    if (st != GVR_OK) return st;
    if (B > 0 && !out_idx) return GVR_ERR_INVALID_ARG;
    // The fused guess: the indexer scores each row's sample of prev_topk and
    // leaves the row's guess statistics in the tail of its out_idx row, where
    // the Top-K reads them (instead of gathering the sample's scores after
    // the indexer). Not with the paper's Phase 2 schedule (which reads every
    // guessed score) or without a guess.
    gvr_host::CallOptions o;
    int dummy = 0;
    st = gvr_host::validate(&dummy, 1, 1, K, &dummy, options, 1, &o);
    if (st != GVR_OK) return st;
    const bool fused = prev_topk && o.use_guess && !o.secant && K >= kGuessWords;
    int32_t* gstats = fused && out_idx ? out_idx + (K - kGuessWords) : nullptr;
    st = indexer_launch(q, w, k, k_scale, B, H, D, group, ld, row_len, scores, prev_topk, K, gstats, stream);
    if (st != GVR_OK) return st;
    if (fused)
        return gvr_internal::topk_with_guess_stats(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options,
                                                   stats);
    return gvr_topk_ex(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats);
}

}  // extern "C"
