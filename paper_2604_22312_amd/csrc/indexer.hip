// indexer.hip -- FP8 indexer scores of DeepSeek Sparse Attention (Sec. 2.1,
// Eq. indexer) on the MI355X matrix cores, behind include/gvr_indexer.h.
//
// One wave computes the scores of one row for a run of 32-key tiles. Per
// tile the logits q[j] . k[s] of all H heads and 32 keys are 32 x 32 blocks
// of v_mfma_f32_32x32x16_fp8_fp8 (heads down the rows, keys across the
// columns, D / 16 steps over the head dimension); the epilogue scales each
// key's column by its k_scale, applies ReLU, weights the heads and sums them.
// In the accumulator layout a lane holds 16 heads of one key (row
// 8 (i / 4) + 4 (lane / 32) + i % 4 of column lane % 32 for register i), so
// the head sum is 16 fused multiply-adds per 32 heads plus one exchange with
// lane ^ 32. The reduction dimension is visited in the order the loads give:
// lane half h holds bytes [h D / 2, (h + 1) D / 2) of its head and of its key,
// k-step t uses 8 of them, and A and B use the same order, so the product is
// the plain dot product.
//
// Each lane keeps its half of its query heads (16-byte aligned) and their
// weights in registers for the whole run; the keys stream through a double
// buffer (a tile's 32 x D bytes are one contiguous block of the cache, read
// with 16-byte loads while the previous tile is on the matrix cores). The
// rows of one cache (group of draft rows) run on waves of one workgroup at
// the same keys, so the cache is read from HBM once for all of them. The
// kernel is HBM-bound: D + 4 bytes per key and cache, 4 bytes per score.

#include <hip/hip_runtime.h>

#include <stdint.h>

#include "gvr_indexer.h"

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;                // waves per workgroup
constexpr int kTile = 32;                // keys per column tile
constexpr int kTilesPerWave = 32;        // tiles of one wave's run (1024 keys)
constexpr int64_t kMaxLd = ((int64_t)1 << 31) - 16;

typedef float v16f __attribute__((ext_vector_type(16)));

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
};

template <int D>
struct KeyHalf {
    uint64_t b[D / 16];   // bytes [h D / 2, (h + 1) D / 2) of one key: 8 per k-step
};

template <int D>
__device__ __forceinline__ KeyHalf<D> load_half(const uint8_t* p) {
    KeyHalf<D> r;
    const uint4* s = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
        const uint4 v = s[j];
        r.b[2 * j] = (uint64_t)v.x | ((uint64_t)v.y << 32);
        r.b[2 * j + 1] = (uint64_t)v.z | ((uint64_t)v.w << 32);
    }
    return r;
}

template <int H, int D>
__global__ __launch_bounds__(kWaves * kWave) void indexer_kernel(IdxParams p) {
    constexpr int MT = H / 32;   // 32-head row tiles
    constexpr int KS = D / 16;   // k-steps of 16 bytes (8 per lane half)
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int G = p.group;
    const int wpr = kWaves / G;               // waves per row (one idle wave when G = 3)
    if (wave >= G * wpr) return;
    const int g = blockIdx.x / p.chunks;      // cache
    const int c = blockIdx.x - g * p.chunks;  // key chunk
    const int r_in = wave % G, sub = wave / G;
    const int64_t row = (int64_t)g * G + r_in;
    if (row >= p.rows) return;
    int64_t n64 = p.row_len ? (int64_t)p.row_len[row] : p.ld;
    n64 = n64 < 0 ? 0 : (n64 > p.ld ? p.ld : n64);
    const int64_t s_begin = (int64_t)c * p.chunk_keys + sub * (kTilesPerWave * kTile);
    const int64_t s_end = min(s_begin + kTilesPerWave * kTile, n64);
    if (s_begin >= s_end) return;
    const int col = lane & 31, h = lane >> 5;

    // Query halves and head weights of the rows this lane's registers hold.
    uint64_t qa[MT][KS];
    float wr[MT][16];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int head = 32 * mt + col;
        const KeyHalf<D> qh = load_half<D>(p.q + ((row * H + head) * D + h * (D / 2)));
#pragma unroll
        for (int t = 0; t < KS; ++t) qa[mt][t] = qh.b[t];
#pragma unroll
        for (int i = 0; i < 16; ++i) wr[mt][i] = p.w[row * H + 32 * mt + 8 * (i / 4) + 4 * h + (i % 4)];
    }

    const uint8_t* kg = p.k + (int64_t)g * p.ld * D + h * (D / 2);
    const float* sg = p.k_scale + (int64_t)g * p.ld;
    float* out = p.scores + row * p.ld;
    auto key_of_tile = [&](int64_t s0) { return min(s0 + col, n64 - 1); };   // clamped: a partial tile re-reads key n - 1
    int64_t s0 = s_begin;
    KeyHalf<D> kb = load_half<D>(kg + key_of_tile(s0) * D);
    float ks = sg[key_of_tile(s0)];
    for (; s0 < s_end; s0 += kTile) {
        // Next tile's loads first (the last iteration re-reads this tile's keys).
        const int64_t s1 = s0 + kTile < s_end ? s0 + kTile : s0;
        const KeyHalf<D> kn = load_half<D>(kg + key_of_tile(s1) * D);
        const float ksn = sg[key_of_tile(s1)];
        v16f acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = (v16f)(0.f);
#pragma unroll
        for (int t = 0; t < KS; ++t) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_fp8_fp8((long)qa[mt][t], (long)kb.b[t], acc[mt], 0, 0, 0);
        }
        float sum = 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
            for (int i = 0; i < 16; ++i) sum += wr[mt][i] * fmaxf(acc[mt][i] * ks, 0.f);
        }
        sum += __shfl_xor(sum, 32, kWave);
        const int64_t s = s0 + col;
        if (h == 0 && s < s_end) out[s] = sum;
        kb = kn;
        ks = ksn;
    }
}

template <int H, int D>
gvr_status launch(const IdxParams& q, unsigned grid, void* stream) {
    hipLaunchKernelGGL((indexer_kernel<H, D>), dim3(grid), dim3(kWaves * kWave), 0, (hipStream_t)stream, q);
    return hipGetLastError() == hipSuccess ? GVR_OK : GVR_ERR_HIP;
}

}  // namespace

extern "C" {

gvr_status gvr_indexer_scores(const uint8_t* q, const float* w, const uint8_t* k, const float* k_scale,
                              int64_t B, int32_t H, int32_t D, int32_t group, int64_t ld,
                              const int32_t* row_len, float* scores, void* stream) {
    if (B < 0 || ld < 0) return GVR_ERR_INVALID_ARG;
    if (!(H == 32 || H == 64 || H == 128) || !(D == 64 || D == 128)) return GVR_ERR_INVALID_ARG;
    if (group < 1 || group > kWaves || B % group != 0) return GVR_ERR_INVALID_ARG;
    if (ld > kMaxLd) return GVR_ERR_TOO_LONG;
    if (B == 0 || ld == 0) return GVR_OK;
    if (!q || !w || !k || !k_scale || !scores) return GVR_ERR_INVALID_ARG;
    if (((uintptr_t)q | (uintptr_t)k) & 15) return GVR_ERR_INVALID_ARG;   // 16-byte loads
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
    const int wpr = kWaves / group;
    p.chunk_keys = wpr * kTilesPerWave * kTile;
    const int64_t chunks = (ld + p.chunk_keys - 1) / p.chunk_keys;
    const int64_t caches = B / group;
    if (chunks * caches > 0x7FFFFFFF) return GVR_ERR_TOO_LONG;
    p.chunks = (int32_t)chunks;
    const unsigned grid = (unsigned)(chunks * caches);
    if (H == 32) return D == 64 ? launch<32, 64>(p, grid, stream) : launch<32, 128>(p, grid, stream);
    if (H == 64) return D == 64 ? launch<64, 64>(p, grid, stream) : launch<64, 128>(p, grid, stream);
    return D == 64 ? launch<128, 64>(p, grid, stream) : launch<128, 128>(p, grid, stream);
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
    st = gvr_indexer_scores(q, w, k, k_scale, B, H, D, group, ld, row_len, scores, stream);
    if (st != GVR_OK) return st;
    return gvr_topk_ex(scores, B, ld, row_len, prev_topk, K, out_idx, stream, options, stats);
}

}  // extern "C"
