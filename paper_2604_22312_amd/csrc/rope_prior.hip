// rope_prior.hip -- the static RoPE/YaRN prior P_static (Sec. 3.2, 3.3) on
// MI355X (gfx950), behind the C ABI declared in include/gvr_rope_prior.h.
//
//   g kernel. One thread per relative position Delta (256-thread
//   workgroups). The first d/2 threads of every workgroup derive the YaRN
//   angles theta'_i into LDS (a few pow/log calls, the same in every
//   workgroup), then each thread sums cos(Delta * theta'_i) over the pairs in
//   float64 and stores g(Delta). Compute-bound on fp64 cos; run once per
//   model and length, not per decode step.
//
//   select kernel. One workgroup of 1024 threads finds the K-th largest g by
//   a radix select over the 64-bit order-preserving key of each float64
//   (digits of 11, 11, 11, 11, 10, 10 bits; an LDS histogram per digit). The
//   first digits read g from global memory (L2-resident at these lengths);
//   as soon as the elements sharing the selected prefix fit in LDS (<= 4096)
//   they are gathered there and the remaining digits never touch memory
//   again. A final pass in index order writes every Delta whose key beats
//   the K-th key, plus the first equal ones, at offsets from two block scans
//   per 4096-element chunk, so the output comes out in ascending order.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "gvr_rope_prior.h"

#define DEV __device__ __forceinline__

namespace {

constexpr int kGBlock = 256;                 // threads of a g workgroup
constexpr int kMaxPairs = 256;               // d <= 512
constexpr int kSBlock = 1024;                // threads of the select workgroup
constexpr int kSWaves = kSBlock / 64;
constexpr int kSelBins = 2048;               // widest digit: 11 bits
constexpr int kGather = 4096;                // keys the select keeps in LDS
constexpr int kDigits = 6;
constexpr int kEmitPer = 4;                  // consecutive elements per thread in the emit pass
constexpr int64_t kMaxN = ((int64_t)1 << 31) - 16;

__constant__ int kDigitShift[kDigits] = {53, 42, 31, 20, 10, 0};
__constant__ int kDigitBits[kDigits] = {11, 11, 11, 11, 10, 10};

struct RopeArgs {
    int d;
    int orig_ctx;
    double base, scale, beta_fast, beta_slow;
};

// theta'_i of one rotary pair (YaRN ramp over the pair index).
DEV double yarn_angle(int i, const RopeArgs& a) {
#pragma clang fp contract(off)
    const double two_pi = 6.283185307179586;
    const double ln_base = log(a.base);
    const double x_fast = a.d * log(a.orig_ctx / (two_pi * a.beta_fast)) / (2.0 * ln_base);
    const double x_slow = a.d * log(a.orig_ctx / (two_pi * a.beta_slow)) / (2.0 * ln_base);
    const double lo = fmax(floor(x_fast), 0.0);
    const double hi = fmin(ceil(x_slow), (double)(a.d - 1));
    const double theta = pow(a.base, -2.0 * i / a.d);
    const double gamma = fmin(fmax((i - lo) / fmax(hi - lo, 1e-3), 0.0), 1.0);
    return theta * (1.0 - gamma) + (theta / a.scale) * gamma;
}

__global__ __launch_bounds__(kGBlock) void rope_g_kernel(int64_t n, RopeArgs a, double* __restrict__ g,
                                                         double* __restrict__ theta_out) {
    __shared__ double th[kMaxPairs];
    const int h = a.d / 2;
    const int t = threadIdx.x;
    if (t < h) {
        const double v = yarn_angle(t, a);
        th[t] = v;
        if (blockIdx.x == 0 && theta_out) theta_out[t] = v;
    }
    __syncthreads();
    const int64_t delta = (int64_t)blockIdx.x * kGBlock + t;
    if (delta >= n) return;
    const double x = (double)delta;
    double acc = 0.0;
    for (int i = 0; i < h; ++i) acc += cos(x * th[i]);
    g[delta] = 2.0 * acc;
}

// Order-preserving 64-bit key of a float64 (-0.0 folded into +0.0 first).
DEV uint64_t order_key(double v) {
    v = v + 0.0;
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Exclusive prefix sum of v over the workgroup's threads in thread order;
// *total receives the sum over all threads. Every thread must call it.
DEV uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint32_t x = v;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    uint32_t base = 0, tot = 0;
    for (int i = 0; i < kSWaves; ++i) {
        const uint32_t s = wsum[i];
        base += (i < w) ? s : 0u;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return base + x - v;
}

__global__ __launch_bounds__(kSBlock) void prior_select_kernel(const double* __restrict__ g, int64_t n, int K,
                                                               int32_t* __restrict__ out) {
    __shared__ uint32_t hist[kSelBins];
    __shared__ uint64_t cand[kGather];
    __shared__ uint32_t wsum[kSWaves];
    __shared__ uint32_t s_bin, s_need, s_cnt, s_ncand;
    const int tid = threadIdx.x;
    if (n <= K) {
        for (int i = tid; i < K; i += kSBlock) out[i] = (i < n) ? i : -1;
        return;
    }
    uint64_t prefix = 0, mask = 0;
    uint32_t need = (uint32_t)K;     // rank of the K-th key among those sharing `prefix`
    uint32_t ncand = 0;
    bool in_lds = false;
    for (int dg = 0; dg < kDigits; ++dg) {
        const int sh = kDigitShift[dg];
        const int nb = 1 << kDigitBits[dg];
        for (int b = tid; b < nb; b += kSBlock) hist[b] = 0;
        __syncthreads();
        if (in_lds) {
            for (uint32_t i = tid; i < ncand; i += kSBlock) {
                const uint64_t k = cand[i];
                if ((k & mask) == prefix) atomicAdd(&hist[(k >> sh) & (uint64_t)(nb - 1)], 1u);
            }
        } else {
            for (int64_t i = tid; i < n; i += kSBlock) {
                const uint64_t k = order_key(g[i]);
                if ((k & mask) == prefix) atomicAdd(&hist[(k >> sh) & (uint64_t)(nb - 1)], 1u);
            }
        }
        __syncthreads();
        // Thread t holds bins nb-1-2t and nb-2-2t (descending), so a scan in
        // thread order counts the keys in higher bins.
        const int b0 = nb - 1 - 2 * tid, b1 = b0 - 1;
        const uint32_t c0 = (b0 >= 0) ? hist[b0] : 0u;
        const uint32_t c1 = (b1 >= 0) ? hist[b1] : 0u;
        uint32_t tot;
        const uint32_t above = block_exclusive_scan(c0 + c1, wsum, &tot);
        if (above < need && need <= above + c0 + c1) {
            if (need <= above + c0) {
                s_bin = (uint32_t)b0; s_need = need - above; s_cnt = c0;
            } else {
                s_bin = (uint32_t)b1; s_need = need - above - c0; s_cnt = c1;
            }
        }
        __syncthreads();
        prefix |= (uint64_t)s_bin << sh;
        mask |= (uint64_t)(nb - 1) << sh;
        need = s_need;
        const uint32_t cnt = s_cnt;
        __syncthreads();
        if (!in_lds && cnt <= (uint32_t)kGather && dg + 1 < kDigits) {
            if (tid == 0) s_ncand = 0;
            __syncthreads();
            for (int64_t i = tid; i < n; i += kSBlock) {
                const uint64_t k = order_key(g[i]);
                if ((k & mask) == prefix) {
                    const uint32_t slot = atomicAdd(&s_ncand, 1u);
                    if (slot < (uint32_t)kGather) cand[slot] = k;
                }
            }
            __syncthreads();
            ncand = s_ncand;
            in_lds = true;
        }
    }
    // prefix is now the K-th largest key; `need` keys equal to it are taken,
    // the lowest indices first.
    const uint64_t kth = prefix;
    uint32_t carry_eq = 0, carry_sel = 0;
    for (int64_t base = 0; base < n; base += (int64_t)kSBlock * kEmitPer) {
        const int64_t i0 = base + (int64_t)tid * kEmitPer;
        uint32_t gt = 0, eq = 0;   // bit j: element i0 + j beats / equals the K-th key
        for (int j = 0; j < kEmitPer; ++j) {
            if (i0 + j < n) {
                const uint64_t k = order_key(g[i0 + j]);
                gt |= (uint32_t)(k > kth) << j;
                eq |= (uint32_t)(k == kth) << j;
            }
        }
        uint32_t tot_eq;
        uint32_t rank = carry_eq + block_exclusive_scan((uint32_t)__builtin_popcount(eq), wsum, &tot_eq);
        uint32_t sel = gt;
        for (int j = 0; j < kEmitPer; ++j) {
            if ((eq >> j) & 1u) {
                if (rank < need) sel |= 1u << j;
                ++rank;
            }
        }
        uint32_t tot_sel;
        uint32_t pos = carry_sel + block_exclusive_scan((uint32_t)__builtin_popcount(sel), wsum, &tot_sel);
        for (int j = 0; j < kEmitPer; ++j) {
            if (((sel >> j) & 1u) && pos < (uint32_t)K) out[pos++] = (int32_t)(i0 + j);
        }
        carry_eq += tot_eq;
        carry_sel += tot_sel;
    }
}

bool finite_pos(double v) { return isfinite(v) && v > 0.0; }

gvr_status read_params(const gvr_rope_params* p, RopeArgs* a) {
    gvr_rope_params d;
    if (!p) {
        gvr_rope_params_default(&d);
        p = &d;
    }
    if (p->d_rope < 2 || p->d_rope > 2 * kMaxPairs || (p->d_rope & 1)) return GVR_ERR_INVALID_ARG;
    if (p->orig_ctx < 1) return GVR_ERR_INVALID_ARG;
    if (!isfinite(p->base) || p->base <= 1.0) return GVR_ERR_INVALID_ARG;
    if (!finite_pos(p->scale) || !finite_pos(p->beta_fast) || !finite_pos(p->beta_slow)) return GVR_ERR_INVALID_ARG;
    a->d = p->d_rope;
    a->orig_ctx = p->orig_ctx;
    a->base = p->base;
    a->scale = p->scale;
    a->beta_fast = p->beta_fast;
    a->beta_slow = p->beta_slow;
    return GVR_OK;
}

gvr_status launch_g(int64_t n, const RopeArgs& a, double* g, double* theta, void* stream) {
    const int64_t blocks = n > 0 ? (n + kGBlock - 1) / kGBlock : 1;
    hipLaunchKernelGGL(rope_g_kernel, dim3((unsigned)blocks), dim3(kGBlock), 0, (hipStream_t)stream, n, a, g,
                       theta);
    return hipGetLastError() == hipSuccess ? GVR_OK : GVR_ERR_HIP;
}

}  // namespace

extern "C" {

void gvr_rope_params_default(gvr_rope_params* p) {
    if (!p) return;
    p->d_rope = 64;
    p->orig_ctx = 4096;
    p->base = 10000.0;
    p->scale = 40.0;
    p->beta_fast = 32.0;
    p->beta_slow = 1.0;
}

gvr_status gvr_rope_g(int64_t n, const gvr_rope_params* params, double* g, double* theta, void* stream) {
    RopeArgs a;
    const gvr_status st = read_params(params, &a);
    if (st != GVR_OK) return st;
    if (n < 0 || (n > 0 && !g)) return GVR_ERR_INVALID_ARG;
    if (n > kMaxN) return GVR_ERR_TOO_LONG;
    if (n == 0 && !theta) return GVR_OK;
    return launch_g(n, a, g, theta, stream);
}

gvr_status gvr_rope_prior(int64_t n, int32_t K, const gvr_rope_params* params, double* g, int32_t* out_delta,
                          void* stream) {
    RopeArgs a;
    const gvr_status st = read_params(params, &a);
    if (st != GVR_OK) return st;
    if (n < 0 || (n > 0 && !g) || !out_delta) return GVR_ERR_INVALID_ARG;
    if (K < 1 || K > GVR_MAX_K) return GVR_ERR_UNSUPPORTED_K;
    if (n > kMaxN) return GVR_ERR_TOO_LONG;
    if (n > 0) {
        const gvr_status s = launch_g(n, a, g, nullptr, stream);
        if (s != GVR_OK) return s;
    }
    hipLaunchKernelGGL(prior_select_kernel, dim3(1), dim3(kSBlock), 0, (hipStream_t)stream, (const double*)g, n,
                       (int)K, out_delta);
    return hipGetLastError() == hipSuccess ? GVR_OK : GVR_ERR_HIP;
}

}  // extern "C"
