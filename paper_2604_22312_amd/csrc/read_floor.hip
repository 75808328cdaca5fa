// read_floor.hip -- the plain read rate of score rows on MI355X (gfx950):
// every element of rows[b][0, n_b) is read once and folded into one xor word
// per row; nothing else is computed. The Top-K streams the same bytes, so this
// kernel is the practical ceiling its streaming pass is measured against. It
// is a measurement helper, not a step of the Top-K (declared in gvr_topk.h).
//
// Each row is read by P workgroups of 16 waves (P chosen so that the grid
// holds about two workgroups per compute unit), the parts of a row on one
// XCD; each wave streams a
// contiguous run of 1 KB slabs (64 lanes x one 16-byte load) with eight
// slabs in flight, using non-temporal loads. Part p of row b writes word
// out[b][p] (the xor of its elements' bits); part 0 also zeroes the words of
// the parts a row does not have, so the xor of a row's 16 words covers every
// element once.

#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "gvr_topk.h"

namespace {

constexpr int kFloorWaves = 16;
constexpr int kFloorRing = 8;
constexpr int kFloorMaxParts = 16;

typedef __attribute__((ext_vector_type(4))) unsigned u32x4;

__global__ __launch_bounds__(kFloorWaves * 64) void read_floor_kernel(const float* __restrict__ scores, int64_t ld,
                                                                       const int32_t* __restrict__ row_len, int rows,
                                                                       int parts, uint32_t* __restrict__ out) {
    // Slots (row, part) in order on one XCD: workgroup i runs on XCD i % 8,
    // so neighbouring parts of the address space share an XCD.
    const int slot = (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8);
    const int row = slot / parts, part = slot - row * parts;
    if (row >= rows) return;
    // the row length through the scalar data cache (the row is wave-uniform)
    int64_t n64 = row_len ? (int64_t)__builtin_amdgcn_readfirstlane(
                                *(const __attribute__((address_space(4))) int32_t*)(row_len + row))
                          : ld;
    n64 = n64 < 0 ? 0 : (n64 > ld ? ld : n64);
    const int n = (int)n64;
    const float* x = scores + (int64_t)row * ld;
    // 16-byte blocks of the row (virtual index = element index + aoff; the
    // first block starts the row's first 128-byte line, so 1 KB slabs are
    // whole lines)
    const int aoff = (int)(((uintptr_t)x >> 2) & 31);
    const u32x4* xa = reinterpret_cast<const u32x4*>(x - aoff);
    const int nq = n > 0 ? (n + aoff + 3) >> 2 : 0;
    const int nslab = (nq + 63) >> 6;
    const int ps = (nslab + parts - 1) / parts;
    const int s0 = std::min(part * ps, nslab), s1 = std::min(s0 + ps, nslab);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int per = (s1 - s0 + kFloorWaves - 1) / kFloorWaves;
    const int a = std::min(s0 + wave * per, s1), b = std::min(a + per, s1);
    const int cnt = b - a;
    uint32_t acc = 0u;
    if (cnt > 0) {
        const int qlast = nq - 1;
        auto block_of = [&](int s) { return std::min((a + std::min(s, cnt - 1)) * 64 + lane, qlast); };
        u32x4 buf[kFloorRing];
#pragma unroll
        for (int u = 0; u < kFloorRing; ++u) buf[u] = __builtin_nontemporal_load(xa + block_of(u));
        for (int s = 0; s < cnt; s += kFloorRing) {
#pragma unroll
            for (int u = 0; u < kFloorRing; ++u) {
                const int sg = a + s + u;   // the row's slab (wave-uniform)
                const int q = sg * 64 + lane;
                if (s + u < cnt) {
                    const u32x4 v = buf[u];
                    if (sg == 0 || 256 * sg + 255 - aoff >= n) {   // an edge slab: mask by element
                        const int e0 = 4 * q - aoff;
                        if (q <= qlast)
                            acc ^= (e0 >= 0 && e0 < n ? v.x : 0u) ^ (e0 + 1 >= 0 && e0 + 1 < n ? v.y : 0u) ^
                                   (e0 + 2 >= 0 && e0 + 2 < n ? v.z : 0u) ^ (e0 + 3 >= 0 && e0 + 3 < n ? v.w : 0u);
                    } else {
                        acc ^= v.x ^ v.y ^ v.z ^ v.w;
                    }
                }
                if (s + u + kFloorRing < cnt) buf[u] = __builtin_nontemporal_load(xa + block_of(s + u + kFloorRing));
            }
        }
    }
    // fold the wave, then the workgroup's waves, into the part's word
    for (int o = 32; o > 0; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
    __shared__ uint32_t wsum[kFloorWaves];
    if (lane == 0) wsum[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0u;
        for (int w = 0; w < kFloorWaves; ++w) t ^= wsum[w];
        out[(int64_t)row * kFloorMaxParts + part] = t;
    }
    if (part == 0 && (int)threadIdx.x >= parts && (int)threadIdx.x < kFloorMaxParts) out[(int64_t)row * kFloorMaxParts + threadIdx.x] = 0u;
}

// Compute units of a device, queried once per device.
int floor_cu_count(int device) {
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

}  // namespace

extern "C" gvr_status gvr_read_floor(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                                     uint32_t* out_words, void* stream) {
    if (B < 0 || ld < 0) return GVR_ERR_INVALID_ARG;
    if (B == 0) return GVR_OK;
    if (!scores || !out_words) return GVR_ERR_INVALID_ARG;
    if (ld > (int64_t)0x7FFFFFF0 || B > ((int64_t)1 << 26)) return GVR_ERR_TOO_LONG;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return GVR_ERR_HIP;
    const int cus = floor_cu_count(device);
    // about two workgroups per compute unit, parts of at least 16 slabs
    int64_t parts = std::max<int64_t>(1, (2 * (int64_t)cus) / B);
    parts = std::min<int64_t>(parts, kFloorMaxParts);
    parts = std::max<int64_t>(1, std::min<int64_t>(parts, (ld / 4 + 64 * 16 - 1) / (64 * 16)));
    const hipStream_t hs = (hipStream_t)stream;
    const int64_t grid = (B * parts + 7) / 8 * 8;   // a multiple of the 8 XCDs
    hipLaunchKernelGGL(read_floor_kernel, dim3((unsigned)grid), dim3(kFloorWaves * 64), 0, hs, scores, ld, row_len,
                       (int)B, (int)parts, out_words);
    return hipGetLastError() == hipSuccess ? GVR_OK : GVR_ERR_HIP;
}
