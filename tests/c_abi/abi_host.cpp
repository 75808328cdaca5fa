// A host program that uses the library through its C ABI alone (no Python,
// no torch): device buffers from the HIP runtime, gvr_topk / radix_topk /
// gvr_topk_ex and the caller-workspace calls on one stream, each result
// compared with the C oracle
// (oracle/oracle_topk.c, linked in as a test dependency).
//
// Inputs: B rows of stride ld from a 64-bit linear congruential generator
// (uniform floats in [0, 1), seeded), ragged lengths including n <= K and
// n = K + 1; the guess is the oracle's Top-K of a perturbed copy of the rows.
// Exit status 0 when every call succeeded and matched, else nonzero.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "gvr_topk.h"

extern "C" int oracle_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                           int32_t* out_idx, uint32_t* kth_key, int32_t* n_gt);

namespace {

uint64_t lcg_state = 0x9E3779B97F4A7C15ull;
float lcg_uniform() {
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    return (float)(lcg_state >> 40) * (1.0f / 16777216.0f);
}

#define HIP_OK(x)                                                                    \
    do {                                                                             \
        hipError_t e_ = (x);                                                         \
        if (e_ != hipSuccess) {                                                      \
            std::fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));             \
            return 3;                                                                \
        }                                                                            \
    } while (0)

}  // namespace

int main() {
    const int64_t B = 6, ld = 20011;
    const int32_t K = 2048;
    std::vector<float> x(B * ld), y(B * ld);
    for (auto& v : x) v = lcg_uniform();
    for (int64_t i = 0; i < B * ld; ++i) y[i] = x[i] + 0.05f * (lcg_uniform() - 0.5f);
    std::vector<int32_t> len = {20011, 2048, 2049, 100, 15000, 4097};
    std::vector<int32_t> exp(B * K), guess(B * K), got(B * K);
    if (oracle_topk(x.data(), B, ld, len.data(), K, exp.data(), nullptr, nullptr) != 0) return 4;
    if (oracle_topk(y.data(), B, ld, len.data(), K, guess.data(), nullptr, nullptr) != 0) return 4;

    std::printf("%s\n", gvr_version());
    // An argument error is reported before anything is enqueued.
    if (gvr_topk(nullptr, B, ld, nullptr, nullptr, 0, nullptr, nullptr) != GVR_ERR_UNSUPPORTED_K) return 5;

    float* dx = nullptr;
    int32_t *dlen = nullptr, *dprev = nullptr, *dout = nullptr;
    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    HIP_OK(hipMalloc(&dx, sizeof(float) * B * ld));
    HIP_OK(hipMalloc(&dlen, sizeof(int32_t) * B));
    HIP_OK(hipMalloc(&dprev, sizeof(int32_t) * B * K));
    HIP_OK(hipMalloc(&dout, sizeof(int32_t) * B * K));
    HIP_OK(hipMemcpy(dx, x.data(), sizeof(float) * B * ld, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dlen, len.data(), sizeof(int32_t) * B, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dprev, guess.data(), sizeof(int32_t) * B * K, hipMemcpyHostToDevice));

    int failures = 0;
    auto check = [&](const char* name, gvr_status st) -> int {
        if (st != GVR_OK) {
            std::fprintf(stderr, "%s: %s\n", name, gvr_status_string(st));
            return 1;
        }
        if (hipStreamSynchronize(stream) != hipSuccess) return 1;
        if (hipMemcpy(got.data(), dout, sizeof(int32_t) * B * K, hipMemcpyDeviceToHost) != hipSuccess) return 1;
        const bool same = std::memcmp(got.data(), exp.data(), sizeof(int32_t) * B * K) == 0;
        std::printf("%s: %s\n", name, same ? "equal to the oracle" : "DIFFERS from the oracle");
        return same ? 0 : 1;
    };
    failures += check("gvr_topk", gvr_topk(dx, B, ld, dlen, dprev, K, dout, stream));
    failures += check("gvr_topk (no guess)", gvr_topk(dx, B, ld, dlen, nullptr, K, dout, stream));
    failures += check("radix_topk", radix_topk(dx, B, ld, dlen, dprev, K, dout, stream));
    gvr_options opt = {};
    const int32_t flags[] = {64, 16, 8, 4};
    for (int32_t f : flags) {
        opt.flags = f;
        char name[64];
        std::snprintf(name, sizeof name, "gvr_topk_ex flags %d", (int)f);
        failures += check(name, gvr_topk_ex(dx, B, ld, dlen, dprev, K, dout, stream, &opt, nullptr));
    }
    // The caller-owned workspace: sized by gvr_workspace_size for a forced
    // two-part split, zero-filled once, used by two calls in a row.
    opt.flags = 0;
    opt.parts = 2;
    size_t ws_bytes = 0;
    if (gvr_workspace_size(B, ld, K, 1, &opt, &ws_bytes) != GVR_OK || ws_bytes == 0) return 6;
    void* ws = nullptr;
    HIP_OK(hipMalloc(&ws, ws_bytes));
    HIP_OK(hipMemset(ws, 0, ws_bytes));
    failures += check("gvr_topk_ex_ws 2 parts", gvr_topk_ex_ws(dx, B, ld, dlen, dprev, K, dout, stream, &opt, nullptr,
                                                                ws, ws_bytes));
    failures += check("gvr_topk_ex_ws 2 parts again", gvr_topk_ex_ws(dx, B, ld, dlen, dprev, K, dout, stream, &opt,
                                                                      nullptr, ws, ws_bytes));
    failures += check("radix_topk_ex_ws 2 parts", radix_topk_ex_ws(dx, B, ld, dlen, K, dout, stream, &opt, nullptr,
                                                                    ws, ws_bytes));
    // a forced split that does not fit is refused before anything is enqueued
    if (gvr_topk_ex_ws(dx, B, ld, dlen, dprev, K, dout, stream, &opt, nullptr, ws, ws_bytes / 2) != GVR_ERR_WORKSPACE)
        ++failures;
    HIP_OK(hipFree(ws));
    HIP_OK(hipFree(dx));
    HIP_OK(hipFree(dlen));
    HIP_OK(hipFree(dprev));
    HIP_OK(hipFree(dout));
    HIP_OK(hipStreamDestroy(stream));
    std::printf(failures ? "FAILED\n" : "ok\n");
    return failures ? 1 : 0;
}
