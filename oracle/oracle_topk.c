/*
 * oracle_topk.c -- CPU oracle for exact per-row Top-K (TEST INFRASTRUCTURE ONLY).
 *
 * Only tests/, the smoke check and the CPU-baseline leg of the benchmark may
 * load this file's library. The GPU product path never calls it, and this file
 * shares no code, header, table or helper with the GPU path.
 *
 * What it computes is the plain definition of the problem, not the
 * Guess-Verify-Refine method: the method provably reaches the same set
 * (Sec. 4.1, Lemma 1: once a threshold T with K <= f(T) <= C is found, the
 * exact Top-K is contained in {i : x_i >= T}; the refine step then selects it
 * exactly), so the oracle is simply "sort everything, take the first K".
 *
 *   Problem statement (Sec. 4.1, "Core Idea"): given x in R^N, return the
 *   index set S* with |S*| = K holding the K largest values.
 *   Threshold count (Sec. 4.1, definition of f(T)): f(T) = |{i : x_i >= T}|.
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - Order: every float is mapped to a 32-bit "sortable key" (the paper's
 *     radix baseline ranks the sortable FP32 key, Sec. 2.2). The map is
 *     monotone on the reals and total on all bit patterns:
 *       -NaN < -inf < ... < -0.0 < +0.0 < ... < +inf < +NaN.
 *     -0.0 and +0.0 are different keys.
 *   - Ties: the paper leaves ties non-deterministic (Sec. 6.2); here the lower
 *     index wins, so the answer is a unique set.
 *   - Row length: n = clamp(row_len[b], 0, ld); only x[0..n) exists.
 *   - n <= K: the answer is 0..n-1 followed by -1 padding.
 *   - Output order: the K indices in ascending order.
 *
 * Built with plain gcc (-O2, no -ffast-math); slow and obvious on purpose.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Sortable key of one fp32 bit pattern: flip all bits of negative numbers,
 * set the sign bit of non-negative ones. Unsigned order of keys is the total
 * order above. */
uint32_t oracle_key(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    if (u & 0x80000000u)
        return ~u;
    return u | 0x80000000u;
}

void oracle_keys(const float* x, int64_t n, uint32_t* out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_key(x[i]);
}

/* f(T) of Sec. 4.1 written out, with "x_i >= T" read as key(x_i) >= key(T). */
int64_t oracle_count_ge(const float* row, int64_t n, uint32_t tkey)
{
    int64_t c = 0;
    for (int64_t i = 0; i < n; ++i)
        if (oracle_key(row[i]) >= tkey)
            ++c;
    return c;
}

typedef struct {
    uint32_t key;
    int32_t idx;
} pair_t;

/* "a comes before b": larger key first, then lower index first. */
static int cmp_pair(const void* pa, const void* pb)
{
    const pair_t* a = (const pair_t*)pa;
    const pair_t* b = (const pair_t*)pb;
    if (a->key != b->key)
        return a->key > b->key ? -1 : 1;
    if (a->idx != b->idx)
        return a->idx < b->idx ? -1 : 1;
    return 0;
}

static int cmp_int(const void* pa, const void* pb)
{
    int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
    return (a > b) - (a < b);
}

/*
 * One row. out[0..K) receives the answer; kth_key / n_gt (nullable) receive the
 * K-th largest key T* and #{key > T*} when n > K (both 0 otherwise).
 * Returns 0, or -1 if a scratch allocation fails.
 */
int oracle_topk_row(const float* row, int64_t n, int32_t K, int32_t* out,
                    uint32_t* kth_key, int32_t* n_gt)
{
    if (kth_key) *kth_key = 0;
    if (n_gt) *n_gt = 0;
    if (n <= K) {
        for (int32_t i = 0; i < K; ++i)
            out[i] = (i < n) ? i : -1;
        return 0;
    }
    pair_t* p = (pair_t*)malloc((size_t)n * sizeof(pair_t));
    if (!p)
        return -1;
    for (int64_t i = 0; i < n; ++i) {
        p[i].key = oracle_key(row[i]);
        p[i].idx = (int32_t)i;
    }
    qsort(p, (size_t)n, sizeof(pair_t), cmp_pair);
    for (int32_t i = 0; i < K; ++i)
        out[i] = p[i].idx;
    qsort(out, (size_t)K, sizeof(int32_t), cmp_int);
    if (kth_key || n_gt) {
        uint32_t t = p[K - 1].key;
        int32_t gt = 0;
        for (int32_t i = 0; i < K; ++i)
            if (p[i].key > t)
                ++gt;
        if (kth_key) *kth_key = t;
        if (n_gt) *n_gt = gt;
    }
    free(p);
    return 0;
}

/*
 * B rows of stride ld. row_len may be NULL (then every row has n = ld).
 * out_idx is [B][K]; kth_key / n_gt are [B] or NULL.
 */
int oracle_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                int32_t K, int32_t* out_idx, uint32_t* kth_key, int32_t* n_gt)
{
    if (B < 0 || ld < 0 || K < 1)
        return -2;
    for (int64_t b = 0; b < B; ++b) {
        int64_t n = row_len ? (int64_t)row_len[b] : ld;
        if (n < 0) n = 0;
        if (n > ld) n = ld;
        int rc = oracle_topk_row(scores + b * ld, n, K, out_idx + b * (int64_t)K,
                                 kth_key ? kth_key + b : NULL, n_gt ? n_gt + b : NULL);
        if (rc)
            return rc;
    }
    return 0;
}
