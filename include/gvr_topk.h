/*
 * gvr_topk.h -- exact per-row Top-K for decode-time sparse-attention indexer
 * scores on AMD Instinct MI355X (gfx950).
 *
 * Problem (Sec. 4.1, "Core Idea"): for each row b, given the fp32 scores
 * x[0..n) and a guessed index set P (the previous decode step's Top-K,
 * Sec. 3.3), return the indices of the K largest scores.
 *
 * gvr_topk  -- Guess-Verify-Refine (Sec. 4): statistics of the guessed scores
 *              (Phase 1), full-row threshold counting passes (Phase 2),
 *              collection of the candidates at or above the accepted threshold
 *              (Phase 3, Lemma 1 of Sec. 4.1 makes this set contain the answer),
 *              exact on-chip selection among them (Phase 4).
 * radix_topk -- distribution-agnostic radix select over the sortable key
 *              (the baseline of Sec. 2.2), same signature, same result.
 *
 * Result definition, shared by both entry points:
 *   - n = clamp(row_len[b], 0, ld); only scores[b*ld + 0 .. b*ld + n) are used
 *     (loads never leave the 128-byte-aligned lines holding those elements,
 *     so they never touch a page the row does not).
 *   - Order: each fp32 bit pattern u maps to the 32-bit key
 *       (u & 0x80000000) ? ~u : (u | 0x80000000)
 *     compared as unsigned, i.e. -NaN < -inf < ... < -0.0 < +0.0 < ... <
 *     +inf < +NaN (NaNs ordered by payload; -0.0 below +0.0).
 *   - Ties: among equal keys the lower index wins, so the answer is unique.
 *   - out_idx[b*K + 0 .. K) receives the K selected indices in ascending
 *     index order. If n <= K it receives 0, 1, ..., n-1 followed by -1.
 *   - The result never depends on prev_topk (exactness): prev_topk only
 *     changes how fast the answer is found.
 *
 * Memory and ownership:
 *   - All array arguments are DEVICE pointers on the current HIP device;
 *     the caller owns them; the library neither frees nor retains them.
 *   - scores: [B][ld] fp32, row stride ld elements, 4-byte aligned.
 *   - row_len: [B] int32 (device-resident, so values are clamped, not checked).
 *   - prev_topk: [B][K] int32 or NULL. Entries outside [0, n) (e.g. -1
 *     padding) are ignored; duplicates are tolerated. It guides calls with
 *     2K < ld <= 2^29 - 4096; for a longer stride the guess-free schedule
 *     runs (same result).
 *   - out_idx: [B][K] int32, written in full; must not overlap the inputs.
 *   - stream: a hipStream_t passed as void* (NULL = the null stream).
 *
 * Errors and synchronisation:
 *   - Argument problems detectable on the host are reported synchronously,
 *     before any work is enqueued. B == 0 is a no-op returning GVR_OK.
 *   - On GVR_OK the work is enqueued on `stream` as one kernel launch;
 *     out_idx is complete when the stream reaches that point. The call does
 *     not synchronise.
 *
 * Workspace:
 *   - gvr_topk and radix_topk may split a long row over several workgroups
 *     (few rows, long rows: see gvr_options.parts). The parts exchange their candidate lists
 *     through a device workspace that the library allocates on the first
 *     such call for each (device, stream) pair (hipMalloc; arrival counters
 *     + 128 KB per row part) and reuses for every later call on that stream.
 *     A call that needs more room allocates a larger one; the outgrown one is
 *     never freed. Every workspace stays allocated until the process ends,
 *     so a graph captured earlier can still be replayed after a later call
 *     has grown the stream's workspace.
 *   - Calls on one stream run in order and share its workspace; calls on
 *     different streams use different workspaces and may overlap.
 *   - A call that has to allocate returns GVR_ERR_HIP while its stream is
 *     being captured into a HIP graph: issue one eager call of the same (or
 *     a larger) shape on that stream before capturing.
 *   - A captured graph keeps the capture stream's workspace. Replayed on
 *     another stream, it must not overlap split calls on the capture stream
 *     (eager calls or replays of other graphs captured there): overlapping
 *     calls that share a workspace corrupt each other's merge.
 *   - Calls that do not split their rows use no workspace.
 *   - gvr_topk_ex_ws / radix_topk_ex_ws take the workspace from the caller
 *     instead (sized by gvr_workspace_size) and allocate nothing.
 */
#ifndef GVR_TOPK_H
#define GVR_TOPK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GVR_OK = 0,
    GVR_ERR_INVALID_ARG = -1,    /* B < 0, ld < 0, NULL required pointer, bad option */
    GVR_ERR_UNSUPPORTED_K = -2,  /* K < 1 or K > GVR_MAX_K */
    GVR_ERR_WORKSPACE = -3,      /* gvr_topk_ex_noalloc, *_ex_ws: a forced split
                                    needs more (row, part) slots than the
                                    call's workspace holds */
    GVR_ERR_HIP = -4,            /* the kernel launch failed */
    GVR_ERR_TOO_LONG = -5        /* ld > 2^31 - 16 */
} gvr_status;

/* Largest supported K (Sec. 5.5: K = M = 2048 in the deployed gate). */
#define GVR_MAX_K 2048
/* Default and largest refine capacity C of Lemma 1 (Sec. 4.1): the number of
 * (key, index) candidates one gfx950 workgroup keeps in LDS (128 KB). The
 * paper's C = 6144 is sized for its B200 shared memory (Sec. 5.3). */
#define GVR_MAX_CANDIDATES 16384

/* Per-row outcome codes reported in gvr_row_stats.path. */
enum {
    GVR_PATH_TRIVIAL = 0,      /* n <= K: iota / -1 padding */
    GVR_PATH_ALL = 1,          /* K < n <= C and no guess, or K < n <= 2K:
                                  every element is a candidate */
    GVR_PATH_GUESS = 2,        /* the guessed threshold held the answer: one pass */
    GVR_PATH_NARROWED = 3,     /* guess fell short; count passes narrowed the threshold */
    GVR_PATH_TIES = 4,         /* the K-th key isolated exactly (ties straddle
                                  [K, C]); selection emitted without refine */
    GVR_PATH_NO_GUESS = 5,     /* prev_topk NULL / without a valid entry, or radix */
    GVR_PATH_SECANT = 6        /* flag bit 2: the secant threshold search accepted a
                                  threshold and one collect pass gathered the list */
};

/* Optional knobs (NULL = defaults). Zero fields mean "default". */
typedef struct gvr_options {
    int32_t capacity;      /* refine capacity C, K <= C <= GVR_MAX_CANDIDATES
                              (default GVR_MAX_CANDIDATES; at most 4096 in
                              the 4-wave and 6144 in the 8-wave shape); a
                              smaller C forces more narrowing passes, never
                              another result */
    int32_t flags;         /* bit 0: ignore prev_topk (run the radix schedule);
                              bit 1: place the parts of a row on different XCDs
                              (a test of the path that does not rely on their
                              shared L2; slower);
                              bit 2: the paper's own threshold search -- every
                              guessed score, T0 = pmean, secant counting passes,
                              a collect pass (one workgroup per row) -- instead
                              of the speculative first pass;
                              bit 3: the paper's own exact selection (Sec. 4.2.4:
                              min / max, 2048-bin histogram with a wave-parallel
                              bin search, snap iterations, partition) instead of
                              the histogram + rank-count refine;
                              bits 4-6 force a workgroup shape (no row
                              splitting except with 16 waves): bit 4: 4 waves,
                              C <= 4096, three workgroups per compute unit;
                              bit 5: 16 waves, one per compute unit; bit 6: 8
                              waves, C <= 6144, two per compute unit. None
                              set: 16 waves when B <= the compute units;
                              above that, with a usable guess (prev_topk and
                              ld > 2K), 8 waves unless ld > 40960 and
                              B <= 2 x the compute units (then 16); without
                              one, 4 waves for ld <= 4096, else 8. Two of
                              bits 4-6 together are an error.
                              bit 7: the parts of a split row hand over
                              through an agent-scope release / acquire on
                              the arrival counter (the memory model's form:
                              an L2 writeback and invalidate per part, 2 to
                              16 % slower on split calls) instead of
                              completed stores read through the XCD's shared
                              L2 (the default: the parts of a row run on one
                              XCD, and the last part of a row whose parts
                              did not reads the row itself).
                              No bit changes the result. */
    int32_t parts;         /* workgroups per row, 1..16 (0 = chosen from B, ld
                              and the device's compute units; a forced value is
                              lowered so that B * parts <= 2048, or refused by
                              the calls whose workspace is too small for it);
                              never changes the result */
    int32_t reserved1;     /* must be 0 */
} gvr_options;

/* Optional per-row diagnostics, written when a device pointer is supplied. */
typedef struct gvr_row_stats {
    int32_t n;             /* clamped row length */
    int32_t path;          /* GVR_PATH_* */
    int32_t passes;        /* full-row passes (1: the guess held the answer) */
    int32_t candidates;    /* candidates handed to the refine = f(threshold) */
    uint32_t threshold;    /* accepted threshold key T (K <= f(T) <= C) */
    uint32_t kth_key;      /* key of the K-th largest score */
    int32_t n_gt;          /* #{key > kth_key} */
    int32_t guess_valid;   /* valid entries of prev_topk used by the guess */
    uint32_t spec_threshold; /* T_spec derived from the guess (0xFFFFFFFF if none) */
    int32_t spec_count;    /* f(T_spec) counted in the first pass (-1 if a
                              candidate list overflowed) */
    float pmean;           /* mean of the guessed scores (T0 of Sec. 4.2.1) */
    int32_t refine_iters;  /* snap iterations of the paper's selection (flag
                              bit 3), else 0 */
    int64_t t_start;       /* stamps of the row's workgroup on the GPU's     */
    int64_t t_guess;       /*   constant-rate clock (s_memrealtime, 100 MHz  */
                           /*   on MI355X): start; guess ready;              */
    int64_t t_search;      /*   threshold accepted (last pass done);           */
    int64_t t_collect;     /*   refine starts;                                 */
    int64_t t_refine;      /*   output written.                                */
} gvr_row_stats;

/* Guess-Verify-Refine Top-K (Sec. 4). See the file comment for semantics. */
gvr_status gvr_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                    const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream);

/* Distribution-agnostic radix-select Top-K (Sec. 2.2); prev_topk is accepted
 * and ignored. Same result as gvr_topk. */
gvr_status radix_topk(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                      const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream);

/* As gvr_topk, with options (NULL = defaults) and per-row stats ([B] device
 * array of gvr_row_stats, or NULL). */
gvr_status gvr_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                       const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                       const gvr_options* options, gvr_row_stats* stats);

/* Largest number of (row, part) slots of one gvr_topk_ex_noalloc call. */
#define GVR_NOALLOC_SLOTS 256

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call and result as gvr_topk_ex, with the split-row workspace taken from a
 * static device array of the library instead of a library allocation. It
 * calls no hipMalloc, hipFree or other allocating routine, so it may be
 * captured into a HIP graph as any call's first, on any stream.
 *   - The array holds GVR_NOALLOC_SLOTS (row, part) slots: 34 MiB per device
 *     the library runs on, held until the process ends. An automatic split
 *     (options->parts == 0) is lowered to fit; a forced split with
 *     B * parts > GVR_NOALLOC_SLOTS returns GVR_ERR_WORKSPACE before
 *     anything is enqueued. Unsplit calls do not touch the array.
 *   - Every call on one device shares that device's array: calls that
 *     overlap on one device (other streams, graph replays, other threads)
 *     race and corrupt each other's merge; serialise them. The array's
 *     arrival words start at zero and every call leaves them at zero.
 *   - All other arguments, errors and semantics as gvr_topk_ex. */
gvr_status gvr_topk_ex_noalloc(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                               const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                               const gvr_options* options, gvr_row_stats* stats);

/* Radix-select counterpart of gvr_topk_ex. */
gvr_status radix_topk_ex(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                         int32_t K, int32_t* out_idx, void* stream, const gvr_options* options,
                         gvr_row_stats* stats);

/* Caller-owned workspace: the graph-capture-safe form of the split
 * schedule (the parts of a split row exchange their counts, thresholds,
 * first refine histograms and candidate lists through it; Sec. 4).
 *
 * gvr_workspace_size writes to *bytes the workspace that a gvr_topk_ex_ws
 * call (use_guess != 0, prev_topk non-NULL) or a radix_topk_ex_ws call
 * (use_guess == 0) of this B, ld, K and options needs on the CURRENT device
 * to split its rows as gvr_topk_ex / radix_topk_ex would (0 when it does not
 * split them). It enqueues nothing. Errors: those of the call's own size and
 * option checks (GVR_ERR_INVALID_ARG also for bytes == NULL);
 * GVR_ERR_WORKSPACE for a forced split of more than 2^24 (row, part) slots;
 * GVR_ERR_HIP if the current device cannot be read. */
gvr_status gvr_workspace_size(int64_t B, int64_t ld, int32_t K, int use_guess, const gvr_options* options,
                              size_t* bytes);

/* gvr_topk_ex / radix_topk_ex with the split-row workspace supplied by the
 * caller: `workspace` is a device buffer of ws_bytes bytes on the current
 * device (8-byte aligned, 256 recommended; NULL only with ws_bytes == 0).
 * The call allocates nothing, clears nothing and does not synchronise, so it
 * may be captured into a HIP graph as any call's first, on any stream.
 *   - Ownership: the caller's. The library keeps no reference once the call
 *     returns; the enqueued kernel uses the buffer until it completes.
 *   - Contents: zero-filled by the caller before its first use (hipMemset,
 *     or a fill kernel inside a graph). Every call leaves it ready for the
 *     next, so reuse needs no clearing as long as every call on the buffer
 *     passes the same ws_bytes (the layout inside depends on it): clear it
 *     again after changing ws_bytes.
 *   - Size: with ws_bytes >= gvr_workspace_size's answer the call splits as
 *     gvr_topk_ex / radix_topk_ex would. With less, an automatic split
 *     (options->parts == 0) is lowered to what fits (down to one workgroup
 *     per row, which uses no workspace), and a forced split that does not
 *     fit returns GVR_ERR_WORKSPACE before anything is enqueued.
 *   - Concurrency: calls that share one buffer must not overlap (one stream
 *     orders them); calls on different buffers may.
 *   - Errors: as gvr_topk_ex / radix_topk_ex, plus GVR_ERR_INVALID_ARG for a
 *     NULL or misaligned workspace with ws_bytes > 0. The result is theirs
 *     whatever the workspace size. */
gvr_status gvr_topk_ex_ws(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                          const int32_t* prev_topk, int32_t K, int32_t* out_idx, void* stream,
                          const gvr_options* options, gvr_row_stats* stats, void* workspace, size_t ws_bytes);
gvr_status radix_topk_ex_ws(const float* scores, int64_t B, int64_t ld, const int32_t* row_len, int32_t K,
                            int32_t* out_idx, void* stream, const gvr_options* options, gvr_row_stats* stats,
                            void* workspace, size_t ws_bytes);

/* Measurement helper, not a step of the Top-K: reads every element of
 * scores[b][0, n_b) once (n_b = clamp(row_len[b], 0, ld), row_len NULL = ld)
 * with the same 16-byte non-temporal loads the Top-K streams with, computing
 * nothing but an xor of the bits: the plain read rate of the rows, the
 * ceiling of the Top-K's streaming pass. out_words [B][16] uint32 (device):
 * row b's part p writes word p and the unused words are zeroed, so the xor of
 * a row's 16 words is the xor of its elements' bit patterns. One launch on
 * `stream`; no allocation. Errors: GVR_ERR_INVALID_ARG (negative sizes, NULL
 * pointers with B > 0), GVR_ERR_TOO_LONG (ld > 2^31 - 16 or B > 2^26),
 * GVR_ERR_HIP. */
gvr_status gvr_read_floor(const float* scores, int64_t B, int64_t ld, const int32_t* row_len,
                          uint32_t* out_words, void* stream);

/* Human-readable name of a status code (static string). */
const char* gvr_status_string(gvr_status status);

/* Library version string (static). */
const char* gvr_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GVR_TOPK_H */
