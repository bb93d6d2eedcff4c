/*
 * hils.h -- C ABI of the MI355X (gfx950) HiLS attention library, libhils.so.
 *
 * HiLS (Hierarchical Landmark Sparse) attention, arXiv 2607.02980:
 *   - Sec. 2.1: keys are cut into chunks of S tokens, c(j) = floor(j / S).  A
 *     query at position i attends a local window [l(i), i] whose left edge is
 *     chunk aligned, l(i) = floor((i - W + 1) / S) * S (clamped at 0), and may
 *     retrieve any chunk of C_i = {0, ..., l(i)/S - 1}.
 *   - Eq. (9): every candidate chunk is scored with its landmark (compressed)
 *     key, s^_ic = scale * <q^_i, k'_c> + b'_c, and the K best chunks I_i are
 *     kept.  Eq. (11): q^ is an optional routing query (Q-Cal); without it q^ = q.
 *   - Sec. 4.1 "HiLS-Attention in GQA" and Appendix C: the G = Hq / Hkv query
 *     heads of a KV group share one selection, ranked by the maximum of their
 *     per-head scores; ties go to the smaller chunk index.
 *   - Eq. (10): softmax attention runs separately inside each retrieved chunk
 *     (intra-chunk softmax) and over the local window; the per-part outputs are
 *     fused with a softmax over {s^_ic : c in I_i} U {log Z_swa} (Eq. (1)), the
 *     local window taking its exact mass Z_swa.
 *   - the backward differentiates Eq. (10) with the selection held fixed, so
 *     gradients reach the landmark keys and biases of the selected chunks only
 *     (Sec. 9 notes that unselected chunks receive no gradient).
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer (hipMalloc'd or equivalent)
 *     unless stated otherwise; `p` (the parameter block) is a HOST pointer.
 *   - The caller owns every buffer.  The library never allocates device
 *     memory, never synchronises the device and keeps no state between calls
 *     other than the thread-local error string (and, only while the optional
 *     timing mode is enabled, its event records) -- except that
 *     hils_decode_fwd_noalloc uses a fixed device array of the library's own
 *     (declared below) and keeps its address per device, and that the prefill
 *     record cap (hils_prefill_record_cap) is one process-wide setting.  All work is enqueued on
 *     `stream` (a hipStream_t; NULL is the default stream) and is complete
 *     when the stream is.
 *   - Layouts are row-major and contiguous ("BHSD"):
 *       q, q_route, out, dout, dq, dq_route : [B, Hq,  N, d]
 *       k, v, dk, dv                        : [B, Hkv, L, d]   (decode: the caches)
 *       lmk, dlmk                           : [B, Hl,  L/S, d] (landmark key of each chunk)
 *       lmk_bias, dlmk_bias                 : [B, Hl,  L/S] float32
 *       lse                                 : [B, Hq,  N] float32
 *       idx                                 : [B, Hkv, N, K] int32
 *     A chunk's K (or V) block is one contiguous S*d span.
 *   - `dtype` fixes the element type of q, k, v, lmk, q_route, out, dout and
 *     of every gradient except dlmk_bias (float32 storage or bf16 storage).
 *     Arithmetic is float32 throughout; outputs are rounded to nearest-even.
 *   - Landmark heads: Hl == Hq (one landmark key per query head, Appendix C)
 *     or Hl == Hkv (one per KV group).  The bias has the landmark heads.
 *   - `idx` rows list the selected chunks in ascending order, padded with -1
 *     when |C_i| < K.
 *   - Return value: HILS_OK (0) or an error code; on error nothing has been
 *     enqueued and hils_last_error() describes the failure.  Argument checks
 *     run entirely on the host before any HIP call, so they work without a GPU.
 *     Values that live in device memory (seqlens, a caller-provided idx) are
 *     not inspected by the host; the kernels clamp them into range (see each
 *     entry point), so they can never cause an out-of-bounds access.
 */
#ifndef HILS_H
#define HILS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { HILS_F32 = 0, HILS_BF16 = 1 } hils_dtype;

typedef enum {
    HILS_OK = 0,
    HILS_ERR_INVALID = 1,     /* a NULL required pointer or an inconsistent shape/value */
    HILS_ERR_UNSUPPORTED = 2, /* valid, but no kernel for this (d, S, G, K, dtype) yet */
    HILS_ERR_WORKSPACE = 3,   /* workspace missing or smaller than hils_workspace_size() */
    HILS_ERR_HIP = 4          /* a HIP launch or runtime call failed */
} hils_status;

/* Forward flag: consume the caller's `idx` instead of selecting (forced-index
 * mode: re-use of a selection, and kernel tests).  Entries < 0 or not in C_i
 * are ignored; entries must be ascending. */
#define HILS_FLAG_GIVEN_IDX 1u

/* Landmark compression flag (hils_landmark_fwd/bwd only): the landmark-token-free
 * variant of Sec. 4.1, one learnable landmark query per landmark head shared by
 * every chunk of every sequence: lq and dlq are [Hl, d] instead of [B, Hl, L/S, d]. */
#define HILS_FLAG_SHARED_LMK_QUERY 2u

/* Forward flag (prefill, decode): rank the chunks by per-head normalised scores,
 * the wording of Sec. 4.1 (each query head's chunk weights are normalised before
 * the maximum over the group's heads): the group score of chunk c becomes
 * max_h (s^_hc - log sum_{c' in C_i} exp(s^_hc')) instead of max_h s^_hc.  Only
 * the selection changes; the fusion weights use the raw s^_hc.  Prefill scores the
 * candidates twice; decode reads the landmarks once (keeping each head's top-K of
 * every slice, ranked once the log-sum-exps are known) and its workspace grows by
 * the kept candidates.  Ignored by hils_bwd (the selection is given). */
#define HILS_FLAG_HEAD_NORM_SELECT 4u

/* Prefill flag (bf16): compute the retrieved-chunk terms by union packing, the
 * one-load-multiple-compute scheme of Sec. 4.2 — each tile of adjacent queries
 * loads the union of their selected chunks once and computes every chunk for
 * all of its rows (rows that did not select a chunk get weight 0).  Same
 * results as the default chunk-major pass; faster when adjacent queries select
 * overlapping chunks (as trained models do), slower when they do not.  Needs no
 * workspace (hils_workspace_size reports 0 under this flag).  Ignored by the
 * fp32 path, decode and the backward. */
#define HILS_FLAG_UNION_PACKING 8u

typedef enum { HILS_OP_PREFILL = 0, HILS_OP_DECODE = 1, HILS_OP_BWD = 2, HILS_OP_LANDMARK = 3 } hils_op;

typedef struct {
    int B;          /* sequences */
    int Hq, Hkv;    /* query heads, KV heads; G = Hq / Hkv query heads share a KV head */
    int Hl;         /* landmark heads: Hq or Hkv */
    int N;          /* queries per sequence (prefill, bwd: query n sits at position n; decode: the
                       new tokens, query n at seqlens[b] - N + n) */
    int L;          /* key positions per sequence (decode: cache capacity); multiple of `chunk` */
    int d;          /* head dimension */
    int chunk;      /* S, tokens per chunk */
    int topk;       /* K, chunks retrieved per query and KV group */
    int window;     /* W >= 1, local window size before chunk alignment */
    float scale;    /* multiplies both the token logits and the landmark scores (1/sqrt(d) in the paper) */
    hils_dtype dtype;
    unsigned flags; /* HILS_FLAG_* */
} hils_params;

/* Library version as 10000*major + 100*minor + patch. */
int hils_version(void);

/* Thread-local description of the last error returned on this thread ("" if none). */
const char* hils_last_error(void);

/* Bytes of device workspace that entry point `op` needs for parameters `p`
 * (0 is a valid answer: then workspace may be NULL).  Writes *bytes and
 * returns HILS_OK, or returns an error code for invalid parameters. */
int hils_workspace_size(const hils_params* p, int op, size_t* bytes);

/*
 * Prefill forward: all N queries of each sequence at once (query n at
 * position n; requires N <= L).  Computes, per (b, KV group, n): the landmark
 * scores of C_n, the group maximum over the G heads, the top-K selection
 * (Eq. (9), App. C), the local-window term (Eq. (1)), the per-chunk softmax
 * terms and their fusion (Eq. (10)).
 *   q        [B,Hq,N,d]     queries (token logits)
 *   k, v     [B,Hkv,L,d]    keys and values
 *   lmk      [B,Hl,L/S,d]   landmark keys k'_c
 *   lmk_bias [B,Hl,L/S] f32 landmark biases b'_c, or NULL for b' = 0
 *   q_route  [B,Hq,N,d]     routing queries q^ (Q-Cal, Eq. (11)), or NULL for q^ = q
 *   out      [B,Hq,N,d]     output (written)
 *   lse      [B,Hq,N] f32   log of the fusion normaliser, LSE of {s^_ic} U {log Z_swa} (written)
 *   idx      [B,Hkv,N,K]    selection (written; read instead under HILS_FLAG_GIVEN_IDX)
 *   workspace, ws_bytes     device scratch of at least hils_workspace_size(p, HILS_OP_PREFILL)
 *   stream                  hipStream_t
 * Deterministic: repeated calls with equal inputs give identical bits.
 */
int hils_prefill_fwd(const hils_params* p, const void* q, const void* k, const void* v, const void* lmk,
                     const float* lmk_bias, const void* q_route, void* out, float* lse, int32_t* idx,
                     void* workspace, size_t ws_bytes, void* stream);

/*
 * Decode forward: N >= 1 new queries per sequence against a KV cache (N = 1:
 * one generated token; N > 1: drafted tokens verified together, as in
 * speculative decoding, each attending causally up to its own position).
 * The caller has already written the new tokens' k/v at the last N positions,
 * so with len = seqlens[b] query n sits at i = len - N + n and attends keys
 * j <= i; every query is computed as a decode row of its own (Eqs. (1), (9),
 * (10) at position i).  Landmark rows exist for every complete chunk.
 *   seqlens  [B] int32 (device) valid tokens per sequence including the new ones,
 *            or NULL for L; values are clamped into [N, L] by the kernels.
 * Other arguments as for hils_prefill_fwd (q, q_route, out [B,Hq,N,d];
 * lse [B,Hq,N]; idx [B,Hkv,N,K]; k, v, lmk, lmk_bias are the caches).
 * Requires N <= L and B * N <= 65535.  Windows above 4032 tokens return
 * HILS_ERR_UNSUPPORTED.  The workspace (hils_workspace_size(p, HILS_OP_DECODE))
 * grows with B * N.
 */
int hils_decode_fwd(const hils_params* p, const void* q, const void* k_cache, const void* v_cache,
                    const void* lmk_cache, const float* lmk_bias, const void* q_route, const int32_t* seqlens,
                    void* out, float* lse, int32_t* idx, void* workspace, size_t ws_bytes, void* stream);

/*
 * Decode forward that allocates nothing, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): hils_decode_fwd with the same arguments minus the
 * workspace, whose role is taken by a fixed array of
 * HILS_DECODE_NOALLOC_SCRATCH_BYTES bytes that the library holds on every GPU
 * it runs on (from the first call on that GPU until the process ends; the
 * first call on a GPU looks up the array's device address, with that GPU
 * current).  Same results as hils_decode_fwd (the same kernels).
 *   Calls whose hils_workspace_size(p, HILS_OP_DECODE) exceeds
 *   HILS_DECODE_NOALLOC_SCRATCH_BYTES return HILS_ERR_WORKSPACE before any
 *   HIP call.  The array keeps the last call's contents; every byte a call
 *   reads it has written first, so nothing needs clearing.  Calls that overlap
 *   on one GPU (other streams or threads) share the array and race: serialise
 *   them.  Nothing is allocated while the optional timing mode is off (its
 *   default; when on, it creates HIP events).
 */
#define HILS_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int hils_decode_fwd_noalloc(const hils_params* p, const void* q, const void* k_cache, const void* v_cache,
                            const void* lmk_cache, const float* lmk_bias, const void* q_route,
                            const int32_t* seqlens, void* out, float* lse, int32_t* idx, void* stream);

/*
 * Decode forward over a paged cache: a page holds one chunk (S tokens) of one
 * sequence, for every KV head and landmark head, and chunk c of sequence b is
 * page block_table[b, c]; pages may be shared between sequences (a common
 * prefix) and need not be in any order.  Same computation and arguments as
 * hils_decode_fwd, with the caches replaced by pools of num_pages pages:
 *   k_pages, v_pages [num_pages, Hkv, S, d]  (dtype)
 *   lmk_pages        [num_pages, Hl, d]      (dtype) landmark k'_c of the page's chunk
 *   bias_pages       [num_pages, Hl] f32     landmark bias b'_c, or NULL
 *   block_table      [B, L/S] int32 (device) page of each chunk; L = the logical
 *                    capacity per sequence.  Entries of chunks at or past a
 *                    sequence's length are not read; an entry outside
 *                    [0, num_pages) is clamped into it (no out-of-bounds access,
 *                    meaningless result).
 * The workspace is hils_workspace_size(p, HILS_OP_DECODE).
 */
int hils_decode_paged_fwd(const hils_params* p, const void* q, const void* k_pages, const void* v_pages,
                          const void* lmk_pages, const float* bias_pages, const void* q_route,
                          const int32_t* block_table, int num_pages, const int32_t* seqlens, void* out, float* lse,
                          int32_t* idx, void* workspace, size_t ws_bytes, void* stream);

/*
 * Backward of the prefill forward with the selection fixed to `idx`.
 *   dout     [B,Hq,N,d]      upstream gradient dL/d(out)
 *   q, k, v, lmk, lmk_bias, q_route: the forward's inputs
 *   out, lse, idx            the forward's outputs (lse and out must come from
 *                            the same forward that produced idx)
 *   dq       [B,Hq,N,d]      written; includes the routing gradient when q_route is NULL
 *   dk, dv   [B,Hkv,L,d]     written (keys no query attends get 0)
 *   dlmk     [B,Hl,L/S,d]    written (chunks no query selected get 0)
 *   dlmk_bias[B,Hl,L/S] f32  written, or NULL to skip
 *   dq_route [B,Hq,N,d]      written when q_route is given (must then be non-NULL)
 * Deterministic: repeated calls with equal inputs produce identical bits (the
 * per-chunk lists of selecting rows are sorted before use, so every gradient sum
 * runs in one fixed order).
 */
int hils_bwd(const hils_params* p, const void* dout, const void* q, const void* k, const void* v,
             const void* lmk, const float* lmk_bias, const void* q_route, const void* out, const float* lse,
             const int32_t* idx, void* dq, void* dk, void* dv, void* dlmk, float* dlmk_bias, void* dq_route,
             void* workspace, size_t ws_bytes, void* stream);

/*
 * Landmark compression, Prop. 3.1: the landmark key k'_c and bias b'_c of every
 * chunk from its landmark query q'_c (in the paper, the query of a landmark
 * token appended to the chunk) and the chunk's own keys:
 *   s_j = scale * <q'_c, k_j> for the S keys j of chunk c (of the landmark
 *   head's KV group), p = softmax(s), k'_c = sum_j p_j k_j (the attention of
 *   q'_c over its chunk), b'_c = -sum_j p_j log p_j (the entropy of p), so that
 *   scale * <q, k'_c> + b'_c is the first-order Taylor expansion of the chunk's
 *   log-sum-exp at q = q'_c.  The outputs are the lmk and lmk_bias inputs of the
 *   attention entry points.
 *   lq       [B, Hl, L/S, d]   landmark queries (dtype)
 *   k        [B, Hkv, L, d]    keys (dtype); landmark head hl uses KV group
 *                              hl / (Hl / Hkv)
 *   lmk      [B, Hl, L/S, d]   written (dtype)
 *   lmk_bias [B, Hl, L/S] f32  written
 * Uses B, Hq, Hkv, Hl, L, d, chunk, scale, dtype and flags of `p`; N, topk and
 * window are not used (they must still be >= 1).  Under HILS_FLAG_SHARED_LMK_QUERY
 * lq is [Hl, d]: q'_c is that head's one query for every chunk.  No workspace.
 */
int hils_landmark_fwd(const hils_params* p, const void* lq, const void* k, void* lmk, float* lmk_bias, void* stream);

/*
 * Backward of hils_landmark_fwd for upstream gradients dlmk (of k'_c) and
 * dlmk_bias (of b'_c, float32, NULL = 0), e.g. the dlmk / dlmk_bias of hils_bwd:
 *   dlq [B, Hl, L/S, d]  written: the gradient of the landmark queries
 *   dk  [B, Hkv, L, d]   written: the compression's gradient of the keys, summed
 *                        over the landmark heads of each KV group (every key
 *                        lies in a chunk, so every row is written); add it to
 *                        the attention's dk for the keys' total gradient.
 * Same parameter use as hils_landmark_fwd.  Under HILS_FLAG_SHARED_LMK_QUERY, lq
 * and dlq are [Hl, d] and dlq is the sum of the per-chunk gradients over every
 * chunk and sequence; that sum needs a workspace of
 * hils_workspace_size(p, HILS_OP_LANDMARK) bytes (B * Hl * L/S * d floats, caller
 * owned, contents on entry ignored).  Without the flag the size is 0 and
 * workspace may be NULL.  Deterministic (fixed summation order, no atomics).
 */
int hils_landmark_bwd(const hils_params* p, const void* lq, const void* k, const void* dlmk,
                      const float* dlmk_bias, void* dlq, void* dk, void* workspace, size_t ws_bytes,
                      void* stream);

/*
 * Prefill (bf16, chunk-major): the most bytes of per-slot records (the chunk
 * outputs o_c and scores s^ of Eq. (10), B * Hq * K * (2 d + 4) bytes per query
 * row) that one pass over the rows may hold.  A longer prefill runs its inverse
 * index, chunk pass and local pass over consecutive segments of rows (multiples of
 * 2048) whose records fit, reusing one workspace, so that the workspace stays
 * bounded whatever N (at 32 query heads, K = 16 and d = 128 the records take 133
 * KB per row: 69 GB for a 512K-token prefill).  Results are bitwise the same for
 * any cap.  The default, 16 GiB, keeps one segment up to 126K rows of that shape.
 * Process-wide; hils_workspace_size reflects the value at the time of the call, so
 * set it before sizing workspaces.  Returns the previous cap; bytes = 0 only
 * reads it.
 */
size_t hils_prefill_record_cap(size_t bytes);

/*
 * Optional per-kernel timing, for profiling (not needed to use the operator).
 * hils_timing_enable(1) makes every kernel that the library launches from the
 * calling thread be bracketed by two HIP events on the launch's stream (state
 * the library keeps per thread while enabled);
 * hils_timing_enable(0) discards the records.
 * hils_timing_read() waits for the recorded events, then reports per kernel
 * name (in first-launch order): names as a '\n'-separated list in `names`
 * (HOST buffer of names_len bytes, NUL-terminated, may be NULL), the summed
 * milliseconds in total_ms[k] and the launch count in launches[k] (HOST arrays
 * of max_kernels entries, may be NULL); *n_kernels receives the number of
 * distinct kernels.  The records are then cleared.
 */
int hils_timing_enable(int on);
int hils_timing_read(char* names, size_t names_len, float* total_ms, int* launches, int max_kernels,
                     int* n_kernels);

#ifdef __cplusplus
}
#endif

#endif /* HILS_H */
