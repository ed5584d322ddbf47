/*
 * splice_attn.h -- C ABI of the MI355X (gfx950) spliced decode-attention library.
 *
 * The method (paper Section 3, "Splice intervention"; Algorithm 1 in the
 * appendix "Splice Intervention Pseudocode"; donor forms in Table 1):
 * a sweep cell (L, W) decodes greedily over a prefilled prompt cache of
 * T_p slots per layer.  For every layer l >= L, from decode step W on, the
 * prompt-span slots are read from a donor cache of the same length (or are
 * all-zero for the ZERO donor) instead of the clean cache; generated entries
 * keep their values.  Readings fixed by this ABI:
 *   - step s is 0-based (s = 0 is the first decode pass after prefill) and
 *     cell c is spliced at (layer, s) iff layer >= L_c and s >= W_c;
 *   - only slots [span_lo, span_hi) are replaced ([0, T_p) is the
 *     paper-literal whole-prompt splice);
 *   - ZERO slots are keys with K = V = 0: they score exactly 0 and are not
 *     masked, and the library never reads memory for them;
 *   - the query of step s sits at position p = T_p + s and sees prompt slots
 *     and generated rows 0..s; a window w > 0 keeps positions > p - w;
 *   - q head h reads KV head floor(h / G) with G = n_q_heads / n_kv_heads.
 * The library never copies a cache to splice it: each cell picks the clean
 * or donor slot by pointer, so all cells of a call share one clean and one
 * donor prompt cache.
 *
 * Memory and ownership.  Every tensor pointer is device memory owned by the
 * caller; the library never allocates, frees or retains it.  Tensors are
 * dense, row-major, 16-byte aligned (lse: 4-byte aligned):
 *   q                        [C][Hq][D]                  dtype
 *   clean_k, clean_v         [Hkv][T_p][D]               dtype (may be NULL if T_p == 0)
 *   donor_k, donor_v         [Hkv][T_p][D]               dtype (NULL for ZERO;
 *                                                        may be NULL if T_p == 0)
 *   gen_k, gen_v             [C][Hkv][gen_capacity][D]   dtype
 *   out                      [C][Hq][D]                  fp32
 *   lse                      [C][Hq]                     fp32, natural log
 * cell_LW is HOST memory: int32 [C][2] = (L_c, W_c), read during the call.
 * Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 * and runs asynchronously; the call returns once it is enqueued.
 *
 * Errors.  Arguments are validated on the host before anything is
 * enqueued: on a negative status nothing was launched and no output byte
 * was written.  SPLICE_EHIP reports a failed HIP launch.
 * Calls are re-entrant (no global mutable state); two calls that share a
 * workspace must be ordered on one stream.  Results are deterministic:
 * identical inputs and the same split give identical bits.
 */
#ifndef SPLICE_ATTN_H
#define SPLICE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define SPLICE_API __attribute__((visibility("default")))
#else
#define SPLICE_API
#endif

#define SPLICE_ABI_VERSION 6
#define SPLICE_MAX_CELLS 256

typedef enum {
    SPLICE_OK = 0,
    SPLICE_EINVAL = -1,        /* NULL pointer, bad enum value, misaligned pointer */
    SPLICE_ESHAPE = -2,        /* sizes inconsistent with each other or with the call */
    SPLICE_EWORKSPACE = -3,    /* workspace NULL or smaller than required */
    SPLICE_EUNSUPPORTED = -4,  /* well-formed but not built: head_dim, group size, cells */
    SPLICE_EHIP = -5           /* a HIP launch failed */
} splice_status;

typedef enum { SPLICE_DONOR_BUFFER = 0, SPLICE_DONOR_ZERO = 1 } splice_donor_kind;
typedef enum { SPLICE_BF16 = 0, SPLICE_F32 = 1 } splice_dtype;
typedef enum {
    SPLICE_SRC_CLEAN = 0, SPLICE_SRC_DONOR = 1, SPLICE_SRC_ZERO = 2, SPLICE_SRC_GEN = 3
} splice_src;

typedef struct {
    int32_t n_cells;       /* C, 0..SPLICE_MAX_CELLS (0: the call does nothing)        */
    int32_t n_layers;      /* N > 0; layer must be < N                                */
    int32_t n_q_heads;     /* Hq > 0                                                  */
    int32_t n_kv_heads;    /* Hkv > 0, Hq % Hkv == 0, G = Hq / Hkv in {1, 2, 4, 8}     */
    int32_t head_dim;      /* D in {64, 128, 256}                                     */
    int32_t prompt_len;    /* T_p >= 0                                                */
    int32_t span_lo;       /* 0 <= span_lo <= span_hi <= T_p                          */
    int32_t span_hi;
    int32_t gen_capacity;  /* rows per generated cache; step < gen_capacity           */
    int32_t donor_kind;    /* splice_donor_kind                                       */
    int32_t dtype;         /* splice_dtype of q and every K/V tensor                  */
} splice_shape;

typedef struct {
    int32_t layer;         /* l, 0 <= l < N: enters only the splice predicate          */
    int32_t step;          /* s, 0 <= s < gen_capacity: 0-based decode step            */
    int32_t window;        /* sliding window w >= 0 (0: every key visible)            */
    float scale;           /* softmax scale applied to q.k: finite and > 0, else
                              SPLICE_EINVAL                                         */
    int32_t split_keys;    /* keys per work item, 0 = library default; else a
                              multiple of 64 in [64, 65536] (tuning and tests)        */
    int32_t merge_wait;    /* bf16 calls with prompt items: how many times a
                              generated-row item polls for the prompt partials of
                              its (cell, KV head) before it leaves the merge to
                              the last item to finish; 0 = library default
                              (about 16 ms), < 0 = never poll (tests)             */
} splice_call;

/* ABI version this library was built with (SPLICE_ABI_VERSION). */
SPLICE_API int32_t splice_abi_version(void);

/* Static string naming a status code; never NULL. */
SPLICE_API const char *splice_status_str(int32_t status);

/*
 * Number of keys one query sees at `call`: visible prompt slots (all of
 * them, spliced or not) plus visible generated rows.  The gather output of
 * splice_kv_build has this many slots.  Negative splice_status on bad input.
 */
SPLICE_API int32_t splice_visible_len(const splice_shape *shape, const splice_call *call);

/*
 * Materialise what each cell attends to at `call` (Section 3, Algorithm 1):
 *   out_k, out_v  device [C][Hkv][n_vis][D], dtype: slot t holds the t-th
 *                 visible key/value -- prompt slots in position order
 *                 (clean, donor or all-zero bits) then generated rows;
 *   out_src       device uint8 [C][n_vis], a splice_src per slot.
 * A bit-exact copy: it is the test hook for the splice selection and the
 * copy-then-attend baseline that splice_decode_attn avoids.
 */
SPLICE_API int32_t splice_kv_build(const splice_shape *shape, const splice_call *call,
                        const int32_t *cell_LW,
                        const void *clean_k, const void *clean_v,
                        const void *donor_k, const void *donor_v,
                        const void *gen_k, const void *gen_v,
                        void *out_k, void *out_v, uint8_t *out_src,
                        void *stream);

/*
 * Workspace bytes splice_decode_attn and splice_decode_forked need for
 * `call` (for a forked sweep, whichever cells have diverged).  With
 * call == NULL: enough for every call on `shape` with split_keys == 0 (any
 * layer, step, window, cells computed).  Negative splice_status on bad input.
 */
SPLICE_API int64_t splice_decode_attn_workspace_bytes(const splice_shape *shape, const splice_call *call);

/*
 * Zero a workspace with a fill kernel enqueued on `stream` (no memset node,
 * so it may be graph-captured).  Required once before a workspace's first
 * splice_decode_attn / splice_decode_step: the workspace starts with a
 * 256-byte statistics block (splice_workspace_handovers) and the
 * per-(cell, KV head) arrival counters, which must start at zero; every call
 * re-arms the counters it used, so later calls need no re-initialisation.
 * workspace must be 256-byte aligned and workspace_bytes a multiple of 4.
 */
SPLICE_API int32_t splice_workspace_init(void *workspace, size_t workspace_bytes, void *stream);

/*
 * Merges handed over since splice_workspace_init: the number of (cell, KV
 * head) pairs of bf16 calls whose generated-row item stopped waiting for the
 * prompt partials (merge_wait ran out, or merge_wait < 0) and left the merge
 * to the last item to finish.  The result does not depend on it (both merge
 * sites fold in one order); it counts how often the slower route ran, which
 * should be 0 with the default bound.  Reads 4 bytes of the workspace's
 * statistics block back to the host on `stream` and waits for the stream.
 * Negative splice_status on a NULL or misaligned workspace, one smaller than
 * 256 bytes, or a failed copy.
 */
SPLICE_API int64_t splice_workspace_handovers(const void *workspace, size_t workspace_bytes, void *stream);

/*
 * Spliced single-query GQA decode attention for C sweep cells at one
 * (layer, step) -- the attention read inside Algorithm 1's forward pass:
 *   score_j = scale * q . k_j over each cell's visible keys,
 *   out     = softmax(score) . V,     lse = log sum_j exp(score_j),
 * with the keys and values chosen per cell as described at the top.
 * q is read in dtype; accumulation is fp32; out and lse are fp32.
 * `workspace` (256-byte aligned, initialised once by splice_workspace_init)
 * must hold splice_decode_attn_workspace_bytes(shape, call) bytes; it holds
 * the split-K partial results and arrival counters of a call, so calls that
 * share a workspace must be ordered on one stream.
 */
SPLICE_API int32_t splice_decode_attn(const splice_shape *shape, const splice_call *call,
                           const int32_t *cell_LW,
                           const void *q,
                           const void *clean_k, const void *clean_v,
                           const void *donor_k, const void *donor_v,
                           const void *gen_k, const void *gen_v,
                           float *out, float *lse,
                           void *workspace, size_t workspace_bytes,
                           void *stream);

/*
 * splice_decode_attn without a workspace argument and without allocating:
 * for callers that cannot call hipMalloc (code under HIP graph capture,
 * serving loops that must not allocate, harnesses that forbid it).  The
 * split-K partials and arrival counters live in a library-owned device
 * array of SPLICE_NOALLOC_WORKSPACE_BYTES bytes, one per GPU, held until
 * the process ends; calls whose splice_decode_attn_workspace_bytes(shape,
 * call) exceeds it return SPLICE_EWORKSPACE before any device work.  The
 * first call on a device takes the array's address and clears it with a
 * fill kernel on `stream` (make that first call outside graph capture);
 * every later call finds the arrival counters at zero, because each call
 * re-arms the counters it uses.  All calls on one GPU share the array:
 * calls that overlap on one GPU (other streams, other threads) race and must
 * be ordered by the caller, e.g. on one stream.  Arguments, results, errors
 * and bits are those of splice_decode_attn (same kernels, same plan).
 */
#define SPLICE_NOALLOC_WORKSPACE_BYTES ((size_t)32 << 20)
SPLICE_API int32_t splice_decode_attn_noalloc(const splice_shape *shape, const splice_call *call,
                           const int32_t *cell_LW,
                           const void *q,
                           const void *clean_k, const void *clean_v,
                           const void *donor_k, const void *donor_v,
                           const void *gen_k, const void *gen_v,
                           float *out, float *lse,
                           void *stream);

/*
 * One decode pass of a batch of cells, each at its own step (Algorithm 1:
 * the forward pass appends the current token's K/V to the generated cache,
 * then attends; a trajectory stops at EOS).  cell_step is host int32 [C]:
 *   cell_step[c] = s_c >= 0  active cell at 0-based step s_c <
 *                            shape->gen_capacity: row s_c of its generated
 *                            caches gen_k, gen_v ([C][Hkv][cap][D]) is set to
 *                            k_new[c], v_new[c] ([C][Hkv][D], dtype), then
 *                            out[c], lse[c] are computed exactly as
 *                            splice_decode_attn at call->step = s_c (the
 *                            splice predicate uses s_c; a sliding window ends
 *                            at T_p + s_c);
 *   cell_step[c] < 0         finished cell (EOS): nothing read or written.
 * call->step is ignored (the other fields of call are validated as usual).
 * The workspace must hold splice_decode_attn_workspace_bytes(shape, NULL)
 * bytes, or with an explicit split_keys, splice_decode_attn_workspace_bytes
 * (shape, call') with call'->step the smallest s_c (the step that sees the
 * most prompt slots).  Only rows s_c of active cells' generated caches are
 * written; the attention of the call takes row s_c from k_new, v_new, so it
 * never depends on when the write lands.  A call with every cell finished is
 * a valid no-op.
 * Errors: as splice_decode_attn, plus SPLICE_EINVAL for a NULL cell_step,
 * k_new or v_new, SPLICE_ESHAPE for s_c >= gen_capacity, and
 * SPLICE_EUNSUPPORTED for f32 inputs (bf16 only).  Other conventions as
 * splice_decode_attn.
 */
SPLICE_API int32_t splice_decode_step(const splice_shape *shape, const splice_call *call,
                           const int32_t *cell_LW, const int32_t *cell_step,
                           const void *q, const void *k_new, const void *v_new,
                           const void *clean_k, const void *clean_v,
                           const void *donor_k, const void *donor_v,
                           void *gen_k, void *gen_v,
                           float *out, float *lse,
                           void *workspace, size_t workspace_bytes,
                           void *stream);

/*
 * The attention of a forked sweep at one (layer, step) (Section 3: a cell
 * (L, W) is the clean run until step W -- nothing is spliced before it --
 * so the clean run is decoded once and each cell forks from it at its onset
 * W).  Cell `trunk` is the clean run: it must never be spliced
 * (L_trunk >= n_layers).  Cell c has diverged from the trunk at call->step
 * iff c == trunk, or L_c < n_layers and call->step >= W_c.
 *   diverged c   attends exactly as splice_decode_attn, except that its
 *                generated rows below W_c are read from the trunk's
 *                generated caches (gen_k, gen_v of cell trunk) and its
 *                rows W_c .. step from its own; its own rows below W_c
 *                are never read (the trunk reads all of its own rows);
 *   other cells  are the clean run at this step: out[c], lse[c] are
 *                written with the trunk's values, bit for bit, and q[c]
 *                and their caches are not read.
 * bf16 only (f32: SPLICE_EUNSUPPORTED).  Errors as splice_decode_attn, plus
 * SPLICE_EINVAL for a negative trunk (with n_cells > 0) and SPLICE_ESHAPE
 * for trunk >= n_cells or a trunk that some layer splices.  Workspace as
 * splice_decode_attn.
 */
SPLICE_API int32_t splice_decode_forked(const splice_shape *shape, const splice_call *call,
                           const int32_t *cell_LW, int32_t trunk,
                           const void *q,
                           const void *clean_k, const void *clean_v,
                           const void *donor_k, const void *donor_v,
                           const void *gen_k, const void *gen_v,
                           float *out, float *lse,
                           void *workspace, size_t workspace_bytes,
                           void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SPLICE_ATTN_H */
