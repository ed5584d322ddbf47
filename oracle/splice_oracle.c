/*
 * splice_oracle.c -- plain, slow fp64 CPU oracle of spliced decode attention.
 *
 * TEST INFRASTRUCTURE ONLY.  The tests, the smoke check and the benchmark's
 * CPU-baseline leg call it; the GPU library never links, loads or calls it,
 * and this file shares no code, header, table or constant with that library.
 *
 * What it computes (the definition, written out):
 *
 *   Splice intervention (paper Section 3, "Splice intervention"; Algorithm 1
 *   in the appendix "Splice Intervention Pseudocode"):
 *     patched layers  P = { l : l >= L }                       (cutoff L)
 *     onset W: decode steps before W use the unmodified cache; from step W on
 *     the prompt-span entries of every patched layer hold the donor's entries
 *     and keep holding them to the end (in-place, permanent replacement).
 *     The rows the decode itself generates stay as written: a splice touches
 *     only prompt slots.
 *   Donors (Table 1): ZERO = all-zero K and V; the other forms are buffers of
 *     the same prompt length, aligned slot for slot with the target prompt.
 *
 *   Readings used here (the paper is silent or ambiguous on these):
 *     - decode step s is 0-based (s = 0 is the first pass after prefill) and
 *       the cell (L, W) is spliced at (layer, s) iff layer >= L and s >= W;
 *     - only the slots in [span_lo, span_hi) are replaced; [0, T_p) is the
 *       paper-literal full-prompt case;
 *     - ZERO slots are ordinary keys whose K and V are zero: they score
 *       exactly 0 and are not masked;
 *     - at step s the query sits at position p = T_p + s and sees the prompt
 *       slots plus generated rows 0..s (its own entry included); a sliding
 *       window w > 0 keeps only positions > p - w;
 *     - q head h reads KV head floor(h / G), G = Hq / Hkv.
 *
 *   Attention over the ordered visible list (textbook softmax, IEEE double on
 *   the exact values of the bf16/f32 inputs):
 *     score_j = scale * sum_d q[d] * k_j[d]          (d ascending)
 *     m = max_j score_j,  Z = sum_j exp(score_j - m)  (list order)
 *     out = sum_j exp(score_j - m) v_j / Z,  lse = m + ln Z  (natural log)
 *
 * Layouts (row-major): q [C][Hq][D]; clean/donor K,V [Hkv][T_p][D];
 * generated K,V [C][Hkv][cap][D]; gathered K,V [C][Hkv][n_vis][D];
 * source map [C][n_vis] (0 clean, 1 donor, 2 zero, 3 generated).
 * Build: gcc -O2 -fopenmp -shared -fPIC (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t n_cells, n_q_heads, n_kv_heads, head_dim;
    int32_t prompt_len, span_lo, span_hi, gen_capacity;
    int32_t donor_zero;   /* 1: ZERO donor (no buffer), 0: donor buffer   */
    int32_t elem_bytes;   /* 2: bf16 bit patterns, 4: IEEE binary32       */
} oracle_shape;

typedef struct {
    int32_t layer, step, window;
    double scale;
} oracle_call;

enum { SRC_CLEAN = 0, SRC_DONOR = 1, SRC_ZERO = 2, SRC_GEN = 3 };

typedef struct { int src; long row; } key_ref;

/* Section 3: layer in P = {l >= L}, and step at or after the onset W. */
int oracle_spliced(int layer, int step, int L, int W)
{
    return layer >= L && step >= W;
}

/* Exact value of one stored element. */
static double load_elem(const void *base, size_t idx, int elem_bytes)
{
    if (elem_bytes == 2) {
        uint16_t h;
        uint32_t u;
        float f;
        memcpy(&h, (const char *)base + 2 * idx, 2);
        u = (uint32_t)h << 16;
        memcpy(&f, &u, 4);
        return (double)f;
    } else {
        float f;
        memcpy(&f, (const char *)base + 4 * idx, 4);
        return (double)f;
    }
}

/* First visible position for the query at p = T_p + step. */
static long first_visible(const oracle_shape *sh, int step, int window)
{
    long p = (long)sh->prompt_len + step;
    return window > 0 ? p - window + 1 : 0;
}

/* The ordered list of keys one cell attends to at (layer, step). */
static int visible_keys(const oracle_shape *sh, int spliced, int step, int window, key_ref *keys)
{
    long j0 = first_visible(sh, step, window);
    long j, i, i0;
    int n = 0;
    for (j = j0 > 0 ? j0 : 0; j < sh->prompt_len; ++j) {
        int in_span = j >= sh->span_lo && j < sh->span_hi;
        int src = SRC_CLEAN;
        if (spliced && in_span)
            src = sh->donor_zero ? SRC_ZERO : SRC_DONOR;
        keys[n].src = src;
        keys[n].row = j;
        ++n;
    }
    i0 = j0 - sh->prompt_len;
    if (i0 < 0)
        i0 = 0;
    for (i = i0; i <= step; ++i) {
        keys[n].src = SRC_GEN;
        keys[n].row = i;
        ++n;
    }
    return n;
}

int oracle_visible_len(const oracle_shape *sh, int step, int window)
{
    long j0 = first_visible(sh, step, window);
    long np = sh->prompt_len - (j0 > 0 ? j0 : 0);
    long i0 = j0 - sh->prompt_len;
    if (np < 0)
        np = 0;
    if (i0 < 0)
        i0 = 0;
    return (int)(np + (step + 1 - i0));
}

/* Element offset of the first element of a key's row, or -1 for ZERO. */
static const void *row_base(const oracle_shape *sh, const key_ref *kr, int c, int g, int want_v,
                            const void *clean_k, const void *clean_v,
                            const void *donor_k, const void *donor_v,
                            const void *gen_k, const void *gen_v, size_t *off)
{
    size_t D = (size_t)sh->head_dim;
    switch (kr->src) {
    case SRC_CLEAN:
        *off = ((size_t)g * sh->prompt_len + (size_t)kr->row) * D;
        return want_v ? clean_v : clean_k;
    case SRC_DONOR:
        *off = ((size_t)g * sh->prompt_len + (size_t)kr->row) * D;
        return want_v ? donor_v : donor_k;
    case SRC_GEN:
        *off = (((size_t)c * sh->n_kv_heads + g) * sh->gen_capacity + (size_t)kr->row) * D;
        return want_v ? gen_v : gen_k;
    default:
        *off = 0;
        return NULL;  /* ZERO: every element is 0 */
    }
}

/*
 * Gather: materialise each cell's visible K and V (the list above, in order)
 * and the source of every slot.  A pure copy of the stored bits; ZERO slots
 * are written as all-zero bits.
 */
int oracle_gather(const oracle_shape *sh, const oracle_call *call, const int32_t *cell_LW,
                  const void *clean_k, const void *clean_v,
                  const void *donor_k, const void *donor_v,
                  const void *gen_k, const void *gen_v,
                  void *out_k, void *out_v, uint8_t *out_src)
{
    int n_vis = oracle_visible_len(sh, call->step, call->window);
    size_t D = (size_t)sh->head_dim, eb = (size_t)sh->elem_bytes;
    key_ref *keys = (key_ref *)malloc(sizeof(key_ref) * (size_t)(n_vis > 0 ? n_vis : 1));
    int c, g, t;
    if (!keys)
        return -1;
    for (c = 0; c < sh->n_cells; ++c) {
        int spliced = oracle_spliced(call->layer, call->step, cell_LW[2 * c], cell_LW[2 * c + 1]);
        int n = visible_keys(sh, spliced, call->step, call->window, keys);
        if (n != n_vis) {
            free(keys);
            return -2;
        }
        for (t = 0; t < n; ++t)
            out_src[(size_t)c * n_vis + t] = (uint8_t)keys[t].src;
        for (g = 0; g < sh->n_kv_heads; ++g) {
            for (t = 0; t < n; ++t) {
                size_t dst = (((size_t)c * sh->n_kv_heads + g) * n_vis + t) * D * eb;
                size_t off;
                const void *bk = row_base(sh, &keys[t], c, g, 0, clean_k, clean_v, donor_k, donor_v, gen_k, gen_v, &off);
                const void *bv = row_base(sh, &keys[t], c, g, 1, clean_k, clean_v, donor_k, donor_v, gen_k, gen_v, &off);
                if (bk) {
                    memcpy((char *)out_k + dst, (const char *)bk + off * eb, D * eb);
                    memcpy((char *)out_v + dst, (const char *)bv + off * eb, D * eb);
                } else {
                    memset((char *)out_k + dst, 0, D * eb);
                    memset((char *)out_v + dst, 0, D * eb);
                }
            }
        }
    }
    free(keys);
    return 0;
}

/*
 * Attention for the requested (cell, q head) rows.  rows = NULL means every
 * row in (c, h) order; otherwise rows holds n_rows pairs (c, h).
 * out: [n_rows][D] doubles, lse: [n_rows] doubles.
 */
int oracle_attn(const oracle_shape *sh, const oracle_call *call, const int32_t *cell_LW,
                const void *q,
                const void *clean_k, const void *clean_v,
                const void *donor_k, const void *donor_v,
                const void *gen_k, const void *gen_v,
                const int32_t *rows, int n_rows, double *out, double *lse, int n_threads)
{
    int n_vis = oracle_visible_len(sh, call->step, call->window);
    int G = sh->n_q_heads / sh->n_kv_heads;
    int total = rows ? n_rows : sh->n_cells * sh->n_q_heads;
    int failed = 0;
    int r;
    size_t D = (size_t)sh->head_dim;
    int eb = sh->elem_bytes;
#ifdef _OPENMP
    int nt = n_threads > 0 ? n_threads : omp_get_max_threads();
#else
    (void)n_threads;
#endif

#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (r = 0; r < total; ++r) {
        int c = rows ? rows[2 * r] : r / sh->n_q_heads;
        int h = rows ? rows[2 * r + 1] : r % sh->n_q_heads;
        int g = h / G;
        int spliced = oracle_spliced(call->layer, call->step, cell_LW[2 * c], cell_LW[2 * c + 1]);
        key_ref *keys = (key_ref *)malloc(sizeof(key_ref) * (size_t)(n_vis > 0 ? n_vis : 1));
        double *score = (double *)malloc(sizeof(double) * (size_t)(n_vis > 0 ? n_vis : 1));
        double *acc = (double *)calloc(D, sizeof(double));
        double *qv = (double *)malloc(sizeof(double) * D);
        size_t qoff = ((size_t)c * sh->n_q_heads + h) * D;
        double m = -INFINITY, Z = 0.0;
        int n, t;
        size_t d;
        if (!keys || !score || !acc || !qv) {
#pragma omp atomic write
            failed = 1;
            free(keys); free(score); free(acc); free(qv);
            continue;
        }
        for (d = 0; d < D; ++d)
            qv[d] = load_elem(q, qoff + d, eb);
        n = visible_keys(sh, spliced, call->step, call->window, keys);
        for (t = 0; t < n; ++t) {
            size_t off;
            const void *bk = row_base(sh, &keys[t], c, g, 0, clean_k, clean_v, donor_k, donor_v, gen_k, gen_v, &off);
            double dot = 0.0;
            for (d = 0; d < D; ++d) {
                double kd = bk ? load_elem(bk, off + d, eb) : 0.0;
                dot += qv[d] * kd;
            }
            score[t] = call->scale * dot;
            if (score[t] > m)
                m = score[t];
        }
        for (t = 0; t < n; ++t) {
            size_t off;
            const void *bv = row_base(sh, &keys[t], c, g, 1, clean_k, clean_v, donor_k, donor_v, gen_k, gen_v, &off);
            double wgt = exp(score[t] - m);
            Z += wgt;
            for (d = 0; d < D; ++d) {
                double vd = bv ? load_elem(bv, off + d, eb) : 0.0;
                acc[d] += wgt * vd;
            }
        }
        for (d = 0; d < D; ++d)
            out[(size_t)r * D + d] = acc[d] / Z;
        lse[r] = m + log(Z);
        free(keys); free(score); free(acc); free(qv);
    }
    return failed ? -1 : 0;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
