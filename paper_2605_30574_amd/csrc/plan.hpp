// plan.hpp -- host-side validation and launch planning for the splice library.
//
// Everything here runs on the CPU before any launch, so a bad argument is
// reported without touching device memory.  The visibility rules implement
// the readings stated in splice_attn.h: the query of step s sits at
// p = T_p + s, sees prompt slots and generated rows 0..s, and a window w > 0
// keeps positions > p - w.
#pragma once

#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "splice_attn.h"

namespace splice {

// What one query sees at (step, window): the visible part of the prompt
// [jp0, T_p), the visible part of the replaced span [sa, sb) and the visible
// generated rows [i0, step].
struct Geometry {
    int jp0;
    int i0;
    int n_prompt;   // T_p - jp0
    int n_gen;      // step + 1 - i0
    int sa, sb;     // span clipped to the visible prompt, sa <= sb
    int n_vis;      // n_prompt + n_gen
};

inline Geometry geometry(const splice_shape &sh, const splice_call &call) {
    const long Tp = sh.prompt_len;
    const long p = Tp + call.step;
    const long j0 = call.window > 0 ? p - call.window + 1 : 0;
    long jp0 = j0 < 0 ? 0 : j0;
    if (jp0 > Tp) jp0 = Tp;
    long i0 = j0 - Tp;
    if (i0 < 0) i0 = 0;
    long sa = sh.span_lo < jp0 ? jp0 : sh.span_lo;
    if (sa > Tp) sa = Tp;
    long sb = sh.span_hi < sa ? sa : sh.span_hi;
    if (sb > Tp) sb = Tp;
    Geometry g;
    g.jp0 = (int)jp0;
    g.i0 = (int)i0;
    g.n_prompt = (int)(Tp - jp0);
    g.n_gen = (int)(call.step + 1 - i0);
    g.sa = (int)sa;
    g.sb = (int)sb;
    g.n_vis = g.n_prompt + g.n_gen;
    return g;
}

inline int group_of(const splice_shape &sh) { return sh.n_q_heads / sh.n_kv_heads; }
inline int elem_bytes(const splice_shape &sh) { return sh.dtype == SPLICE_BF16 ? 2 : 4; }

inline int32_t validate_shape(const splice_shape *sh) {
    if (!sh) return SPLICE_EINVAL;
    if (sh->donor_kind != SPLICE_DONOR_BUFFER && sh->donor_kind != SPLICE_DONOR_ZERO) return SPLICE_EINVAL;
    if (sh->dtype != SPLICE_BF16 && sh->dtype != SPLICE_F32) return SPLICE_EINVAL;
    if (sh->n_cells < 0 || sh->n_layers <= 0 || sh->n_q_heads <= 0 || sh->n_kv_heads <= 0 ||
        sh->head_dim <= 0 || sh->prompt_len < 0 || sh->gen_capacity <= 0)
        return SPLICE_ESHAPE;
    if (sh->n_q_heads % sh->n_kv_heads != 0) return SPLICE_ESHAPE;
    if (sh->span_lo < 0 || sh->span_lo > sh->span_hi || sh->span_hi > sh->prompt_len) return SPLICE_ESHAPE;
    if ((int64_t)sh->prompt_len + sh->gen_capacity > (int64_t)1 << 28) return SPLICE_EUNSUPPORTED;
    if (sh->n_cells > SPLICE_MAX_CELLS) return SPLICE_EUNSUPPORTED;
    const int G = group_of(*sh);
    if (G != 1 && G != 2 && G != 4 && G != 8) return SPLICE_EUNSUPPORTED;
    if (sh->head_dim != 64 && sh->head_dim != 128 && sh->head_dim != 256) return SPLICE_EUNSUPPORTED;
    return SPLICE_OK;
}

inline int32_t validate_call(const splice_shape &sh, const splice_call *call) {
    if (!call) return SPLICE_EINVAL;
    if (call->layer < 0 || call->layer >= sh.n_layers) return SPLICE_ESHAPE;
    if (call->step < 0 || call->step >= sh.gen_capacity) return SPLICE_ESHAPE;
    if (call->window < 0) return SPLICE_ESHAPE;
    if (!isfinite(call->scale)) return SPLICE_EINVAL;
    if (call->split_keys != 0 &&
        (call->split_keys < 64 || call->split_keys > 65536 || call->split_keys % 64 != 0))
        return SPLICE_EINVAL;
    return SPLICE_OK;
}

inline int32_t validate_cells(const splice_shape &sh, const int32_t *cell_LW) {
    if (sh.n_cells == 0) return SPLICE_OK;
    if (!cell_LW) return SPLICE_EINVAL;
    for (int c = 0; c < sh.n_cells; ++c)
        if (cell_LW[2 * c] < 0 || cell_LW[2 * c + 1] < 0) return SPLICE_ESHAPE;
    return SPLICE_OK;
}

inline bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// The splice predicate (Section 3): layer in {l >= L} and step >= W.
inline bool cell_spliced(const int32_t *cell_LW, int c, int layer, int step) {
    return layer >= cell_LW[2 * c] && step >= cell_LW[2 * c + 1];
}

// ---------------------------------------------------------------- attention plan

constexpr int kTargetItems = 2048;   // work items a default split aims for
constexpr int kMinSplit = 256;       // default split never goes below this
constexpr int kMaxSplit = 2048;      // ... nor above this

inline int default_split(int n_keys, int n_cells, int n_kv_heads) {
    const int64_t pairs = (int64_t)n_cells * n_kv_heads;
    int64_t want = ((int64_t)n_keys * pairs + kTargetItems - 1) / kTargetItems;   // ceil
    want = (want + 63) / 64 * 64;
    if (want < kMinSplit) want = kMinSplit;
    if (want > kMaxSplit) want = kMaxSplit;
    return (int)want;
}

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Floats per partial-result slot: o[G][D], m[G], l[G], padded to 256 bytes.
inline int slot_floats(int G, int D) { return (G * D + 2 * G + 63) / 64 * 64; }

struct WorkspaceLayout {
    size_t part_off, part_bytes;
    size_t total;
};

// The workspace holds one partial-result slot per (cell, KV head, chunk).
inline WorkspaceLayout workspace_layout(const splice_shape &sh, int max_chunks) {
    WorkspaceLayout w;
    const int64_t pairs = (int64_t)sh.n_cells * sh.n_kv_heads;
    w.part_off = 0;
    w.part_bytes = max_chunks > 1 ? (size_t)pairs * (size_t)max_chunks *
                                        (size_t)slot_floats(group_of(sh), sh.head_dim) * sizeof(float)
                                  : 0;
    w.total = w.part_off + w.part_bytes;
    if (w.total < 256) w.total = 256;
    return w;
}

// Largest number of work items per (cell, KV head) of any default-split call
// on this shape.  A call has n <= T_p + gen_capacity keys and split(n) is
// either >= n * pairs / kTargetItems (so n / split <= kTargetItems / pairs)
// or clamped to kMaxSplit (so n / split <= (T_p + gen_capacity) / kMaxSplit).
inline int worst_default_chunks(const splice_shape &sh) {
    const int64_t pairs = (int64_t)sh.n_cells * sh.n_kv_heads;
    if (pairs <= 0) return 1;
    const int64_t n_max = (int64_t)sh.prompt_len + sh.gen_capacity;
    const int a = ceil_div(kTargetItems, pairs);
    const int b = ceil_div(n_max, kMaxSplit);
    const int worst = a > b ? a : b;
    const int cap = ceil_div(n_max, kMinSplit);   // split >= kMinSplit always
    return worst < cap ? worst : cap;
}

}  // namespace splice
