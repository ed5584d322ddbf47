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
    // the bf16 kernels mask raw q.k with -inf and scale afterwards, which
    // needs a positive scale; a softmax scale is positive in every model
    if (!isfinite(call->scale) || !(call->scale > 0.f)) return SPLICE_EINVAL;
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
//
// bf16 inputs: one launch of two kinds of items:
//     prompt items: work groups (KV head, group of group_rows(D) rows, prompt
//       chunk); the rows of a KV head are the (cell, q head) pairs of every
//       cell, clean cells first, and each K/V tile is staged in LDS once for
//       all of a group's rows; every row gets one partial result per chunk;
//     generated-row items: one work group per (cell, KV head) streams the
//       cell's generated rows into one more partial result;
//   the last item of a (cell, KV head) to finish merges its partials.
// f32 inputs (vector ALUs, one launch): prompts of at most
//   kCellwiseMaxPrompt visible keys take one work group per (cell, KV head)
//   streaming the cell's whole list; longer ones prompt items (cell, KV head,
//   prompt chunk) and generated items (cell, KV head, generated chunk),
//   merged the same way.

constexpr int kRowBlock = 64;              // rows of the f32 merge staging
constexpr int kMinChunk = 256;             // a default chunk is at least this long
constexpr int kMaxChunks = 32;             // default chunks per part (prompt, generated)
constexpr int kMaxSlots = 64;              // partial results per (cell, KV head)
constexpr int kPromptItemsTarget = 512;    // f32 prompt items a default split aims for
constexpr int kGenItemsTarget = 2048;      // f32 generated items a default split aims for
constexpr int kWideItemsTarget = 512;      // bf16 prompt work groups a default split aims for
constexpr int kWideMinChunk = 128;         // a default bf16 prompt chunk is at least this long
constexpr int kWideLongChunk = 256;        // ... and this long when that leaves enough work groups
constexpr int kWideLongChunkItems = 96;    // prompt work groups the longer chunks must still give

// bf16 items: waves per work group, 16-row MFMA blocks per wave (a wave's
// output accumulators, RB * D / 4 registers, stay at 32 for D <= 128) and
// rows per prompt item.
constexpr int fused_waves(int) { return 4; }
constexpr int fused_row_blocks(int) { return 1; }
constexpr int group_rows(int D) { return fused_waves(D) * 16 * fused_row_blocks(D); }

// Work groups are handed to the GPU's eight XCDs in turn (block b to XCD
// b mod 8); the bf16 prompt grid is laid out in rounds of this many blocks.
constexpr int kXcds = 8;

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }
inline int round_up(int64_t a, int64_t m) { return (int)((a + m - 1) / m * m); }

// Floats per partial-result slot: o[G][D], m[G], l[G], padded to 256 bytes.
inline int slot_floats(int G, int D) { return (G * D + 2 * G + 63) / 64 * 64; }

inline bool bf16_path(const splice_shape &sh) { return sh.dtype == SPLICE_BF16; }

// Bytes per prompt slot: an fp32 slot, or for bf16 inputs a 16-bit one
// (o[G][D] in fp16, then a 16-byte record (m, l, w, 0) per row, padded to
// 256 bytes), never larger than an fp32 slot.
inline int prompt_slot_bytes(const splice_shape &sh) {
    const int G = group_of(sh), D = sh.head_dim;
    return bf16_path(sh) ? round_up((int64_t)G * D * 2 + 16 * G, 256) : slot_floats(G, D) * 4;
}

// bf16 row groups of one KV head: the rows of unspliced cells and the rows
// of spliced cells are grouped separately (group_rows(D) rows per group), so
// no group needs both the clean and the donor span.  n_clean of the call's
// n_active cells (C, or the unfinished cells of a decode step) are unspliced.
inline int clean_row_groups(const splice_shape &sh, int n_clean) {
    return ceil_div((int64_t)n_clean * group_of(sh), group_rows(sh.head_dim));
}
inline int row_groups(const splice_shape &sh, int n_clean, int n_active) {
    return clean_row_groups(sh, n_clean) +
           ceil_div((int64_t)(n_active - n_clean) * group_of(sh), group_rows(sh.head_dim));
}

// Prompt work groups per prompt chunk.  The bf16 count depends on the call's
// split of cells; the default chunking uses the split-independent bound
// (one more row group than an unsplit grid).
inline int prompt_items_per_chunk(const splice_shape &sh, int n_clean) {
    return sh.n_kv_heads * (bf16_path(sh) ? row_groups(sh, n_clean, sh.n_cells) : sh.n_cells);
}
// n_active: the cells the call computes (bf16; a decode step with finished
// cells has fewer, and then takes more, shorter chunks for its prompt items).
inline int prompt_items_bound(const splice_shape &sh, int n_active) {
    if (!bf16_path(sh)) return sh.n_kv_heads * sh.n_cells;
    return sh.n_kv_heads * (ceil_div((int64_t)n_active * group_of(sh), group_rows(sh.head_dim)) + 1);
}

// Keys per prompt tile of the bf16 kernel (one K and one V tile per step of
// a prompt work group's chain).
constexpr int kPromptTileKeys = 32;

// Cost model of the sparse prompt grid (plan_from_geo), measured on MI355X:
// a prompt work group alone on its compute unit (beside one generated-row
// work group) takes about 0.44 us per 32-key tile at D = 128 (16 KiB of K
// and V), i.e. ~27.5 ns per KiB of its tiles, and the generated rows of a
// call stream at about 6.8 TB/s.
constexpr double kPromptChainNsPerKiB = 27.5;
constexpr double kGenBytesPerNs = 6800.0;

// bf16: at most this many prompt chunks by default, so that a generated-row
// item merges every prompt slot in one round of loads.
constexpr int kWideMaxChunks = 16;

inline int prompt_chunk_target(const splice_shape &sh, int n_active) {
    const int per = prompt_items_bound(sh, n_active);
    const int want = bf16_path(sh) ? kWideItemsTarget : kPromptItemsTarget;
    const int cap = bf16_path(sh) ? kWideMaxChunks : kMaxChunks;
    const int t = per > 0 ? want / per : 1;
    return t < 1 ? 1 : (t > cap ? cap : t);
}

inline int gen_chunk_target(const splice_shape &sh) {
    if (bf16_path(sh)) return 1;   // one generated-row item per (cell, KV head)
    const int64_t pairs = (int64_t)sh.n_cells * sh.n_kv_heads;
    const int64_t t = pairs > 0 ? kGenItemsTarget / pairs : 1;
    return t < 1 ? 1 : (t > kMaxChunks ? kMaxChunks : (int)t);
}

// Cut n keys into chunks.  Default: k = min(ceil(n / min_chunk), target)
// chunks of equal length rounded up to 64; split > 0 fixes the length.
inline void cut(int n, int target, int split, int *k, int *len, int min_chunk = kMinChunk) {
    if (n <= 0) {
        *k = 0;
        *len = 64;
        return;
    }
    if (split > 0) {
        *len = split;
        *k = ceil_div(n, split);
        return;
    }
    int kk = ceil_div(n, min_chunk);
    if (kk > target) kk = target;
    *len = round_up(ceil_div(n, kk), 64);
    *k = ceil_div(n, *len);
}

// f32 prompts up to this many visible keys take the cellwise path: each
// (cell, KV head) streams its own list, re-reading the shared prompt from L2,
// which costs less than the split and merge of the item path.
constexpr int kCellwiseMaxPrompt = 512;

struct AttnPlan {
    bool cellwise;           // one work group per (cell, KV head), no partials
    Geometry geo;
    int n_p, p_len;          // prompt chunks over the visible prompt
    int n_g, g_len;          // chunks over the visible generated rows
    int n_slots;             // partial results per (cell, KV head)
    int n_prompt_items, n_gen_items;
    int gen_pairs;           // bf16: (cell, KV head) pairs per generated-row work group
};

// bf16 generated-row items: a work group of fused_waves(D) waves serves P
// consecutive cells of one KV head, NW / P waves each (P = 1, 2 or 4).
//
// With an explicit split_keys the grouping depends on the generated length
// alone, so a cell's bits do not depend on its batch-mates: each wave
// streams at least two 16-row tiles.
inline int gen_pairs_fixed(const splice_shape &sh, int n_gen) {
    const int nw = fused_waves(sh.head_dim);
    const int tiles = ceil_div(n_gen, 16);
    int wpp = nw;
    while (wpp > 1 && tiles < 2 * wpp) wpp /= 2;
    return nw / wpp;
}

// What one GPU holds of the bf16 kernel at once: its compute units and the
// work groups resident on each (0 when unknown).
struct Residency {
    int n_cu = 0;
    int per_cu = 0;
};

// Default grouping.  The generated-row streams run fastest when every work
// group of the launch is resident from the start (no second round whose last
// groups stream alone), when the groups spread evenly over the compute units
// (a unit holding one more group than the others finishes last), and when
// each wave streams enough rows to hide its first loads.  So P is the
// smallest grouping whose waves stream at least kGenWaveBytes among those
// that fit beside the prompt items in one round with at most 1.2 times
// the mean groups per unit (kGenImbalanceNum / kGenImbalanceDen); if no
// wave gets that many bytes, the
// largest such grouping; if none fits, NW.  When the cells stream different
// numbers of rows (a decode step with cells at their own steps; n_gen is the
// longest, and `same_rows` is false), rounds and balance matter less: the
// longest streams are dispatched first, so the groups that wait are the
// shortest, and the groups differ in length anyway; what sets the pass is
// the longest stream, so P is the smallest grouping whose waves stream at
// least kGenWaveBytes of it.  prompt_items is a bound that does not depend on
// the clean/spliced split of the cells, so the grouping (and the bits) of a
// call do not either.
constexpr int64_t kGenWaveBytes = 48 << 10;
constexpr int kGenImbalanceNum = 6, kGenImbalanceDen = 5;   // 1.2

inline int gen_pairs_default(const splice_shape &sh, int n_gen, int n_active, int64_t prompt_items,
                             const Residency &res, bool same_rows) {
    const int nw = fused_waves(sh.head_dim);
    if (res.n_cu <= 0 || res.per_cu <= 0) return gen_pairs_fixed(sh, n_gen);
    const int64_t resident = (int64_t)res.n_cu * res.per_cu;
    const int64_t row_bytes = 2LL * sh.head_dim * elem_bytes(sh);   // a K row and a V row
    int long_enough = 0, largest = 0;
    for (int P = 1; P <= nw; P *= 2) {
        const int64_t groups = (int64_t)ceil_div(n_active, P) * sh.n_kv_heads;
        if (same_rows) {
            if (prompt_items + groups > resident) continue;
            const int64_t per_unit = ceil_div(groups, res.n_cu);
            if (groups > res.n_cu && per_unit * res.n_cu * kGenImbalanceDen > groups * kGenImbalanceNum) continue;
        }
        largest = P;
        if (!long_enough && (int64_t)n_gen * row_bytes * P >= kGenWaveBytes * nw) long_enough = P;
    }
    return long_enough ? long_enough : (largest ? largest : nw);
}

// Validation of a decode step's per-cell steps (host int32 [C]): each is
// < gen_capacity; negative marks a finished cell.
inline int32_t validate_steps(const splice_shape &sh, const int32_t *cell_step) {
    if (sh.n_cells == 0) return SPLICE_OK;
    if (!cell_step) return SPLICE_EINVAL;
    for (int c = 0; c < sh.n_cells; ++c)
        if (cell_step[c] >= sh.gen_capacity) return SPLICE_ESHAPE;
    return SPLICE_OK;
}

// Cells of the call that are not spliced.
inline int count_clean(const splice_shape &sh, const splice_call &call, const int32_t *cell_LW) {
    int n = 0;
    for (int c = 0; c < sh.n_cells; ++c) n += cell_spliced(cell_LW, c, call.layer, call.step) ? 0 : 1;
    return n;
}

// Plan a call whose keys span `geo` (for a decode step with cells at
// different steps: the widest visible prompt and the longest generated part)
// over n_active cells, n_clean of them unspliced.
inline AttnPlan plan_from_geo(const splice_shape &sh, const splice_call &call, const Geometry &geo, int n_clean,
                              int n_active, const Residency &res = Residency(), bool same_rows = true) {
    AttnPlan p;
    p.geo = geo;
    p.cellwise = !bf16_path(sh) && call.split_keys == 0 && p.geo.n_prompt <= kCellwiseMaxPrompt;
    if (p.cellwise) {
        p.n_p = p.n_g = 0;
        p.p_len = p.g_len = 64;
        p.n_slots = 0;
        p.n_prompt_items = p.n_gen_items = 0;
        p.gen_pairs = 1;
        return p;
    }
    cut(p.geo.n_prompt, prompt_chunk_target(sh, n_active), call.split_keys, &p.n_p, &p.p_len,
        bf16_path(sh) ? kWideMinChunk : kMinChunk);
    if (bf16_path(sh) && call.split_keys == 0) {
        // chunks of a few tiles spend much of their time starting up and
        // storing partials: take longer ones when the grid stays wide enough
        int n_long, len_long;
        cut(p.geo.n_prompt, prompt_chunk_target(sh, n_active), 0, &n_long, &len_long, kWideLongChunk);
        const int64_t groups = prompt_items_bound(sh, n_active);
        if (n_long < p.n_p && n_long * groups >= kWideLongChunkItems) {
            p.n_p = n_long;
            p.p_len = len_long;
        }
        // a long generated part: fewer, longer chunks, at most one prompt
        // work group per compute unit, when their chains still end before
        // the generated rows are streamed
        if (same_rows && res.n_cu > 0 && groups > 0) {
            const int n_sparse = (int)(res.n_cu / groups);
            if (n_sparse >= 1 && n_sparse < p.n_p) {
                int k, len;
                cut(p.geo.n_prompt, n_sparse, 0, &k, &len, kWideMinChunk);
                const double tile_kib = 2.0 * kPromptTileKeys * sh.head_dim * elem_bytes(sh) / 1024.0;   // K and V
                const double prompt_ns = (double)ceil_div(len, kPromptTileKeys) * tile_kib * kPromptChainNsPerKiB;
                const double gen_ns = (double)n_active * sh.n_kv_heads * p.geo.n_gen * 2.0 * sh.head_dim *
                                      elem_bytes(sh) / kGenBytesPerNs;
                if (gen_ns >= prompt_ns) {
                    p.n_p = k;
                    p.p_len = len;
                }
            }
        }
    }
    if (bf16_path(sh)) {
        // one generated-row partial per (cell, KV head)
        p.n_g = 1;
        p.g_len = p.geo.n_gen;
    } else {
        cut(p.geo.n_gen, gen_chunk_target(sh), call.split_keys, &p.n_g, &p.g_len);
    }
    p.n_slots = p.n_p + p.n_g;
    if (bf16_path(sh)) {
        // units (KV head, chunk) padded to whole rounds of kXcds, times row groups
        p.n_prompt_items = p.n_p > 0 ? kXcds * row_groups(sh, n_clean, n_active) *
                                            ceil_div((int64_t)sh.n_kv_heads * p.n_p, kXcds)
                                      : 0;
    } else {
        p.n_prompt_items = prompt_items_per_chunk(sh, n_clean) * p.n_p;
    }
    if (bf16_path(sh)) {
        // the prompt items of the call's grid with one more row group per
        // KV head than an unsplit one (the most any split of the cells gives)
        const int64_t prompt_bound =
            p.n_p > 0 ? (int64_t)kXcds *
                            (ceil_div((int64_t)n_active * group_of(sh), group_rows(sh.head_dim)) + 1) *
                            ceil_div((int64_t)sh.n_kv_heads * p.n_p, kXcds)
                      : 0;
        p.gen_pairs = call.split_keys > 0 ? gen_pairs_fixed(sh, p.geo.n_gen)
                                          : gen_pairs_default(sh, p.geo.n_gen, n_active, prompt_bound, res,
                                                              same_rows);
        p.n_gen_items = ceil_div(n_active, p.gen_pairs) * sh.n_kv_heads;   // active cells only
    } else {
        p.gen_pairs = 1;
        p.n_gen_items = sh.n_cells * sh.n_kv_heads * p.n_g;
    }
    return p;
}

// bf16: the generated-row items load V non-temporally, so that the rows,
// read once, do not push the shared prompt tiles out of the caches, when
// the prompt caches a call reads (clean, plus donor when the donor is a
// buffer) exceed kGenNtPromptBytes or the call streams at least
// kGenNtRows generated rows per cell; short calls with small prompts
// measured faster with normal loads.
constexpr int64_t kGenNtPromptBytes = (int64_t)16 << 20;
constexpr int kGenNtRows = 128;

inline bool gen_v_nontemporal(const splice_shape &sh, int n_gen) {
    const int64_t per_cache = (int64_t)sh.prompt_len * sh.n_kv_heads * sh.head_dim * elem_bytes(sh) * 2;
    const int64_t bytes = per_cache * (sh.donor_kind == SPLICE_DONOR_BUFFER ? 2 : 1);
    return bytes > kGenNtPromptBytes || n_gen >= kGenNtRows;
}

struct WorkspaceLayout {
    size_t stats_off;   // kStatsBytes of statistics (the hand-over count), kept across calls
    size_t counters_off, counters_bytes;
    size_t part_off, part_bytes;
    size_t total;
};

// Statistics words at the start of a workspace (int32): [0] the number of
// (cell, KV head) merges handed over by a generated-row item whose bounded
// wait ran out, counted since splice_workspace_init.
constexpr size_t kStatsBytes = 256;

// Statistics, counters [C][Hkv] (int32), then the partial results: one
// slot per (cell, KV head, chunk) -- for bf16 inputs the 16-bit prompt slots
// [C][Hkv][n_slots - 1] followed by the fp32 generated-row slots [C][Hkv]
// (one each), otherwise fp32 slots.
inline WorkspaceLayout workspace_layout(const splice_shape &sh, int n_slots) {
    WorkspaceLayout w;
    const int64_t pairs = (int64_t)sh.n_cells * sh.n_kv_heads;
    w.stats_off = 0;
    w.counters_off = kStatsBytes;
    w.counters_bytes = (size_t)round_up(pairs * 4, 256);
    w.part_off = w.counters_off + w.counters_bytes;
    const size_t f32_slot = (size_t)slot_floats(group_of(sh), sh.head_dim) * 4;
    w.part_bytes = bf16_path(sh) && n_slots > 0
                       ? (size_t)pairs * ((size_t)(n_slots - 1) * (size_t)prompt_slot_bytes(sh) + f32_slot)
                       : (size_t)pairs * (size_t)n_slots * f32_slot;
    w.total = w.part_off + w.part_bytes;
    if (w.total < 256) w.total = 256;
    return w;
}

// Most slots any default-split call on this shape uses.  For n keys the
// default cut makes at most min(ceil(n / kMinChunk), target) chunks (each
// chunk is at least n / that many keys long), and that bound grows with n;
// a call sees at most T_p prompt keys and gen_capacity generated rows.
inline int max_default_chunks(int n, int target, int min_chunk = kMinChunk) {
    if (n <= 0) return 0;
    const int k = ceil_div(n, min_chunk);
    return k < target ? k : target;
}

inline int worst_default_slots(const splice_shape &sh) {
    // bf16: a decode step with one active cell takes the most chunks
    const int prompt = max_default_chunks(sh.prompt_len, prompt_chunk_target(sh, bf16_path(sh) ? 1 : sh.n_cells),
                                          bf16_path(sh) ? kWideMinChunk : kMinChunk);
    return bf16_path(sh) ? prompt + 1 : prompt + max_default_chunks(sh.gen_capacity, gen_chunk_target(sh));
}

}  // namespace splice
