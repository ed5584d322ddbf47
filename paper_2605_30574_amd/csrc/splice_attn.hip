// splice_attn.hip -- gfx950 kernels and C-ABI entry points of the splice library.
//
// Hot path: single-query grouped-query decode attention for C sweep cells at
// one (layer, step), each cell reading its prompt-span slots from the clean
// or the donor cache (paper Section 3, Algorithm 1, Table 1).  A cell picks
// each slot by pointer: no cache is copied, and all cells of a call share
// one clean and one donor prompt cache.
//
// Kernels
//   gather_kernel   splice_kv_build: bit-exact copy of each cell's visible
//                   keys/values plus a source code per slot (16-byte moves).
//   fused_kernel    splice_decode_attn, bf16 inputs (attn_kernels.hpp): one
//                   launch per call of two kinds of work item --
//     prompt items  (KV head, 64 rows, prompt chunk): the rows are the
//                   (cell, q head) pairs of all cells, clean cells first;
//                   each 32-key tile of the clean (and, for spliced rows,
//                   the donor) prompt cache is staged in LDS once for all 64
//                   rows, and both products run on v_mfma_f32_16x16x32_bf16;
//                   every row gets one partial (m, l, o) per chunk;
//     generated-row items (KV head, a few cells): each cell's own rows
//                   streamed on the matrix cores, never spliced, read once;
//                   the item waits (bounded) for its cells' prompt partials
//                   and merges them into out and lse.
//                   splice_decode_step runs the same kernel with each cell
//                   at its own step: the generated-row items first write the
//                   current token's K/V row into the cell's cache, the prompt
//                   items cover the widest visible prompt of the call and
//                   mask, per row, what that row's step does not see, and
//                   finished cells get no rows and no work.
//   items_kernel, cellwise_kernel   f32 inputs, vector ALUs.
//   fill_kernel     splice_workspace_init.
//
// ZERO donor: a ZERO slot has K = V = 0, so its score is exactly 0 and it
// adds no value mass.  The kernel drops those slots from the key list and
// adds n_zero keys of score 0 in the combine: m' = max(m, 0),
// l' = l 2^(m - m') + n_zero 2^(-m'), o' = o 2^(m - m').  No byte is read.
//
// Numerics: bf16 (or f32) inputs, fp32 accumulation, scores kept in base-2
// units (q.k * scale * log2 e) so that exp2 maps to v_exp_f32.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "attn_kernels.hpp"
#include "plan.hpp"
#include "splice_attn.h"

namespace {

using namespace splice_dev;

// ------------------------------------------------------------------ gather

struct GatherArgs {
    const char *ck, *cv, *dk, *dv, *gk, *gv;
    char *ok, *ov;
    uint8_t *src;
    int Hkv, Tp, cap, row_bytes, zero_donor;
    int jp0, i0, n_prompt, n_vis, sa, sb;
    uint32_t spliced[SPLICE_MAX_CELLS / 32];
};

__global__ __launch_bounds__(kThreads) void gather_kernel(GatherArgs a) {
    const int g = blockIdx.y, c = blockIdx.z;
    const bool spl = bit_set(a.spliced, c);
    const int units = a.row_bytes / 16;
    const int64_t total = (int64_t)a.n_vis * units;
    const size_t out_base = ((size_t)c * a.Hkv + g) * (size_t)a.n_vis * a.row_bytes;
    for (int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x; u < total;
         u += (int64_t)gridDim.x * kThreads) {
        const int t = (int)(u / units), part = (int)(u % units);
        uint8_t code;
        const char *kb, *vb;
        size_t off;
        bool read = true;
        if (t < a.n_prompt) {
            const int j = a.jp0 + t;
            const bool in_span = j >= a.sa && j < a.sb;
            const bool from_donor = spl && in_span;
            off = ((size_t)g * a.Tp + j) * a.row_bytes;
            code = from_donor ? (a.zero_donor ? SPLICE_SRC_ZERO : SPLICE_SRC_DONOR) : SPLICE_SRC_CLEAN;
            read = !(from_donor && a.zero_donor);
            kb = pick_base(from_donor && !a.zero_donor, a.ck, a.dk);
            vb = pick_base(from_donor && !a.zero_donor, a.cv, a.dv);
        } else {
            const int i = a.i0 + (t - a.n_prompt);
            off = (((size_t)c * a.Hkv + g) * a.cap + i) * a.row_bytes;
            code = SPLICE_SRC_GEN;
            kb = a.gk;
            vb = a.gv;
        }
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (read) {
            kv = *reinterpret_cast<const uint4 *>(kb + off + (size_t)part * 16);
            vv = *reinterpret_cast<const uint4 *>(vb + off + (size_t)part * 16);
        }
        const size_t dst = out_base + (size_t)t * a.row_bytes + (size_t)part * 16;
        *reinterpret_cast<uint4 *>(a.ok + dst) = kv;
        *reinterpret_cast<uint4 *>(a.ov + dst) = vv;
        if (g == 0 && part == 0) a.src[(size_t)c * a.n_vis + t] = code;
    }
}

__global__ __launch_bounds__(kThreads) void fill_kernel(uint32_t *p, size_t n_words) {
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n_words;
         i += (size_t)gridDim.x * kThreads)
        p[i] = 0u;
}

// ------------------------------------------------------------ dispatch

AttnKernels pick_attn(int D, int G, int dtype) {
    const bool bf16 = dtype == SPLICE_BF16;
    switch (D) {
    case 64: return bf16 ? attn_kernels_d64_bf16(G) : attn_kernels_d64_f32(G);
    case 128: return bf16 ? attn_kernels_d128_bf16(G) : attn_kernels_d128_f32(G);
    case 256: return bf16 ? attn_kernels_d256_bf16(G) : attn_kernels_d256_f32(G);
    default: return AttnKernels{nullptr, nullptr};
    }
}

void fill_mask(const splice_shape &sh, const splice_call &call, const int32_t *cell_LW, uint32_t *mask) {
    for (int i = 0; i < SPLICE_MAX_CELLS / 32; ++i) mask[i] = 0u;
    for (int c = 0; c < sh.n_cells; ++c)
        if (splice::cell_spliced(cell_LW, c, call.layer, call.step)) mask[c >> 5] |= 1u << (c & 31);
}

// Compute units of the current device and work groups of `kernel` (at
// `threads` threads) resident on each, asked of HIP once per device and
// kernel; zeros when HIP cannot tell, and the planner then groups the
// generated rows by their length alone.
splice::Residency residency(const void *kernel, int threads) {
    struct Entry {
        int dev;
        const void *kernel;
        splice::Residency res;
    };
    static std::mutex mu;
    static Entry cache[64];
    static int n_cache = 0;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return splice::Residency();
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < n_cache; ++i)
        if (cache[i].dev == dev && cache[i].kernel == kernel) return cache[i].res;
    splice::Residency res;
    int n_cu = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) == hipSuccess && n_cu > 0 &&
        per_cu > 0) {
        res.n_cu = n_cu;
        res.per_cu = per_cu;
    } else {
        (void)hipGetLastError();   // the call itself has not failed: clear what the queries left
    }
    if (n_cache < 64) cache[n_cache++] = Entry{dev, kernel, res};
    return res;
}

// Workspace bytes of `call` on `shape` (call == NULL: every default-split
// call).  With every_count the bytes cover any number of computed cells:
// a forked sweep plans over its diverged cells only, and by default fewer
// computed cells take more prompt chunks (with an explicit split_keys the
// chunks do not depend on them); without it, a call that computes every cell.
int64_t attn_workspace_bytes(const splice_shape *shape, const splice_call *call, bool every_count) {
    int32_t rc = splice::validate_shape(shape);
    if (rc != SPLICE_OK) return rc;
    int n_slots;
    if (call) {
        rc = splice::validate_call(*shape, call);
        if (rc != SPLICE_OK) return rc;
        const splice::Geometry geo = splice::geometry(*shape, *call);
        const int n_hi = shape->n_cells > 0 ? shape->n_cells : 1;
        const int n_lo = every_count && call->split_keys == 0 ? 1 : n_hi;
        n_slots = 0;
        for (int n = n_lo; n <= n_hi; ++n) {   // the slots do not depend on the cell split
            const int k = splice::plan_from_geo(*shape, *call, geo, 0, n).n_slots;
            n_slots = k > n_slots ? k : n_slots;
        }
        if (n_slots > splice::kMaxSlots) return SPLICE_EUNSUPPORTED;
    } else {
        n_slots = splice::worst_default_slots(*shape);
    }
    return (int64_t)splice::workspace_layout(*shape, n_slots).total;
}

int32_t launch_status() {
    const hipError_t err = hipGetLastError();
    return err == hipSuccess ? SPLICE_OK : SPLICE_EHIP;
}

}  // namespace

// ================================================================== C ABI

extern "C" {

int32_t splice_abi_version(void) { return SPLICE_ABI_VERSION; }

const char *splice_status_str(int32_t status) {
    switch (status) {
    case SPLICE_OK: return "ok";
    case SPLICE_EINVAL: return "invalid argument (NULL pointer, enum value, alignment)";
    case SPLICE_ESHAPE: return "inconsistent shape or call";
    case SPLICE_EWORKSPACE: return "workspace missing or too small";
    case SPLICE_EUNSUPPORTED: return "unsupported head_dim, group size or cell count";
    case SPLICE_EHIP: return "HIP launch failed";
    default: return "unknown status";
    }
}

int32_t splice_visible_len(const splice_shape *shape, const splice_call *call) {
    int32_t rc = splice::validate_shape(shape);
    if (rc != SPLICE_OK) return rc;
    rc = splice::validate_call(*shape, call);
    if (rc != SPLICE_OK) return rc;
    return splice::geometry(*shape, *call).n_vis;
}

int32_t splice_kv_build(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                        const void *clean_k, const void *clean_v, const void *donor_k,
                        const void *donor_v, const void *gen_k, const void *gen_v, void *out_k,
                        void *out_v, uint8_t *out_src, void *stream) {
    int32_t rc = splice::validate_shape(shape);
    if (rc != SPLICE_OK) return rc;
    const splice_shape &sh = *shape;
    rc = splice::validate_call(sh, call);
    if (rc != SPLICE_OK) return rc;
    rc = splice::validate_cells(sh, cell_LW);
    if (rc != SPLICE_OK) return rc;
    if (sh.n_cells == 0) return SPLICE_OK;
    const bool zero = sh.donor_kind == SPLICE_DONOR_ZERO;
    const bool has_prompt = sh.prompt_len > 0;   // an empty prompt has no prompt buffers to read
    if (!gen_k || !gen_v || !out_k || !out_v || !out_src) return SPLICE_EINVAL;
    if (has_prompt && (!clean_k || !clean_v)) return SPLICE_EINVAL;
    if (zero ? (donor_k || donor_v) : (has_prompt && (!donor_k || !donor_v))) return SPLICE_EINVAL;
    const void *ptrs[] = {clean_k, clean_v, gen_k, gen_v, out_k, out_v};
    for (const void *p : ptrs)
        if (!splice::aligned(p, 16)) return SPLICE_EINVAL;
    if (!zero && (!splice::aligned(donor_k, 16) || !splice::aligned(donor_v, 16))) return SPLICE_EINVAL;

    const splice::Geometry geo = splice::geometry(sh, *call);
    GatherArgs a;
    a.ck = (const char *)clean_k; a.cv = (const char *)clean_v;
    a.dk = (const char *)donor_k; a.dv = (const char *)donor_v;
    a.gk = (const char *)gen_k; a.gv = (const char *)gen_v;
    a.ok = (char *)out_k; a.ov = (char *)out_v; a.src = out_src;
    a.Hkv = sh.n_kv_heads; a.Tp = sh.prompt_len; a.cap = sh.gen_capacity;
    a.row_bytes = sh.head_dim * splice::elem_bytes(sh);
    a.zero_donor = zero ? 1 : 0;
    a.jp0 = geo.jp0; a.i0 = geo.i0; a.n_prompt = geo.n_prompt; a.n_vis = geo.n_vis;
    a.sa = geo.sa; a.sb = geo.sb;
    fill_mask(sh, *call, cell_LW, a.spliced);
    const int64_t units = (int64_t)geo.n_vis * (a.row_bytes / 16);
    int bx = (int)((units + kThreads - 1) / kThreads);
    if (bx > 1024) bx = 1024;
    dim3 grid(bx, sh.n_kv_heads, sh.n_cells);
    hipLaunchKernelGGL(gather_kernel, grid, dim3(kThreads), 0, (hipStream_t)stream, a);
    return launch_status();
}

int64_t splice_decode_attn_workspace_bytes(const splice_shape *shape, const splice_call *call) {
    return attn_workspace_bytes(shape, call, true);
}

int32_t splice_workspace_init(void *workspace, size_t workspace_bytes, void *stream) {
    if (!workspace || !splice::aligned(workspace, 256) || workspace_bytes % 4 != 0) return SPLICE_EINVAL;
    const size_t words = workspace_bytes / 4;
    if (words == 0) return SPLICE_OK;
    size_t blocks = (words + kThreads - 1) / kThreads;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, (hipStream_t)stream,
                       (uint32_t *)workspace, words);
    return launch_status();
}

int64_t splice_workspace_handovers(const void *workspace, size_t workspace_bytes, void *stream) {
    if (!workspace || !splice::aligned(workspace, 256)) return SPLICE_EINVAL;
    if (workspace_bytes < splice::kStatsBytes) return SPLICE_EWORKSPACE;
    int32_t count = 0;
    if (hipMemcpyAsync(&count, workspace, sizeof(count), hipMemcpyDeviceToHost, (hipStream_t)stream) != hipSuccess)
        return SPLICE_EHIP;
    if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return SPLICE_EHIP;
    return count;
}

}  // extern "C"

namespace {

// splice_decode_attn (cell_step == nullptr, trunk < 0: every cell at
// call->step), splice_decode_step (each cell at cell_step[c], k_new/v_new
// appended) and splice_decode_forked (trunk >= 0: cells that have not
// diverged from the trunk by call->step take its result).
int32_t decode_attn_impl(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                         const int32_t *cell_step, int trunk, const void *q, const void *k_new, const void *v_new,
                         const void *clean_k, const void *clean_v, const void *donor_k, const void *donor_v,
                         const void *gen_k, const void *gen_v, float *out, float *lse, void *workspace,
                         size_t workspace_bytes, void *stream) {
    int32_t rc = splice::validate_shape(shape);
    if (rc != SPLICE_OK) return rc;
    const splice_shape &sh = *shape;
    if (!call) return SPLICE_EINVAL;
    splice_call checked = *call;
    if (cell_step) checked.step = 0;   // a decode step takes each cell's own step
    rc = splice::validate_call(sh, &checked);
    if (rc != SPLICE_OK) return rc;
    rc = splice::validate_cells(sh, cell_LW);
    if (rc != SPLICE_OK) return rc;
    const bool ragged = cell_step != nullptr;
    if (ragged) {
        rc = splice::validate_steps(sh, cell_step);
        if (rc != SPLICE_OK) return rc;
    }
    if (sh.n_cells == 0) return SPLICE_OK;
    const bool zero = sh.donor_kind == SPLICE_DONOR_ZERO;
    const bool has_prompt = sh.prompt_len > 0;   // an empty prompt has no prompt buffers to read
    if (!q || !gen_k || !gen_v || !out || !lse) return SPLICE_EINVAL;
    if (ragged && (!k_new || !v_new)) return SPLICE_EINVAL;
    if (has_prompt && (!clean_k || !clean_v)) return SPLICE_EINVAL;
    if (zero ? (donor_k || donor_v) : (has_prompt && (!donor_k || !donor_v))) return SPLICE_EINVAL;
    const void *ptrs[] = {q, clean_k, clean_v, gen_k, gen_v};
    for (const void *p : ptrs)
        if (!splice::aligned(p, 16)) return SPLICE_EINVAL;
    if (!zero && (!splice::aligned(donor_k, 16) || !splice::aligned(donor_v, 16))) return SPLICE_EINVAL;
    if (!splice::aligned(out, 16) || !splice::aligned(lse, 4)) return SPLICE_EINVAL;
    if (ragged && (!splice::aligned(k_new, 16) || !splice::aligned(v_new, 16))) return SPLICE_EINVAL;
    const bool forked = trunk >= 0;
    if (forked && (trunk >= sh.n_cells || cell_LW[2 * trunk] < sh.n_layers)) return SPLICE_ESHAPE;
    if ((ragged || forked) && !splice::bf16_path(sh)) return SPLICE_EUNSUPPORTED;

    // a forked sweep's cell has diverged from the trunk once it has been
    // spliced at some layer, i.e. from step W_c on if L_c < n_layers
    auto diverged = [&](int c) {
        return c == trunk || (cell_LW[2 * c] < sh.n_layers && call->step >= cell_LW[2 * c + 1]);
    };
    // the steps of the call: one for every cell, each cell's own, or (forked)
    // the call's for diverged cells and none for the others
    auto step_of = [&](int c) {
        return ragged ? cell_step[c] : (forked && !diverged(c) ? -1 : call->step);
    };
    int s_min = INT32_MAX, s_max = -1, n_active = 0;
    for (int c = 0; c < sh.n_cells; ++c) {
        const int s = step_of(c);
        if (s < 0) continue;
        ++n_active;
        s_min = s < s_min ? s : s_min;
        s_max = s > s_max ? s : s_max;
    }
    if (n_active == 0) return SPLICE_OK;   // every cell finished
    splice_call lo_call = *call, hi_call = *call;
    lo_call.step = s_min;
    hi_call.step = s_max;
    const splice::Geometry g_lo = splice::geometry(sh, lo_call), g_hi = splice::geometry(sh, hi_call);
    // widest visible prompt (the smallest step) and longest generated part (the largest)
    splice::Geometry geo = g_hi;
    geo.jp0 = g_lo.jp0;
    geo.sa = g_lo.sa;
    geo.sb = g_lo.sb;
    geo.n_prompt = g_lo.n_prompt;
    geo.n_vis = geo.n_prompt + geo.n_gen;

    int n_clean = 0;
    uint32_t spliced[SPLICE_MAX_CELLS / 32] = {0};
    for (int c = 0; c < sh.n_cells; ++c) {
        const int s = step_of(c);
        if (s < 0) continue;
        if (splice::cell_spliced(cell_LW, c, call->layer, s))
            spliced[c >> 5] |= 1u << (c & 31);
        else
            ++n_clean;
    }
    const int G = splice::group_of(sh);
    const AttnKernels kern = pick_attn(sh.head_dim, G, sh.dtype);
    if (!kern.items) return SPLICE_EUNSUPPORTED;
    const int threads = splice::bf16_path(sh) ? 64 * splice::fused_waves(sh.head_dim) : kThreads;

    const splice::AttnPlan plan = splice::plan_from_geo(
        sh, hi_call, geo, n_clean, n_active,
        splice::bf16_path(sh) ? residency((const void *)kern.items, threads) : splice::Residency(),
        g_lo.n_gen == g_hi.n_gen);
    if (plan.n_slots > splice::kMaxSlots) return SPLICE_EUNSUPPORTED;
    const splice::WorkspaceLayout wl = splice::workspace_layout(sh, plan.n_slots);
    if (!workspace || !splice::aligned(workspace, 256)) return SPLICE_EWORKSPACE;
    if (workspace_bytes < wl.total) return SPLICE_EWORKSPACE;

    AttnArgs a;
    a.q = (const char *)q;
    a.ck = (const char *)clean_k; a.cv = (const char *)clean_v;
    a.dk = (const char *)donor_k; a.dv = (const char *)donor_v;
    a.gk = (const char *)gen_k; a.gv = (const char *)gen_v;
    a.kn = (const char *)k_new; a.vn = (const char *)v_new;
    a.out = out; a.lse = lse;
    a.counters = (int *)((char *)workspace + wl.counters_off);
    a.stats = (int *)((char *)workspace + wl.stats_off);
    a.part = (float *)((char *)workspace + wl.part_off);
    if (wl.part_bytes >= ((size_t)1 << 31)) return SPLICE_EUNSUPPORTED;
    a.part_bytes = (uint32_t)(wl.part_bytes > 0 ? wl.part_bytes : 16);
    a.C = sh.n_cells; a.Hq = sh.n_q_heads; a.Hkv = sh.n_kv_heads; a.Tp = sh.prompt_len;
    a.cap = sh.gen_capacity;
    a.jp0 = geo.jp0; a.i0 = geo.i0; a.n_gen = geo.n_gen; a.sa = geo.sa; a.sb = geo.sb;
    a.zero_donor = zero ? 1 : 0;
    a.n_p = plan.n_p; a.p_len = plan.p_len; a.n_g = plan.n_g; a.g_len = plan.g_len;
    a.n_slots = plan.n_slots;
    // prompt slots [C][Hkv][n_p], then generated-row slots [C][Hkv][n_g]
    a.p_slot_bytes = (uint32_t)splice::prompt_slot_bytes(sh);
    a.g_slot_bytes = (uint32_t)splice::slot_floats(G, sh.head_dim) * 4u;
    a.gen_base = (uint32_t)((int64_t)sh.n_cells * sh.n_kv_heads * plan.n_p * a.p_slot_bytes);
    a.n_rb = 0; a.n_rg_clean = 0;
    a.n_prompt_items = plan.n_prompt_items;
    a.gen_pairs = plan.gen_pairs;
    a.gen_v_nt = splice::gen_v_nontemporal(sh, geo.n_gen) ? 1 : 0;
    a.wait_polls = call->merge_wait == 0 ? kDefaultWaitPolls : (call->merge_wait < 0 ? 0 : call->merge_wait);
    a.qk_scale = call->scale * kLog2e;
    a.ragged = ragged || forked ? 1 : 0;
    a.trunk = forked ? trunk : -1;
    a.window = call->window;
    a.span_lo = sh.span_lo; a.span_hi = sh.span_hi;
    a.row_lo = ragged && g_lo.jp0 != g_hi.jp0 ? 1 : 0;
    for (int i = 0; i < SPLICE_MAX_CELLS / 32; ++i) a.spliced[i] = spliced[i];
    for (int c = 0; c < SPLICE_MAX_CELLS; ++c) a.cstep[c] = c < sh.n_cells ? step_of(c) : -1;
    // row-block order: active clean cells first, then active spliced cells (each by index)
    int n = 0;
    for (int c = 0; c < sh.n_cells; ++c)
        if (step_of(c) >= 0 && !(spliced[c >> 5] >> (c & 31) & 1u)) a.order[n++] = (uint8_t)c;
    a.n_clean = n;
    for (int c = 0; c < sh.n_cells; ++c)
        if (step_of(c) >= 0 && (spliced[c >> 5] >> (c & 31) & 1u)) a.order[n++] = (uint8_t)c;
    a.n_active = n;
    a.n_dormant = 0;
    if (forked) {   // then the cells that take the trunk's result
        for (int c = 0; c < sh.n_cells; ++c)
            if (step_of(c) < 0) a.order[n++] = (uint8_t)c;
        a.n_dormant = n - a.n_active;
    }
    for (int c = 0; c < SPLICE_MAX_CELLS; ++c) a.wfork[c] = forked && c < sh.n_cells ? cell_LW[2 * c + 1] : 0;
    // generated-row items serve the cells with rows to stream (active, and
    // diverged under a forked sweep), longest generated part first
    {
        int gen_len[SPLICE_MAX_CELLS];
        int n_gc = 0;
        for (int c = 0; c < sh.n_cells; ++c) {
            const int s = step_of(c);
            if (s < 0) continue;
            splice_call cc = *call;
            cc.step = s;
            gen_len[c] = splice::geometry(sh, cc).n_gen;
            a.gorder[n_gc++] = (uint8_t)c;
        }
        std::stable_sort(a.gorder, a.gorder + n_gc,
                         [&](uint8_t x, uint8_t y) { return gen_len[x] > gen_len[y]; });
        a.n_gen_cells = n_gc;
        for (int i = n_gc; i < SPLICE_MAX_CELLS; ++i) a.gorder[i] = 0;
    }
    for (; n < SPLICE_MAX_CELLS; ++n) a.order[n] = 0;
    if (splice::bf16_path(sh)) {
        a.n_rb = splice::row_groups(sh, a.n_clean, a.n_active);
        a.n_rg_clean = splice::clean_row_groups(sh, a.n_clean);
    }

    if (plan.cellwise) {
        hipLaunchKernelGGL(kern.cellwise, dim3((unsigned)(sh.n_cells * sh.n_kv_heads)), dim3(kThreads), 0,
                           (hipStream_t)stream, a);
        return launch_status();
    }
    const int64_t items = (int64_t)plan.n_prompt_items + plan.n_gen_items;
    if (items > INT32_MAX) return SPLICE_EUNSUPPORTED;
    hipLaunchKernelGGL(kern.items, dim3((unsigned)items), dim3((unsigned)threads), 0, (hipStream_t)stream, a);
    return launch_status();
}

}  // namespace

extern "C" {

int32_t splice_decode_attn(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                           const void *q, const void *clean_k, const void *clean_v,
                           const void *donor_k, const void *donor_v, const void *gen_k,
                           const void *gen_v, float *out, float *lse, void *workspace,
                           size_t workspace_bytes, void *stream) {
    return decode_attn_impl(shape, call, cell_LW, nullptr, -1, q, nullptr, nullptr, clean_k, clean_v, donor_k,
                            donor_v, gen_k, gen_v, out, lse, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {

// The allocation-free entry point's workspace: one array per GPU, held until
// the process ends.  In host code `scratch` is only a stand-in for the
// symbol; its device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) char scratch[SPLICE_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` on each device, set once

// The current device's scratch array.  The first call on a device takes its
// address and clears it with the fill kernel on `stream` (the arrival
// counters must start at zero; every call re-arms the counters it used, so
// the array is left zeroed for the next call).
int32_t device_scratch(void *stream, void **ptr) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SPLICE_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SPLICE_EHIP;
        const size_t words = SPLICE_NOALLOC_WORKSPACE_BYTES / 4;
        hipLaunchKernelGGL(fill_kernel, dim3(4096), dim3(kThreads), 0, (hipStream_t)stream, (uint32_t *)p, words);
        if (hipGetLastError() != hipSuccess) return SPLICE_EHIP;
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return SPLICE_OK;
}

}  // namespace

extern "C" {

int32_t splice_decode_attn_noalloc(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                                   const void *q, const void *clean_k, const void *clean_v, const void *donor_k,
                                   const void *donor_v, const void *gen_k, const void *gen_v, float *out, float *lse,
                                   void *stream) {
    // validation and the size check come first: a call that does not fit is
    // rejected before any device work
    const int64_t need = attn_workspace_bytes(shape, call, false);   // every cell is computed
    if (need < 0) return (int32_t)need;
    if (need > (int64_t)SPLICE_NOALLOC_WORKSPACE_BYTES) return SPLICE_EWORKSPACE;
    void *ws = nullptr;
    const int32_t rc = device_scratch(stream, &ws);
    if (rc != SPLICE_OK) return rc;
    return decode_attn_impl(shape, call, cell_LW, nullptr, -1, q, nullptr, nullptr, clean_k, clean_v, donor_k,
                            donor_v, gen_k, gen_v, out, lse, ws, SPLICE_NOALLOC_WORKSPACE_BYTES, stream);
}

int32_t splice_decode_step(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                           const int32_t *cell_step, const void *q, const void *k_new, const void *v_new,
                           const void *clean_k, const void *clean_v, const void *donor_k,
                           const void *donor_v, void *gen_k, void *gen_v, float *out, float *lse,
                           void *workspace, size_t workspace_bytes, void *stream) {
    if (!cell_step && shape && shape->n_cells > 0) return SPLICE_EINVAL;
    return decode_attn_impl(shape, call, cell_LW, cell_step, -1, q, k_new, v_new, clean_k, clean_v, donor_k,
                            donor_v, gen_k, gen_v, out, lse, workspace, workspace_bytes, stream);
}

int32_t splice_decode_forked(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                             int32_t trunk, const void *q, const void *clean_k, const void *clean_v,
                             const void *donor_k, const void *donor_v, const void *gen_k, const void *gen_v,
                             float *out, float *lse, void *workspace, size_t workspace_bytes, void *stream) {
    if (shape && shape->n_cells > 0 && trunk < 0) return SPLICE_EINVAL;
    if (shape && shape->n_cells == 0) trunk = -1;
    return decode_attn_impl(shape, call, cell_LW, nullptr, trunk, q, nullptr, nullptr, clean_k, clean_v, donor_k,
                            donor_v, gen_k, gen_v, out, lse, workspace, workspace_bytes, stream);
}

}  // extern "C"
