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
//   attn_kernel     splice_decode_attn: one work item = (cell, KV head,
//                   chunk of the cell's key list).  Lanes stream K/V rows
//                   from HBM with coalesced 16-byte loads, D/16 lanes per
//                   row; q.k uses v_dot2_f32_bf16 and a DPP butterfly inside
//                   the row group; every row group keeps its own online
//                   softmax state (max, sum, weighted V) for the G query
//                   heads of the KV head.  States merge across row groups
//                   (lane shuffles) and waves (LDS).  A cell whose list fits
//                   one chunk is finished here; otherwise the item writes a
//                   partial (m, l, o) to the workspace.
//   combine_kernel  merges the partials of each (cell, KV head) with a
//                   log-sum-exp combine in chunk order, adds the ZERO
//                   donor's closed-form term and writes out/lse.  It is a
//                   separate launch: the kernel boundary makes the partials
//                   visible across XCDs without device-scope fences, whose
//                   L2 write-back and invalidate cost every other work item
//                   its cached prompt tiles.
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

#include "plan.hpp"
#include "splice_attn.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

// Sum over the LPK consecutive lanes of a row group (LPK in {4, 8, 16}), every
// lane of the group ending with the same bits.  DPP: quad_perm [1,0,3,2],
// quad_perm [2,3,0,1], row_half_mirror, row_mirror.
template <int LPK>
__device__ __forceinline__ float group_sum(float x) {
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));
    if constexpr (LPK >= 8)
        x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, false));
    if constexpr (LPK >= 16)
        x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xF, 0xF, false));
    return x;
}

// 2^x with v_exp_f32 (results below 2^-126 flush to zero: negligible weights).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bool bit_set(const uint32_t *mask, int c) {
    return (mask[c >> 5] >> (c & 31)) & 1u;
}

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
        const char *kb = nullptr, *vb = nullptr;
        size_t off;
        if (t < a.n_prompt) {
            const int j = a.jp0 + t;
            const bool in_span = j >= a.sa && j < a.sb;
            off = ((size_t)g * a.Tp + j) * a.row_bytes;
            if (spl && in_span) {
                code = a.zero_donor ? SPLICE_SRC_ZERO : SPLICE_SRC_DONOR;
                if (!a.zero_donor) { kb = a.dk; vb = a.dv; }
            } else {
                code = SPLICE_SRC_CLEAN;
                kb = a.ck; vb = a.cv;
            }
        } else {
            const int i = a.i0 + (t - a.n_prompt);
            off = (((size_t)c * a.Hkv + g) * a.cap + i) * a.row_bytes;
            code = SPLICE_SRC_GEN;
            kb = a.gk; vb = a.gv;
        }
        uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
        if (kb) {
            kv = *reinterpret_cast<const uint4 *>(kb + off + (size_t)part * 16);
            vv = *reinterpret_cast<const uint4 *>(vb + off + (size_t)part * 16);
        }
        const size_t dst = out_base + (size_t)t * a.row_bytes + (size_t)part * 16;
        *reinterpret_cast<uint4 *>(a.ok + dst) = kv;
        *reinterpret_cast<uint4 *>(a.ov + dst) = vv;
        if (g == 0 && part == 0) a.src[(size_t)c * a.n_vis + t] = code;
    }
}

// --------------------------------------------------------------- attention

struct AttnArgs {
    const void *q;
    const char *ck, *cv, *dk, *dv, *gk, *gv;
    float *out, *lse;
    float *part;
    int Hq, Hkv, Tp, cap, step;
    int jp0, i0, sa, sb, n_gen;
    int zero_donor;
    int split, max_chunks, slot_floats;
    float qk_scale;   // scale * log2(e)
    uint32_t spliced[SPLICE_MAX_CELLS / 32];
};

// Length of cell c's key list: visible prompt slots (without the ZERO slots of
// a spliced cell, which never enter the list) plus visible generated rows.
__device__ __forceinline__ int list_len(const AttnArgs &a, int c) {
    const bool zskip = a.zero_donor && bit_set(a.spliced, c);
    return (a.Tp - a.jp0) - (zskip ? a.sb - a.sa : 0) + a.n_gen;
}

// Lane layout for one K/V row of D elements (EB bytes each):
//   LPK = D / 16 lanes per row ("row group"), KPW = 64 / LPK rows per wave;
//   lane lj of a row group owns NP = EB pieces of 16 bytes at byte offsets
//   p * (D * EB / NP) + lj * 16, i.e. 16 elements.  Each load instruction
//   of a wave reads KPW rows x D bytes, fully coalesced.
template <int D, int G, bool BF16>
__global__ __launch_bounds__(kThreads) void attn_kernel(AttnArgs a) {
    constexpr int EB = BF16 ? 2 : 4;
    constexpr int LPK = D / 16;
    constexpr int KPW = 64 / LPK;
    constexpr int NP = EB;
    constexpr int EPP = 16 / EB;            // elements per piece
    constexpr int PIECE_STRIDE = D * EB / NP;
    constexpr int ROW_BYTES = D * EB;
    constexpr int U = (BF16 && G <= 4) ? 4 : 2;   // rows per row group per iteration
    constexpr int QW = BF16 ? 8 : 16;             // q registers per head per lane

    __shared__ float s_o[kWaves][G][D];
    __shared__ float s_m[kWaves][G];
    __shared__ float s_l[kWaves][G];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lj = lane % LPK, rg = lane / LPK;

    int item = blockIdx.x;
    const int ch = item % a.max_chunks;
    item /= a.max_chunks;
    const int g = item % a.Hkv;
    const int c = item / a.Hkv;

    const bool spl = bit_set(a.spliced, c);
    const bool zskip = spl && a.zero_donor;
    const int nsv = a.sb - a.sa;
    const int n_prompt = (a.Tp - a.jp0) - (zskip ? nsv : 0);
    const int n_list = n_prompt + a.n_gen;
    const int n_chunks = (n_list + a.split - 1) / a.split;
    if (ch >= n_chunks) return;
    const int kbeg = ch * a.split;
    const int kend = min(kbeg + a.split, n_list);

    // q of the G heads of KV head g, this lane's 16 elements each
    uint32_t qr[G][QW];
    {
        const char *qb = reinterpret_cast<const char *>(a.q) +
                         ((size_t)c * a.Hq + (size_t)g * G) * ROW_BYTES;
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                const uint4 w = *reinterpret_cast<const uint4 *>(qb + (size_t)h * ROW_BYTES +
                                                                 p * PIECE_STRIDE + lj * 16);
                qr[h][p * 4 + 0] = w.x; qr[h][p * 4 + 1] = w.y;
                qr[h][p * 4 + 2] = w.z; qr[h][p * 4 + 3] = w.w;
            }
    }

    const size_t prompt_off = (size_t)g * a.Tp * ROW_BYTES;
    const char *ckb = a.ck + prompt_off, *cvb = a.cv + prompt_off;
    const char *dkb = a.zero_donor ? ckb : a.dk + prompt_off;
    const char *dvb = a.zero_donor ? cvb : a.dv + prompt_off;
    const size_t gen_off = ((size_t)c * a.Hkv + g) * (size_t)a.cap * ROW_BYTES;
    const char *gkb = a.gk + gen_off, *gvb = a.gv + gen_off;

    // online softmax state of this row group (identical in its LPK lanes)
    float m[G], l[G], o[G][16];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) o[h][e] = 0.f;
    }

    for (int base = kbeg + wave * (U * KPW); base < kend; base += kWaves * U * KPW) {
        uint4 kr[U][NP], vr[U][NP];
        bool valid[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int v = base + u * KPW + rg;
            valid[u] = v < kend;
            if (!valid[u]) v = kbeg;   // a row that exists; its score is masked below
            const char *kp, *vp;
            if (v < n_prompt) {
                int j = v + a.jp0;
                if (zskip && j >= a.sa) j += nsv;
                const bool from_donor = spl && j >= a.sa && j < a.sb;
                const size_t off = (size_t)j * ROW_BYTES;
                kp = (from_donor ? dkb : ckb) + off;
                vp = (from_donor ? dvb : cvb) + off;
            } else {
                const size_t off = (size_t)(a.i0 + (v - n_prompt)) * ROW_BYTES;
                kp = gkb + off;
                vp = gvb + off;
            }
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                kr[u][p] = *reinterpret_cast<const uint4 *>(kp + p * PIECE_STRIDE + lj * 16);
                vr[u][p] = *reinterpret_cast<const uint4 *>(vp + p * PIECE_STRIDE + lj * 16);
            }
        }

        float s[U][G];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int h = 0; h < G; ++h) {
                float acc = 0.f;
#pragma unroll
                for (int p = 0; p < NP; ++p) {
                    const uint32_t kw[4] = {kr[u][p].x, kr[u][p].y, kr[u][p].z, kr[u][p].w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if constexpr (BF16) {
                            acc = dot2_bf16(qr[h][p * 4 + i], kw[i], acc);
                        } else {
                            acc = fmaf(__uint_as_float(qr[h][p * 4 + i]), __uint_as_float(kw[i]), acc);
                        }
                    }
                }
                acc = group_sum<LPK>(acc) * a.qk_scale;
                s[u][h] = valid[u] ? acc : -INFINITY;
            }

        // values of this lane's 16 elements for the U rows
        float vf[U][16];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                const uint32_t vw[4] = {vr[u][p].x, vr[u][p].y, vr[u][p].z, vr[u][p].w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if constexpr (BF16) {
                        vf[u][p * EPP + 2 * i] = bf16_lo(vw[i]);
                        vf[u][p * EPP + 2 * i + 1] = bf16_hi(vw[i]);
                    } else {
                        vf[u][p * EPP + i] = __uint_as_float(vw[i]);
                    }
                }
            }

#pragma unroll
        for (int h = 0; h < G; ++h) {
            float mx = m[h];
#pragma unroll
            for (int u = 0; u < U; ++u) mx = fmaxf(mx, s[u][h]);
            const float ms = mx == -INFINITY ? 0.f : mx;
            const float alpha = fast_exp2(m[h] - ms);
            l[h] *= alpha;
#pragma unroll
            for (int e = 0; e < 16; ++e) o[h][e] *= alpha;
            m[h] = mx;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float pw = fast_exp2(s[u][h] - ms);
                l[h] += pw;
#pragma unroll
                for (int e = 0; e < 16; ++e) o[h][e] = fmaf(pw, vf[u][e], o[h][e]);
            }
        }
    }

    // merge the KPW row-group states of this wave (butterfly over lanes)
#pragma unroll
    for (int off = LPK; off < 64; off <<= 1) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float mo = __shfl_xor(m[h], off);
            const float lo = __shfl_xor(l[h], off);
            const float mx = fmaxf(m[h], mo);
            const float ms = mx == -INFINITY ? 0.f : mx;
            const float fa = fast_exp2(m[h] - ms), fb = fast_exp2(mo - ms);
            l[h] = l[h] * fa + lo * fb;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float oo = __shfl_xor(o[h][e], off);
                o[h][e] = o[h][e] * fa + oo * fb;
            }
            m[h] = mx;
        }
    }
    if (rg == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
#pragma unroll
            for (int p = 0; p < NP; ++p)
#pragma unroll
                for (int i = 0; i < EPP; ++i)
                    s_o[wave][h][p * (D / NP) + lj * EPP + i] = o[h][p * EPP + i];
            if (lj == 0) {
                s_m[wave][h] = m[h];
                s_l[wave][h] = l[h];
            }
        }
    }
    __syncthreads();

    // merge the waves; a single-chunk list finishes here, otherwise the
    // work item writes its partial slot
    const bool zero_term = zskip && nsv > 0;
    const int row0 = c * a.Hq + g * G;
    float *slot_base = a.part + ((size_t)(c * a.Hkv + g) * a.max_chunks) * a.slot_floats;
    for (int e = tid; e < G * D; e += kThreads) {
        const int h = e / D, d = e % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][h]);
        const float Ms = M == -INFINITY ? 0.f : M;
        float L = 0.f, O = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float f = fast_exp2(s_m[w][h] - Ms);
            L = fmaf(s_l[w][h], f, L);
            O = fmaf(s_o[w][h][d], f, O);
        }
        if (n_chunks == 1) {
            if (zero_term) {
                const float Mz = fmaxf(M, 0.f);
                const float f = fast_exp2(M - Mz);
                L = L * f + (float)nsv * fast_exp2(-Mz);
                O *= f;
                M = Mz;
            }
            a.out[(size_t)(row0 + h) * D + d] = O / L;
            if (d == 0) a.lse[row0 + h] = (M + log2f(L)) * kLn2;
        } else {
            float *slot = slot_base + (size_t)ch * a.slot_floats;
            slot[h * D + d] = O;
            if (d == 0) {
                slot[G * D + h] = M;
                slot[G * D + G + h] = L;
            }
        }
    }
}

// Merge the partials of one (cell, KV head) in chunk order (grid: C * Hkv).
template <int D, int G>
__global__ __launch_bounds__(kThreads) void combine_kernel(AttnArgs a) {
    const int g = blockIdx.x % a.Hkv;
    const int c = blockIdx.x / a.Hkv;
    const int n_chunks = (list_len(a, c) + a.split - 1) / a.split;
    if (n_chunks <= 1) return;   // finished by the attention kernel
    const bool zero_term = a.zero_donor && bit_set(a.spliced, c) && a.sb > a.sa;
    const float nsv = (float)(a.sb - a.sa);
    const float *slot_base = a.part + ((size_t)(c * a.Hkv + g) * a.max_chunks) * a.slot_floats;
    const int row0 = c * a.Hq + g * G;
    for (int e = threadIdx.x; e < G * D; e += kThreads) {
        const int h = e / D, d = e % D;
        float M = zero_term ? 0.f : -INFINITY;
        for (int k = 0; k < n_chunks; ++k)
            M = fmaxf(M, slot_base[(size_t)k * a.slot_floats + G * D + h]);
        float L = zero_term ? nsv * fast_exp2(-M) : 0.f;
        float O = 0.f;
        for (int k = 0; k < n_chunks; ++k) {
            const float *slot = slot_base + (size_t)k * a.slot_floats;
            const float f = fast_exp2(slot[G * D + h] - M);
            L = fmaf(slot[G * D + G + h], f, L);
            O = fmaf(slot[h * D + d], f, O);
        }
        a.out[(size_t)(row0 + h) * D + d] = O / L;
        if (d == 0) a.lse[row0 + h] = (M + log2f(L)) * kLn2;
    }
}

__global__ __launch_bounds__(kThreads) void fill_kernel(uint32_t *p, size_t n_words) {
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n_words;
         i += (size_t)gridDim.x * kThreads)
        p[i] = 0u;
}

// ------------------------------------------------------------ dispatch

typedef void (*attn_fn)(AttnArgs);
struct AttnKernels {
    attn_fn attn, combine;
};

template <int D, int G, bool BF16>
AttnKernels kernels_of() {
    return AttnKernels{attn_kernel<D, G, BF16>, combine_kernel<D, G>};
}

template <int D, bool BF16>
AttnKernels pick_g(int G) {
    switch (G) {
    case 1: return kernels_of<D, 1, BF16>();
    case 2: return kernels_of<D, 2, BF16>();
    case 4: return kernels_of<D, 4, BF16>();
    case 8: return kernels_of<D, 8, BF16>();
    default: return AttnKernels{nullptr, nullptr};
    }
}

template <bool BF16>
AttnKernels pick_d(int D, int G) {
    switch (D) {
    case 64: return pick_g<64, BF16>(G);
    case 128: return pick_g<128, BF16>(G);
    case 256: return pick_g<256, BF16>(G);
    default: return AttnKernels{nullptr, nullptr};
    }
}

AttnKernels pick_attn(int D, int G, int dtype) {
    return dtype == SPLICE_BF16 ? pick_d<true>(D, G) : pick_d<false>(D, G);
}

void fill_mask(const splice_shape &sh, const splice_call &call, const int32_t *cell_LW, uint32_t *mask) {
    for (int i = 0; i < SPLICE_MAX_CELLS / 32; ++i) mask[i] = 0u;
    for (int c = 0; c < sh.n_cells; ++c)
        if (splice::cell_spliced(cell_LW, c, call.layer, call.step)) mask[c >> 5] |= 1u << (c & 31);
}

int plan_chunks(const splice_shape &sh, const splice_call &call, const splice::Geometry &geo, int *split) {
    *split = call.split_keys > 0 ? call.split_keys
                                 : splice::default_split(geo.n_vis, sh.n_cells, sh.n_kv_heads);
    return splice::ceil_div(geo.n_vis, *split);
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
    int32_t rc = splice::validate_shape(shape);
    if (rc != SPLICE_OK) return rc;
    int max_chunks;
    if (call) {
        rc = splice::validate_call(*shape, call);
        if (rc != SPLICE_OK) return rc;
        int split;
        max_chunks = plan_chunks(*shape, *call, splice::geometry(*shape, *call), &split);
    } else {
        max_chunks = splice::worst_default_chunks(*shape);
    }
    return (int64_t)splice::workspace_layout(*shape, max_chunks).total;
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

int32_t splice_decode_attn(const splice_shape *shape, const splice_call *call, const int32_t *cell_LW,
                           const void *q, const void *clean_k, const void *clean_v,
                           const void *donor_k, const void *donor_v, const void *gen_k,
                           const void *gen_v, float *out, float *lse, void *workspace,
                           size_t workspace_bytes, void *stream) {
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
    if (!q || !gen_k || !gen_v || !out || !lse) return SPLICE_EINVAL;
    if (has_prompt && (!clean_k || !clean_v)) return SPLICE_EINVAL;
    if (zero ? (donor_k || donor_v) : (has_prompt && (!donor_k || !donor_v))) return SPLICE_EINVAL;
    const void *ptrs[] = {q, clean_k, clean_v, gen_k, gen_v};
    for (const void *p : ptrs)
        if (!splice::aligned(p, 16)) return SPLICE_EINVAL;
    if (!zero && (!splice::aligned(donor_k, 16) || !splice::aligned(donor_v, 16))) return SPLICE_EINVAL;
    if (!splice::aligned(out, 4) || !splice::aligned(lse, 4)) return SPLICE_EINVAL;

    const splice::Geometry geo = splice::geometry(sh, *call);
    int split;
    const int max_chunks = plan_chunks(sh, *call, geo, &split);
    const splice::WorkspaceLayout wl = splice::workspace_layout(sh, max_chunks);
    if (!workspace || !splice::aligned(workspace, 256)) return SPLICE_EWORKSPACE;
    if (workspace_bytes < wl.total) return SPLICE_EWORKSPACE;

    const int G = splice::group_of(sh);
    const AttnKernels kern = pick_attn(sh.head_dim, G, sh.dtype);
    if (!kern.attn) return SPLICE_EUNSUPPORTED;

    AttnArgs a;
    a.q = q;
    a.ck = (const char *)clean_k; a.cv = (const char *)clean_v;
    a.dk = (const char *)donor_k; a.dv = (const char *)donor_v;
    a.gk = (const char *)gen_k; a.gv = (const char *)gen_v;
    a.out = out; a.lse = lse;
    a.part = (float *)((char *)workspace + wl.part_off);
    a.Hq = sh.n_q_heads; a.Hkv = sh.n_kv_heads; a.Tp = sh.prompt_len; a.cap = sh.gen_capacity;
    a.step = call->step;
    a.jp0 = geo.jp0; a.i0 = geo.i0; a.sa = geo.sa; a.sb = geo.sb; a.n_gen = geo.n_gen;
    a.zero_donor = zero ? 1 : 0;
    a.split = split;
    a.max_chunks = max_chunks;
    a.slot_floats = splice::slot_floats(G, sh.head_dim);
    a.qk_scale = call->scale * kLog2e;
    fill_mask(sh, *call, cell_LW, a.spliced);

    const int64_t items = (int64_t)sh.n_cells * sh.n_kv_heads * max_chunks;
    if (items > INT32_MAX) return SPLICE_EUNSUPPORTED;
    hipLaunchKernelGGL(kern.attn, dim3((unsigned)items), dim3(kThreads), 0, (hipStream_t)stream, a);
    if (max_chunks > 1)
        hipLaunchKernelGGL(kern.combine, dim3((unsigned)(sh.n_cells * sh.n_kv_heads)), dim3(kThreads), 0,
                           (hipStream_t)stream, a);
    return launch_status();
}

}  // extern "C"
