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
//   attn_kernel     splice_decode_attn, one launch per call, two kinds of
//                   work item in one grid:
//     prompt items  (KV head, 64 rows, prompt chunk): the rows are the
//                   (cell, q head) pairs of all cells, clean cells first.
//                   Each 64-key tile of the clean (and, for spliced rows,
//                   the donor) prompt cache is staged in LDS once -- K
//                   row-major, V transposed -- and feeds all 64 rows through
//                   v_mfma_f32_16x16x32_bf16 for q.k and p.v.  (f32 inputs
//                   take a per-cell vector-ALU variant.)
//     generated items (cell, KV head, chunk of generated rows): lanes stream
//                   the cell's own rows with coalesced 16-byte loads, D/16
//                   lanes per row, v_dot2_f32_bf16 and a DPP butterfly for
//                   q.k, per-row-group online softmax with lazy rescaling.
//                   Generated rows are never spliced and are read once.
//     Each item stores one partial (m, l, o) per row it serves; the last item
//     of a (cell, KV head) to finish -- found with a device-scope counter --
//     merges the partials and writes out and lse.
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

#include <type_traits>

#include "plan.hpp"
#include "splice_attn.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
using splice::kMaxSlots;
using splice::kRowBlock;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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
    // update_dpp with old = 0 lets the compiler fold each move into v_add_f32_dpp
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
    if constexpr (LPK >= 8)
        x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));
    if constexpr (LPK >= 16)
        x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));
    return x;
}

// x + (x of the lane r places further on in its 16-lane DPP row), r in {4, 8}.
template <int R>
__device__ __forceinline__ float add_row_ror(float x) {
    return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x120 + R, 0xF, 0xF, false));
}

// 2^x with v_exp_f32 (results below 2^-126 flush to zero: negligible weights).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bool bit_set(const uint32_t *mask, int c) {
    return (mask[c >> 5] >> (c & 31)) & 1u;
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E), so
// register arrays are only ever indexed by constants.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
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
    const char *q;
    const char *ck, *cv, *dk, *dv, *gk, *gv;
    float *out, *lse, *part;
    int *counters;
    uint32_t part_bytes;   // size of the partial-result region (< 2^31)
    int C, Hq, Hkv, Tp, cap;
    int jp0, i0, n_gen, sa, sb;
    int zero_donor;
    int n_p, p_len, n_g, g_len, n_slots, slot_floats;
    int n_rb, n_prompt_items, n_clean;
    float qk_scale;   // scale * log2(e)
    uint32_t spliced[SPLICE_MAX_CELLS / 32];
    uint8_t order[SPLICE_MAX_CELLS];   // clean cells, then spliced cells
};

// Lazy rescaling: a running maximum is only raised when a score exceeds it
// by more than this many powers of two, so weights stay <= 2^kSlack and the
// rescale of the accumulators is rare.  The result is exact either way: a
// partial result only needs its (m, l, o) to share one reference m.
constexpr float kSlack = 8.f;

// Partial results are written and read with the sc1 cache policy -- the
// policy of agent-scope atomics: a store is written through to the device
// coherence point before it counts as performed, and a load is served from
// there rather than from a possibly stale L2 line of another XCD.  They go
// through one buffer descriptor over the partial region (16-byte accesses;
// dword 3 = 0x00020000 is the gfx9-family raw-buffer format).
constexpr int kSc1 = 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t part_rsrc(const AttnArgs &a) {
    return __builtin_amdgcn_make_buffer_rsrc(a.part, 0, a.part_bytes, 0x00020000);
}
__device__ __forceinline__ void part_store4(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4_t v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kSc1);
}
__device__ __forceinline__ void part_store1(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, kSc1);
}
__device__ __forceinline__ f32x4_t part_load4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kSc1));
}
__device__ __forceinline__ float part_load1(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSc1));
}

// ---------------------------------------------------------- vector-ALU rows
//
// Streams K/V rows for the G query heads of one KV head on the vector ALUs.
// A row of D elements is cut into 16-byte pieces; LPK = D / 16 lanes share a
// row (a "row group") and lane lj owns the NP pieces at byte offsets
// p * LPK * 16 + lj * 16 (16 elements in all), so each load instruction of a
// wave covers whole rows.  A row group takes U consecutive rows per
// iteration.  q.k: v_dot2_f32_bf16 over the lane's
// elements, then a DPP butterfly inside the row group.  The running maximum
// of each head is wave-uniform (row groups combine with DPP, ds_swizzle and
// readlane), so row groups never rescale against each other and the rescale
// is a scalar branch; at the end their (l, o) are plain sums.
template <int D, int G, bool BF16>
struct Valu {
    static constexpr int EB = BF16 ? 2 : 4;
    static constexpr int EPP = 16 / EB;                        // elements per piece
    static constexpr int LPK = D / 16;                         // lanes per row: 16 elements each
    static constexpr int NP = EB;                              // pieces per lane
    static constexpr int EL = 16;                              // elements per lane
    static constexpr int KPW = 64 / LPK;                       // row groups per wave
    static constexpr int RGR = 16 / LPK;                       // row groups per 16-lane DPP row
    static constexpr int ROW = D * EB;
    static constexpr int PSTRIDE = LPK * 16;
    static constexpr int U = 4;
    static constexpr int QW = NP * 4;                          // q dwords per head per lane
    // element index of piece p, element e of lane lj
    static __device__ __forceinline__ int elem(int lj, int p, int e) { return p * LPK * EPP + lj * EPP + e; }
};

// LDS budget of one work group.
template <int D, int G, bool BF16>
struct Lds {
    static constexpr int KT = 64;                  // keys per staged prompt tile
    static constexpr int KROW = D * 2 + 16;        // K tile row stride (bytes), padded
    static constexpr int VROW = KT * 2 + 8;        // V^T tile row stride (bytes), padded
    static constexpr int TILES = BF16 ? KT * KROW + D * VROW : 0;
    static constexpr int MERGE = kWaves * 4 * G * (D + 1) * 4 + kWaves * G * 4;
    static constexpr int STAGE = 2 * kMaxSlots * kRowBlock * 4;
    static constexpr int BYTES = TILES > MERGE ? (TILES > STAGE ? TILES : STAGE)
                                               : (MERGE > STAGE ? MERGE : STAGE);
};

// Maximum over the row groups of a wave of a value that is the same in all
// lanes of a row group; the result is wave-uniform.
template <int LPK>
__device__ __forceinline__ float wave_max_rows(float x) {
    // row groups of a 16-lane DPP row (rotations keep a max all-reduce exact)
    if constexpr (LPK <= 4)
        x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false)));
    if constexpr (LPK <= 8)
        x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false)));
    x = fmaxf(x, __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x401F)));   // lane ^ 16
    return fmaxf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0)),
                 __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32)));
}

template <int D, int G, bool BF16>
__device__ __forceinline__ void load_q(const AttnArgs &a, int c, int g, uint32_t (&qr)[G][Valu<D, G, BF16>::QW]) {
    using V = Valu<D, G, BF16>;
    const int lj = (threadIdx.x & 63) % V::LPK;
    const char *qb = a.q + ((size_t)c * a.Hq + (size_t)g * G) * V::ROW;
    static_for<0, G>([&](auto h) {
        static_for<0, V::NP>([&](auto p) {
            const u32x4_t w = *reinterpret_cast<const u32x4_t *>(qb + (size_t)h * V::ROW + p * V::PSTRIDE + lj * 16);
            static_for<0, 4>([&](auto i) { qr[h][p * 4 + i] = w[(int)i]; });
        });
    });
}

// row_of(key, &k_row, &v_row) -> false if the key is not to be attended
// (its pointers must still be readable).  m is wave-uniform on return.
template <int D, int G, bool BF16, class RowFn>
__device__ __forceinline__ void valu_stream(const uint32_t (&qr)[G][Valu<D, G, BF16>::QW], int kbeg, int kend,
                                            float qk_scale, RowFn row_of, float (&m)[G], float (&l)[G],
                                            float (&o)[G][Valu<D, G, BF16>::EL]) {
    using V = Valu<D, G, BF16>;
    constexpr int U = V::U;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lj = lane % V::LPK, rg = lane / V::LPK;
    static_for<0, G>([&](auto h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
        static_for<0, V::EL>([&](auto e) { o[h][e] = 0.f; });
    });
    for (int base = kbeg + wave * (V::KPW * U); base < kend; base += kWaves * V::KPW * U) {
        const int kf = base + rg * U;
        u32x4_t kr[U][V::NP], vr[U][V::NP];
        bool ok[U];
        static_for<0, U>([&](auto u) {
            const int key = kf + u;
            const bool inr = key < kend;
            const char *kp;
            const char *vp;
            const bool use = row_of(inr ? key : kend - 1, kp, vp);
            ok[u] = inr && use;
            static_for<0, V::NP>([&](auto p) {
                kr[u][p] = *reinterpret_cast<const u32x4_t *>(kp + p * V::PSTRIDE + lj * 16);
                vr[u][p] = *reinterpret_cast<const u32x4_t *>(vp + p * V::PSTRIDE + lj * 16);
            });
        });
        float s[U][G];
        static_for<0, U>([&](auto u) {
            static_for<0, G>([&](auto h) {
                float acc = 0.f;
                static_for<0, V::NP>([&](auto p) {
                    static_for<0, 4>([&](auto i) {
                        if constexpr (BF16)
                            acc = dot2_bf16(qr[h][p * 4 + i], kr[u][p][(int)i], acc);
                        else
                            acc = fmaf(__uint_as_float(qr[h][p * 4 + i]), __uint_as_float(kr[u][p][(int)i]), acc);
                    });
                });
                acc = group_sum<V::LPK>(acc) * qk_scale;
                s[u][h] = ok[u] ? acc : -INFINITY;
            });
        });
        float mt[G];
        bool need = false;
        static_for<0, G>([&](auto h) {
            float x = s[0][h];
            static_for<1, U>([&](auto u) { x = fmaxf(x, s[u][h]); });
            mt[h] = wave_max_rows<V::LPK>(x);
            need |= mt[h] > m[h] + kSlack;
        });
        if (need) {   // wave-uniform
            static_for<0, G>([&](auto h) {
                const float mn = fmaxf(m[h], mt[h]);
                const float al = fast_exp2(m[h] - (mn == -INFINITY ? 0.f : mn));
                l[h] *= al;
                static_for<0, V::EL>([&](auto e) { o[h][e] *= al; });
                m[h] = mn;
            });
        }
        float pw[U][G];
        static_for<0, G>([&](auto h) {
            const float ms = m[h] == -INFINITY ? 0.f : m[h];
            static_for<0, U>([&](auto u) {
                pw[u][h] = fast_exp2(s[u][h] - ms);
                l[h] += pw[u][h];
            });
        });
        static_for<0, U>([&](auto u) {
            static_for<0, V::NP>([&](auto p) {
                static_for<0, 4>([&](auto i) {
                    constexpr int pp = decltype(p)::value, ii = decltype(i)::value;
                    if constexpr (BF16) {
                        const float v0 = bf16_lo(vr[u][p][ii]), v1 = bf16_hi(vr[u][p][ii]);
                        static_for<0, G>([&](auto h) {
                            o[h][pp * 8 + 2 * ii] = fmaf(pw[u][h], v0, o[h][pp * 8 + 2 * ii]);
                            o[h][pp * 8 + 2 * ii + 1] = fmaf(pw[u][h], v1, o[h][pp * 8 + 2 * ii + 1]);
                        });
                    } else {
                        const float v0 = __uint_as_float(vr[u][p][ii]);
                        static_for<0, G>([&](auto h) { o[h][pp * 4 + ii] = fmaf(pw[u][h], v0, o[h][pp * 4 + ii]); });
                    }
                });
            });
        });
    }
}

// Sum the row groups (same maximum within a wave) and merge the waves
// (LDS); sink(h, d, M, L, O) receives four consecutive outputs of head h.
template <int D, int G, bool BF16, typename StoreFn, int EL = Valu<D, G, BF16>::EL>
__device__ __forceinline__ void valu_merge(float (&m)[G], float (&l)[G], float (&o)[G][EL],
                                           char *buf, StoreFn sink) {
    using V = Valu<D, G, BF16>;
    float *s_o = reinterpret_cast<float *>(buf);              // [kWaves][4][G][D]
    float *s_l = s_o + kWaves * 4 * G * D;                     // [kWaves][4][G]
    float *s_m = s_l + kWaves * 4 * G;                         // [kWaves][G]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lj = lane % V::LPK, rg = lane / V::LPK;
    const int drow = lane >> 4;                                // 16-lane DPP row of this lane
    // sum the row groups that share a DPP row (same maximum: plain sums)
    static_for<0, G>([&](auto h) {
        if constexpr (V::RGR >= 4) l[h] = add_row_ror<4>(l[h]);
        if constexpr (V::RGR >= 2) l[h] = add_row_ror<8>(l[h]);
        static_for<0, V::EL>([&](auto e) {
            if constexpr (V::RGR >= 4) o[h][e] = add_row_ror<4>(o[h][e]);
            if constexpr (V::RGR >= 2) o[h][e] = add_row_ror<8>(o[h][e]);
        });
    });
    __syncthreads();   // buf may still be read by a previous phase
    if (rg % V::RGR == 0) {   // the first row group of each DPP row holds its sum
        static_for<0, G>([&](auto h) {
            float *dst = s_o + ((wave * 4 + drow) * G + h) * D;
            static_for<0, V::NP>([&](auto p) {
                constexpr int pp = decltype(p)::value;
                static_for<0, V::EPP / 4>([&](auto q4) {
                    constexpr int qq = decltype(q4)::value;
                    *reinterpret_cast<f32x4_t *>(dst + V::elem(lj, pp, 4 * qq)) =
                        f32x4_t{o[h][pp * V::EPP + 4 * qq + 0], o[h][pp * V::EPP + 4 * qq + 1],
                                o[h][pp * V::EPP + 4 * qq + 2], o[h][pp * V::EPP + 4 * qq + 3]};
                });
            });
            if (lj == 0) s_l[(wave * 4 + drow) * G + h] = l[h];
        });
    }
    if (lane == 0) static_for<0, G>([&](auto h) { s_m[wave * G + h] = m[h]; });
    __syncthreads();
    for (int e = tid; e < G * D / 4; e += kThreads) {   // four consecutive d per thread
        const int h = e / (D / 4), d = 4 * (e % (D / 4));
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w * G + h]);
        const float Ms = M == -INFINITY ? 0.f : M;
        float L = 0.f;
        f32x4_t O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float f = fast_exp2(s_m[w * G + h] - Ms);
            float lw = 0.f;
            f32x4_t ow = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                lw += s_l[(w * 4 + r4) * G + h];
                ow += *reinterpret_cast<const f32x4_t *>(s_o + ((w * 4 + r4) * G + h) * D + d);
            }
            L = fmaf(lw, f, L);
            O += ow * f;
        }
        sink(h, d, M, L, O);
    }
}

// Store the merged state as the item's partial result (sc1 stores):
// o[G][D], m[G], l[G].
template <int D, int G, bool BF16>
__device__ __forceinline__ void valu_store_partial(const AttnArgs &a, float (&m)[G], float (&l)[G],
                                                   float (&o)[G][Valu<D, G, BF16>::EL], char *buf, uint32_t slot) {
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    valu_merge<D, G, BF16>(m, l, o, buf, [&](int h, int d, float M, float L, f32x4_t O) {
        part_store4(r, slot + (uint32_t)(h * D + d) * 4u, O);
        if (d == 0) {
            part_store1(r, slot + (uint32_t)(G * D + h) * 4u, M);
            part_store1(r, slot + (uint32_t)(G * D + G + h) * 4u, L);
        }
    });
}

// Byte offset of slot k of (cell c, KV head g) in the partial region.
__device__ __forceinline__ uint32_t slot_off(const AttnArgs &a, int c, int g, int k) {
    return (uint32_t)((((c * a.Hkv + g) * a.n_slots) + k) * a.slot_floats) * 4u;
}

// Generated rows of one (cell, KV head): contiguous, never spliced.
template <int D, int G, bool BF16>
__device__ void gen_item(const AttnArgs &a, int c, int g, int gk, char *buf) {
    using V = Valu<D, G, BF16>;
    uint32_t qr[G][V::QW];
    load_q<D, G, BF16>(a, c, g, qr);
    const int r0 = a.i0 + gk * a.g_len;
    const int r1 = min(r0 + a.g_len, a.i0 + a.n_gen);
    const size_t off = ((size_t)c * a.Hkv + g) * (size_t)a.cap * V::ROW;
    const char *kb = a.gk + off, *vb = a.gv + off;
    float m[G], l[G], o[G][V::EL];
    valu_stream<D, G, BF16>(qr, r0, r1, a.qk_scale,
                            [&](int key, const char *&kp, const char *&vp) {
                                kp = kb + (size_t)key * V::ROW;
                                vp = vb + (size_t)key * V::ROW;
                                return true;
                            },
                            m, l, o);
    valu_store_partial<D, G, BF16>(a, m, l, o, buf, slot_off(a, c, g, a.n_p + gk));
}

// Prompt chunk of one (cell, KV head) on the vector ALUs (f32 inputs): each
// key is read from the clean or the donor cache by pointer; ZERO slots are
// skipped (their closed-form term is added when the partials are merged).
template <int D, int G, bool BF16>
__device__ void prompt_item_valu(const AttnArgs &a, int c, int g, int pk, char *buf) {
    using V = Valu<D, G, BF16>;
    uint32_t qr[G][V::QW];
    load_q<D, G, BF16>(a, c, g, qr);
    const int k0 = a.jp0 + pk * a.p_len;
    const int k1 = min(k0 + a.p_len, a.Tp);
    const bool spl = bit_set(a.spliced, c);
    const size_t head = (size_t)g * a.Tp * V::ROW;
    float m[G], l[G], o[G][V::EL];
    valu_stream<D, G, BF16>(qr, k0, k1, a.qk_scale,
                            [&](int j, const char *&kp, const char *&vp) {
                                const bool in_span = j >= a.sa && j < a.sb;
                                const bool donor = spl && in_span && !a.zero_donor;
                                const size_t off = head + (size_t)j * V::ROW;
                                kp = (donor ? a.dk : a.ck) + off;
                                vp = (donor ? a.dv : a.cv) + off;
                                return !(spl && in_span && a.zero_donor);
                            },
                            m, l, o);
    valu_store_partial<D, G, BF16>(a, m, l, o, buf, slot_off(a, c, g, pk));
}

// One thread's share of staging a KT-key prompt tile: K in 16-byte units
// (row-major in LDS), V in units of 4 keys x 8 d (transposed in LDS, so the
// p.v operand reads key-contiguous words).
template <int D>
struct TileIo {
    static constexpr int KT = 64;
    static constexpr int KROW = D * 2 + 16;
    static constexpr int VROW = KT * 2 + 8;
    static constexpr int KUNITS = KT * (D / 8);
    static constexpr int VUNITS = (D / 8) * (KT / 4);
    static constexpr int NKU = KUNITS / kThreads;
    static constexpr int NVU = VUNITS >= kThreads ? VUNITS / kThreads : 1;
};

template <int D>
__device__ __forceinline__ void tile_fetch(u32x4_t (&kreg)[TileIo<D>::NKU], u32x4_t (&vreg)[TileIo<D>::NVU][4],
                                           const char *Kg, const char *Vg, int t0, int t1) {
    using T = TileIo<D>;
    const int tid = threadIdx.x;
    static_for<0, T::NKU>([&](auto n) {
        const int u = tid + n * kThreads;
        const int r = u / (D / 8), part = u % (D / 8);
        const int key = min(t0 + r, t1 - 1);
        kreg[n] = *reinterpret_cast<const u32x4_t *>(Kg + (size_t)key * (D * 2) + part * 16);
    });
    static_for<0, T::NVU>([&](auto n) {
        const int u = tid + n * kThreads;
        const int dg = u % (D / 8), kq = (u / (D / 8)) % (T::KT / 4);   // in range for every lane
        static_for<0, 4>([&](auto kk) {
            const int key = min(t0 + 4 * kq + kk, t1 - 1);
            vreg[n][kk] = *reinterpret_cast<const u32x4_t *>(Vg + (size_t)key * (D * 2) + dg * 16);
        });
    });
}

template <int D>
__device__ __forceinline__ void tile_stage(const u32x4_t (&kreg)[TileIo<D>::NKU], const u32x4_t (&vreg)[TileIo<D>::NVU][4],
                                           char *sK, char *sV) {
    using T = TileIo<D>;
    const int tid = threadIdx.x;
    static_for<0, T::NKU>([&](auto n) {
        const int u = tid + n * kThreads;
        const int r = u / (D / 8), part = u % (D / 8);
        *reinterpret_cast<u32x4_t *>(sK + r * T::KROW + part * 16) = kreg[n];
    });
    static_for<0, T::NVU>([&](auto n) {
        const int u = tid + n * kThreads;
        if (u < T::VUNITS) {
            const int dg = u % (D / 8), kq = u / (D / 8);
            static_for<0, 8>([&](auto j) {
                constexpr int jj = decltype(j)::value;
                constexpr uint32_t sel = (jj & 1) ? 0x07060302u : 0x05040100u;
                const uint32_t lo = __builtin_amdgcn_perm(vreg[n][1][jj >> 1], vreg[n][0][jj >> 1], sel);
                const uint32_t hi = __builtin_amdgcn_perm(vreg[n][3][jj >> 1], vreg[n][2][jj >> 1], sel);
                *reinterpret_cast<u32x2_t *>(sV + (8 * dg + jj) * T::VROW + 8 * kq) = u32x2_t{lo, hi};
            });
        }
    });
}

template <int D, int G>
__device__ void prompt_item_mfma(const AttnArgs &a, int g, int rb, int pk, char *buf) {
    using L = Lds<D, G, true>;
    constexpr int KT = L::KT, KROW = L::KROW, VROW = L::VROW;
    constexpr int NDS = D / 32;   // k-steps of q.k
    constexpr int NDT = D / 16;   // 16-wide d tiles of the output
    char *sK = buf;
    char *sV = buf + KT * KROW;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, quad = lane >> 4;

    const int R = rb * kRowBlock + wave * 16 + col;
    const int cidx = R / G;
    const bool row_ok = cidx < a.C;
    const int cell = row_ok ? a.order[cidx] : 0;
    const int hl = R % G;
    const bool spl = row_ok && bit_set(a.spliced, cell);
    const bool row_clean = row_ok && !spl;
    const bool row_donor = spl && !a.zero_donor;
    const int first = rb * kRowBlock / G;
    const int last = min(a.C, (rb + 1) * kRowBlock / G) - 1;
    const bool blk_clean = first < a.n_clean;
    const bool blk_donor = !a.zero_donor && last >= a.n_clean;

    bf16x8_t qf[NDS];
    {
        const char *qrow = a.q + ((size_t)cell * a.Hq + (size_t)g * G + hl) * (D * 2);
        static_for<0, NDS>([&](auto st) {
            uint4 w = make_uint4(0, 0, 0, 0);
            if (row_ok) w = *reinterpret_cast<const uint4 *>(qrow + (32 * st + 8 * quad) * 2);
            qf[st] = __builtin_bit_cast(bf16x8_t, w);
        });
    }
    f32x4_t o[NDT];
    static_for<0, NDT>([&](auto t) { o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f}; });
    float m = -INFINITY, lsum = 0.f;

    const int k0 = a.jp0 + pk * a.p_len;
    const int k1 = min(k0 + a.p_len, a.Tp);
    const size_t head = (size_t)g * a.Tp * (D * 2);

    // The chunk is a sequence of steps (tile, source).  Tiles hold up to KT
    // keys and never straddle a span boundary (a tile is all span or all
    // not), so a row's keys are grouped the same whether it is spliced or
    // not.  A tile runs a clean pass if any row reads it from the clean cache
    // and a donor pass if any spliced row reads it from the donor cache.
    auto tile_end = [&](int t0) __attribute__((always_inline)) {
        int t1 = min(t0 + KT, k1);
        if (t0 < a.sa) t1 = min(t1, a.sa);
        else if (t0 < a.sb) t1 = min(t1, a.sb);
        return t1;
    };
    auto needed = [&](int t0, int dpass) __attribute__((always_inline)) {
        const bool span = t0 >= a.sa && t0 < a.sb;
        return dpass ? (span && blk_donor) : (!span || blk_clean);
    };
    auto advance = [&](int &t0, int &dpass) __attribute__((always_inline)) {   // to the next needed step, t0 = k1 at the end
        for (;;) {
            if (dpass == 0) {
                dpass = 1;
            } else {
                t0 = tile_end(t0);
                dpass = 0;
            }
            if (t0 >= k1 || needed(t0, dpass)) return;
        }
    };

    // this thread's share of a tile: K units (16 bytes) and V units (4 keys x 8 d)
    u32x4_t kreg[TileIo<D>::NKU];
    u32x4_t vreg[TileIo<D>::NVU][4];

    int t0 = k0, dpass = 0;
    if (t0 < k1 && !needed(t0, 0)) advance(t0, dpass);
    if (t0 < k1)
        tile_fetch<D>(kreg, vreg, (dpass ? a.dk : a.ck) + head, (dpass ? a.dv : a.cv) + head, t0, tile_end(t0));
    while (t0 < k1) {
        const int t1 = tile_end(t0);
        const int cur_dpass = dpass;
        __syncthreads();   // the previous step no longer reads the LDS tiles
        tile_stage<D>(kreg, vreg, sK, sV);
        __syncthreads();
        int nt0 = t0, ndpass = dpass;
        advance(nt0, ndpass);
        if (nt0 < k1)   // in flight while this step computes
            tile_fetch<D>(kreg, vreg, (ndpass ? a.dk : a.ck) + head, (ndpass ? a.dv : a.cv) + head, nt0,
                          tile_end(nt0));

        f32x4_t s[4];
        static_for<0, 4>([&](auto sub) {
            s[sub] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            static_for<0, NDS>([&](auto st) {
                const bf16x8_t kf = *reinterpret_cast<const bf16x8_t *>(
                    sK + (16 * sub + col) * KROW + (32 * st + 8 * quad) * 2);
                s[sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[st], s[sub], 0, 0, 0);
            });
        });
        float p[4][4];
        float mt = -INFINITY;
#pragma unroll
        for (int sub = 0; sub < 4; ++sub)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = t0 + 16 * sub + 4 * quad + i;
                const bool in_span = key >= a.sa && key < a.sb;
                const bool ok = row_ok && key < t1 &&
                                (cur_dpass ? (in_span && row_donor) : (!in_span || row_clean));
                p[sub][i] = ok ? s[sub][i] * a.qk_scale : -INFINITY;
                mt = fmaxf(mt, p[sub][i]);
            }
        mt = fmaxf(mt, __shfl_xor(mt, 16));
        mt = fmaxf(mt, __shfl_xor(mt, 32));
        const bool need = mt > m + kSlack;
        if (__any(need)) {
            // only rows that need it move their maximum: a row's arithmetic
            // never depends on the other rows of its wave
            const float mn = need ? fmaxf(m, mt) : m;
            const float al = need ? fast_exp2(m - (mn == -INFINITY ? 0.f : mn)) : 1.f;
            lsum *= al;
            static_for<0, NDT>([&](auto t) { o[t] *= al; });
            m = mn;
        }
        const float ms = m == -INFINITY ? 0.f : m;
#pragma unroll
        for (int sub = 0; sub < 4; ++sub)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                p[sub][i] = fast_exp2(p[sub][i] - ms);
                lsum += p[sub][i];
            }
        static_for<0, 2>([&](auto kg) {
            bf16x8_t ph, pl;
            static_for<0, 8>([&](auto j) {
                constexpr int jj = decltype(j)::value;
                const float x = p[2 * kg + (jj >> 2)][jj & 3];
                const __bf16 hb = (__bf16)x;
                ph[jj] = hb;
                pl[jj] = (__bf16)(x - (float)hb);
            });
            static_for<0, NDT>([&](auto t) {
                const char *vrow = sV + (16 * t + col) * VROW;
                const uint2 va = *reinterpret_cast<const uint2 *>(vrow + (32 * kg + 4 * quad) * 2);
                const uint2 vb = *reinterpret_cast<const uint2 *>(vrow + (32 * kg + 16 + 4 * quad) * 2);
                const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, make_uint4(va.x, va.y, vb.x, vb.y));
                o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, ph, o[t], 0, 0, 0);
                o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl, o[t], 0, 0, 0);
            });
        });
        t0 = nt0;
        dpass = ndpass;
    }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    if (row_ok) {
        const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
        const uint32_t slot = slot_off(a, cell, g, pk);
        static_for<0, NDT>([&](auto t) {
            part_store4(r, slot + (uint32_t)(hl * D + 16 * t + 4 * quad) * 4u, o[t]);
        });
        if (quad == 0) {
            part_store1(r, slot + (uint32_t)(G * D + hl) * 4u, m);
            part_store1(r, slot + (uint32_t)(G * D + G + hl) * 4u, lsum);
        }
    }
}

// ----------------------------------------------------------- merging
//
// Every work item stores its partial results with agent-scope (L2
// write-through) stores, waits until they are performed, and then counts
// itself on each (cell, KV head) it fed with a device-scope atomic.  The item
// that brings a counter to n_slots merges that (cell, KV head): it reads the
// slots with agent-scope loads (which do not trust a stale L2 line), merges
// them in slot order with a log-sum-exp combine, adds the ZERO term, writes
// out and lse, and re-arms the counter.  No cache-wide write-back or
// invalidate is needed, so the cached tiles of other items survive.

__device__ __forceinline__ void stores_performed() {
    __builtin_amdgcn_s_waitcnt(0);   // every outstanding memory operation of this lane is done
    __syncthreads();
}

__device__ __forceinline__ bool arrive(const AttnArgs &a, int c, int g) {
    const int prev = __hip_atomic_fetch_add(&a.counters[c * a.Hkv + g], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    return prev == a.n_slots - 1;
}

// Merge the partial results of cells list[0..n) of KV head g.  One round of
// loads stages every (m, l) in LDS; then each thread owns up to kMergeUnits
// groups of four consecutive outputs and loads them two slots at a time, so
// a merge costs a few memory round trips whatever the cell count.
constexpr int kMergeUnits = 4;

template <int D, int G>
__device__ void combine_cells(const AttnArgs &a, const int *list, int n, int g, char *buf) {
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    float *s_m = reinterpret_cast<float *>(buf);           // [n][n_slots][G]
    float *s_l = s_m + kRowBlock * kMaxSlots;               // [n][n_slots][G]
    const int per_cell = a.n_slots * G;
    for (int t = threadIdx.x; t < n * per_cell; t += kThreads) {
        const int i = t / per_cell, rem = t % per_cell;
        const int k = rem / G, h = rem % G;
        const uint32_t slot = slot_off(a, list[i], g, k);
        s_m[t] = part_load1(r, slot + (uint32_t)(G * D + h) * 4u);
        s_l[t] = part_load1(r, slot + (uint32_t)(G * D + G + h) * 4u);
    }
    __syncthreads();
    constexpr int UPC = G * D / 4;                           // 4-wide units per cell
    const int total = n * UPC;
    const uint32_t slot_bytes = (uint32_t)a.slot_floats * 4u;
    for (int u0 = threadIdx.x; u0 < total; u0 += kThreads * kMergeUnits) {
        float M[kMergeUnits], L[kMergeUnits];
        f32x4_t O[kMergeUnits];
        uint32_t base[kMergeUnits];
        int sm_off[kMergeUnits];
#pragma unroll
        for (int b = 0; b < kMergeUnits; ++b) {
            const int u = min(u0 + b * kThreads, total - 1);   // tail units repeat a valid one
            const int i = u / UPC, rem = u % UPC;
            const int h = rem / (D / 4), d = 4 * (rem % (D / 4));
            const int c = list[i];
            sm_off[b] = i * per_cell + h;
            base[b] = slot_off(a, c, g, 0) + (uint32_t)(h * D + d) * 4u;
            const bool zero_term = a.zero_donor && bit_set(a.spliced, c) && a.sb > a.sa;
            float mx = zero_term ? 0.f : -INFINITY;
            for (int k = 0; k < a.n_slots; ++k) mx = fmaxf(mx, s_m[sm_off[b] + k * G]);
            M[b] = mx;
            L[b] = zero_term ? (float)(a.sb - a.sa) * fast_exp2(-mx) : 0.f;
            O[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        int k = 0;
        for (; k + 2 <= a.n_slots; k += 2) {
            f32x4_t v0[kMergeUnits], v1[kMergeUnits];
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) {
                v0[b] = part_load4(r, base[b] + (uint32_t)k * slot_bytes);
                v1[b] = part_load4(r, base[b] + (uint32_t)(k + 1) * slot_bytes);
            }
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) {
                const float f0 = fast_exp2(s_m[sm_off[b] + k * G] - M[b]);
                const float f1 = fast_exp2(s_m[sm_off[b] + (k + 1) * G] - M[b]);
                L[b] = fmaf(s_l[sm_off[b] + k * G], f0, L[b]);
                L[b] = fmaf(s_l[sm_off[b] + (k + 1) * G], f1, L[b]);
                O[b] += v0[b] * f0;
                O[b] += v1[b] * f1;
            }
        }
        if (k < a.n_slots) {
            f32x4_t v0[kMergeUnits];
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) v0[b] = part_load4(r, base[b] + (uint32_t)k * slot_bytes);
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) {
                const float f0 = fast_exp2(s_m[sm_off[b] + k * G] - M[b]);
                L[b] = fmaf(s_l[sm_off[b] + k * G], f0, L[b]);
                O[b] += v0[b] * f0;
            }
        }
#pragma unroll
        for (int b = 0; b < kMergeUnits; ++b) {
            const int u = u0 + b * kThreads;
            if (u < total) {
                const int i = u / UPC, rem = u % UPC;
                const int h = rem / (D / 4), d = 4 * (rem % (D / 4));
                const int row = list[i] * a.Hq + g * G + h;
                *reinterpret_cast<f32x4_t *>(a.out + (size_t)row * D + d) = O[b] * (1.f / L[b]);
                if (d == 0) a.lse[row] = (M[b] + log2f(L[b])) * kLn2;
            }
        }
    }
    if (threadIdx.x < n)
        __hip_atomic_store(&a.counters[list[threadIdx.x] * a.Hkv + g], 0, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// One launch per call: blocks [0, n_prompt_items) are prompt items, the
// rest generated-row items.
template <int D, int G, bool BF16>
__global__ __launch_bounds__(kThreads) void attn_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char buf[Lds<D, G, BF16>::BYTES];
    __shared__ int s_list[kRowBlock + 1];
    const int tid = threadIdx.x;
    int item = blockIdx.x;
    if (item < a.n_prompt_items) {
        const int pk = item % a.n_p;
        item /= a.n_p;
        if constexpr (BF16) {
            const int rb = item % a.n_rb;
            const int g = item / a.n_rb;
            prompt_item_mfma<D, G>(a, g, rb, pk, buf);
            if (tid == 0) s_list[0] = 0;
            stores_performed();
            const int first = rb * kRowBlock / G;
            const int n_cells = min(a.C, first + kRowBlock / G) - first;
            if (tid < n_cells) {
                const int cell = a.order[first + tid];
                if (arrive(a, cell, g)) s_list[1 + atomicAdd(&s_list[0], 1)] = cell;
            }
            __syncthreads();
            if (s_list[0] > 0) combine_cells<D, G>(a, s_list + 1, s_list[0], g, buf);
        } else {
            const int g = item % a.Hkv;
            const int c = item / a.Hkv;
            prompt_item_valu<D, G, BF16>(a, c, g, pk, buf);
            stores_performed();
            if (tid == 0) {
                s_list[0] = arrive(a, c, g) ? 1 : 0;
                s_list[1] = c;
            }
            __syncthreads();
            if (s_list[0]) combine_cells<D, G>(a, s_list + 1, 1, g, buf);
        }
    } else {
        item -= a.n_prompt_items;
        const int gk = item % a.n_g;
        item /= a.n_g;
        const int g = item % a.Hkv;
        const int c = item / a.Hkv;
        gen_item<D, G, BF16>(a, c, g, gk, buf);
        stores_performed();
        if (tid == 0) {
            s_list[0] = arrive(a, c, g) ? 1 : 0;
            s_list[1] = c;
        }
        __syncthreads();
        if (s_list[0]) combine_cells<D, G>(a, s_list + 1, 1, g, buf);
    }
}

// ------------------------------------------------------- cellwise kernel
//
// Short prompts: one work group per (cell, KV head) streams the cell's
// whole visible list -- prompt slots read from the clean or the donor cache
// by pointer (a ZERO cell skips its span), then its generated rows -- and
// writes out and lse itself.  No partial results and no merge; the prompt
// tiles the cells share are re-read from L2.  Chosen by the host when the
// prompt is short enough for that to be cheaper than the row-block path.
template <int D, int G, bool BF16>
__global__ __launch_bounds__(kThreads) void cellwise_kernel(AttnArgs a) {
    using V = Valu<D, G, BF16>;
    __shared__ __attribute__((aligned(16))) char buf[kWaves * 4 * G * (D + 1) * 4 + kWaves * G * 4];
    const int g = blockIdx.x % a.Hkv;
    const int c = blockIdx.x / a.Hkv;
    uint32_t qr[G][V::QW];
    load_q<D, G, BF16>(a, c, g, qr);
    const bool spl = bit_set(a.spliced, c);
    const bool zskip = spl && a.zero_donor;
    const int nsv = a.sb - a.sa;
    const int n_pl = (a.Tp - a.jp0) - (zskip ? nsv : 0);   // prompt part of the list
    const int n_list = n_pl + a.n_gen;
    const size_t head = (size_t)g * a.Tp * V::ROW;
    const char *gkb = a.gk + ((size_t)c * a.Hkv + g) * (size_t)a.cap * V::ROW;
    const char *gvb = a.gv + ((size_t)c * a.Hkv + g) * (size_t)a.cap * V::ROW;
    float m[G], l[G], o[G][V::EL];
    valu_stream<D, G, BF16>(qr, 0, n_list, a.qk_scale,
                            [&](int v, const char *&kp, const char *&vp) {
                                if (v < n_pl) {
                                    int j = a.jp0 + v;
                                    if (zskip && j >= a.sa) j += nsv;
                                    const bool donor = spl && !a.zero_donor && j >= a.sa && j < a.sb;
                                    const size_t off = head + (size_t)j * V::ROW;
                                    kp = (donor ? a.dk : a.ck) + off;
                                    vp = (donor ? a.dv : a.cv) + off;
                                } else {
                                    const size_t off = (size_t)(a.i0 + (v - n_pl)) * V::ROW;
                                    kp = gkb + off;
                                    vp = gvb + off;
                                }
                                return true;
                            },
                            m, l, o);
    const bool zero_term = zskip && nsv > 0;
    valu_merge<D, G, BF16>(m, l, o, buf, [&](int h, int d, float M, float L, f32x4_t O) {
        if (zero_term) {   // nsv keys of score 0 and value 0
            const float Mz = fmaxf(M, 0.f);
            const float f = fast_exp2(M - Mz);
            L = L * f + (float)nsv * fast_exp2(-Mz);
            O *= f;
            M = Mz;
        }
        const int row = c * a.Hq + g * G + h;
        *reinterpret_cast<f32x4_t *>(a.out + (size_t)row * D + d) = O * (1.f / L);
        if (d == 0) a.lse[row] = (M + log2f(L)) * kLn2;
    });
}

__global__ __launch_bounds__(kThreads) void fill_kernel(uint32_t *p, size_t n_words) {
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n_words;
         i += (size_t)gridDim.x * kThreads)
        p[i] = 0u;
}

// ------------------------------------------------------------ dispatch

typedef void (*attn_fn)(AttnArgs);
struct AttnKernels {
    attn_fn rowblock, cellwise;
};

template <int D, int G, bool BF16>
AttnKernels kernels_of() {
    return AttnKernels{attn_kernel<D, G, BF16>, cellwise_kernel<D, G, BF16>};
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
    int n_slots;
    if (call) {
        rc = splice::validate_call(*shape, call);
        if (rc != SPLICE_OK) return rc;
        n_slots = splice::plan_attn(*shape, *call).n_slots;
        if (n_slots > splice::kMaxSlots) return SPLICE_EUNSUPPORTED;
    } else {
        n_slots = splice::worst_default_slots(*shape);
    }
    return (int64_t)splice::workspace_layout(*shape, n_slots).total;
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
    if (!splice::aligned(out, 16) || !splice::aligned(lse, 4)) return SPLICE_EINVAL;

    const splice::AttnPlan plan = splice::plan_attn(sh, *call);
    if (plan.n_slots > splice::kMaxSlots) return SPLICE_EUNSUPPORTED;
    const splice::WorkspaceLayout wl = splice::workspace_layout(sh, plan.n_slots);
    if (!workspace || !splice::aligned(workspace, 256)) return SPLICE_EWORKSPACE;
    if (workspace_bytes < wl.total) return SPLICE_EWORKSPACE;

    const int G = splice::group_of(sh);
    const AttnKernels kern = pick_attn(sh.head_dim, G, sh.dtype);
    if (!kern.rowblock) return SPLICE_EUNSUPPORTED;

    const splice::Geometry &geo = plan.geo;
    AttnArgs a;
    a.q = (const char *)q;
    a.ck = (const char *)clean_k; a.cv = (const char *)clean_v;
    a.dk = (const char *)donor_k; a.dv = (const char *)donor_v;
    a.gk = (const char *)gen_k; a.gv = (const char *)gen_v;
    a.out = out; a.lse = lse;
    a.counters = (int *)((char *)workspace + wl.counters_off);
    a.part = (float *)((char *)workspace + wl.part_off);
    if (wl.part_bytes >= ((size_t)1 << 31)) return SPLICE_EUNSUPPORTED;
    a.part_bytes = (uint32_t)(wl.part_bytes > 0 ? wl.part_bytes : 16);
    a.C = sh.n_cells; a.Hq = sh.n_q_heads; a.Hkv = sh.n_kv_heads; a.Tp = sh.prompt_len;
    a.cap = sh.gen_capacity;
    a.jp0 = geo.jp0; a.i0 = geo.i0; a.n_gen = geo.n_gen; a.sa = geo.sa; a.sb = geo.sb;
    a.zero_donor = zero ? 1 : 0;
    a.n_p = plan.n_p; a.p_len = plan.p_len; a.n_g = plan.n_g; a.g_len = plan.g_len;
    a.n_slots = plan.n_slots;
    a.slot_floats = splice::slot_floats(G, sh.head_dim);
    a.n_rb = splice::row_blocks(sh);
    a.n_prompt_items = plan.n_prompt_items;
    a.qk_scale = call->scale * kLog2e;
    fill_mask(sh, *call, cell_LW, a.spliced);
    // row-block order: clean cells first, then spliced cells (each by index)
    int n = 0;
    for (int c = 0; c < sh.n_cells; ++c)
        if (!splice::cell_spliced(cell_LW, c, call->layer, call->step)) a.order[n++] = (uint8_t)c;
    a.n_clean = n;
    for (int c = 0; c < sh.n_cells; ++c)
        if (splice::cell_spliced(cell_LW, c, call->layer, call->step)) a.order[n++] = (uint8_t)c;
    for (; n < SPLICE_MAX_CELLS; ++n) a.order[n] = 0;

    if (plan.cellwise) {
        hipLaunchKernelGGL(kern.cellwise, dim3((unsigned)(sh.n_cells * sh.n_kv_heads)), dim3(kThreads), 0,
                           (hipStream_t)stream, a);
        return launch_status();
    }
    const int64_t items = (int64_t)plan.n_prompt_items + plan.n_gen_items;
    if (items > INT32_MAX) return SPLICE_EUNSUPPORTED;
    hipLaunchKernelGGL(kern.rowblock, dim3((unsigned)items), dim3(kThreads), 0, (hipStream_t)stream, a);
    return launch_status();
}

}  // extern "C"
