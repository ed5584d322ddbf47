// attn_kernels.hpp -- the spliced decode-attention kernels (templates over
// head_dim D, group size G and element type).  Each attn_*.hip translation
// unit instantiates one (D, element type) pair, so the six pairs compile in
// parallel and no kernel is instantiated twice.
#pragma once

#include "device_common.hpp"
#include "prompt_wide.hpp"
#include "wave_mfma.hpp"

namespace splice_dev {

// --------------------------------------------------------------- attention

struct AttnArgs {
    const char *q;
    const char *ck, *cv, *dk, *dv, *gk, *gv;
    float *out, *lse, *part;
    int *counters;
    int *stats;            // workspace statistics: [0] merges handed over (see fused_gen_item)
    uint32_t part_bytes;   // size of the partial-result region (< 2^31)
    int C, Hq, Hkv, Tp, cap;
    int jp0, i0, n_gen, sa, sb;
    int zero_donor;
    int n_p, p_len, n_g, g_len, n_slots;
    // partial-result region: the prompt slots [C][Hkv][n_p] of p_slot_bytes
    // each, then from byte gen_base the generated-row slots [C][Hkv][n_g] of
    // g_slot_bytes each
    uint32_t p_slot_bytes, g_slot_bytes, gen_base;
    int n_rb, n_prompt_items, n_clean;
    int n_rg_clean;   // bf16 prompt row groups of unspliced cells (the rest: spliced cells)
    int wait_polls;   // bf16 generated-row items: most polls for the prompt partials
    int n_active;     // cells in `order` (all cells, or the unfinished ones of a decode step)
    int ragged;       // bf16: each cell at its own step cstep[c] (< 0: finished, skipped)
    int window;       // sliding window of the call (0: every key visible)
    int span_lo, span_hi;
    int row_lo;       // prompt items mask the keys before each row's first visible slot
    const char *kn, *vn;   // bf16 decode step: the current token's K, V [C][Hkv][D], appended
    int32_t cstep[SPLICE_MAX_CELLS];
    int trunk;        // forked sweep: the cell of the clean run (-1: none); see fused_gen_item
    int n_dormant;    // forked sweep: cells not yet diverged, order[n_active ..], given the trunk's result
    int32_t wfork[SPLICE_MAX_CELLS];   // forked sweep: a cell's generated rows below wfork are the trunk's
    int gen_pairs;    // bf16 generated-row items: (cell, KV head) pairs per work group
    int gen_v_nt;     // bf16 generated-row items: V rows loaded non-temporally
    float qk_scale;   // scale * log2(e)
    uint32_t spliced[SPLICE_MAX_CELLS / 32];
    uint8_t order[SPLICE_MAX_CELLS];   // clean cells, then spliced cells
    // bf16 generated-row items: the cells that have generated rows to stream
    // (active, and under a forked sweep diverged), longest first; item i
    // serves gorder[i * gen_pairs ..]
    int n_gen_cells;
    uint8_t gorder[SPLICE_MAX_CELLS];
};


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

// fp16 partial values (converted from fp32 rounding to nearest even): four
// outputs in 8 bytes, or a group of eight in 16.
typedef _Float16 h16x4_t __attribute__((ext_vector_type(4)));
typedef _Float16 h16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f32x4_t part_load4h(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const u32x2_t w = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kSc1);
    return __builtin_convertvector(__builtin_bit_cast(h16x4_t, w), f32x4_t);
}

// One partial-result slot of a (cell, KV head): o[G][D], then m[G] and l[G]
// in fp32.  A 16-bit slot (the prompt chunks of a bf16 call) holds
// o / (l sc) in fp16, then per row a 16-byte record (m, l, w, 0) with
// w = l sc, the weight its o enters the merge with; sc is a power of two, 1
// unless the largest |o / l| of the row is above kH16Limit.  Since o / l is
// a convex combination of V rows, the stored values are bounded by the
// largest |v| of the chunk.
//
// A 16-bit row is stored in groups of eight values, d0 .. d0 + 3 and
// d0 + 16 .. d0 + 19 for d0 = 32 u + 4 q (q < 4), at group 4 u + q: the
// outputs one lane of a prompt item holds for two adjacent 16-row MFMA
// tiles, so the lane writes a group with one 16-byte store and a reader of
// 8 outputs loads it with one.  o(h, d) is the byte offset of the four
// outputs d .. d + 3 (d a multiple of 4).
template <int D, int G, bool H16>
struct Slot {
    static constexpr uint32_t OE = H16 ? 2 : 4;
    static constexpr uint32_t ML = (uint32_t)(G * D) * OE;
    __device__ static uint32_t o(int h, int d) {
        if constexpr (H16) {
            const int t = d >> 4, u = t >> 1, hf = t & 1, q = (d & 15) >> 2;
            return (uint32_t)(h * D) * 2u + (uint32_t)((u * 4 + q) * 16 + hf * 8);
        } else {
            return (uint32_t)(h * D + d) * 4u;
        }
    }
    __device__ static uint32_t m(int h) { return H16 ? ML + 16u * (uint32_t)h : ML + 4u * (uint32_t)h; }
    __device__ static uint32_t l(int h) { return H16 ? ML + 16u * (uint32_t)h + 4u : ML + 4u * (uint32_t)(G + h); }
    __device__ static uint32_t w(int h) { return ML + 16u * (uint32_t)h + 8u; }   // H16 only
};
constexpr float kH16Limit = 32768.f;

// Byte offsets of prompt slot k and generated-row slot j of (cell c, KV head g).
__device__ __forceinline__ uint32_t pslot_off(const AttnArgs &a, int c, int g, int k) {
    return ((uint32_t)(c * a.Hkv + g) * (uint32_t)a.n_p + (uint32_t)k) * a.p_slot_bytes;
}
__device__ __forceinline__ uint32_t gslot_off(const AttnArgs &a, int c, int g, int j) {
    return a.gen_base + ((uint32_t)(c * a.Hkv + g) * (uint32_t)a.n_g + (uint32_t)j) * a.g_slot_bytes;
}

// (o, m, l, w) of four outputs of a prompt slot at byte offset base.
template <int D, int G, bool H16>
__device__ __forceinline__ void load_pslot(__amdgpu_buffer_rsrc_t r, uint32_t base, int h, int d, f32x4_t &o,
                                           float &m, float &l, float &w) {
    using SL = Slot<D, G, H16>;
    if constexpr (H16) {
        o = part_load4h(r, base + SL::o(h, d));
        const f32x4_t mlw = part_load4(r, base + SL::m(h));
        m = mlw.x;
        l = mlw.y;
        w = mlw.z;
    } else {
        o = part_load4(r, base + SL::o(h, d));
        m = part_load1(r, base + SL::m(h));
        l = part_load1(r, base + SL::l(h));
        w = l;
    }
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
// LDS of the f32 items kernel: row-group sums of the vector-ALU stream and
// the merge staging.
template <int D, int G, bool BF16>
struct Lds {
    static constexpr int MERGE = kWaves * 4 * G * (D + 1) * 4 + kWaves * G * 4;
    static constexpr int STAGE = 2 * kMaxSlots * kRowBlock * 4;
    static constexpr int BYTES = cmax(MERGE, STAGE);
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
    valu_store_partial<D, G, BF16>(a, m, l, o, buf, gslot_off(a, c, g, gk));
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
                                kp = pick_base(donor, a.ck, a.dk) + off;
                                vp = pick_base(donor, a.cv, a.dv) + off;
                                return !(spl && in_span && a.zero_donor);
                            },
                            m, l, o);
    valu_store_partial<D, G, BF16>(a, m, l, o, buf, pslot_off(a, c, g, pk));
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
//
// The combine of one (row, four outputs) is fixed: M = the maximum of the
// slots' m (and 0 with a ZERO term); L starts at the ZERO term
// n_zero 2^-M (or 0); then slot k = 0, 1, ... adds l_k 2^(m_k - M) to L and
// o_k 2^(m_k - M) to O with one fused multiply-add per value (a 16-bit
// prompt slot: its stored o times w_k 2^(m_k - M), the product rounded
// once); out = O / L.  Every merge site below follows it, so a result does
// not depend on which item merged it.

__device__ __forceinline__ void stores_performed() {
    __builtin_amdgcn_s_waitcnt(0);   // every outstanding memory operation of this lane is done
    __syncthreads();
}

__device__ __forceinline__ bool arrive(const AttnArgs &a, int c, int g) {
    const int prev = __hip_atomic_fetch_add(&a.counters[c * a.Hkv + g], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    return prev == a.n_slots - 1;
}

__device__ __forceinline__ void fold_slot(float mk, float lk, f32x4_t ok, float M, float &L, f32x4_t &O) {
    const float f = fast_exp2(mk - M);
    L = fmaf(lk, f, L);
    O.x = fmaf(ok.x, f, O.x);
    O.y = fmaf(ok.y, f, O.y);
    O.z = fmaf(ok.z, f, O.z);
    O.w = fmaf(ok.w, f, O.w);
}

// A prompt slot: l enters with 2^(m - M), o with w 2^(m - M) (a 16-bit slot
// holds o / w); an fp32 slot has w = l and folds exactly as fold_slot.
template <bool H16>
__device__ __forceinline__ void fold_pslot(float mk, float lk, float wk, f32x4_t ok, float M, float &L, f32x4_t &O) {
    if constexpr (H16) {
        const float f = fast_exp2(mk - M);
        L = fmaf(lk, f, L);
        const float fw = wk * f;
        O.x = fmaf(ok.x, fw, O.x);
        O.y = fmaf(ok.y, fw, O.y);
        O.z = fmaf(ok.z, fw, O.z);
        O.w = fmaf(ok.w, fw, O.w);
    } else {
        fold_slot(mk, lk, ok, M, L, O);
    }
}

// What cell c sees: its step, visible generated rows [i0, i0 + n_gen), first
// visible prompt slot jp0 and visible span [sa, sb) -- the call's values, or
// the cell's own under a decode step with cells at different steps.
struct CellGeo {
    int s, i0, n_gen, jp0, sa, sb;
};

__device__ __forceinline__ CellGeo cell_geo(const AttnArgs &a, int c) {
    if (!a.ragged) return CellGeo{a.i0 + a.n_gen - 1, a.i0, a.n_gen, a.jp0, a.sa, a.sb};
    const int s = a.cstep[c];
    const int j0 = a.window > 0 ? a.Tp + s - a.window + 1 : 0;
    const int jp0 = min(max(j0, 0), a.Tp);
    const int i0 = max(j0 - a.Tp, 0);
    const int sa = min(max(a.span_lo, jp0), a.Tp);
    const int sb = min(max(a.span_hi, sa), a.Tp);
    return CellGeo{s, i0, s + 1 - i0, jp0, sa, sb};
}

__device__ __forceinline__ bool cell_active(const AttnArgs &a, int c) { return !a.ragged || a.cstep[c] >= 0; }

// ZERO-donor slots cell c sees (0 without a ZERO term): keys of score 0 and
// value 0, added in closed form by the merge.
__device__ __forceinline__ int zero_slots(const AttnArgs &a, int c) {
    if (!a.zero_donor || !bit_set(a.spliced, c)) return 0;
    const CellGeo geo = cell_geo(a, c);
    return geo.sb - geo.sa;
}

__device__ __forceinline__ bool has_zero_term(const AttnArgs &a, int c) { return zero_slots(a, c) > 0; }

// Set (in LDS) when this work group has written rows of a forked sweep's
// trunk: the work group then copies them to the cells that have not yet
// diverged from it (dormant_copy).
__device__ __forceinline__ int &trunk_written() {
    __shared__ int flag;
    return flag;
}

// Output row (cell c, q head hq): four outputs at d, and lse.
__device__ __forceinline__ void write_row(const AttnArgs &a, int c, int hq, int d, int D, float M, float L,
                                          f32x4_t O) {
    const f32x4_t o = O * (1.f / L);
    const float lse = (M + log2f(L)) * kLn2;
    const size_t row = (size_t)c * a.Hq + hq;
    *reinterpret_cast<f32x4_t *>(a.out + row * D + d) = o;
    if (d == 0) a.lse[row] = lse;
    if (c == a.trunk) trunk_written() = 1;
}

// Under a forked sweep the trunk's rows are also the rows of every cell that
// has not yet diverged from it.  The work group that wrote the trunk's rows
// of KV head g copies them, all its threads at once: it stages the dormant
// cells' indices in LDS (buf) and reads the trunk's rows once, each thread
// keeping its units in registers, then only stores.  The rows were written
// by this work group, so a work-group fence and barrier make them readable
// (they are in this compute unit's L2, and its L1 holds no older copy: out
// is only ever written).
template <int D, int G, int NT>
__device__ void dormant_copy(const AttnArgs &a, int g, char *buf) {
    constexpr int U = G * D / 4;                     // 16-byte units of one cell's rows of KV head g
    constexpr int GROUPS = U <= NT ? NT / U : 1;     // thread groups taking every GROUPS-th cell
    constexpr int UPT = U <= NT ? 1 : U / NT;        // units per thread
    static_assert(U <= NT ? NT % U == 0 : U % NT == 0, "whole units per thread");
    __threadfence_block();
    __syncthreads();
    int *cells = reinterpret_cast<int *>(buf);
    for (int i = threadIdx.x; i < a.n_dormant; i += NT) cells[i] = a.order[a.n_active + i];
    const int grp = U <= NT ? (int)threadIdx.x / U : 0;
    const int u0 = U <= NT ? (int)threadIdx.x % U : (int)threadIdx.x;
    const size_t src = ((size_t)a.trunk * a.Hq + (size_t)g * G) * D;
    f32x4_t v[UPT];
    static_for<0, UPT>([&](auto j) {
        v[j] = *reinterpret_cast<const f32x4_t *>(a.out + src + 4 * (u0 + (int)j * NT));
    });
    const float l = u0 < G ? a.lse[(size_t)a.trunk * a.Hq + (size_t)g * G + u0] : 0.f;
    __syncthreads();
    for (int i = grp; i < a.n_dormant; i += GROUPS) {
        const size_t row = (size_t)cells[i] * a.Hq + (size_t)g * G;
        static_for<0, UPT>([&](auto j) {
            *reinterpret_cast<f32x4_t *>(a.out + row * D + 4 * (u0 + (int)j * NT)) = v[j];
        });
        if (u0 < G) a.lse[row + u0] = l;
    }
}

// Merge the partial results of cells list[0..n) of KV head g.  One round of
// loads stages every (m, l) in LDS; then each thread owns up to kMergeUnits
// groups of four consecutive outputs and loads them two slots at a time.
constexpr int kMergeUnits = 4;

template <int D, int G, int NT, bool H16>
__device__ void combine_cells(const AttnArgs &a, const int *list, int n, int g, char *buf) {
    using SP = Slot<D, G, H16>;     // prompt slots
    using SG = Slot<D, G, false>;   // generated-row slots
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    float *s_m = reinterpret_cast<float *>(buf);           // [n][n_slots][G]
    float *s_l = s_m + kRowBlock * kMaxSlots;               // [n][n_slots][G]
    float *s_w = H16 ? s_l + kRowBlock * kMaxSlots : s_l;  // [n][n_slots][G]: weights of o (H16 only)
    const int per_cell = a.n_slots * G;
    for (int t = threadIdx.x; t < n * per_cell; t += NT) {
        const int i = t / per_cell, rem = t % per_cell;
        const int k = rem / G, h = rem % G;
        if (k < a.n_p) {
            const uint32_t slot = pslot_off(a, list[i], g, k);
            s_m[t] = part_load1(r, slot + SP::m(h));
            s_l[t] = part_load1(r, slot + SP::l(h));
            if constexpr (H16) s_w[t] = part_load1(r, slot + SP::w(h));
        } else {
            const uint32_t slot = gslot_off(a, list[i], g, k - a.n_p);
            s_m[t] = part_load1(r, slot + SG::m(h));
            s_l[t] = part_load1(r, slot + SG::l(h));
            if constexpr (H16) s_w[t] = 1.f;   // fp32 slot: o itself, weight 2^(m - M)
        }
    }
    __syncthreads();
    constexpr int UPC = G * D / 4;                           // 4-wide units per cell
    const int total = n * UPC;
    // slot k of unit b: its four outputs, in the slot's own format
    auto load_o = [&](int c, int h, int d, int k) -> f32x4_t {
        if (k < a.n_p) {
            const uint32_t off = pslot_off(a, c, g, k) + SP::o(h, d);
            if constexpr (H16) return part_load4h(r, off);
            else return part_load4(r, off);
        }
        return part_load4(r, gslot_off(a, c, g, k - a.n_p) + SG::o(h, d));
    };
    for (int u0 = threadIdx.x; u0 < total; u0 += NT * kMergeUnits) {
        float M[kMergeUnits], L[kMergeUnits];
        f32x4_t O[kMergeUnits];
        int cb[kMergeUnits], hb[kMergeUnits], db[kMergeUnits];
        int sm_off[kMergeUnits];
#pragma unroll
        for (int b = 0; b < kMergeUnits; ++b) {
            const int u = min(u0 + b * NT, total - 1);   // tail units repeat a valid one
            const int i = u / UPC, rem = u % UPC;
            hb[b] = rem / (D / 4);
            db[b] = 4 * (rem % (D / 4));
            const int c = list[i];
            cb[b] = c;
            sm_off[b] = i * per_cell + hb[b];
            const bool zero_term = has_zero_term(a, c);
            float mx = zero_term ? 0.f : -INFINITY;
            for (int k = 0; k < a.n_slots; ++k) mx = fmaxf(mx, s_m[sm_off[b] + k * G]);
            M[b] = mx;
            L[b] = zero_term ? (float)zero_slots(a, c) * fast_exp2(-mx) : 0.f;
            O[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        int k = 0;
        for (; k + 2 <= a.n_slots; k += 2) {
            f32x4_t v0[kMergeUnits], v1[kMergeUnits];
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) {
                v0[b] = load_o(cb[b], hb[b], db[b], k);
                v1[b] = load_o(cb[b], hb[b], db[b], k + 1);
            }
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) {
                const int s0 = sm_off[b] + k * G, s1 = sm_off[b] + (k + 1) * G;
                fold_pslot<H16>(s_m[s0], s_l[s0], s_w[s0], v0[b], M[b], L[b], O[b]);
                fold_pslot<H16>(s_m[s1], s_l[s1], s_w[s1], v1[b], M[b], L[b], O[b]);
            }
        }
        if (k < a.n_slots) {
            f32x4_t v0[kMergeUnits];
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) v0[b] = load_o(cb[b], hb[b], db[b], k);
#pragma unroll
            for (int b = 0; b < kMergeUnits; ++b) {
                const int s0 = sm_off[b] + k * G;
                fold_pslot<H16>(s_m[s0], s_l[s0], s_w[s0], v0[b], M[b], L[b], O[b]);
            }
        }
#pragma unroll
        for (int b = 0; b < kMergeUnits; ++b) {
            const int u = u0 + b * NT;
            if (u < total) {
                const int i = u / UPC, rem = u % UPC;
                const int h = rem / (D / 4), d = 4 * (rem % (D / 4));
                write_row(a, list[i], g * G + h, d, D, M[b], L[b], O[b]);
            }
        }
    }
    if (threadIdx.x < n)
        __hip_atomic_store(&a.counters[list[threadIdx.x] * a.Hkv + g], 0, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Cache policies of the generated-row loads.  Each K load instruction covers
// 64 bytes of 16 rows (the MFMA operand layout), so the other half of every
// 128-byte line arrives with the next instruction: K loads stay normal
// (non-temporal ones, which do not keep the line, measured slower).  V
// loads cover whole lines; with a long prompt they are non-temporal, so that
// the generated rows, read once, do not push the prompt tiles the prompt
// items share out of the caches (the host sets AttnArgs::gen_v_nt).
constexpr int kAuxNormal = 0;
constexpr int kAuxStream = 2;

// f32 inputs, one launch per call: blocks [0, n_prompt_items) are prompt
// items (cell, KV head, prompt chunk), the rest generated-row items; the
// last item of a (cell, KV head) merges its partials.
template <int D, int G>
__global__ __launch_bounds__(kThreads) void items_kernel(AttnArgs a) {
    constexpr bool BF16 = false;
    __shared__ __attribute__((aligned(16))) char buf[Lds<D, G, BF16>::BYTES];
    __shared__ int s_list[2];
    const int tid = threadIdx.x;
    int item = blockIdx.x;
    int c, g;
    if (item < a.n_prompt_items) {
        const int pk = item % a.n_p;
        item /= a.n_p;
        g = item % a.Hkv;
        c = item / a.Hkv;
        prompt_item_valu<D, G, BF16>(a, c, g, pk, buf);
    } else {
        item -= a.n_prompt_items;
        const int gk = item % a.n_g;
        item /= a.n_g;
        g = item % a.Hkv;
        c = item / a.Hkv;
        gen_item<D, G, BF16>(a, c, g, gk, buf);
    }
    stores_performed();
    if (tid == 0) {
        s_list[0] = arrive(a, c, g) ? 1 : 0;
        s_list[1] = c;
    }
    __syncthreads();
    if (s_list[0]) combine_cells<D, G, kThreads, false>(a, s_list + 1, 1, g, buf);
}

// ------------------------------------------------------- bf16, long prompts
//
// One launch per call, two kinds of work group:
//   shared-prompt items (prompt_wide.hpp), work group = (KV head, group of
//     Fused::ROWS rows, prompt chunk), where the rows of a KV head are the
//     (cell, q head) pairs of every cell, unspliced cells first, and a group
//     holds rows of one class only -- each K/V tile of the chunk is staged
//     in LDS once for all of the group's rows, and every row gets one
//     partial result;
//   generated-row items, work group = (KV head, a few consecutive cells),
//     whose waves stream each cell's generated rows into one more partial;
//     the item waits for the prompt partials of its cells and merges them
//     (slot order: prompt chunks, then the generated rows; then the ZERO
//     term) into out and lse.
// Blocks [0, n_prompt_items) are the prompt items.  Work groups start in
// block order, so the prompt items a generated-row item waits for have
// started before it.

// Default bound of a generated-row item's wait for the prompt partials: a
// poll is one agent-scope load (about a microsecond under load) plus a short
// sleep, so 16384 polls stay around 16 ms -- far beyond any prompt item.
constexpr int kDefaultWaitPolls = 16384;

// Work-group shape: NW waves (splice::fused_waves), NT threads, ROWS rows
// of a prompt item.  Tiles in flight: the prompt items' LDS ring, and the
// registers of each generated-row wave, within the registers a lane has at
// WAVES_PER_SIMD waves per SIMD (168 at 3, 256 at 2).
template <int D>
struct Fused {
    static constexpr int NW = splice::fused_waves(D);
    static constexpr int NT = NW * 64;
    static constexpr int RB = splice::fused_row_blocks(D);
    static constexpr int ROWS = splice::group_rows(D);
    static constexpr int GEN_DEPTH = D <= 128 ? 2 : 1;
    static constexpr int WAVES_PER_SIMD = D <= 128 ? 3 : 2;
    static_assert(ROWS == NW * 16 * RB, "host and device agree on the row groups");
};

// The prompt slots 0 .. n_p - 1 (n_p <= B) of one (row, four outputs) in one
// round of loads: M over the slots and this item's own maximum Mg, the ZERO
// term, then the slots folded in order (the fixed fold order).
template <int D, int G, int B>
__device__ __forceinline__ void merge_slots_once(const AttnArgs &a, __amdgpu_buffer_rsrc_t r, uint32_t sbase, int h,
                                                 int d, int nz, float Mg, float &M, float &Ls, f32x4_t &O) {
    f32x4_t ok[B];
    float mk[B], lk[B], wk[B];
#pragma unroll
    for (int j = 0; j < B; ++j)
        if (j < a.n_p) load_pslot<D, G, true>(r, sbase + (uint32_t)j * a.p_slot_bytes, h, d, ok[j], mk[j], lk[j], wk[j]);
#pragma unroll
    for (int j = 0; j < B; ++j)
        if (j < a.n_p) M = fmaxf(M, mk[j]);
    M = fmaxf(M, Mg);
    if (nz > 0) Ls = (float)nz * fast_exp2(-M);
#pragma unroll
    for (int j = 0; j < B; ++j)
        if (j < a.n_p) fold_pslot<true>(mk[j], lk[j], wk[j], ok[j], M, Ls, O);
}

template <int D, int G>
struct FusedLds {
    static constexpr int NW = Fused<D>::NW;
    static constexpr int PROMPT = Direct<D>::LDS;
    static constexpr int WAVE_MERGE = NW * G * (D + 2) * 4;                     // waves_merge buffer
    static constexpr int GEN = cmax(NW * WaveMfma<D>::LDS, WAVE_MERGE);         // V^T tiles, wave merge
    static constexpr int MERGE = 3 * kRowBlock * kMaxSlots * 4;                 // combine_cells staging (m, l, w)
    static constexpr int BYTES = cmax(cmax(PROMPT, GEN), MERGE);
    static_assert(BYTES <= 160 * 1024 - 4096, "fits the LDS of a compute unit");
};

// Most cells one item can complete: the cells of one row group.
template <int D, int G>
constexpr int fused_max_merge() { return Fused<D>::ROWS / G; }

// Each item returns its KV head and leaves in s_list the count and the list
// of the cells it completed (a merge handed over by a generated-row item).
//
// Work groups are handed to the eight XCDs in turn (block b to XCD b mod
// 8).  Prompt block b serves unit u = (KV head, chunk) and row group rg with
// b mod 8 = u mod 8, so every row group of a unit runs on one XCD and the
// unit's tiles come from that XCD's L2 after the first read.  Blocks with u
// past the last unit (a grid padded to whole rounds of eight) do nothing.
template <int D, int G>
__device__ int fused_prompt_item(const AttnArgs &a, int item, char *lds, int *s_list) {
    constexpr int RB = Fused<D>::RB, ROWS = Fused<D>::ROWS;
    constexpr int X8 = splice::kXcds;
    using X = Direct<D>;
    const int rg = (item / X8) % a.n_rb;
    const int u = (item / X8 / a.n_rb) * X8 + item % X8;
    if (u >= a.n_p * a.Hkv) return 0;   // s_list[0] stays 0: nothing to merge
    const int g = u / a.n_p, pk = u % a.n_p;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const char *qrow[RB];
    int cell[RB], hh[RB], lo[RB];
    bool ok[RB];
    // row groups of unspliced cells come first; a group never mixes classes
    const bool clean_group = rg < a.n_rg_clean;
    const int first_cell = clean_group ? 0 : a.n_clean;
    const int end_cell = clean_group ? a.n_clean : a.n_active;
    const int grp = clean_group ? rg : rg - a.n_rg_clean;
    static_for<0, RB>([&](auto rb) {
        const int R = grp * ROWS + (wave * RB + rb) * 16 + col;
        const int cidx = first_cell + R / G;
        ok[rb] = cidx < end_cell;
        cell[rb] = ok[rb] ? a.order[cidx] : 0;
        hh[rb] = R % G;
        lo[rb] = a.row_lo && ok[rb] ? cell_geo(a, cell[rb]).jp0 : 0;
        qrow[rb] = ok[rb] ? a.q + ((size_t)cell[rb] * a.Hq + (size_t)g * G + hh[rb]) * X::ROW : nullptr;
    });

    // the prompt chunk: clean before and after the span; the span from the
    // clean cache (unspliced rows), the donor cache (spliced rows) or not at
    // all (ZERO splice: its closed-form term is added by the merge)
    const int k0 = a.jp0 + pk * a.p_len;
    const int k1 = min(k0 + a.p_len, a.Tp);
    const size_t head = (size_t)g * a.Tp * X::ROW;
    const char *ck = a.ck + head, *cv = a.cv + head;
    const int pre1 = min(k1, a.sa), sp0 = max(k0, a.sa), sp1 = min(k1, a.sb), post0 = max(k0, a.sb);
    KeyList L;
    list_init(L);
    list_add<X::TK>(L, ck + (size_t)k0 * X::ROW, cv + (size_t)k0 * X::ROW, pre1 - k0, kColsAll, k0);
    if (clean_group) {
        list_add<X::TK>(L, ck + (size_t)sp0 * X::ROW, cv + (size_t)sp0 * X::ROW, sp1 - sp0, kColsAll, sp0);
    } else if (!a.zero_donor) {
        const char *dk = a.dk + head, *dv = a.dv + head;
        list_add<X::TK>(L, dk + (size_t)sp0 * X::ROW, dv + (size_t)sp0 * X::ROW, sp1 - sp0, kColsAll, sp0);
    }
    list_add<X::TK>(L, ck + (size_t)post0 * X::ROW, cv + (size_t)post0 * X::ROW, k1 - post0, kColsAll, post0);

    WideState<D, RB> S;
    static_for<0, RB>([&](auto rb) {
        static_for<0, X::NDT>([&](auto t) { S.o[rb][t] = f32x4_t{0.f, 0.f, 0.f, 0.f}; });
        S.m[rb] = -INFINITY;
        S.lsum[rb] = 0.f;
    });
    direct_stream<D, RB, Fused<D>::NW>(L, qrow, a.qk_scale, a.row_lo != 0, lo, lds, S);

    // each row's partial as a 16-bit slot: o / (l sc) in fp16, m, l, w = l sc
    using SL = Slot<D, G, true>;
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    static_for<0, RB>([&](auto rb) {
        float l = S.lsum[rb];
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        float amax = 0.f;
        static_for<0, X::NDT>([&](auto t) {
            static_for<0, 4>([&](auto i) { amax = fmaxf(amax, fabsf(S.o[rb][t][(int)i])); });
        });
        amax = fmaxf(amax, __shfl_xor(amax, 16));
        amax = fmaxf(amax, __shfl_xor(amax, 32));
        const float inv_l = l > 0.f ? 1.f / l : 0.f;
        const float big = amax * inv_l;
        const float sc = big > kH16Limit ? exp2f(ceilf(log2f(big / kH16Limit))) : 1.f;
        const float mul = inv_l / sc;
        if (ok[rb]) {
            const uint32_t slot = pslot_off(a, cell[rb], g, pk);
            static_for<0, X::NDT / 2>([&](auto u) {
                const f32x4_t lo = S.o[rb][2 * u] * mul, hi = S.o[rb][2 * u + 1] * mul;
                const h16x8_t h = __builtin_convertvector(
                    (f32x8_t{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w}), h16x8_t);
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, h), r,
                                                       slot + SL::o(hh[rb], 32 * u + 4 * quad), 0, kSc1);
            });
            if (quad == 0) part_store4(r, slot + SL::m(hh[rb]), f32x4_t{S.m[rb], l, l * sc, 0.f});
        }
    });
    stores_performed();
    // count this chunk on each cell of the group
    const int c0 = first_cell + grp * (ROWS / G);
    const int n_cells = min(ROWS / G, end_cell - c0);
    if ((int)threadIdx.x < n_cells) {
        const int c = a.order[c0 + threadIdx.x];
        if (arrive(a, c, g)) s_list[1 + atomicAdd(&s_list[0], 1)] = c;
    }
    __syncthreads();
    return g;
}

// In-place merge of a generated-row item whose cells' prompt partials are
// all stored: the item's own partial (its waves combined through LDS) is
// the last slot and never leaves the chip.  A unit is eight outputs of one
// (cell, q head), d0 .. d0 + 3 and d0 + 16 .. d0 + 19: one 16-byte load per
// prompt slot.  Each thread owns up to U units per round; the loads of
// every prompt slot of a round's units are issued before the waves'
// partials are combined, so their latency overlaps the LDS work.  Fold
// order (fixed, as in combine_cells): the ZERO term, the prompt slots in
// order, this item's slot; each output is folded exactly as there.
template <int D, int G, int NW, int B, int U>
__device__ __forceinline__ void gen_merge_in_place(const AttnArgs &a, const WaveState<D> &S, char *buf, int wpp,
                                                   int n_pairs, int c0, int g) {
    using W = WaveMfma<D>;
    using SL = Slot<D, G, true>;
    constexpr int NT = NW * 64;
    constexpr int UPR = D / 8;       // units per (cell, q head)
    constexpr int UPG = G * UPR;     // units per (cell, KV head)
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, quad = lane >> 4;
    const int total = n_pairs * UPG;
    float *s_o = reinterpret_cast<float *>(buf);   // [NW][G][D]
    float *s_m = s_o + NW * G * D;                  // [NW][G]
    float *s_l = s_m + NW * G;                      // [NW][G]
    // the waves' partials into LDS (every wave is done with its V^T tile)
    if (col < G) {
        static_for<0, W::NDT>([&](auto t) {
            *reinterpret_cast<f32x4_t *>(s_o + (wave * G + col) * D + 16 * t + 4 * quad) = S.o[t];
        });
        if (quad == 0) {
            s_m[wave * G + col] = S.m;
            s_l[wave * G + col] = S.lsum;
        }
    }
    for (int e0 = 0; e0 < total; e0 += NT * U) {
        u32x4_t ok[U][B];   // eight fp16 outputs
        float mk[U][B], lk[U][B], wk[U][B];
        int pe[U], he[U], de[U];
        static_for<0, U>([&](auto u) {
            const int e = min(e0 + (int)u * NT + tid, total - 1);   // past the end: repeat a valid unit
            pe[u] = e / UPG;
            he[u] = (e % UPG) / UPR;
            const int r8 = e % UPR;
            de[u] = 32 * (r8 >> 2) + 4 * (r8 & 3);
            const uint32_t sbase = pslot_off(a, a.gorder[c0 + pe[u]], g, 0);
#pragma unroll
            for (int j = 0; j < B; ++j) {
                if (j < a.n_p) {
                    const uint32_t off = sbase + (uint32_t)j * a.p_slot_bytes;
                    ok[u][j] = __builtin_amdgcn_raw_buffer_load_b128(r, off + SL::o(he[u], de[u]), 0, kSc1);
                    const f32x4_t mlw = part_load4(r, off + SL::m(he[u]));
                    mk[u][j] = mlw.x;
                    lk[u][j] = mlw.y;
                    wk[u][j] = mlw.z;
                }
            }
        });
        __syncthreads();   // the staged partials are visible (first round); no-op ordering after
        static_for<0, U>([&](auto u) {
            const int e = e0 + (int)u * NT + tid;
            const int cq = a.gorder[c0 + pe[u]];
            if (e < total) {
                const int h = he[u], d0 = de[u], d1 = d0 + 16, w0 = pe[u] * wpp;
                // this item's partial: its waves combined
                float Mg = -INFINITY;
#pragma unroll
                for (int i = 0; i < NW; ++i)
                    if (i < wpp) Mg = fmaxf(Mg, s_m[(w0 + i) * G + h]);
                const float Mgs = Mg == -INFINITY ? 0.f : Mg;
                float Lg = 0.f;
                f32x4_t Og0 = {0.f, 0.f, 0.f, 0.f}, Og1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int i = 0; i < NW; ++i) {
                    if (i < wpp) {
                        const int w = w0 + i;
                        const float f = fast_exp2(s_m[w * G + h] - Mgs);
                        Lg = fmaf(s_l[w * G + h], f, Lg);
                        Og0 += *reinterpret_cast<const f32x4_t *>(s_o + (w * G + h) * D + d0) * f;
                        Og1 += *reinterpret_cast<const f32x4_t *>(s_o + (w * G + h) * D + d1) * f;
                    }
                }
                const int nz = zero_slots(a, cq);
                float M = nz > 0 ? 0.f : -INFINITY;
#pragma unroll
                for (int j = 0; j < B; ++j)
                    if (j < a.n_p) M = fmaxf(M, mk[u][j]);
                M = fmaxf(M, Mg);
                float Ls = nz > 0 ? (float)nz * fast_exp2(-M) : 0.f, Ls1 = Ls;
                f32x4_t O0 = {0.f, 0.f, 0.f, 0.f}, O1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    if (j < a.n_p) {
                        const f32x8_t v = __builtin_convertvector(__builtin_bit_cast(h16x8_t, ok[u][j]), f32x8_t);
                        fold_pslot<true>(mk[u][j], lk[u][j], wk[u][j], f32x4_t{v[0], v[1], v[2], v[3]}, M, Ls, O0);
                        fold_pslot<true>(mk[u][j], lk[u][j], wk[u][j], f32x4_t{v[4], v[5], v[6], v[7]}, M, Ls1, O1);
                    }
                }
                fold_slot(Mg, Lg, Og0, M, Ls, O0);   // this item's slot, a.n_p, comes last
                fold_slot(Mg, Lg, Og1, M, Ls1, O1);
                write_row(a, cq, g * G + h, d0, D, M, Ls, O0);
                write_row(a, cq, g * G + h, d1, D, M, Ls1, O1);
            }
        });
    }
}

// Generated-row item: KV head g and P = a.gen_pairs consecutive cells of
// a.gorder (the cells with generated rows to stream, longest first, so the
// grid holds no empty items and the longest streams are dispatched first),
// wpp = NW / P waves per (cell, KV head) pair streaming that cell's generated
// rows (interleaved tiles).  After streaming, the first wave polls the pairs' counters (a lane per pair)
// until every prompt chunk has stored its partial (at most a.wait_polls polls
// in all; prompt items have lower block indices and never wait, so they are
// dispatched first and finish).  Then this item merges in place: its own
// partial is the last slot and never leaves the chip.  Past the bound it
// stores its partials and counts itself like any other item, and the last
// arrival merges.  Under a decode step the item first appends each active
// cell's new row (a.kn, a.vn) to its generated caches, and streams that row
// from a.kn, a.vn rather than reading it back; finished cells are skipped.
template <int D, int G>
__device__ int fused_gen_item(const AttnArgs &a, int item, char *lds, int *s_list) {
    using W = WaveMfma<D>;
    constexpr int NW = Fused<D>::NW, NT = Fused<D>::NT;
    const int P = a.gen_pairs, wpp = NW / P;
    const int g = item % a.Hkv;
    const int c0 = (item / a.Hkv) * P;   // first of the item's cells in gorder
    const int n_pairs = min(P, a.n_gen_cells - c0);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const bool valid = wave / wpp < n_pairs;
    const int c = valid ? a.gorder[c0 + wave / wpp] : 0;   // this wave's cell
    const int col = threadIdx.x & 15;
    if (a.kn) {   // append: row s of each active cell's generated K and V
        constexpr int U = W::ROW / 16;   // 16-byte units of a row
        for (int t = threadIdx.x; t < n_pairs * 2 * U; t += NT) {
            const int cq = a.gorder[c0 + t / (2 * U)], kv = (t / U) & 1, u = t % U;
            const size_t src = ((size_t)cq * a.Hkv + g) * W::ROW + 16 * u;
            const size_t dst = (((size_t)cq * a.Hkv + g) * (size_t)a.cap + cell_geo(a, cq).s) * W::ROW + 16 * u;
            char *to = const_cast<char *>(kv ? a.gv : a.gk);
            *reinterpret_cast<u32x4_t *>(to + dst) = *reinterpret_cast<const u32x4_t *>((kv ? a.vn : a.kn) + src);
        }
    }
    bf16x8_t qb[W::NDS];
    load_q_cols<D>(valid ? a.q + ((size_t)c * a.Hq + (size_t)g * G + col % G) * W::ROW : nullptr, qb);
    KeyList L;
    list_init(L);
    if (valid) {
        const CellGeo geo = cell_geo(a, c);
        const size_t goff = (((size_t)c * a.Hkv + g) * (size_t)a.cap + geo.i0) * W::ROW;
        if (a.kn) {   // rows before the current one from the cache, the current one as given
            list_add(L, a.gk + goff, a.gv + goff, geo.n_gen - 1);
            const size_t noff = ((size_t)c * a.Hkv + g) * W::ROW;
            list_add(L, a.kn + noff, a.vn + noff, 1);
        } else if (a.trunk >= 0 && c != a.trunk) {
            // forked sweep: rows below the fork step are the trunk's, the rest the cell's own
            const int i1 = geo.i0 + geo.n_gen, wf = min(max(a.wfork[c], geo.i0), i1);
            const size_t toff = (((size_t)a.trunk * a.Hkv + g) * (size_t)a.cap + geo.i0) * W::ROW;
            list_add(L, a.gk + toff, a.gv + toff, wf - geo.i0);
            const size_t ooff = (((size_t)c * a.Hkv + g) * (size_t)a.cap + wf) * W::ROW;
            list_add(L, a.gk + ooff, a.gv + ooff, i1 - wf);
        } else {
            list_add(L, a.gk + goff, a.gv + goff, geo.n_gen);
        }
    }
    WaveState<D> S;
    state_init(S);
    const ColMask cm{true, true, true};
    if (a.gen_v_nt)
        wave_stream<D, Fused<D>::GEN_DEPTH, kAuxNormal, kAuxStream>(L, wave % wpp, wpp, cm, qb, a.qk_scale,
                                                                     lds + wave * W::LDS, S);
    else
        wave_stream<D, Fused<D>::GEN_DEPTH, kAuxNormal, kAuxNormal>(L, wave % wpp, wpp, cm, qb, a.qk_scale,
                                                                     lds + wave * W::LDS, S);
    state_finish(S);

    if (threadIdx.x < 64) {   // wave 0: lane q polls the counter of pair q, all pairs at once
        const int lane = threadIdx.x;
        const bool mine = lane < n_pairs && a.n_p > 0;
        const int *cnt = a.counters + (int)a.gorder[c0 + (mine ? lane : 0)] * a.Hkv + g;
        bool done = !mine;
        // wait_polls == 0: never look, so every pair of the item is handed
        // over (the counter is not read even when the partials are in)
        for (int polls = 0; polls < a.wait_polls; ++polls) {   // polls: the same in every lane
            if (!done) done = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= a.n_p;
            if (__all(done)) break;
            __builtin_amdgcn_s_sleep(4);
        }
        const bool ready = __all(done);
        if (lane == 0) s_list[0] = ready ? -1 : 0;
        // count the pairs this item hands over (the ones that have prompt
        // partials to wait for); a fallback the caller can read back
        const uint64_t handed = __ballot(mine);
        if (!ready && lane == 0 && handed)
            __hip_atomic_fetch_add(a.stats, (int)__popcll(handed), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();   // also: every wave is done with its V^T tile
    const bool ready = s_list[0] < 0;
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    if (ready) {
        if (a.n_p <= 8) {
            gen_merge_in_place<D, G, NW, 8, 1>(a, S, lds, wpp, n_pairs, c0, g);
        } else {
        waves_merge<D, G, NW>(S, lds, wpp, n_pairs, [&](int q, int h, int d, float Mg, float Lg, f32x4_t Og) {
            const int cq = a.gorder[c0 + q];
            const uint32_t sbase = pslot_off(a, cq, g, 0);
            const int nz = zero_slots(a, cq);
            float M = nz > 0 ? 0.f : -INFINITY;
            float Ls = 0.f;
            f32x4_t O = {0.f, 0.f, 0.f, 0.f};
            if (a.n_p <= 8) {
                merge_slots_once<D, G, 8>(a, r, sbase, h, d, nz, Mg, M, Ls, O);
            } else if (a.n_p <= 16) {
                merge_slots_once<D, G, 16>(a, r, sbase, h, d, nz, Mg, M, Ls, O);
            } else {
                using SL = Slot<D, G, true>;
                constexpr int B = 8;
                for (int k = 0; k < a.n_p; ++k)
                    M = fmaxf(M, part_load1(r, sbase + (uint32_t)k * a.p_slot_bytes + SL::m(h)));
                M = fmaxf(M, Mg);
                if (nz > 0) Ls = (float)nz * fast_exp2(-M);
                for (int k0 = 0; k0 < a.n_p; k0 += B) {
                    f32x4_t ok[B];
                    float mk[B], lk[B], wk[B];
#pragma unroll
                    for (int j = 0; j < B; ++j)
                        load_pslot<D, G, true>(r, sbase + (uint32_t)min(k0 + j, a.n_p - 1) * a.p_slot_bytes, h, d, ok[j],
                                               mk[j], lk[j], wk[j]);
#pragma unroll
                    for (int j = 0; j < B; ++j)
                        if (k0 + j < a.n_p) fold_pslot<true>(mk[j], lk[j], wk[j], ok[j], M, Ls, O);
                }
            }
            fold_slot(Mg, Lg, Og, M, Ls, O);   // this item's slot, a.n_p, comes last
            write_row(a, cq, g * G + h, d, D, M, Ls, O);
        });
        }
        if ((int)threadIdx.x < n_pairs)
            __hip_atomic_store(a.counters + (int)a.gorder[c0 + threadIdx.x] * a.Hkv + g, 0, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        if (threadIdx.x == 0) s_list[0] = 0;   // nothing left to merge
    } else {
        waves_merge<D, G, NW>(S, lds, wpp, n_pairs, [&](int q, int h, int d, float M, float Lsum, f32x4_t O) {
            using SG = Slot<D, G, false>;
            const uint32_t slot = gslot_off(a, a.gorder[c0 + q], g, 0);
            part_store4(r, slot + SG::o(h, d), O);
            if (d == 0) {
                part_store1(r, slot + SG::m(h), M);
                part_store1(r, slot + SG::l(h), Lsum);
            }
        });
        stores_performed();
        if ((int)threadIdx.x < n_pairs && arrive(a, a.gorder[c0 + threadIdx.x], g))
            s_list[1 + atomicAdd(&s_list[0], 1)] = a.gorder[c0 + threadIdx.x];
    }
    __syncthreads();
    return g;
}

template <int D, int G>
__global__ __launch_bounds__(Fused<D>::NT) __attribute__((amdgpu_waves_per_eu(Fused<D>::WAVES_PER_SIMD)))
void fused_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) char lds[FusedLds<D, G>::BYTES];
    constexpr int MAXM = fused_max_merge<D, G>();
    __shared__ int s_list[1 + MAXM];   // [0] count, [1..] cells to merge
    static_assert(MAXM <= Fused<D>::NT, "one thread per cell of a row group");
    if (threadIdx.x == 0) {
        s_list[0] = 0;
        trunk_written() = 0;
    }
    __syncthreads();
    const int g = (int)blockIdx.x < a.n_prompt_items
                      ? fused_prompt_item<D, G>(a, blockIdx.x, lds, s_list)
                      : fused_gen_item<D, G>(a, blockIdx.x - a.n_prompt_items, lds, s_list);
    const int n = s_list[0];
    // merge in batches whose (m, l) staging fits
    const int per = max(1, (kRowBlock * kMaxSlots) / (a.n_slots * G));
    for (int i = 0; i < n; i += per) {
        combine_cells<D, G, Fused<D>::NT, true>(a, s_list + 1 + i, min(per, n - i), g, lds);
        __syncthreads();
    }
    if (a.trunk >= 0 && a.n_dormant > 0) {   // uniform: a forked sweep
        __syncthreads();
        if (trunk_written()) dormant_copy<D, G, Fused<D>::NT>(a, g, lds);
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
                                    kp = pick_base(donor, a.ck, a.dk) + off;
                                    vp = pick_base(donor, a.cv, a.dv) + off;
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

// ------------------------------------------------------------ dispatch

typedef void (*attn_fn)(AttnArgs);
struct AttnKernels {
    attn_fn items;      // one launch of prompt and generated-row items with merge
    attn_fn cellwise;   // f32, short prompts: one work group per (cell, KV head)
};

template <int D, int G, bool BF16>
AttnKernels kernels_of() {
    if constexpr (BF16)
        return AttnKernels{fused_kernel<D, G>, nullptr};
    else
        return AttnKernels{items_kernel<D, G>, cellwise_kernel<D, G, BF16>};
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

// One per instantiation unit (attn_d<D>_<type>.hip).
AttnKernels attn_kernels_d64_bf16(int G);
AttnKernels attn_kernels_d128_bf16(int G);
AttnKernels attn_kernels_d256_bf16(int G);
AttnKernels attn_kernels_d64_f32(int G);
AttnKernels attn_kernels_d128_f32(int G);
AttnKernels attn_kernels_d256_f32(int G);

}  // namespace splice_dev
