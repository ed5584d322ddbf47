// attn_kernels.hpp -- the spliced decode-attention kernels (templates over
// head_dim D, group size G and element type).  Each attn_*.hip translation
// unit instantiates one (D, element type) pair, so the six pairs compile in
// parallel and no kernel is instantiated twice.
#pragma once

#include "device_common.hpp"
#include "wave_mfma.hpp"

namespace splice_dev {

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
    // bf16 generated-row items: one V^T tile per wave, then the wave merge
    static constexpr int GEN_TILES = BF16 ? kWaves * WaveMfma<D>::LDS : 0;
    static constexpr int GEN_MERGE = BF16 ? kWaves * G * (D + 2) * 4 : 0;
    static constexpr int BYTES = cmax(cmax(TILES, MERGE), cmax(STAGE, cmax(GEN_TILES, GEN_MERGE)));
};

// LDS of the bf16 cellwise kernel.
template <int D, int G>
struct CellwiseLds {
    static constexpr int BYTES = cmax(kWaves * WaveMfma<D>::LDS, kWaves * G * (D + 2) * 4);
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

// Generated rows of one (cell, KV head) on the matrix cores (bf16): the four
// waves take interleaved 32-row tiles of the chunk and merge in LDS.
template <int D, int G>
__device__ void gen_item_mfma(const AttnArgs &a, int c, int g, int gk, char *buf) {
    using W = WaveMfma<D>;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: tile pointers stay scalar
    bf16x8_t qb[W::NDS];
    load_q_mfma<D, G>(a.q + ((size_t)c * a.Hq + (size_t)g * G) * W::ROW, qb);
    const int r0 = a.i0 + gk * a.g_len;
    const int r1 = min(r0 + a.g_len, a.i0 + a.n_gen);
    const size_t off = (((size_t)c * a.Hkv + g) * (size_t)a.cap + r0) * W::ROW;
    KeyList L;
    list_init(L);
    list_add(L, a.gk + off, a.gv + off, r1 - r0);
    WaveState<D> S;
    state_init(S);
    wave_stream<D>(L, wave, kWaves, qb, a.qk_scale, buf + wave * W::LDS, S);
    state_finish(S);
    const __amdgpu_buffer_rsrc_t r = part_rsrc(a);
    const uint32_t slot = slot_off(a, c, g, a.n_p + gk);
    waves_merge<D, G>(S, buf, [&](int h, int d, float M, float L, f32x4_t O) {
        part_store4(r, slot + (uint32_t)(h * D + d) * 4u, O);
        if (d == 0) {
            part_store1(r, slot + (uint32_t)(G * D + h) * 4u, M);
            part_store1(r, slot + (uint32_t)(G * D + G + h) * 4u, L);
        }
    });
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
        tile_fetch<D>(kreg, vreg, pick_base(dpass, a.ck, a.dk) + head, pick_base(dpass, a.cv, a.dv) + head, t0,
                      tile_end(t0));
    while (t0 < k1) {
        const int t1 = tile_end(t0);
        const int cur_dpass = dpass;
        __syncthreads();   // the previous step no longer reads the LDS tiles
        tile_stage<D>(kreg, vreg, sK, sV);
        __syncthreads();
        int nt0 = t0, ndpass = dpass;
        advance(nt0, ndpass);
        if (nt0 < k1)   // in flight while this step computes
            tile_fetch<D>(kreg, vreg, pick_base(ndpass, a.ck, a.dk) + head, pick_base(ndpass, a.cv, a.dv) + head, nt0,
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
        if constexpr (BF16)
            gen_item_mfma<D, G>(a, c, g, gk, buf);
        else
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

// bf16 cellwise kernel: the same per-(cell, KV head) work group, streaming
// the cell's list on the matrix cores.  The list is cut into segments that
// are contiguous in memory -- prompt before the span, the span (clean or
// donor; absent for a ZERO splice), prompt after the span, generated rows --
// and the span segment exists whether or not the cell is spliced, so a
// splice never moves a tile boundary.
template <int D, int G>
__global__ __launch_bounds__(kThreads) void cellwise_mfma_kernel(AttnArgs a) {
    using W = WaveMfma<D>;
    __shared__ __attribute__((aligned(16))) char buf[CellwiseLds<D, G>::BYTES];
    const int g = blockIdx.x % a.Hkv;
    const int c = blockIdx.x / a.Hkv;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: tile pointers stay scalar
    bf16x8_t qb[W::NDS];
    load_q_mfma<D, G>(a.q + ((size_t)c * a.Hq + (size_t)g * G) * W::ROW, qb);
    const bool spl = bit_set(a.spliced, c);
    const bool zskip = spl && a.zero_donor;
    const bool from_donor = spl && !a.zero_donor;
    const size_t head = (size_t)g * a.Tp * W::ROW;
    KeyList L;
    list_init(L);
    if (a.Tp > 0) {
        list_add(L, a.ck + head + (size_t)a.jp0 * W::ROW, a.cv + head + (size_t)a.jp0 * W::ROW, a.sa - a.jp0);
        if (!zskip)
            list_add(L, pick_base(from_donor, a.ck, a.dk) + head + (size_t)a.sa * W::ROW,
                     pick_base(from_donor, a.cv, a.dv) + head + (size_t)a.sa * W::ROW, a.sb - a.sa);
        list_add(L, a.ck + head + (size_t)a.sb * W::ROW, a.cv + head + (size_t)a.sb * W::ROW, a.Tp - a.sb);
    }
    const size_t goff = (((size_t)c * a.Hkv + g) * (size_t)a.cap + a.i0) * W::ROW;
    list_add(L, a.gk + goff, a.gv + goff, a.n_gen);
    WaveState<D> S;
    state_init(S);
    wave_stream<D>(L, wave, kWaves, qb, a.qk_scale, buf + wave * W::LDS, S);
    state_finish(S);
    const int nsv = a.sb - a.sa;
    const bool zero_term = zskip && nsv > 0;
    waves_merge<D, G>(S, buf, [&](int h, int d, float M, float L, f32x4_t O) {
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
    attn_fn rowblock, cellwise;
};

template <int D, int G, bool BF16>
AttnKernels kernels_of() {
    if constexpr (BF16)
        return AttnKernels{attn_kernel<D, G, BF16>, cellwise_mfma_kernel<D, G>};
    else
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

// One per instantiation unit (attn_d<D>_<type>.hip).
AttnKernels attn_kernels_d64_bf16(int G);
AttnKernels attn_kernels_d128_bf16(int G);
AttnKernels attn_kernels_d256_bf16(int G);
AttnKernels attn_kernels_d64_f32(int G);
AttnKernels attn_kernels_d128_f32(int G);
AttnKernels attn_kernels_d256_f32(int G);

}  // namespace splice_dev
