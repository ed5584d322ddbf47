// prompt_wide.hpp -- the shared-prompt contraction: many (cell, q head) rows
// of one KV head against the same prompt tiles, on the matrix cores.
//
// A work group of NW waves owns NW * 16 * RB rows; each wave owns RB blocks
// of 16 rows.  A 32-key tile of the prompt (K row-major, V transposed) is
// staged in LDS once per work group and then, per wave,
//   S  = K Q^T  : the K operand (16 keys x 32 d) is read from LDS once and
//                 multiplied into all RB row blocks (v_mfma_f32_16x16x32_bf16);
//   online softmax per row (column of S), masked per segment class;
//   O^T += V^T P: each 16 d x 32 keys V^T operand is read once and multiplied
//                 into all RB row blocks, P rounded to bf16 (the sums of P
//                 stay in fp32).
// The LDS tiles are double-buffered and the global loads of the next
// DEPTH - 1 tiles are in flight while one is computed; one barrier per tile
// orders the buffers.
#pragma once

#include "plan.hpp"
#include "wave_mfma.hpp"

namespace splice_dev {

template <int D, int RB_>
struct Wide {
    static constexpr int RB = RB_;                          // 16-row blocks per wave
    static constexpr int TK = 32;                           // keys per tile
    static constexpr int ROW = D * 2;                       // bytes per K or V row
    static constexpr int NDS = D / 32;                      // k-steps of q.k
    static constexpr int NDT = D / 16;                      // 16-row d tiles of the output
    static constexpr int KROW = ROW + 16;                   // K tile row stride in LDS (padded)
    static constexpr int VROW = TK * 2 + 8;                 // V^T tile row stride in LDS (padded)
    static constexpr int KTILE = TK * KROW;
    static constexpr int BUF = KTILE + D * VROW;            // one staged tile
    static constexpr int LDS = 2 * BUF;                     // double buffer
};

// How NT threads share the loads of one tile: KU 16-byte K units (unit u is
// bytes 16 (u mod D/8) of key row u / (D/8)) owned by threads 0, 1, ...;
// VU V units of 2 keys x 8 d (keys 2 kp, 2 kp + 1 with kp = u mod 16, bytes
// 16 dg with dg = u / 16) owned by the last VU threads (all threads in
// turn when VU >= NT), so that a thread owning both is rare.
template <int D, int NT>
struct TileShare {
    static constexpr int KU = Wide<D, 1>::TK * (D / 8);
    static constexpr int VU = (D / 8) * (Wide<D, 1>::TK / 2);
    static constexpr int NKU = (KU + NT - 1) / NT;
    static constexpr int NVU = (VU + NT - 1) / NT;
    static constexpr int VSHIFT = VU < NT ? NT - VU : 0;
    static_assert(NVU <= 2 && NKU <= 4, "tile staging assumes 64 <= D <= 256");
};

// One thread's share of a tile in flight.
template <int D, int NT>
struct WideRegs {
    u32x4_t k[TileShare<D, NT>::NKU];
    u32x4_t v[TileShare<D, NT>::NVU][2];
};

template <int D, int NT>
__device__ __forceinline__ void wide_fetch(const TileRef &t, WideRegs<D, NT> &r) {
    using X = Wide<D, 1>;
    using T = TileShare<D, NT>;
    const int tid = threadIdx.x;
    const __amdgpu_buffer_rsrc_t rk = rows_rsrc(t.k, t.n * X::ROW);
    const __amdgpu_buffer_rsrc_t rv = rows_rsrc(t.v, t.n * X::ROW);
    static_for<0, T::NKU>([&](auto i) {
        const int u = tid + NT * i;
        if (T::KU % NT == 0 || u < T::KU) r.k[i] = row_load<0>(rk, (u / (D / 8)) * X::ROW + (u % (D / 8)) * 16);
    });
    static_for<0, T::NVU>([&](auto i) {
        const int u = tid - T::VSHIFT + NT * i;
        if ((T::VSHIFT == 0 && T::VU % NT == 0) || (u >= 0 && u < T::VU)) {
            const int kp = u & 15, dg = u >> 4;
            r.v[i][0] = row_load<0>(rv, (2 * kp) * X::ROW + 16 * dg);
            r.v[i][1] = row_load<0>(rv, (2 * kp + 1) * X::ROW + 16 * dg);
        }
    });
}

// K row-major (16-byte units), V transposed: row d holds the tile's keys.
// The 16 lanes of one dg fill a 64-byte V^T row segment; the four dg of a
// wave land 8 rows apart, 16 banks apart.
template <int D, int NT>
__device__ __forceinline__ void wide_stage(const WideRegs<D, NT> &r, char *buf) {
    using X = Wide<D, 1>;
    using T = TileShare<D, NT>;
    const int tid = threadIdx.x;
    char *sK = buf;
    char *sV = buf + X::KTILE;
    static_for<0, T::NKU>([&](auto i) {
        const int u = tid + NT * i;
        if (T::KU % NT == 0 || u < T::KU)
            *reinterpret_cast<u32x4_t *>(sK + (u / (D / 8)) * X::KROW + (u % (D / 8)) * 16) = r.k[i];
    });
    static_for<0, T::NVU>([&](auto i) {
        const int u = tid - T::VSHIFT + NT * i;
        if ((T::VSHIFT == 0 && T::VU % NT == 0) || (u >= 0 && u < T::VU)) {
            const int kp = u & 15, dg = u >> 4;
            static_for<0, 8>([&](auto j) {
                constexpr int jj = decltype(j)::value;
                constexpr uint32_t sel = (jj & 1) ? 0x07060302u : 0x05040100u;
                *reinterpret_cast<uint32_t *>(sV + (8 * dg + jj) * X::VROW + 4 * kp) =
                    __builtin_amdgcn_perm(r.v[i][1][jj >> 1], r.v[i][0][jj >> 1], sel);
            });
        }
    });
}

// Streaming state of one wave: RB row blocks, lane (quad, col) holding row
// block rb's column col (o[rb][t][i] = O^T[16 t + 4 quad + i][col]).
template <int D, int RB>
struct WideState {
    f32x4_t o[RB][Wide<D, RB>::NDT];
    float m[RB];
    float lsum[RB];
};

// One staged tile for this wave's RB row blocks.  A work group's rows all
// belong to one class (unspliced or spliced cells), so every tile of its list
// is visible to every row; rows past the last cell compute values that are
// never stored.  A partial tile (n_valid < TK) masks its missing keys; with
// row_lo set, a row also masks the keys before its own first visible slot
// lo[rb] (rows of cells at different steps under a sliding window), the
// tile's first key being slot key0.
template <int D, int RB>
__device__ __forceinline__ void wide_compute(const char *buf, int n_valid, int key0, bool row_lo,
                                             const int (&lo)[RB],
                                             const bf16x8_t (&qb)[RB][Wide<D, RB>::NDS], float qk_scale,
                                             WideState<D, RB> &S) {
    using X = Wide<D, RB>;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    const char *sK = buf;
    const char *sV = buf + X::KTILE;
    f32x4_t s[X::RB][2];
    static_for<0, X::RB>([&](auto rb) {
        s[rb][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        s[rb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    });
    static_for<0, 2>([&](auto h) {
        static_for<0, X::NDS>([&](auto st) {
            const bf16x8_t kf = *reinterpret_cast<const bf16x8_t *>(
                sK + (16 * h + col) * X::KROW + (32 * st + 8 * quad) * 2);
            static_for<0, X::RB>([&](auto rb) {
                s[rb][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qb[rb][st], s[rb][h], 0, 0, 0);
            });
        });
    });
    bf16x8_t pb[X::RB];
    static_for<0, X::RB>([&](auto rb) {
        float x[2][4];
        static_for<0, 2>([&](auto h) {
            static_for<0, 4>([&](auto i) { x[h][i] = s[rb][h][(int)i] * qk_scale; });
        });
        if (n_valid < X::TK) {   // uniform: only the last tile of a segment
            static_for<0, 2>([&](auto h) {
                static_for<0, 4>([&](auto i) {
                    if (16 * h + 4 * quad + i >= n_valid) x[h][i] = -INFINITY;
                });
            });
        }
        if (row_lo) {   // uniform
            static_for<0, 2>([&](auto h) {
                static_for<0, 4>([&](auto i) {
                    if (key0 + 16 * h + 4 * quad + i < lo[rb]) x[h][i] = -INFINITY;
                });
            });
        }
        float mt = -INFINITY;
        static_for<0, 2>([&](auto h) { static_for<0, 4>([&](auto i) { mt = fmaxf(mt, x[h][i]); }); });
        mt = fmaxf(mt, __shfl_xor(mt, 16));
        mt = fmaxf(mt, __shfl_xor(mt, 32));
        const bool need = mt > S.m[rb] + kSlack;
        if (__any(need)) {
            const float mn = need ? fmaxf(S.m[rb], mt) : S.m[rb];
            const float al = need ? fast_exp2(S.m[rb] - (mn == -INFINITY ? 0.f : mn)) : 1.f;
            S.lsum[rb] *= al;
            static_for<0, X::NDT>([&](auto t) { S.o[rb][t] *= al; });
            S.m[rb] = mn;
        }
        const float ms = S.m[rb] == -INFINITY ? 0.f : S.m[rb];
        static_for<0, 8>([&](auto j) {
            constexpr int jj = decltype(j)::value;
            const float p = fast_exp2(x[jj >> 2][jj & 3] - ms);
            S.lsum[rb] += p;
            pb[rb][jj] = (__bf16)p;
        });
    });
    // k-slot 8 quad + j is key 4 quad + j (j < 4) or 16 + 4 quad + (j - 4):
    // the keys whose scores this lane holds
    static_for<0, X::NDT>([&](auto t) {
        const char *vrow = sV + (16 * t + col) * X::VROW;
        const uint2 va = *reinterpret_cast<const uint2 *>(vrow + 8 * quad);
        const uint2 vb = *reinterpret_cast<const uint2 *>(vrow + 32 + 8 * quad);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, make_uint4(va.x, va.y, vb.x, vb.y));
        static_for<0, X::RB>([&](auto rb) {
            S.o[rb][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb[rb], S.o[rb][t], 0, 0, 0);
        });
    });
}

template <int D, int RB, int DEPTH, int NT>
__device__ __forceinline__ void wide_stream(const KeyList &L, const bf16x8_t (&qb)[RB][Wide<D, RB>::NDS],
                                            float qk_scale, bool row_lo, const int (&lo)[RB], char *lds,
                                            WideState<D, RB> &S) {
    using X = Wide<D, RB>;
    const int n_tiles = list_tiles(L);
    if (n_tiles == 0) return;
    WideRegs<D, NT> r[DEPTH];
    TileRef ref[DEPTH];
    static_for<0, DEPTH>([&](auto i) {
        ref[i] = list_tile_or_empty<X::TK>(L, i, n_tiles, X::ROW);
        wide_fetch<D, NT>(ref[i], r[i]);
    });
    wide_stage<D, NT>(r[0], lds);
    __syncthreads();
    for (int base = 0; base < n_tiles; base += DEPTH) {
        static_for<0, DEPTH>([&](auto j) {
            constexpr int jn = (decltype(j)::value + 1) % DEPTH;
            const int t = base + j;
            const bool live = t < n_tiles;   // false only in the last round
            const TileRef cur = ref[j];
            // registers of tile t are free (staged last iteration): refill them
            // with tile t + DEPTH, or an empty tile past the end, on every
            // path, so the count of loads in flight never depends on `live`
            ref[j] = list_tile_or_empty<X::TK>(L, t + DEPTH, n_tiles, X::ROW);
            wide_fetch<D, NT>(ref[j], r[j]);
            if (live) {
                wide_compute<D, RB>(lds + (t & 1) * X::BUF, cur.n, cur.key0, row_lo, lo, qb, qk_scale, S);
                if (t + 1 < n_tiles) wide_stage<D, NT>(r[jn], lds + ((t + 1) & 1) * X::BUF);
                __syncthreads();   // the next buffer is staged; nobody reads this one any more
            }
        });
    }
}

}  // namespace splice_dev
