// wave_mfma.hpp -- one wave streams the K/V rows of one (cell, KV head)
// through the matrix cores (bf16 inputs, fp32 accumulation).
//
// The keys of a list are processed in tiles of 32.  For a tile the wave
// computes, for all G query heads of the KV head at once,
//   S = K Q^T   with v_mfma_f32_16x16x32_bf16: A = 16 keys x 32 d of K, loaded
//               from memory straight into the operand layout; B = Q^T with
//               the 16 columns holding heads (column j -> head j mod G);
//   online softmax per column (running maximum shared by the column's lanes);
//   O^T += V^T P with the same instruction: A = 16 d x 32 keys of V^T, read
//               from a per-wave LDS tile that holds V transposed; B = P, which
//               stays in the lanes where S came out (split into a bf16 high
//               part and a bf16 remainder, so p is carried to ~2^-17).
// Waves never synchronise with each other while streaming: each owns its
// LDS tile, and the next tile's loads are in flight while the current one is
// computed.
#pragma once

#include "device_common.hpp"

namespace splice_dev {

constexpr int kTileKeys = 32;
constexpr int kMaxSeg = 4;

// An ordered key list made of up to kMaxSeg segments; the rows of a segment
// are contiguous (row stride D bf16) from k[s] / v[s].  Tiles never straddle
// a segment, so tile boundaries depend only on the segment lengths.
struct KeyList {
    const char *k[kMaxSeg];
    const char *v[kMaxSeg];
    int len[kMaxSeg];
    int first_tile[kMaxSeg + 1];   // tiles before segment s; [n_seg] = total
    int n_seg;
};

__device__ __forceinline__ void list_init(KeyList &L) {
    L.n_seg = 0;
#pragma unroll
    for (int s = 0; s <= kMaxSeg; ++s) L.first_tile[s] = 0;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s) {
        L.k[s] = nullptr;
        L.v[s] = nullptr;
        L.len[s] = 0;
    }
}

// Appends n rows starting at (k, v); empty segments are dropped.  The
// segment index only ever takes constant values after unrolling, so the
// list stays in scalar registers.
__device__ __forceinline__ void list_add(KeyList &L, const char *k, const char *v, int n) {
    if (n <= 0) return;
    const int tiles = (n + kTileKeys - 1) / kTileKeys;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s) {
        if (s == L.n_seg) {
            L.k[s] = k;
            L.v[s] = v;
            L.len[s] = n;
            L.first_tile[s + 1] = L.first_tile[s] + tiles;
        } else if (s > L.n_seg) {
            L.first_tile[s + 1] = L.first_tile[s] + tiles;
        }
    }
    L.n_seg += 1;
}

__device__ __forceinline__ int list_tiles(const KeyList &L) {
    int t = 0;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s)
        if (s < L.n_seg) t = L.first_tile[s + 1];
    return t;
}

// Where tile t lies: base pointers of its first key and the number of keys.
struct TileRef {
    const char *k, *v;
    int n;
};

__device__ __forceinline__ TileRef list_tile(const KeyList &L, int t, int row_bytes) {
    TileRef r{L.k[0], L.v[0], 0};
    int off = t;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s) {
        if (s < L.n_seg && t >= L.first_tile[s]) {
            off = t - L.first_tile[s];
            r.k = L.k[s];
            r.v = L.v[s];
            r.n = L.len[s];
        }
    }
    const int t0 = off * kTileKeys;
    r.k += (size_t)t0 * row_bytes;
    r.v += (size_t)t0 * row_bytes;
    r.n = min(kTileKeys, r.n - t0);
    return r;
}

template <int D>
struct WaveMfma {
    static constexpr int ROW = D * 2;               // bytes per K or V row
    static constexpr int NDS = D / 32;              // k-steps of q.k
    static constexpr int NDT = D / 16;              // 16-row d tiles of the output
    static constexpr int NVU = D / 64;              // V units (4 keys x 8 d) per lane per tile
    static constexpr int VROW = kTileKeys * 2 + 8;  // bytes per d row of the V^T tile (padded)
    static constexpr int LDS = D * VROW;            // V^T tile of one wave
};

// Registers of one tile in flight.
template <int D>
struct TileRegs {
    u32x4_t k[2][WaveMfma<D>::NDS];   // [16-key half][k-step]
    u32x4_t v[WaveMfma<D>::NVU][4];   // [unit][key of the unit]
};

// Raw buffer resource over [base, base + bytes): loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const char *base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(base), 0, bytes, 0x00020000);
}

template <int D>
__device__ __forceinline__ void tile_load(const TileRef &t, TileRegs<D> &r) {
    using W = WaveMfma<D>;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    const __amdgpu_buffer_rsrc_t rk = rows_rsrc(t.k, t.n * W::ROW);
    const __amdgpu_buffer_rsrc_t rv = rows_rsrc(t.v, t.n * W::ROW);
    static_for<0, 2>([&](auto h) {
        const int off = (16 * h + col) * W::ROW + 16 * quad;
        static_for<0, W::NDS>([&](auto st) {
            r.k[h][st] = __builtin_amdgcn_raw_buffer_load_b128(rk, off + 64 * st, 0, 0);
        });
    });
    static_for<0, W::NVU>([&](auto n) {
        const int u = lane + 64 * n;
        const int dg = u % (D / 8), kq = u / (D / 8);
        static_for<0, 4>([&](auto kk) {
            r.v[n][kk] = __builtin_amdgcn_raw_buffer_load_b128(rv, (4 * kq + kk) * W::ROW + 16 * dg, 0, 0);
        });
    });
}

// V^T tile: row d holds the tile's 32 keys (bf16) at byte 2 * key.
template <int D>
__device__ __forceinline__ void tile_stage_vt(const TileRegs<D> &r, char *sVt) {
    using W = WaveMfma<D>;
    const int lane = threadIdx.x & 63;
    static_for<0, W::NVU>([&](auto n) {
        const int u = lane + 64 * n;
        const int dg = u % (D / 8), kq = u / (D / 8);
        static_for<0, 8>([&](auto j) {
            constexpr int jj = decltype(j)::value;
            constexpr uint32_t sel = (jj & 1) ? 0x07060302u : 0x05040100u;
            const uint32_t lo = __builtin_amdgcn_perm(r.v[n][1][jj >> 1], r.v[n][0][jj >> 1], sel);
            const uint32_t hi = __builtin_amdgcn_perm(r.v[n][3][jj >> 1], r.v[n][2][jj >> 1], sel);
            *reinterpret_cast<u32x2_t *>(sVt + (8 * dg + jj) * W::VROW + 8 * kq) = u32x2_t{lo, hi};
        });
    });
}

// Streaming state of one wave.  Lane (quad, col) holds column col (head
// col mod G): o[t][i] = O^T[16 t + 4 quad + i][col] relative to m; lsum is
// this lane's share of the column's sum (the four quads add up at the end).
template <int D>
struct WaveState {
    f32x4_t o[WaveMfma<D>::NDT];
    float m;
    float lsum;
};

template <int D>
__device__ __forceinline__ void state_init(WaveState<D> &S) {
    static_for<0, WaveMfma<D>::NDT>([&](auto t) { S.o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f}; });
    S.m = -INFINITY;
    S.lsum = 0.f;
}

// B operand of q.k: lane (quad, col) holds q[head col mod G][32 st + 8 quad ..+8].
template <int D, int G>
__device__ __forceinline__ void load_q_mfma(const char *q_heads, bf16x8_t (&qb)[WaveMfma<D>::NDS]) {
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    const char *row = q_heads + (size_t)(col % G) * (D * 2);
    static_for<0, WaveMfma<D>::NDS>([&](auto st) {
        qb[st] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4 *>(row + (32 * st + 8 * quad) * 2));
    });
}

// One tile: q.k, online softmax, p.v.  `kr` holds the tile's K rows; its V
// rows have been staged in sVt by this wave.
template <int D>
__device__ __forceinline__ void tile_compute(const u32x4_t (&kr)[2][WaveMfma<D>::NDS], int n_valid,
                                             const bf16x8_t (&qb)[WaveMfma<D>::NDS], float qk_scale,
                                             const char *sVt, WaveState<D> &S) {
    using W = WaveMfma<D>;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    f32x4_t s[2];
    static_for<0, 2>([&](auto h) {
        s[h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        static_for<0, W::NDS>([&](auto st) {
            s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[h][st]), qb[st], s[h], 0, 0, 0);
        });
    });
    float x[2][4];
    float mt = -INFINITY;
    static_for<0, 2>([&](auto h) {
        static_for<0, 4>([&](auto i) {
            const int key = 16 * h + 4 * quad + i;
            x[h][i] = key < n_valid ? s[h][(int)i] * qk_scale : -INFINITY;
            mt = fmaxf(mt, x[h][i]);
        });
    });
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    // lazy rescale: a column moves its maximum only when a score exceeds it
    // by more than kSlack (weights stay <= 2^kSlack); every lane of a column
    // takes the same decision
    const bool need = mt > S.m + kSlack;
    if (__any(need)) {
        const float mn = need ? fmaxf(S.m, mt) : S.m;
        const float al = need ? fast_exp2(S.m - (mn == -INFINITY ? 0.f : mn)) : 1.f;
        S.lsum *= al;
        static_for<0, W::NDT>([&](auto t) { S.o[t] *= al; });
        S.m = mn;
    }
    const float ms = S.m == -INFINITY ? 0.f : S.m;
    bf16x8_t ph, pl;
    static_for<0, 2>([&](auto h) {
        static_for<0, 4>([&](auto i) {
            constexpr int jj = 4 * decltype(h)::value + decltype(i)::value;
            const float p = fast_exp2(x[h][i] - ms);
            S.lsum += p;
            const __bf16 hb = (__bf16)p;
            ph[jj] = hb;
            pl[jj] = (__bf16)(p - (float)hb);
        });
    });
    // k-slot 8 quad + j of the p.v product is key 4 quad + j (j < 4) or
    // 16 + 4 quad + (j - 4): the keys whose scores this lane holds
    static_for<0, W::NDT>([&](auto t) {
        const char *vrow = sVt + (16 * t + col) * W::VROW;
        const uint2 va = *reinterpret_cast<const uint2 *>(vrow + 8 * quad);
        const uint2 vb = *reinterpret_cast<const uint2 *>(vrow + 32 + 8 * quad);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, make_uint4(va.x, va.y, vb.x, vb.y));
        S.o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, ph, S.o[t], 0, 0, 0);
        S.o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl, S.o[t], 0, 0, 0);
    });
}

// Stream tiles t = first, first + step, ... of the list through one wave.
template <int D>
__device__ __forceinline__ void wave_stream(const KeyList &L, int first, int step, const bf16x8_t (&qb)[WaveMfma<D>::NDS],
                                            float qk_scale, char *sVt, WaveState<D> &S) {
    const int n_tiles = list_tiles(L);
    int t = first;
    if (t >= n_tiles) return;
    TileRegs<D> r;
    TileRef cur = list_tile(L, t, WaveMfma<D>::ROW);
    tile_load<D>(cur, r);
    for (;;) {
        // V goes to LDS and K is kept aside, so the next tile's loads can be
        // issued into `r` before this tile is computed
        tile_stage_vt<D>(r, sVt);
        u32x4_t kr[2][WaveMfma<D>::NDS];
        static_for<0, 2>([&](auto h) { static_for<0, WaveMfma<D>::NDS>([&](auto st) { kr[h][st] = r.k[h][st]; }); });
        const int n_valid = cur.n;
        const int nt = t + step;
        if (nt < n_tiles) {
            cur = list_tile(L, nt, WaveMfma<D>::ROW);
            tile_load<D>(cur, r);
        }
        tile_compute<D>(kr, n_valid, qb, qk_scale, sVt, S);
        if (nt >= n_tiles) break;
        t = nt;
    }
}

// Column sums: after this every lane of a column holds the column's sum.
template <int D>
__device__ __forceinline__ void state_finish(WaveState<D> &S) {
    S.lsum += __shfl_xor(S.lsum, 16);
    S.lsum += __shfl_xor(S.lsum, 32);
}

// Merge the waves of a work group (each with its WaveState, finished) through
// LDS and hand every group of four consecutive outputs of each head to
// sink(h, d, M, L, O) -- M and L in base-2 units, O not yet divided by L.
// `buf` needs kWaves * G * (D + 2) floats and may alias the V^T tiles.
template <int D, int G, typename Sink>
__device__ __forceinline__ void waves_merge(WaveState<D> &S, char *buf, Sink sink) {
    using W = WaveMfma<D>;
    float *s_o = reinterpret_cast<float *>(buf);          // [kWaves][G][D]
    float *s_m = s_o + kWaves * G * D;                      // [kWaves][G]
    float *s_l = s_m + kWaves * G;                          // [kWaves][G]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, quad = lane >> 4;
    __syncthreads();   // every wave is done with its V^T tile
    if (col < G) {
        static_for<0, W::NDT>([&](auto t) {
            *reinterpret_cast<f32x4_t *>(s_o + (wave * G + col) * D + 16 * t + 4 * quad) = S.o[t];
        });
        if (quad == 0) {
            s_m[wave * G + col] = S.m;
            s_l[wave * G + col] = S.lsum;
        }
    }
    __syncthreads();
    for (int e = tid; e < G * D / 4; e += kThreads) {
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
            L = fmaf(s_l[w * G + h], f, L);
            O += *reinterpret_cast<const f32x4_t *>(s_o + (w * G + h) * D + d) * f;
        }
        sink(h, d, M, L, O);
    }
}

}  // namespace splice_dev
