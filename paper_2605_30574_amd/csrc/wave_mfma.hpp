// wave_mfma.hpp -- one wave streams K/V rows through the matrix cores for 16
// query rows at once (bf16 inputs, fp32 accumulation).
//
// The keys of a list are processed in tiles of 16.  For a tile the wave
// computes, for its 16 query rows ("columns"),
//   S = K Q^T   with v_mfma_f32_16x16x32_bf16: A = 16 keys x 32 d of K, loaded
//               from memory straight into the operand layout; B = Q^T;
//   online softmax per column (running maximum shared by the column's lanes);
//   O^T += V^T P with v_mfma_f32_16x16x16_bf16: A = 16 d x 16 keys of V^T,
//               read from a per-wave LDS tile that holds V transposed; B = P
//               rounded to bf16, which stays in the lanes where S came out
//               (the running sums of P stay in fp32).
// The 16 columns are either the G heads of one (cell, KV head) repeated
// (column j -> head j mod G), or 16 different (cell, head) rows of one KV
// head reading a shared prompt.  Waves never synchronise with each other
// while streaming: each owns its LDS tile, and the next tile's loads are in
// flight while the current one is computed.
#pragma once

#include "device_common.hpp"

namespace splice_dev {

constexpr int kTileKeys = 16;
constexpr int kMaxSeg = 4;

typedef short i16x4_t __attribute__((ext_vector_type(4)));

// Which columns a segment's keys are visible to.
enum SegCols : int {
    kColsAll = 0,     // every valid column
    kColsClean = 1,   // columns of unspliced cells (span read from the clean cache)
    kColsDonor = 2,   // columns of spliced cells (span read from the donor cache)
};

// An ordered key list made of up to kMaxSeg segments; the rows of a segment
// are contiguous (row stride D bf16) from k[s] / v[s].  Tiles never straddle
// a segment, so tile boundaries depend only on the segment lengths.
struct KeyList {
    const char *k[kMaxSeg];
    const char *v[kMaxSeg];
    int len[kMaxSeg];
    int cols[kMaxSeg];             // SegCols
    int key0[kMaxSeg];             // position of the segment's first key (prompt slots)
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
        L.cols[s] = kColsAll;
        L.key0[s] = 0;
    }
}

// Appends n rows starting at (k, v); empty segments are dropped.  Tiles hold
// TK keys (a list is built and walked with one TK).  The segment index only
// takes constant values after unrolling, so the list stays in scalar
// registers.
template <int TK = kTileKeys>
__device__ __forceinline__ void list_add(KeyList &L, const char *k, const char *v, int n, int cols = kColsAll,
                                         int key0 = 0) {
    if (n <= 0) return;
    const int tiles = (n + TK - 1) / TK;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s) {
        if (s == L.n_seg) {
            L.k[s] = k;
            L.v[s] = v;
            L.len[s] = n;
            L.cols[s] = cols;
            L.key0[s] = key0;
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

// Where tile t lies: base pointers of its first key, its valid key count,
// which columns see it and the position of its first key.
struct TileRef {
    const char *k, *v;
    int n;
    int cols;
    int key0;
};

template <int TK = kTileKeys>
__device__ __forceinline__ TileRef list_tile(const KeyList &L, int t, int row_bytes) {
    TileRef r{L.k[0], L.v[0], 0, kColsAll, 0};
    int off = t;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s) {
        if (s < L.n_seg && t >= L.first_tile[s]) {
            off = t - L.first_tile[s];
            r.k = L.k[s];
            r.v = L.v[s];
            r.n = L.len[s];
            r.cols = L.cols[s];
            r.key0 = L.key0[s];
        }
    }
    const int t0 = off * TK;
    r.k += (size_t)t0 * row_bytes;
    r.v += (size_t)t0 * row_bytes;
    r.n = min(TK, r.n - t0);
    r.key0 += t0;
    return r;
}

// A tile reference that loads nothing: its buffer range is empty, so every
// row load returns 0 without a memory access.  Issuing loads for it keeps the
// number of loads in flight the same on every path, which lets the compiler
// wait for exactly the tile it needs instead of for all of them.
__device__ __forceinline__ TileRef empty_tile(const KeyList &L) { return TileRef{L.k[0], L.v[0], 0, kColsAll, 0}; }

template <int TK = kTileKeys>
__device__ __forceinline__ TileRef list_tile_or_empty(const KeyList &L, int t, int n_tiles, int row_bytes) {
    return t < n_tiles ? list_tile<TK>(L, t, row_bytes) : empty_tile(L);
}

template <int D>
struct WaveMfma {
    static constexpr int ROW = D * 2;               // bytes per K or V row
    static constexpr int NDS = D / 32;              // k-steps of q.k
    static constexpr int NDT = D / 16;              // 16-row d tiles of the output
    static constexpr int DG = D / 8;                // 16-byte groups of a row
    static constexpr int UNITS = 4 * DG;            // V units (4 keys x 8 d) per tile
    static constexpr int NVU = (UNITS + 63) / 64;   // V units per lane
    static constexpr int VROW = kTileKeys * 2 + 8;  // bytes per d row of the V^T tile (padded)
    static constexpr int LDS = D * VROW;            // V^T tile of one wave
};

// Registers of one tile in flight.
template <int D>
struct TileRegs {
    u32x4_t k[WaveMfma<D>::NDS];      // [k-step]
    u32x4_t v[WaveMfma<D>::NVU][4];   // [unit][key of the unit]
};

// Raw buffer resource over [base, base + bytes): loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const char *base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(base), 0, bytes, 0x00020000);
}

// Row load with cache policy AUX (0 normal, 2 non-temporal).
template <int AUX>
__device__ __forceinline__ u32x4_t row_load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX));
}

template <int D, int KAUX, int VAUX>
__device__ __forceinline__ void tile_load_aux(const TileRef &t, TileRegs<D> &r) {
    using W = WaveMfma<D>;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    const __amdgpu_buffer_rsrc_t rk = rows_rsrc(t.k, t.n * W::ROW);
    const __amdgpu_buffer_rsrc_t rv = rows_rsrc(t.v, t.n * W::ROW);
    const int koff = col * W::ROW + 16 * quad;
    static_for<0, W::NDS>([&](auto st) { r.k[st] = row_load<KAUX>(rk, koff + 64 * st); });
    static_for<0, W::NVU>([&](auto n) {
        const int u = lane + 64 * n;
        const int kq = u & 3, dg = u >> 2;   // unit: keys 4 kq .. 4 kq + 3, bytes 16 dg .. 16 dg + 15
        if (u < W::UNITS) {
            static_for<0, 4>([&](auto kk) { r.v[n][kk] = row_load<VAUX>(rv, (4 * kq + kk) * W::ROW + 16 * dg); });
        }
    });
}


// V^T tile: row d holds the tile's 16 keys (bf16) at byte 2 * key.  The
// four lanes of a unit row write one 32-byte row segment together.
template <int D>
__device__ __forceinline__ void tile_stage_vt(const TileRegs<D> &r, char *sVt) {
    using W = WaveMfma<D>;
    const int lane = threadIdx.x & 63;
    static_for<0, W::NVU>([&](auto n) {
        const int u = lane + 64 * n;
        const int kq = u & 3, dg = u >> 2;
        if (u < W::UNITS) {
            static_for<0, 8>([&](auto j) {
                constexpr int jj = decltype(j)::value;
                constexpr uint32_t sel = (jj & 1) ? 0x07060302u : 0x05040100u;
                const uint32_t lo = __builtin_amdgcn_perm(r.v[n][1][jj >> 1], r.v[n][0][jj >> 1], sel);
                const uint32_t hi = __builtin_amdgcn_perm(r.v[n][3][jj >> 1], r.v[n][2][jj >> 1], sel);
                *reinterpret_cast<u32x2_t *>(sVt + (8 * dg + jj) * W::VROW + 8 * kq) = u32x2_t{lo, hi};
            });
        }
    });
}

// Streaming state of one wave.  Lane (quad, col) holds column col:
// o[t][i] = O^T[16 t + 4 quad + i][col] relative to m; lsum is this lane's
// share of the column's sum (the four quads add up at the end).
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

// B operand of q.k: lane (quad, col) holds q_row[32 st + 8 quad ..+8] of the
// query row that column col stands for (zeros when q_row is null).
template <int D>
__device__ __forceinline__ void load_q_cols(const char *q_row, bf16x8_t (&qb)[WaveMfma<D>::NDS]) {
    const int quad = (threadIdx.x & 63) >> 4;
    static_for<0, WaveMfma<D>::NDS>([&](auto st) {
        uint4 w = make_uint4(0, 0, 0, 0);
        if (q_row) w = *reinterpret_cast<const uint4 *>(q_row + (32 * st + 8 * quad) * 2);
        qb[st] = __builtin_bit_cast(bf16x8_t, w);
    });
}

// Per-lane visibility of the three segment classes for this lane's column.
struct ColMask {
    bool all, clean, donor;
    __device__ __forceinline__ bool on(int cols) const {
        return cols == kColsAll ? all : (cols == kColsClean ? clean : donor);
    }
};

// One tile: q.k, online softmax, p.v.  `kr` holds the tile's K rows; its V
// rows have been staged in sVt by this wave.
template <int D>
__device__ __forceinline__ void tile_compute(const u32x4_t (&kr)[WaveMfma<D>::NDS], int n_valid, bool col_on,
                                             const bf16x8_t (&qb)[WaveMfma<D>::NDS], float qk_scale,
                                             const char *sVt, WaveState<D> &S) {
    using W = WaveMfma<D>;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
    static_for<0, W::NDS>([&](auto st) {
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[st]), qb[st], s, 0, 0, 0);
    });
    // raw q.k; the scale (> 0) enters the maximum once and each weight's
    // exponent as one fma
    float x[4];
    float mt = -INFINITY;
    static_for<0, 4>([&](auto i) {
        const int key = 4 * quad + i;
        x[i] = (col_on && key < n_valid) ? s[(int)i] : -INFINITY;
        mt = fmaxf(mt, x[i]);
    });
    mt *= qk_scale;
    // lazy rescale: a column moves its maximum only when a score exceeds it
    // by more than kSlack (weights stay <= 2^kSlack).  Each lane checks its
    // own scores first; only then are the column's four lanes combined, so
    // that every lane of a column takes the same decision (other columns
    // multiply by exactly 1)
    if (__any(mt > S.m + kSlack)) {
        mt = fmaxf(mt, __shfl_xor(mt, 16));
        mt = fmaxf(mt, __shfl_xor(mt, 32));
        const bool need = mt > S.m + kSlack;
        const float mn = need ? fmaxf(S.m, mt) : S.m;
        const float al = need ? fast_exp2(S.m - (mn == -INFINITY ? 0.f : mn)) : 1.f;
        S.lsum *= al;
        static_for<0, W::NDT>([&](auto t) { S.o[t] *= al; });
        S.m = mn;
    }
    const float ms = S.m == -INFINITY ? 0.f : S.m;
    i16x4_t pb;
    static_for<0, 4>([&](auto i) {
        const float p = fast_exp2(fmaf(x[i], qk_scale, -ms));
        S.lsum += p;
        pb[(int)i] = __builtin_bit_cast(short, (__bf16)p);
    });
    // k-slot 4 quad + i of the p.v product is key 4 quad + i: the keys whose
    // scores this lane holds
    static_for<0, W::NDT>([&](auto t) {
        const uint2 va = *reinterpret_cast<const uint2 *>(sVt + (16 * t + col) * W::VROW + 8 * quad);
        const i16x4_t vf = __builtin_bit_cast(i16x4_t, va);
        S.o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vf, pb, S.o[t], 0, 0, 0);
    });
}

// Stream tiles t = first, first + step, ... of the list through one wave,
// keeping DEPTH tiles in flight: when tile t is computed, the loads of the
// next DEPTH - 1 tiles are outstanding.  The loop is unrolled DEPTH times so
// the register sets are only ever indexed by constants.  KAUX and VAUX are
// the cache policies of the K and the V row loads (0 normal, 2
// non-temporal); they are constants so that every path issues the same
// loads.
template <int D, int DEPTH, int KAUX, int VAUX>
__device__ __forceinline__ void wave_stream(const KeyList &L, int first, int step, const ColMask &cm,
                                            const bf16x8_t (&qb)[WaveMfma<D>::NDS], float qk_scale, char *sVt,
                                            WaveState<D> &S) {
    const int n_tiles = list_tiles(L);
    if (first >= n_tiles) return;
    TileRegs<D> r[DEPTH];
    TileRef ref[DEPTH];
    static_for<0, DEPTH>([&](auto i) {
        ref[i] = list_tile_or_empty(L, first + i * step, n_tiles, WaveMfma<D>::ROW);
        tile_load_aux<D, KAUX, VAUX>(ref[i], r[i]);
    });
    for (int base = first; base < n_tiles; base += DEPTH * step) {
        static_for<0, DEPTH>([&](auto j) {
            const int t = base + j * step;
            const bool live = t < n_tiles;   // false only in the last round
            // V goes to LDS and K is kept aside, so the loads of tile
            // t + DEPTH * step are issued into these registers before the tile
            // is computed.  The loads are issued on every path (an empty tile
            // past the end), so the count in flight never depends on `live`.
            if (live) tile_stage_vt<D>(r[j], sVt);
            u32x4_t kr[WaveMfma<D>::NDS];
            static_for<0, WaveMfma<D>::NDS>([&](auto st) { kr[st] = r[j].k[st]; });
            const TileRef cur = ref[j];
            ref[j] = list_tile_or_empty(L, t + DEPTH * step, n_tiles, WaveMfma<D>::ROW);
            tile_load_aux<D, KAUX, VAUX>(ref[j], r[j]);
            if (live) tile_compute<D>(kr, cur.n, cm.on(cur.cols), qb, qk_scale, sVt, S);
        });
    }
}

// Column sums: after this every lane of a column holds the column's sum.
template <int D>
__device__ __forceinline__ void state_finish(WaveState<D> &S) {
    S.lsum += __shfl_xor(S.lsum, 16);
    S.lsum += __shfl_xor(S.lsum, 32);
}

// Merge the waves of a work group in groups of wpp consecutive waves (each
// wave with its WaveState, finished; a group's waves stream the same G heads,
// in columns j mod G) through LDS, and hand every group of four consecutive
// outputs of head h of group p < n_groups to sink(p, h, d, M, L, O) -- M and
// L in base-2 units, O not yet divided by L.  `buf` needs NW * G * (D + 2)
// floats and may alias the V^T tiles.  Called by all threads.
template <int D, int G, int NW, typename Sink>
__device__ __forceinline__ void waves_merge(WaveState<D> &S, char *buf, int wpp, int n_groups, Sink sink) {
    using W = WaveMfma<D>;
    float *s_o = reinterpret_cast<float *>(buf);          // [NW][G][D]
    float *s_m = s_o + NW * G * D;                          // [NW][G]
    float *s_l = s_m + NW * G;                              // [NW][G]
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
    constexpr int UPG = G * D / 4;   // units of four outputs per group
    for (int e = tid; e < n_groups * UPG; e += NW * 64) {
        const int p = e / UPG, h = (e % UPG) / (D / 4), d = 4 * (e % (D / 4));
        const int w0 = p * wpp;
        float M = -INFINITY;
#pragma unroll
        for (int i = 0; i < NW; ++i)
            if (i < wpp) M = fmaxf(M, s_m[(w0 + i) * G + h]);
        const float Ms = M == -INFINITY ? 0.f : M;
        float L = 0.f;
        f32x4_t O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            if (i < wpp) {
                const int w = w0 + i;
                const float f = fast_exp2(s_m[w * G + h] - Ms);
                L = fmaf(s_l[w * G + h], f, L);
                O += *reinterpret_cast<const f32x4_t *>(s_o + (w * G + h) * D + d) * f;
            }
        }
        sink(p, h, d, M, L, O);
    }
}

}  // namespace splice_dev
