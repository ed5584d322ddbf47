// prompt_wide.hpp -- the shared-prompt contraction: many (cell, q head) rows
// of one KV head against the same prompt tiles, on the matrix cores.
//
// A work group of NW waves owns NW * 16 * RB rows; each wave owns RB blocks
// of 16 rows.  A 32-key tile of the prompt is loaded into LDS once per work
// group, straight from memory (no registers, no staging instructions), and
// then, per wave,
//   S  = K Q^T  : the K operand (16 keys x 32 d) is read from LDS once and
//                 multiplied into all RB row blocks (v_mfma_f32_16x16x32_bf16);
//   online softmax per row (column of S);
//   O^T += V^T P: each 16 d x 32 keys V^T operand is read with transposing
//                 LDS reads and multiplied into all RB row blocks, P rounded
//                 to bf16 (the sums of P stay in fp32).
// A ring of tile buffers keeps the next tiles in flight while one is
// computed; one barrier per tile orders the ring.
#pragma once

#include "plan.hpp"
#include "wave_mfma.hpp"

namespace splice_dev {

// Streaming state of one wave: RB row blocks, lane (quad, col) holding row
// block rb's column col (o[rb][t][i] = O^T[16 t + 4 quad + i][col]).
template <int D, int RB>
struct WideState {
    f32x4_t o[RB][D / 16];
    float m[RB];
    float lsum[RB];
};

// ------------------------------------------------- direct-to-LDS prompt tiles
//
// The tiles go from memory straight into LDS (buffer_load_dwordx4 ... lds:
// lane L of a wave instruction writes 16 bytes at the instruction's LDS base
// + 16 L, from any global address the lane names), so a tile in flight holds
// no registers and needs no staging instructions.  K and V both stay
// row-major; within a row, 16-byte chunk c of key r sits at chunk slot
// c ^ swz(r) (K) or c ^ swz_v(r) (V), which spreads the rows one operand
// read touches over all banks.  The p.v operand (keys along the MFMA k
// dimension) is read with ds_read_b64_tr_b16: in each 16-lane group, lane
// 4a + b receives element b of the 8-byte vectors named by lanes a, a + 4,
// a + 8 and a + 12.  A ring of NB tile buffers keeps NB - 1 tiles in
// flight; one barrier per tile.
template <int D>
struct Direct {
    static constexpr int TK = splice::kPromptTileKeys;             // keys per tile
    static constexpr int ROW = D * 2;                              // bytes per K or V row
    static constexpr int CH = ROW / 16;                            // 16-byte chunks per row
    static constexpr int TILE = TK * ROW;                          // K (or V) tile bytes
    static constexpr int BUF = 2 * TILE;                           // K tile, then V tile
    static constexpr int NB = D <= 64 ? 4 : (D <= 128 ? 3 : 2);    // buffers in the ring
    static constexpr int LDS = NB * BUF;
    static constexpr int NDS = D / 32;                             // k-steps of q.k
    static constexpr int NDT = D / 16;                             // 16-row d tiles of the output
};

// Chunk-slot swizzles (XOR on the 16-byte chunk index) of key row r.  K:
// the 16 rows of one 16-lane quarter-wave read land in 16 different bank
// groups (rows of 128 bytes, D = 64, pair up in one 256-byte bank line, so
// they use r / 2).  V: a half-wave of transposed reads touches 8 keys x 2
// adjacent chunks, so the XOR leaves chunk bit 0 alone and spreads the 8
// keys over the other bits.
template <int D>
__device__ __forceinline__ int swz(int r) {
    return D == 64 ? (r >> 1) & 7 : r & 15;
}
template <int D>
__device__ __forceinline__ int swz_v(int r) {
    return D == 64 ? ((r >> 1) & 3) << 1 : (r & 7) << 1;
}

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

// Wait until at most N vector-memory operations of this wave are in flight
// (s_waitcnt vmcnt(N); expcnt and lgkmcnt left alone).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is six bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Loads of one tile per thread (K and V): the tile's TK * CH chunks of each
// operand are spread over the NW waves, 64 chunks per wave instruction.
template <int D, int NW>
constexpr int direct_loads_per_thread() { return 2 * Direct<D>::TK * Direct<D>::CH / 64 / NW; }

// Raw buffer descriptor over [base, base + bytes) as four words (the form
// make_buffer_rsrc builds: stride 0, dword 3 = 0x00020000).
__device__ __forceinline__ u32x4_t rows_desc(const char *base, int bytes) {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    return u32x4_t{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)p),
                   (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xffffu)),
                   (uint32_t)__builtin_amdgcn_readfirstlane(bytes), 0x00020000u};
}

// One 16-byte-per-lane load into LDS at lds_addr + 16 * lane.  Written as
// inline assembly on purpose: the compiler, which cannot tell the ring's
// buffers apart, would otherwise wait for every load in flight before each
// LDS read (s_waitcnt vmcnt(0)) and undo the prefetch; the stream waits on
// vmcnt itself.  M0 holds the LDS base; the statement declares M0 clobbered,
// so the compiler keeps nothing in it across the load.
__device__ __forceinline__ void lds_dma16(u32x4_t desc, uint32_t lds_addr, int voff) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "buffer_load_dwordx4 %1, %2, 0 offen lds"
        :
        : "s"(lds_addr), "v"(voff), "s"(desc)
        : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_offset(const char *p) {
    return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char *)p);
}

// The part of a tile one thread loads: PER wave instructions per operand;
// instruction i of wave w fills chunk slots 64 (i NW + w) .. + 63, and the
// lane's source offsets within the tile (K and V swizzles) are fixed.
template <int D, int NW>
struct DirectLanes {
    static constexpr int PER = Direct<D>::TK * Direct<D>::CH / 64 / NW;
    static_assert(PER * 64 * NW == Direct<D>::TK * Direct<D>::CH, "whole wave instructions per tile");
    int koff[PER], voff[PER];
    uint32_t slot0[PER];   // byte offset of the instruction's first slot (wave-uniform)
};

template <int D, int NW>
__device__ __forceinline__ DirectLanes<D, NW> direct_lanes() {
    using X = Direct<D>;
    DirectLanes<D, NW> dl;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    static_for<0, DirectLanes<D, NW>::PER>([&](auto i) {
        const int q0 = ((int)i * NW + wave) * 64;
        const int q = q0 + lane;
        const int r = q / X::CH, sl = q % X::CH;
        dl.koff[i] = r * X::ROW + (sl ^ swz<D>(r)) * 16;
        dl.voff[i] = r * X::ROW + (sl ^ swz_v<D>(r)) * 16;
        dl.slot0[i] = (uint32_t)q0 * 16u;
    });
    return dl;
}

// Issue the loads of tile t into the buffer at LDS offset base (rows past
// t.n read as zero: the buffer range of an n-row tile is n rows long).
template <int D, int NW>
__device__ __forceinline__ void direct_issue(const TileRef &t, uint32_t base, const DirectLanes<D, NW> &dl) {
    using X = Direct<D>;
    const u32x4_t rk = rows_desc(t.k, t.n * X::ROW);
    const u32x4_t rv = rows_desc(t.v, t.n * X::ROW);
    static_for<0, DirectLanes<D, NW>::PER>([&](auto i) {
        lds_dma16(rk, base + dl.slot0[i], dl.koff[i]);
        lds_dma16(rv, base + X::TILE + dl.slot0[i], dl.voff[i]);
    });
}

// One tile from LDS for this wave's RB row blocks: q.k, the online softmax
// of each row, p.v.
template <int D, int RB>
__device__ __forceinline__ void direct_compute(const char *buf, int n_valid, int key0, bool row_lo,
                                               const int (&lo)[RB],
                                               const bf16x8_t (&qb)[RB][D / 32], float qk_scale,
                                               WideState<D, RB> &S) {
    using X = Direct<D>;
    const int lane = threadIdx.x & 63, col = lane & 15, quad = lane >> 4;
    const char *sK = buf;
    const char *sV = buf + X::TILE;
    // every operand read of the tile is issued up front: the V reads do not
    // depend on the scores and land while q.k and the softmax run.  V operand
    // of d tile t: lane (quad, col) names key 16 hf + 4 quad + col / 4,
    // elements 16 t + 4 (col mod 4) .. + 3, and receives keys 16 hf + 4 quad
    // + 0..3 at element 16 t + col -- k-slots 8 quad + 4 hf + 0..3, the keys
    // whose scores this lane holds
    bf16x8_t kf[2][X::NDS];
    static_for<0, 2>([&](auto h) {
        const int r = 16 * h + col;
        static_for<0, X::NDS>([&](auto st) {
            const int c = 4 * st + quad;
            kf[h][st] = *reinterpret_cast<const bf16x8_t *>(sK + r * X::ROW + (c ^ swz<D>(r)) * 16);
        });
    });
    const int kr0 = 4 * quad + (col >> 2);
    i16x4_t vt[X::NDT][2];
    static_for<0, X::NDT>([&](auto t) {
        const int c = 2 * t + ((col & 3) >> 1);
        const int b8 = (col & 1) * 8;
        vt[t][0] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4_t *)(sV + kr0 * X::ROW + (c ^ swz_v<D>(kr0)) * 16 + b8));
        vt[t][1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4_t *)(sV + (kr0 + 16) * X::ROW + (c ^ swz_v<D>(kr0 + 16)) * 16 + b8));
    });
    f32x4_t s[RB][2];
    static_for<0, RB>([&](auto rb) {
        s[rb][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        s[rb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    });
    static_for<0, 2>([&](auto h) {
        static_for<0, X::NDS>([&](auto st) {
            static_for<0, RB>([&](auto rb) {
                s[rb][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[h][st], qb[rb][st], s[rb][h], 0, 0, 0);
            });
        });
    });
    bf16x8_t pb[RB];
    static_for<0, RB>([&](auto rb) {
        // raw q.k here; the scale (> 0) enters the maximum once and each
        // weight's exponent as one fma
        float x[2][4];
        static_for<0, 2>([&](auto h) {
            static_for<0, 4>([&](auto i) { x[h][i] = s[rb][h][(int)i]; });
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
        // the running maximum of a row moves only when one of its scores
        // passes it by more than kSlack; each lane checks its own eight
        // scores, and only then are the row's four lanes combined
        float mt = -INFINITY;
        static_for<0, 2>([&](auto h) { static_for<0, 4>([&](auto i) { mt = fmaxf(mt, x[h][i]); }); });
        mt *= qk_scale;
        if (__any(mt > S.m[rb] + kSlack)) {
            mt = fmaxf(mt, __shfl_xor(mt, 16));
            mt = fmaxf(mt, __shfl_xor(mt, 32));
            const bool need = mt > S.m[rb] + kSlack;   // the same in the row's four lanes
            const float mn = need ? fmaxf(S.m[rb], mt) : S.m[rb];
            const float al = need ? fast_exp2(S.m[rb] - (mn == -INFINITY ? 0.f : mn)) : 1.f;
            S.lsum[rb] *= al;
            static_for<0, X::NDT>([&](auto t) { S.o[rb][t] *= al; });
            S.m[rb] = mn;
        }
        const float ms = S.m[rb] == -INFINITY ? 0.f : S.m[rb];
        static_for<0, 8>([&](auto j) {
            constexpr int jj = decltype(j)::value;
            const float p = fast_exp2(fmaf(x[jj >> 2][jj & 3], qk_scale, -ms));
            S.lsum[rb] += p;
            pb[rb][jj] = (__bf16)p;
        });
    });
    static_for<0, X::NDT>([&](auto t) {
        const u32x2_t v0 = __builtin_bit_cast(u32x2_t, vt[t][0]);
        const u32x2_t v1 = __builtin_bit_cast(u32x2_t, vt[t][1]);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, u32x4_t{v0.x, v0.y, v1.x, v1.y});
        static_for<0, RB>([&](auto rb) {
            S.o[rb][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb[rb], S.o[rb][t], 0, 0, 0);
        });
    });
}

// Walks a key list tile by tile in order (segments are never empty), so a
// tile costs a few scalar additions rather than a search of the segments.
struct TileIter {
    const char *k, *v;
    int rem;    // rows left in the current segment (0: past the end)
    int key0;   // position of the next tile's first key
    int seg;
};

__device__ __forceinline__ void iter_seg(const KeyList &L, TileIter &it) {
    it.rem = 0;
#pragma unroll
    for (int s = 0; s < kMaxSeg; ++s)
        if (s == it.seg && s < L.n_seg) {
            it.k = L.k[s];
            it.v = L.v[s];
            it.rem = L.len[s];
            it.key0 = L.key0[s];
        }
}

// The next tile (an empty one past the end).
template <int TK>
__device__ __forceinline__ TileRef iter_next(const KeyList &L, TileIter &it, int row_bytes) {
    if (it.rem <= 0) return empty_tile(L);
    const TileRef r{it.k, it.v, min(TK, it.rem), kColsAll, it.key0};
    it.k += (size_t)TK * row_bytes;
    it.v += (size_t)TK * row_bytes;
    it.rem -= TK;
    it.key0 += TK;
    if (it.rem <= 0) {
        ++it.seg;
        iter_seg(L, it);
    }
    return r;
}

// Stream a key list through the ring.  Every iteration issues one tile (an
// empty one past the end), so the count of loads in flight is the same in
// every iteration and one vmcnt wait finds tile t complete.
template <int D, int RB, int NW>
__device__ __forceinline__ void direct_stream(const KeyList &L, const char *const (&qrow)[RB], float qk_scale,
                                              bool row_lo, const int (&lo)[RB], char *lds, WideState<D, RB> &S) {
    using X = Direct<D>;
    constexpr int NB = X::NB;
    constexpr int LPT = direct_loads_per_thread<D, NW>();
    const int n_tiles = list_tiles(L);
    if (n_tiles == 0) return;
    const DirectLanes<D, NW> dl = direct_lanes<D, NW>();
    const uint32_t lds0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds_offset(lds));
    TileIter it;
    it.k = L.k[0];
    it.v = L.v[0];
    it.key0 = 0;
    it.seg = 0;
    iter_seg(L, it);
    TileRef ref[NB];
    static_for<0, NB - 1>([&](auto i) {
        ref[i] = iter_next<X::TK>(L, it, X::ROW);
        direct_issue<D, NW>(ref[i], lds0 + i * X::BUF, dl);
    });
    // q (the rows' MFMA operands; a NULL row reads zeros) is loaded while the
    // first tiles are in flight, and the ring starts once both are in: the
    // compiler, which does not see the tile loads, places no wait of its own
    // inside the loop after this one
    bf16x8_t qb[RB][X::NDS];
    static_for<0, RB>([&](auto rb) { load_q_cols<D>(qrow[rb], qb[rb]); });
    wait_vmcnt<0>();
    for (int base = 0; base < n_tiles; base += NB) {
        static_for<0, NB>([&](auto j) {
            constexpr int jj = decltype(j)::value;
            constexpr int jn = (jj + NB - 1) % NB;   // the buffer of tile t - 1, free after the barrier
            const int t = base + jj;
            if (t < n_tiles) {   // uniform
                wait_vmcnt<LPT * (NB - 2)>();   // this wave's loads of tile t are done
                __syncthreads();                // every wave's are; every wave is done with tile t - 1
                ref[jn] = iter_next<X::TK>(L, it, X::ROW);   // tile t + NB - 1
                direct_issue<D, NW>(ref[jn], lds0 + jn * X::BUF, dl);
                direct_compute<D, RB>(lds + jj * X::BUF, ref[jj].n, ref[jj].key0, row_lo, lo, qb, qk_scale, S);
            }
        });
    }
    wait_vmcnt<0>();   // the trailing empty tiles are done with the ring
    __syncthreads();
}

}  // namespace splice_dev
