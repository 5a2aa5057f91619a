// verify_common.h -- building blocks shared by the verify kernels: the MFMA
// operand layouts for K, V and the verify rows, and the register-ring tile
// pipeline.  Internal to the library.
#pragma once

#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace vc {

constexpr int kThreads = 256;  // 4 waves
constexpr int kWaves = 4;
constexpr int kTile = 32;      // keys per wave step
constexpr int kRowCap = 64;    // rows per item slot in the workspace

// Tile-local key assigned to A row m of a 16-key half tile.  The accumulator
// rows lane group G receives are 4G + i, which then hold keys G + 4i: the same
// keys lane group G loads as full 256-byte rows for the V^T operand.
__device__ __forceinline__ int a_row_key(int m) { return (m >> 2) + 4 * (m & 3); }

// The verify rows a lane owns: row rt*16 + (lane & 15) of each row tile.
template <int NRT>
struct Rows {
    int plim[NRT];      // last key the row may see; -1 for padding rows
    bool inwin[NRT];    // row contributes to the scores
    u32x4 q[NRT][4];    // B operand (Q^T): row's head-dim slice per 32-wide k-block
};

// Row rt*16 + m16 of a launch is verify position qoff + row / group of the
// sequence (of its qfull positions) and query head c*group + row % group.
template <int NRT>
__device__ __forceinline__ void load_rows(const VerifyArgs& a, int b, int c, int T, int nq, int qoff,
                                          int qfull, int m16, int G, Rows<NRT>& r) {
    const int g = a.group;
    const int R = nq * g;
    const int wn = min(a.window, qfull);
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        const int row = rt * 16 + m16;
        if (row < R) {
            const int j = qoff + row / g;
            const int hh = row - (j - qoff) * g;
            r.plim[rt] = T - qfull + j;
            r.inwin[rt] = j >= qfull - wn;
            const uint16_t* qp =
                a.q + (((size_t)b * a.max_q + j) * a.n_q_heads + c * g + hh) * kHeadDim + 8 * G;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) r.q[rt][kb] = ld_u32x4(qp + 32 * kb);
        } else {
            r.plim[rt] = -1;
            r.inwin[rt] = false;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) r.q[rt][kb] = u32x4{0u, 0u, 0u, 0u};
        }
    }
}

// K operand of a 32-key tile: lane (m16, G) holds key a_row_key(m16) (+16 for
// the second half) and head-dim elements 32kb + 8G .. +8 of k-block kb.
// With kStream the loads carry the non-temporal hint.  It streams faster when
// the rows are read once by a single round of workgroups; the two-sweep
// statistics pass leaves it off so that the second pass finds K in the
// memory-side cache, and so does a one-sweep launch of several rounds, where
// it measured slower.
template <bool kStream = true>
__device__ __forceinline__ void load_k(const uint16_t* kbase, int key0, int T, int m16, int G,
                                       u32x4 (&kr)[2][4]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int key = min(key0 + 16 * t + a_row_key(m16), T - 1);
        const uint16_t* p = kbase + (size_t)key * kHeadDim + 8 * G;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) kr[t][kb] = kStream ? ld_stream_u32x4(p + 32 * kb) : ld_u32x4(p + 32 * kb);
    }
}

// V rows of a 32-key tile: slot e = 4t + i is key 16t + G + 4i, and lane
// (m16, G) holds its head-dim elements 8*m16 .. +8; one load instruction
// covers four whole consecutive rows.
template <bool kStream = true>
__device__ __forceinline__ void load_v(const uint16_t* vbase, int key0, int T, int m16, int G,
                                       u32x4 (&vr)[8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int key = min(key0 + 16 * (e >> 2) + G + 4 * (e & 3), T - 1);
        const uint16_t* p = vbase + (size_t)key * kHeadDim + 8 * m16;
        vr[e] = kStream ? ld_stream_u32x4(p) : ld_u32x4(p);
    }
}

// Paged cache.  Pages hold a multiple of kTile keys, so a tile (starting at a
// multiple of kTile; its rows clamped to the sequence's last key) lies in one
// page.  A wave's tiles are first, first + kWaves, ...: lane l of
// wave_pages() holds the page of the wave's tile l, loaded once before the
// sweep, and a tile reads it back with readlane instead of waiting for a
// table load in front of its own loads.
__device__ __forceinline__ int wave_pages(const VerifyArgs& a, int b, int key_begin, int ntile,
                                          int first, int lane) {
    const int t = min(first + kWaves * lane, ntile - 1);
    return a.block_table[(size_t)b * a.max_blocks + (key_begin + t * kTile) / a.page_size];
}

__device__ __forceinline__ size_t paged_row(const VerifyArgs& a, int page, int c, int key0) {
    return ((size_t)page * a.n_kv_heads + c) * a.page_size + key0 % a.page_size;
}

// The page of tile t (wave-uniform) from wave_pages()' lanes.
__device__ __forceinline__ int tile_page(int pages, int t, int first) {
    return __builtin_amdgcn_readlane(pages, (t - first) / kWaves);
}

// Loads the K and V tile at key0 from the dense cache (unit bases kbase,
// vbase) or, with kPaged, from page `page`.
template <bool kPaged, bool kStream, typename Tile>
__device__ __forceinline__ void load_kv_tile(const VerifyArgs& a, const uint16_t* kbase,
                                             const uint16_t* vbase, int page, int c, int key0,
                                             int T, int m16, int G, Tile& bf) {
    if constexpr (kPaged) {
        const size_t r0 = paged_row(a, page, c, key0) * kHeadDim;
        load_k<kStream>(a.k + r0, 0, T - key0, m16, G, bf.k);
        load_v<kStream>(a.v + r0, 0, T - key0, m16, G, bf.v);
    } else {
        load_k<kStream>(kbase, key0, T, m16, G, bf.k);
        load_v<kStream>(vbase, key0, T, m16, G, bf.v);
    }
}

// Logits^T tile: acc[t][rt][i] = q(row rt*16+m16) . k(key 16t + G + 4i).
template <int NRT>
__device__ __forceinline__ void qk_tile(const u32x4 (&kr)[2][4], const Rows<NRT>& r,
                                        f32x4 (&acc)[2][NRT]) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) {
            f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) s = mfma_bf16(kr[t][kb], r.q[rt][kb], s);
            acc[t][rt] = s;
        }
}

// Runs compute(tile) over the wave's tiles first, first + step, ... < ntile
// with a ring of NBUF register buffers: while one tile is computed, the loads
// of the next NBUF - 1 tiles are in flight.  load(buf, tile) issues loads only.
// The steady-state loop issues its loads unconditionally: a load under a
// branch makes the compiler's wait counts assume the path without it, so the
// wait for the current tile would also wait for the tiles in flight.  The
// last tiles are peeled off into a tail where the loads may be skipped.
template <int NBUF, typename Buf, typename Load, typename Compute, typename Pre>
__device__ __forceinline__ void tile_pipeline(int first, int ntile, int step, Load&& load,
                                              Compute&& compute, Pre&& pre) {
    const int n = first < ntile ? (ntile - first + step - 1) / step : 0;
    Buf buf[NBUF];
#pragma unroll
    for (int p = 0; p < NBUF - 1; ++p)
        if (p < n) load(buf[p], first + p * step);
    // Every wave runs pre() once, with the first tiles' loads already in flight.
    pre();
    int i = 0;
    for (; i + 2 * NBUF - 1 <= n; i += NBUF) {
#pragma unroll
        for (int p = 0; p < NBUF; ++p) {
            load(buf[(p + NBUF - 1) % NBUF], first + (i + p + NBUF - 1) * step);
            compute(buf[p], first + (i + p) * step);
        }
    }
#pragma unroll
    for (int q = 0; q < 2 * NBUF - 2; ++q) {
        if (i + q < n) {
            if (i + q + NBUF - 1 < n) load(buf[(q + NBUF - 1) % NBUF], first + (i + q + NBUF - 1) * step);
            compute(buf[q % NBUF], first + (i + q) * step);
        }
    }
}

template <int NBUF, typename Buf, typename Load, typename Compute>
__device__ __forceinline__ void tile_pipeline(int first, int ntile, int step, Load&& load,
                                              Compute&& compute) {
    tile_pipeline<NBUF, Buf>(first, ntile, step, load, compute, [] {});
}

struct KTile {
    u32x4 k[2][4];
};
struct KVTile {
    u32x4 k[2][4];
    u32x4 v[8];
};

// A work item: (sequence b, KV head c, key chunk s) of a launch whose items
// are numbered sequence by sequence, head by head, chunk by chunk.  bt is the
// sequence's entry in the launch's tables, b the sequence itself (a.sid[bt]).
// A launch over whole sequences (kBlocks false: sid[bt] = bt, qoff 0, qfull
// the sequence's q_len) skips those tables, so that the first K/V addresses do
// not wait for one more dependent load of the launch arguments.
struct Item {
    int b, bt, c, s, nchunk, T, nq, qoff, qfull, key_begin, key_end, unit, item0;
};

template <bool kBlocks>
__device__ __forceinline__ Item decode_item(const VerifyArgs& a, const SeqTable& st, int item,
                                            int chunk) {
    const int n_kv = a.n_kv_heads;
    Item it;
    int bt = 0;
    while (bt + 1 < st.n_seq && item >= st.item_start[bt + 1]) ++bt;
    const int b = kBlocks ? a.sid[bt] : bt;
    it.b = b;
    it.bt = bt;
    it.T = st.ctx[bt];
    it.nq = st.qlen[bt];
    it.qoff = kBlocks ? a.qoff[bt] : 0;
    it.qfull = kBlocks ? a.qfull[bt] : it.nq;
    it.nchunk = (it.T + chunk - 1) / chunk;
    const int local = item - st.item_start[bt];
    it.c = local / it.nchunk;
    it.s = local - it.c * it.nchunk;
    it.key_begin = it.s * chunk;
    it.key_end = min(it.key_begin + chunk, it.T);
    it.unit = b * n_kv + it.c;
    it.item0 = st.item_start[bt] + it.c * it.nchunk;
    return it;
}

}  // namespace vc
}  // namespace ssl
