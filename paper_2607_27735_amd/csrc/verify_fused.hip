// verify_fused.hip -- single-sweep verify attention with fused Eq. 3 scores
// (Sec. 3.1 verification, Sec. 3.2 Eq. 3).
//
// The Eq. 3 score of a key needs the final normalizer of every verify row,
// which no split of the context knows while it streams.  When every chunk of
// a (sequence, KV head) can be resident at once, one sweep suffices:
//
//   1. each workgroup streams its chunk of K and V once and runs an online
//      softmax per verify row (P.V on the MFMA, as in the two-sweep kernel);
//      it keeps in LDS the probabilities of its keys relative to the running
//      row maxima, and those maxima for every 32-key tile;
//   2. it publishes its partial P.V relative to the running maxima and, once
//      those stores have landed, its (running max, sum) per row, each 64-bit
//      word carrying the low 32 bits of the call's exchange tag above the
//      value; it then polls the (max, sum) words of every chunk of its head
//      until all carry the tag, so the poll that finds them delivers them;
//   3. from the merged (max, sum) of all chunks it forms one factor per tile
//      and row, so that a stashed probability times its factor is the exact
//      probability, and writes the scores of its keys;
//   4. the workgroup of chunk s adds the partials of rows s, s + nchunk, ...,
//      each scaled to the exact normalizer, and writes them.
//
// Publication avoids agent-scope fences, which write back a whole L2 per wave
// on this multi-XCD part: the published statistics and partials are written
// and read with device-coherent (agent-scope relaxed atomic) stores and
// loads, and every wave waits for its partial-output stores to complete
// before the tagged statistics are written.  The tags need no initialisation:
// the host draws a fresh tag for every call from a process-wide sequence with
// a clock-seeded start (consecutive calls differ in the low 32 bits for 2^32
// calls), so a stale or uninitialised word matches only by a 2^-32 accident.
//
// Two kernels run these steps.  verify_fused_kernel gives each chunk its own
// workgroup (fp32 stash; with kStep it then selects and drafts too).  Its wait
// ends: workgroups are dispatched in index order and the chunks of one head
// are consecutive, so when the lowest unfinished head waits, every workgroup
// ahead of its chunks has finished and its chunks are resident (the host
// plans at most half of what the device's CUs hold at once per head).
// verify_pipe_kernel, for calls whose chunks would take several rounds of
// workgroups, is a resident grid that takes every grid-th chunk with two
// 16-bit stash buffers and runs steps 2-4 of one chunk while the next one
// streams (its own comment gives the order and why its waits end).  Every
// wait is also bounded: a workgroup whose wait gives up reports it on the
// device's status word and leaves without writing scores or outputs.
#include <algorithm>
#include <atomic>

#include "select_common.h"
#include "verify_common.h"

namespace ssl {
namespace {

using namespace vc;

constexpr int kParkStride = kHeadDim + 4;                 // floats per parked output row
constexpr int kParkFloats = 2 * 16 * kParkStride;         // two waves' slices of a row tile
constexpr float kLazy = 8.f;          // reference-maximum slack, log2 units
// The decode step's row-sum scratch (256 f32x4) in the dynamic LDS, past the
// select's.
constexpr size_t kStepRedOffset = (sizeof(SelLds) + 15) / 16 * 16;
constexpr size_t kStepLdsMin = kStepRedOffset + 256 * sizeof(f32x4);
static_assert(kStepLdsMin + 8 * 1024 <= 160 * 1024, "the step's LDS fits beside the static arrays");

// The LDS stash holds each key's probability per verify row, relative to the
// row's reference maximum (at most 2^kLazy).  Two element formats:
//  - StashF32: the fp32 value (the kernel that runs one chunk per workgroup);
//  - StashU16: a 16-bit code, half the LDS, so that the persistent kernel can
//    keep two chunks' stashes: 6 exponent bits (2^-54 .. 2^9) above the top 10
//    mantissa bits, rounded to nearest (relative error at most 2^-11, so a
//    score, a sum of such terms times exact factors, keeps that bound); values
//    below 2^-54 of the reference are coded 0.
struct StashF32 {
    using T = float;
    static constexpr int kPad = 4;   // elements of padding per row
    static __device__ __forceinline__ void put(T* p, float v) { *p = v; }
    // keys k4 .. k4 + 3 of a row (k4 a multiple of 4)
    static __device__ __forceinline__ f32x4 get4(const T* row, int k4) {
        return *reinterpret_cast<const f32x4*>(row + k4);
    }
};

struct StashU16 {
    using T = uint16_t;
    static constexpr int kPad = 8;
    static constexpr uint32_t kBias = 72u << 10;   // exponent field 72 at code 0
    static __device__ __forceinline__ uint32_t enc(float v) {
        const uint32_t r = (__float_as_uint(v) + 0x1000u) >> 13;   // 10 mantissa bits, rounded
        return r >= kBias + 1024u ? min(r - kBias, 0xFFFFu) : 0u;
    }
    static __device__ __forceinline__ float dec(uint32_t c) {
        return c ? __uint_as_float((c + kBias) << 13) : 0.f;
    }
    static __device__ __forceinline__ void put(T* p, float v) { *p = (uint16_t)enc(v); }
    static __device__ __forceinline__ f32x4 get4(const T* row, int k4) {
        const uint2 w = *reinterpret_cast<const uint2*>(row + k4);
        return f32x4{dec(w.x & 0xFFFFu), dec(w.x >> 16), dec(w.y & 0xFFFFu), dec(w.y >> 16)};
    }
};

template <int NRT>
constexpr int static_lds_bytes() {
    return kWaves * NRT * 16 * 8            // wml
           + kRowCap * 4                    // row_lse
           + kWaves * kRowCap * 8           // slack kept: the chunk limits below were tuned with it
           + 64;
}

// The largest chunk whose stash (probabilities, padding, one running maximum
// per tile and row) fits in LDS beside the static arrays and the parking
// slices.
template <int NRT>
constexpr int max_fused_chunk() {
    constexpr int kLds = 160 * 1024;
    constexpr int floats_per_row =
        (kLds - static_lds_bytes<NRT>() - kParkFloats * 4 - 1024) / 4 / (16 * NRT);
    return (floats_per_row - StashF32::kPad) * kTile / (kTile + 1) / 128 * 128;
}

__device__ __forceinline__ float safe_max(float m) { return m == -INFINITY ? 0.f : m; }

// One 32-key tile: online softmax and P.V; the tile's probabilities relative
// to the rows' reference maxima go to the LDS stash, those maxima to mtile.
template <int NRT, typename Codec>
__device__ __forceinline__ void fused_tile(const VerifyArgs& a, const Rows<NRT>& r,
                                           const KVTile& tl, int key0, int kl0,
                                           typename Codec::T* stash, int stride, float* mtile,
                                           int mts, int m16, int G, float (&M)[NRT],
                                           float (&L)[NRT], f32x4 (&oacc)[8][NRT]) {
    f32x4 acc[2][NRT];
    qk_tile<NRT>(tl.k, r, acc);
    float p[2][NRT][4];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        float y[8];
        float mt = -INFINITY;
        typename Codec::T* srow = stash + (rt * 16 + m16) * stride + kl0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int t = e >> 2, i = e & 3;
            const int key = key0 + 16 * t + G + 4 * i;
            y[e] = key <= r.plim[rt] ? acc[t][rt][i] * a.scale_log2 : -INFINITY;
            mt = fmaxf(mt, y[e]);
        }
        mt = fmaxf(mt, shfl_xor_f(mt, 16));
        mt = fmaxf(mt, shfl_xor_f(mt, 32));
        // M is a reference maximum that moves only when a tile's maximum
        // exceeds it by more than kLazy (log2 units): the accumulators are then
        // rescaled, for the whole row tile at once, and rarely; probabilities
        // relative to it stay below 2^kLazy.
        const bool grow = mt > M[rt] + kLazy;   // M = -inf: any finite mt
        if (__any(grow)) {
            const float alpha = grow ? fast_exp2(M[rt] - mt) : 1.f;
            M[rt] = grow ? mt : M[rt];
            L[rt] *= alpha;
#pragma unroll
            for (int jd = 0; jd < 8; ++jd) oacc[jd][rt] *= alpha;
        }
        const float Mr = safe_max(M[rt]);
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            p[e >> 2][rt][e & 3] = fast_exp2(y[e] - Mr);
            sum += p[e >> 2][rt][e & 3];
            Codec::put(srow + 16 * (e >> 2) + G + 4 * (e & 3), p[e >> 2][rt][e & 3]);
        }
        if (G == 0) mtile[(rt * 16 + m16) * mts + kl0 / kTile] = Mr;
        L[rt] += sum;
    }
    u32x4 pb[NRT];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        pb[rt][0] = pack_bf16(p[0][rt][0], p[0][rt][1]);
        pb[rt][1] = pack_bf16(p[0][rt][2], p[0][rt][3]);
        pb[rt][2] = pack_bf16(p[1][rt][0], p[1][rt][1]);
        pb[rt][3] = pack_bf16(p[1][rt][2], p[1][rt][3]);
    }
#pragma unroll
    for (int jd = 0; jd < 8; ++jd) {
        u32x4 av;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            const uint32_t x = tl.v[2 * s2][jd >> 1], yv = tl.v[2 * s2 + 1][jd >> 1];
            av[s2] = (jd & 1) ? perm_hi(x, yv) : perm_lo(x, yv);
        }
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) oacc[jd][rt] = mfma_bf16(av, pb[rt], oacc[jd][rt]);
    }
}

// The decode step's select (partition p of unit u): the keys in the select
// layout from the chunk's score bits in skeys (LDS), then the one-kernel
// select and draft step (select_common.h) with the stash as their LDS.
template <int NR, typename Mid>
__device__ __forceinline__ bool step_select(const SelectArgs& sa, const Geom& g, int p, int u,
                                            const uint32_t* skeys, int nk, int key_begin,
                                            SelLds& L, uint64_t want, Mid&& mid) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t keys[4 * NR];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int x = r * kRound + wave * 256 + e * 64 + lane;   // chunk-local position
            const int pos = key_begin + x;
            uint32_t v = x < nk ? skeys[x] : kNone;
            v = v == 0x80000000u ? 0u : v;   // -0 ranks as +0, as select reads it
            keys[4 * r + e] = (x < nk && pos >= g.s_end && pos < g.r_start) ? v : kNone;
        }
    __syncthreads();   // every key is read: the stash becomes the select's
    select_local_hist<NR>(keys, L);
    return select_partition<NR, true>(sa, g, p, u, keys, L, want, mid);
}

// A chunk of one (sequence, KV head): work item `slot` of the launch.
struct Chunk {
    int slot, unit, b, c, s, slot0, nchunk, T, nq, R, key_begin, key_end;
};

__device__ __forceinline__ Chunk chunk_of(const VerifyArgs& a, int slot) {
    const Item it = decode_item<false>(a, a.seq, slot, a.chunk);
    Chunk k;
    k.slot = slot;
    k.unit = it.unit;
    k.b = it.b;
    k.c = it.c;
    k.s = it.s;
    k.slot0 = it.item0;
    k.nchunk = it.nchunk;
    k.T = it.T;
    k.nq = it.nq;
    k.R = it.nq * a.group;
    k.key_begin = it.key_begin;
    k.key_end = it.key_end;
    return k;
}

template <int NRT>
__device__ __forceinline__ void clear_state(float (&M)[NRT], float (&L)[NRT], f32x4 (&oacc)[8][NRT]) {
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        M[rt] = -INFINITY;
        L[rt] = 0.f;
#pragma unroll
        for (int jd = 0; jd < 8; ++jd) oacc[jd][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
}

// ---- 1. the sweep: the chunk's K and V once, online softmax, P.V ----------
// pre() runs once per wave with each wave's first tile already in flight.
template <int NRT, bool kStream, bool kPaged, typename Codec, typename Pre>
__device__ __forceinline__ void sweep_chunk(const VerifyArgs& a, const Chunk& k, const Rows<NRT>& r,
                                            typename Codec::T* stash, int stride, float* mtile,
                                            int mts, float (&M)[NRT], float (&L)[NRT],
                                            f32x4 (&oacc)[8][NRT], Pre&& pre) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m16 = lane & 15, G = lane >> 4;
    const size_t cache_off = (size_t)k.unit * a.max_ctx * kHeadDim;
    const uint16_t* kbase = a.k + cache_off;
    const uint16_t* vbase = a.v + cache_off;
    const int ntile = (k.key_end - k.key_begin + kTile - 1) / kTile;
    const int pages = kPaged ? wave_pages(a, k.b, k.key_begin, ntile, wave, lane) : 0;
    tile_pipeline<2, KVTile>(
        wave, ntile, kWaves,
        [&](KVTile& bf, int t) {
            load_kv_tile<kPaged, kStream>(a, kbase, vbase, kPaged ? tile_page(pages, t, wave) : 0,
                                          k.c, k.key_begin + t * kTile, k.T, m16, G, bf);
        },
        [&](const KVTile& bf, int t) {
            fused_tile<NRT, Codec>(a, r, bf, k.key_begin + t * kTile, t * kTile, stash, stride, mtile,
                                   mts, m16, G, M, L, oacc);
        },
        pre);
}

// ---- 2. publish the chunk's partial output, then its row statistics ------
// Every thread calls this.  Returns the exchange tag; *clean is false when an
// earlier captured call on this workspace gave up (the epoch is marked), and
// then nothing is published.  Uses L (summed over the wave's lanes here).
template <int NRT>
__device__ __forceinline__ uint64_t publish_chunk(const FusedArgs& fa, const Chunk& k,
                                                  const float (&M)[NRT], float (&L)[NRT],
                                                  const f32x4 (&oacc)[8][NRT],
                                                  float2 (*wml)[NRT * 16], float* park,
                                                  int* wait_failed, bool* clean) {
    const VerifyArgs& a = fa.v;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m16 = lane & 15, G = lane >> 4;
    // The unit's exchange epoch (exchange_tag), loaded here so that its round
    // trip overlaps the stores below (the tag is formed only after the wait
    // for them); the unit's chunk 0 advances it once it has every chunk's
    // statistics, i.e. once every chunk has read it.
    const uint64_t ep = fa.epoch ? ld_dev64(fa.epoch + k.unit) : 0ull;
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        L[rt] += shfl_xor_f(L[rt], 16);
        L[rt] += shfl_xor_f(L[rt], 32);
        if (G == 0) wml[wave][rt * 16 + m16] = make_float2(M[rt], L[rt]);
    }
    if (tid == 0) *wait_failed = 0;
    __syncthreads();
    // the workgroup's row statistics, merged over its waves (published below,
    // once the partial output has landed)
    float own_m = -INFINITY, own_l = 0.f;
    if (tid < k.R) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) own_m = fmaxf(own_m, wml[w][tid].x);
#pragma unroll
        for (int w = 0; w < kWaves; ++w) own_l += wml[w][tid].y * fast_exp2(wml[w][tid].x - safe_max(own_m));
    }
    // the partial P.V relative to the workgroup's row maxima: per row tile,
    // waves 2 and 3 park theirs, waves 0 and 1 add them, park the sums, and
    // all threads add the two slices and store the rows device-coherently
    {
        float* po = a.part_o + (size_t)k.slot * kRowCap * kHeadDim;
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) {
            const int row = rt * 16 + m16;
            float mw = -INFINITY;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) mw = fmaxf(mw, wml[w][row].x);
            const float f = fast_exp2(M[rt] - safe_max(mw));
            float* slice = park + ((wave & 1) * 16 + m16) * kParkStride;
            if (wave >= 2) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int c4 = 32 * G + 8 * i;
                    *reinterpret_cast<f32x4*>(slice + c4) =
                        f32x4{oacc[0][rt][i], oacc[1][rt][i], oacc[2][rt][i], oacc[3][rt][i]} * f;
                    *reinterpret_cast<f32x4*>(slice + c4 + 4) =
                        f32x4{oacc[4][rt][i], oacc[5][rt][i], oacc[6][rt][i], oacc[7][rt][i]} * f;
                }
            }
            __syncthreads();
            if (wave < 2) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int c4 = 32 * G + 8 * i;
                    f32x4 lo = *reinterpret_cast<const f32x4*>(slice + c4);
                    f32x4 hi = *reinterpret_cast<const f32x4*>(slice + c4 + 4);
                    lo += f32x4{oacc[0][rt][i], oacc[1][rt][i], oacc[2][rt][i], oacc[3][rt][i]} * f;
                    hi += f32x4{oacc[4][rt][i], oacc[5][rt][i], oacc[6][rt][i], oacc[7][rt][i]} * f;
                    *reinterpret_cast<f32x4*>(slice + c4) = lo;
                    *reinterpret_cast<f32x4*>(slice + c4 + 4) = hi;
                }
            }
            __syncthreads();
            const int rows_here = min(16, k.R - rt * 16);
            f32x4 o[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {   // both halves' reads in flight
                const int x = tid + h * kThreads, rr = x >> 5, q4 = x & 31;
                o[h] = *reinterpret_cast<const f32x4*>(park + rr * kParkStride + 4 * q4) +
                       *reinterpret_cast<const f32x4*>(park + (16 + rr) * kParkStride + 4 * q4);
            }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int x = tid + h * kThreads, rr = x >> 5, q4 = x & 31;
                if (rr < rows_here) {
                    uint64_t* d64 = reinterpret_cast<uint64_t*>(po + (size_t)(rt * 16 + rr) * kHeadDim + 4 * q4);
                    st_dev64(d64, __builtin_bit_cast(uint64_t, make_float2(o[h][0], o[h][1])));
                    st_dev64(d64 + 1, __builtin_bit_cast(uint64_t, make_float2(o[h][2], o[h][3])));
                }
            }
            if (rt + 1 < NRT) __syncthreads();   // (the last one: the barrier below)
        }
    }
    // Each (max, sum) word carries the low 32 bits of the exchange tag above
    // the value, and is stored only once this workgroup's partial output has
    // landed: a reader that finds every chunk's words tagged has the head's
    // statistics from that one poll, and may then load the partial outputs.
    wait_stores_done();
    __syncthreads();
    const uint64_t epv = scalar_here(ep);
    const uint64_t want = exchange_tag(fa.call_tag, epv);
    // a dirty epoch: an earlier captured call on this workspace gave up
    *clean = !epoch_is_dirty(epv);
    if (*clean && tid < k.R) {
        uint64_t* ml64 = reinterpret_cast<uint64_t*>(a.part_ml);   // [slot][kRowCap][2]
        const uint64_t pub = ((want ^ fa.xc.tag_flip) & 0xFFFFFFFFull) << 32;
        uint64_t* e = ml64 + ((size_t)k.slot * kRowCap + tid) * 2;
        st_dev64(e, pub | __float_as_uint(own_m));
        st_dev64(e + 1, pub | __float_as_uint(own_l));
    }
    return want;
}

// Partial outputs and maxima of row `row` of chunks s0, s0 + 8, ... (kSum of
// them; past the unit's chunks: zero and -inf), columns 4 d4 .. 4 d4 + 3.
template <int kSum>
__device__ __forceinline__ void load_part(const VerifyArgs& a, const Chunk& k, int row, int s0, int d4,
                                          f32x4 (&v)[kSum], float (&m)[kSum]) {
    const uint64_t* ml64 = reinterpret_cast<const uint64_t*>(a.part_ml);   // [slot][kRowCap][2]
#pragma unroll
    for (int uu = 0; uu < kSum; ++uu) {
        const int s2 = s0 + 8 * uu;
        if (s2 < k.nchunk) {
            const size_t rw = (size_t)(k.slot0 + s2) * kRowCap + row;
            const uint64_t* s64 = reinterpret_cast<const uint64_t*>(a.part_o + rw * kHeadDim + 4 * d4);
            const float2 lo = __builtin_bit_cast(float2, ld_dev64(s64));
            const float2 hi = __builtin_bit_cast(float2, ld_dev64(s64 + 1));
            v[uu] = f32x4{lo.x, lo.y, hi.x, hi.y};
            m[uu] = __uint_as_float((uint32_t)ld_dev64(ml64 + rw * 2));
        } else {
            v[uu] = f32x4{0.f, 0.f, 0.f, 0.f};
            m[uu] = -INFINITY;
        }
    }
}

// ---- 4. rows s, s + nchunk, ... summed over the unit's chunks ----------
// Every thread calls this, with the normalizers in row_lse; red: 256 f32x4
// of free LDS.  A chunk's partial is relative to its maxima m: it enters with
// 2^(m - lse).  Chunks are added in index order within eight interleaved
// groups, then the groups in order.  pre_v / pre_m (or null): the first batch
// of row s, already loaded.
template <int kSum>
__device__ __forceinline__ void row_sums(const VerifyArgs& a, const Chunk& k, const float* row_lse,
                                         f32x4* red, const f32x4 (*pre_v)[kSum],
                                         const float (*pre_m)[kSum]) {
    const int tid = threadIdx.x, d4 = tid & 31, sg = tid >> 5;
    const int R = k.R, nchunk = k.nchunk;
    for (int row = k.s; row < R; row += nchunk) {
        const float lse = row_lse[row];
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int s0 = sg; s0 < nchunk; s0 += kSum * 8) {
            f32x4 v[kSum];
            float m[kSum];
            if (pre_v && row == k.s && s0 == sg) {
#pragma unroll
                for (int uu = 0; uu < kSum; ++uu) {
                    v[uu] = (*pre_v)[uu];
                    m[uu] = (*pre_m)[uu];
                }
            } else {
                load_part<kSum>(a, k, row, s0, d4, v, m);
            }
#pragma unroll
            for (int uu = 0; uu < kSum; ++uu) acc += v[uu] * fast_exp2(m[uu] - lse);
        }
        red[sg * 32 + d4] = acc;
        __syncthreads();
        if (sg == 0) {
            f32x4 o = red[d4];
#pragma unroll
            for (int gq = 1; gq < 8; ++gq) o += red[gq * 32 + d4];
            const int j = row / a.group;
            const int h = k.c * a.group + (row - j * a.group);
            const size_t base = (((size_t)k.b * a.max_q + j) * a.n_q_heads + h) * kHeadDim + 4 * d4;
            if (a.out_fp32) {
                *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + base) = o;
            } else {
                const uint2 pk = make_uint2(pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3]));
                *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + base) = pk;
            }
        }
        __syncthreads();
    }
}

// ---- 3, 4. the chunk's scores and its rows' outputs ----------------------
// Every thread calls this.  Waits for every chunk's statistics of the unit
// (false: the wait gave up, reported on the status word; nothing written),
// then writes the scores of the chunk's keys from its stash and the outputs
// of rows s, s + nchunk, ... (kDefer: the caller runs row_sums later).  With
// kStep the score bits also go to skeys.
template <int NRT, typename Codec, bool kStep, int kPoll = 8, int kSum = 4, bool kDefer = false>
__device__ __forceinline__ bool finish_chunk(const FusedArgs& fa, const Chunk& k, uint64_t want,
                                             bool clean, typename Codec::T* stash, int stride,
                                             const float* mtile, int mts, float* row_lse,
                                             int* wait_failed, uint32_t* skeys) {
    const VerifyArgs& a = fa.v;
    const int tid = threadIdx.x, lane = tid & 63;
    const int R = k.R, nchunk = k.nchunk, slot0 = k.slot0;
    const uint64_t tag_hi = (want & 0xFFFFFFFFull) << 32;
    const uint64_t* ml64 = reinterpret_cast<const uint64_t*>(a.part_ml);   // [slot][kRowCap][2]

    // ---- 3a. exact row statistics over every chunk of the head -------------
    // Wave w takes rows 16 w .. 16 w + 15 (those below R): lane (c4, r16)
    // polls row 16 w + r16 of chunks c4, c4 + 4, ... (kPoll of them per round
    // trip) until all their words carry the tag, merges them, and the four
    // chunk groups are merged across lanes, so each row's normalizer is
    // formed in the wave that polled it.  (One poll in flight per wave: two,
    // issued half a round trip apart, load the memory system enough to cost
    // more than the earlier sight gains.)
    {
        const int ph = tid >> 6, r16 = lane & 15, c4 = lane >> 4;
        const int row = ph * 16 + r16;
        float Mx = -INFINITY, Lx = 0.f;
        bool in_all = clean;
        if (ph * 16 < R) {   // wave-uniform
            for (int b0 = 0; in_all && b0 < nchunk; b0 += kPoll * 4) {   // wave-uniform
                uint64_t w0[kPoll], w1[kPoll];
                // every lane loads (lanes past the rows or chunks re-read valid
                // entries): no branch around the loads
                const uint64_t* e[kPoll];
#pragma unroll
                for (int uu = 0; uu < kPoll; ++uu)
                    e[uu] = ml64 + ((size_t)(slot0 + min(b0 + c4 + 4 * uu, nchunk - 1)) * kRowCap + min(row, R - 1)) * 2;
                int spins = 0;
                bool all_in;
                do {
                    bool in = true;
#pragma unroll
                    for (int uu = 0; uu < kPoll; ++uu) {
                        w0[uu] = ld_dev64(e[uu]);
                        w1[uu] = ld_dev64(e[uu] + 1);
                    }
#pragma unroll
                    for (int uu = 0; uu < kPoll; ++uu)
                        in &= ((w0[uu] & ~0xFFFFFFFFull) == tag_hi && (w1[uu] & ~0xFFFFFFFFull) == tag_hi);
                    all_in = __all(in);
                    if (!all_in) __builtin_amdgcn_s_sleep(1);
                } while (!all_in && ++spins < fa.xc.spin_limit);
                in_all = all_in;
                if (all_in && row < R) {
#pragma unroll
                    for (int uu = 0; uu < kPoll; ++uu)
                        if (b0 + c4 + 4 * uu < nchunk)
                            ml_merge(Mx, Lx, __uint_as_float((uint32_t)w0[uu]), __uint_as_float((uint32_t)w1[uu]));
                }
            }
            ml_merge(Mx, Lx, shfl_xor_f(Mx, 16), shfl_xor_f(Lx, 16));
            ml_merge(Mx, Lx, shfl_xor_f(Mx, 32), shfl_xor_f(Lx, 32));
            if (c4 == 0 && row < R) row_lse[row] = Lx > 0.f ? Mx + fast_log2(Lx) : INFINITY;
        }
        if (!in_all && lane == 0) *wait_failed = 1;
    }
    __syncthreads();
    if (*wait_failed) {
        if (tid == 0) exchange_gave_up(fa.xc, kStatusVerify, fa.epoch ? fa.epoch + k.unit : nullptr);
        return false;
    }

    // The first chunks of this workgroup's first row in step 4 (all of them
    // for up to 32 chunks), loaded now so that the round trip overlaps 3b
    // (kDefer: step 4 is left to the caller).
    const int d4 = tid & 31, sg = tid >> 5;
    f32x4 pv[kSum];
    float pm[kSum];
    if (!kDefer && k.s < R) load_part<kSum>(a, k, k.s, sg, d4, pv, pm);

    const int nk = k.key_end - k.key_begin;

    // ---- 3b. scores of this chunk's keys from the stashed probabilities ----
    {
        const int wn = min(a.window, k.nq);
        const int r0 = (k.nq - wn) * a.group;   // first window row
        float* srow = a.scores + (size_t)k.unit * a.max_ctx;
        // four consecutive keys per thread (one LDS read per row, several rows
        // in flight); the stash row stride and the chunk are multiples of 4
        // elements, and 4 consecutive keys share one tile.
        // A stashed probability times its tile's factor 2^(m_tile - lse) is
        // exact; the tile maxima are [row][tile], so the lanes of a wave
        // (eight tiles, one row) read distinct banks.
        // one index set per query head: head hh of the group sums its own
        // window rows r0 + hh, r0 + hh + group, ...
        for (int k4 = 4 * tid; a.per_head && k4 < nk; k4 += 4 * kThreads) {
            const float* mt = mtile + k4 / kTile;
            for (int hh = 0; hh < a.group; ++hh) {
                f32x4 sc = {0.f, 0.f, 0.f, 0.f};
                for (int row = r0 + hh; row < R; row += a.group)
                    sc += Codec::get4(stash + row * stride, k4) * fast_exp2(mt[row * mts] - row_lse[row]);
                float* hrow = a.scores + ((size_t)k.b * a.n_q_heads + k.c * a.group + hh) * a.max_ctx;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (k4 + i < nk) hrow[k.key_begin + k4 + i] = sc[i];
            }
        }
        for (int k4 = 4 * tid; !a.per_head && k4 < nk; k4 += 4 * kThreads) {
            const float* mt = mtile + k4 / kTile;   // mt[row * mts]
            f32x4 sc = {0.f, 0.f, 0.f, 0.f};
            int row = r0;
            for (; row + 8 <= R; row += 8) {   // eight rows' reads in flight
                f32x4 pr[8];
                float cr[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    pr[j] = Codec::get4(stash + (row + j) * stride, k4);
                    cr[j] = mt[(row + j) * mts] - row_lse[row + j];
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) sc += pr[j] * fast_exp2(cr[j]);
            }
            for (; row + 4 <= R; row += 4) {
                f32x4 pr[4];
                float cr[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    pr[j] = Codec::get4(stash + (row + j) * stride, k4);
                    cr[j] = fast_exp2(mt[(row + j) * mts] - row_lse[row + j]);
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) sc += pr[j] * cr[j];
            }
            for (; row < R; ++row)
                sc += Codec::get4(stash + row * stride, k4) * fast_exp2(mt[row * mts] - row_lse[row]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (k4 + i < nk) srow[k.key_begin + k4 + i] = sc[i];
            if constexpr (kStep) *reinterpret_cast<f32x4*>(skeys + k4) = sc;   // k4 + 3 < chunk
        }
    }

    // ---- 4. rows s, s + nchunk, ... summed over the unit's chunks ----------
    if constexpr (!kDefer) {
        __syncthreads();   // the stash is free once every thread's scores are out
        row_sums<kSum>(a, k, row_lse, reinterpret_cast<f32x4*>(stash), &pv, &pm);
    }
    return true;
}

// The unit's chunk 0, once it has every chunk's statistics: every chunk has
// published, so has read the epoch; advanced after the workgroup's final wait
// for loads.
__device__ __forceinline__ void chunk0_done(const FusedArgs& fa, const Chunk& k) {
    if (threadIdx.x != 0 || k.slot != k.slot0) return;
    if (fa.epoch) epoch_advance(fa.epoch + k.unit);
    if (fa.heal) st_dev64(fa.heal + k.unit, fa.heal_value + k.unit);
}

// One workgroup per chunk (fp32 stash): sweep, publish, then the scores and
// outputs; with kStep it goes on as partition s of its unit's select and draft.
template <int NRT, bool kStream, bool kPaged, bool kStep>
__global__ __launch_bounds__(kThreads) void verify_fused_kernel(FusedArgs fa) {
    const VerifyArgs& a = fa.v;
    extern __shared__ __attribute__((aligned(16))) float stash[];   // [NRT*16][chunk + pad]
    __shared__ float2 wml[kWaves][NRT * 16];
    __shared__ float row_lse[kRowCap];
    __shared__ int wait_failed;

    const Chunk k = chunk_of(a, blockIdx.x);
    const int chunk = a.chunk;
    const int stride = chunk + StashF32::kPad;
    const int mts = chunk / kTile;
    float* mtile = stash + NRT * 16 * stride;   // [NRT*16][mts] reference row maxima per tile
    float* park = mtile + mts * (NRT * 16);     // [2][16][kParkStride]
    const int lane = threadIdx.x & 63;
    const int m16 = lane & 15, G = lane >> 4;

    Rows<NRT> r;
    load_rows<NRT>(a, k.b, k.c, k.T, k.nq, 0, k.nq, m16, G, r);
    float M[NRT], L[NRT];
    f32x4 oacc[8][NRT];
    clear_state<NRT>(M, L, oacc);
    sweep_chunk<NRT, kStream, kPaged, StashF32>(a, k, r, stash, stride, mtile, mts, M, L, oacc, [] {});
    bool clean;
    const uint64_t want = publish_chunk<NRT>(fa, k, M, L, oacc, wml, park, &wait_failed, &clean);
    // (decode step: the chunk's score bits also go to skeys, in the parking
    // slices, free once the partial output is out)
    uint32_t* skeys = reinterpret_cast<uint32_t*>(park);
    // (decode step: the output rows are summed later, see below)
    if (!finish_chunk<NRT, StashF32, kStep, 8, 4, kStep>(fa, k, want, clean, stash, stride, mtile, mts,
                                                         row_lse, &wait_failed, skeys))
        return;
    if constexpr (kStep) {
        // ---- 5. select (Eq. 4) and the first draft step (Eq. 5) ------------
        // The verify output rows of the chunk are summed once its select
        // histogram is out, while that exchange is in flight (rows summed
        // first would hold up the unit's exchange for the chunks that have
        // one), in 4 KB of LDS past the select's.
        const SelectArgs& sa = fa.sel;
        const Geom g = geom_of(sa, k.b);
        SelLds& SL = *reinterpret_cast<SelLds*>(stash);
        f32x4* red = reinterpret_cast<f32x4*>(reinterpret_cast<char*>(stash) + kStepRedOffset);
        auto sums = [&]() __attribute__((always_inline)) { row_sums<4>(a, k, row_lse, red, nullptr, nullptr); };
        const int nk = k.key_end - k.key_begin;
        bool done;
        if (g.simple) {
            __syncthreads();   // the stash becomes the select's
            sums();
            done = select_simple<true>(sa, g, k.s, k.unit, SL, want);
        } else if (NRT > 1 || chunk <= kRound) {
            done = step_select<1>(sa, g, k.s, k.unit, skeys, nk, k.key_begin, SL, want, sums);
        } else {
            done = step_select<NRT == 1 ? 2 : 1>(sa, g, k.s, k.unit, skeys, nk, k.key_begin, SL, want, sums);
        }
        // chunk 0 goes on only when every exchange of the step completed
        if (!done) return;
    }
    chunk0_done(fa, k);
}

// Chunks per lane per statistics poll, and per thread per row-sum pass, in
// the persistent kernel's finish (its units may have more chunks).
constexpr int kPipePoll = 16, kPipeSum = 8;

// Persistent one-sweep kernel (16-bit stash, two chunk buffers): workgroup w
// takes chunks w, w + G, w + 2G, ... (round j: its chunk w + jG; G = the grid,
// all resident at once).  At the start of round j + 1's sweep, with each
// wave's first tile of it in flight, the workgroup publishes its round-j chunk
// and finishes its round j - 1 chunk (whose stash buffer the new sweep then
// fills), so each chunk's exchange runs a round behind its streaming.  The
// host keeps a unit's chunks within two consecutive rounds (at most G per
// unit), so that finish waits only for chunks of rounds j - 1 and j, which
// every workgroup publishes at the start of rounds j and j + 1, before it
// waits on anything there: no wait depends on a workgroup that is itself
// waiting.
template <int NRT, bool kPaged>
__global__ __launch_bounds__(kThreads) void verify_pipe_kernel(FusedArgs fa) {
    using Codec = StashU16;
    const VerifyArgs& a = fa.v;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ float2 wml[kWaves][NRT * 16];
    __shared__ float row_lse[kRowCap];
    __shared__ int wait_failed;

    const int chunk = a.chunk;
    const int stride = chunk + Codec::kPad;
    const int mts = chunk / kTile;
    const int code_bytes = NRT * 16 * stride * 2;                 // a multiple of 16
    const int buf_bytes = code_bytes + NRT * 16 * mts * 4;
    char* base = reinterpret_cast<char*>(lds);
    float* park = reinterpret_cast<float*>(base + 2 * buf_bytes);   // [2][16][kParkStride]
    auto codes = [&](int j) { return reinterpret_cast<uint16_t*>(base + (j & 1) * buf_bytes); };
    auto tiles = [&](int j) { return reinterpret_cast<float*>(base + (j & 1) * buf_bytes + code_bytes); };
    const int lane = threadIdx.x & 63;
    const int m16 = lane & 15, G = lane >> 4;
    const int grid = gridDim.x, w = blockIdx.x;
    const int n = (fa.n_tasks - w + grid - 1) / grid;   // >= 1: the grid is at most the task count

    float M[NRT], L[NRT];
    f32x4 oacc[8][NRT];
    clear_state<NRT>(M, L, oacc);
    Chunk k1 = chunk_of(a, w), k2 = k1;   // chunks j - 1 and j - 2
    uint64_t want1 = 0, want2 = 0;
    bool clean1 = false, clean2 = false, failed = false;
    // (the finish calls are written out: a lambda around them is not inlined
    // and puts the kernel's locals on the scratch stack)
    for (int j = 0; j < n; ++j) {
        const Chunk k = chunk_of(a, w + j * grid);
        Rows<NRT> r;
        load_rows<NRT>(a, k.b, k.c, k.T, k.nq, 0, k.nq, m16, G, r);
        sweep_chunk<NRT, false, kPaged, Codec>(a, k, r, codes(j), stride, tiles(j), mts, M, L, oacc, [&] {
            if (j >= 1) {
                want1 = publish_chunk<NRT>(fa, k1, M, L, oacc, wml, park, &wait_failed, &clean1);
                clear_state<NRT>(M, L, oacc);
            }
            if (j >= 2) {   // chunk j - 2's stash: buffer (j - 2) & 1 = j & 1
                if (finish_chunk<NRT, Codec, false, kPipePoll, kPipeSum>(fa, k2, want2, clean2, codes(j), stride,
                                                                         tiles(j), mts, row_lse,
                                                                         &wait_failed, nullptr))
                    chunk0_done(fa, k2);
                else
                    failed = true;
            }
        });
        if (failed) return;
        k2 = k1;
        want2 = want1;
        clean2 = clean1;
        k1 = k;
    }
    want1 = publish_chunk<NRT>(fa, k1, M, L, oacc, wml, park, &wait_failed, &clean1);
    if (n >= 2) {
        if (!finish_chunk<NRT, Codec, false, kPipePoll, kPipeSum>(fa, k2, want2, clean2, codes(n), stride, tiles(n),
                                                                  mts, row_lse, &wait_failed, nullptr))
            return;
        chunk0_done(fa, k2);
    }
    if (!finish_chunk<NRT, Codec, false, kPipePoll, kPipeSum>(fa, k1, want1, clean1, codes(n - 1), stride,
                                                              tiles(n - 1), mts, row_lse, &wait_failed,
                                                              nullptr))
        return;
    chunk0_done(fa, k1);
}

template <int NRT>
constexpr size_t fused_lds_bytes(int chunk) {
    // the probability stash with its tile maxima, then the parking slices
    return ((size_t)NRT * 16 * (chunk + StashF32::kPad + chunk / kTile) + kParkFloats) * sizeof(float);
}

constexpr int kPipeMaxRowTiles = 3;   // 48 rows: more spill the persistent kernel's registers

template <int NRT>
constexpr size_t pipe_lds_bytes(int chunk) {
    // two buffers of 16-bit codes and tile maxima, then the parking slices
    const size_t codes = (size_t)NRT * 16 * (chunk + StashU16::kPad) * 2;
    const size_t tiles = (size_t)NRT * 16 * (chunk / kTile) * sizeof(float);
    return 2 * (codes + tiles) + kParkFloats * sizeof(float);
}

// The largest chunk (a multiple of 128 keys) whose two buffers fit in LDS.
template <int NRT>
constexpr int max_pipe_chunk() {
    int c = 128;
    while (pipe_lds_bytes<NRT>(c + 128) + static_lds_bytes<NRT>() + 1024 <= 160 * 1024) c += 128;
    return c;
}

// Once per device and row-tile count: the kernels' dynamic LDS limits are
// raised to the largest stashes, and the CU count and the workgroups a CU
// holds at that LDS use are read (doing this twice is harmless, so a race
// between threads is too).
struct FusedDevice {
    int n_cu, per_cu, pipe_per_cu;
};

template <int NRT>
hipError_t fused_setup(FusedDevice* out) {
    constexpr int kMaxDevices = 64;
    // packed (n_cu * 16 + per_cu) * 16 + pipe_per_cu, plus 1; 0: not set up yet
    static std::atomic<int> state[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    int st = dev >= 0 && dev < kMaxDevices ? state[dev].load(std::memory_order_relaxed) : 0;
    if (st == 0) {
        const int lds = (int)std::max(fused_lds_bytes<NRT>(max_fused_chunk<NRT>()), kStepLdsMin);
        const void* fns[6] = {reinterpret_cast<const void*>(verify_fused_kernel<NRT, true, false, false>),
                              reinterpret_cast<const void*>(verify_fused_kernel<NRT, false, false, false>),
                              reinterpret_cast<const void*>(verify_fused_kernel<NRT, true, true, false>),
                              reinterpret_cast<const void*>(verify_fused_kernel<NRT, false, true, false>),
                              reinterpret_cast<const void*>(verify_fused_kernel<NRT, true, false, true>),
                              reinterpret_cast<const void*>(verify_fused_kernel<NRT, false, false, true>)};
        for (const void* f : fns) {
            e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
            if (e != hipSuccess) return e;
        }
        int cu = 0, blocks = 0, pipe_blocks = 0;
        if constexpr (NRT <= kPipeMaxRowTiles) {
            const int pipe_lds = (int)pipe_lds_bytes<NRT>(max_pipe_chunk<NRT>());
            const void* pfns[2] = {reinterpret_cast<const void*>(verify_pipe_kernel<NRT, false>),
                                   reinterpret_cast<const void*>(verify_pipe_kernel<NRT, true>)};
            for (const void* f : pfns) {
                e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, pipe_lds);
                if (e != hipSuccess) return e;
            }
            e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&pipe_blocks, verify_pipe_kernel<NRT, false>,
                                                             kThreads, pipe_lds);
            if (e != hipSuccess) return e;
        }
        e = hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, verify_fused_kernel<NRT, true, false, false>,
                                                         kThreads, lds);
        if (e != hipSuccess) return e;
        st = (std::min(cu, (1 << 20) - 1) * 16 + std::min(blocks, 15)) * 16 + std::min(pipe_blocks, 15) + 1;
        if (dev >= 0 && dev < kMaxDevices) state[dev].store(st, std::memory_order_relaxed);
    }
    out->n_cu = (st - 1) / 256;
    out->per_cu = ((st - 1) / 16) % 16;
    out->pipe_per_cu = (st - 1) % 16;
    return hipSuccess;
}

template <int NRT>
hipError_t launch_fused_nrt(const FusedArgs& a, int n_slots, hipStream_t stream) {
    FusedDevice fd;
    const hipError_t e = fused_setup<NRT>(&fd);
    if (e != hipSuccess) return e;
    const bool paged = a.v.block_table != nullptr;
    const dim3 grid(n_slots), block(kThreads);
    if (a.n_tasks > 0) {   // persistent: n_slots workgroups over n_tasks chunks
        if constexpr (NRT <= kPipeMaxRowTiles) {
            const size_t dyn = pipe_lds_bytes<NRT>(a.v.chunk);
            if (paged)
                hipLaunchKernelGGL((verify_pipe_kernel<NRT, true>), grid, block, dyn, stream, a);
            else
                hipLaunchKernelGGL((verify_pipe_kernel<NRT, false>), grid, block, dyn, stream, a);
            return hipGetLastError();
        } else {
            return hipErrorInvalidValue;   // (the host plans it only up to kPipeMaxRowTiles)
        }
    }
    // non-temporal K/V loads when every workgroup runs in the first round
    const bool stream1 = n_slots <= fd.n_cu;
    if (a.step) {   // (dense caches only; the host checks)
        const size_t dyn = std::max(fused_lds_bytes<NRT>(a.v.chunk), kStepLdsMin);
        if (stream1)
            hipLaunchKernelGGL((verify_fused_kernel<NRT, true, false, true>), grid, block, dyn, stream, a);
        else
            hipLaunchKernelGGL((verify_fused_kernel<NRT, false, false, true>), grid, block, dyn, stream, a);
        return hipGetLastError();
    }
    const size_t dyn = fused_lds_bytes<NRT>(a.v.chunk);
    if (stream1) {
        if (paged)
            hipLaunchKernelGGL((verify_fused_kernel<NRT, true, true, false>), grid, block, dyn, stream, a);
        else
            hipLaunchKernelGGL((verify_fused_kernel<NRT, true, false, false>), grid, block, dyn, stream, a);
    } else {
        if (paged)
            hipLaunchKernelGGL((verify_fused_kernel<NRT, false, true, false>), grid, block, dyn, stream, a);
        else
            hipLaunchKernelGGL((verify_fused_kernel<NRT, false, false, false>), grid, block, dyn, stream, a);
    }
    return hipGetLastError();
}

template <int NRT>
FusedDevice fused_device() {
    FusedDevice fd = {0, 0, 0};
    if (fused_setup<NRT>(&fd) != hipSuccess) {
        (void)hipGetLastError();
        return FusedDevice{0, 0, 0};
    }
    return fd;
}

}  // namespace

int fused_max_chunk(int row_tiles) {
    switch (row_tiles) {
        case 1: return max_fused_chunk<1>();
        case 2: return max_fused_chunk<2>();
        case 3: return max_fused_chunk<3>();
        default: return max_fused_chunk<4>();
    }
}

int fused_blocks_per_cu(int row_tiles) {
    switch (row_tiles) {
        case 1: return fused_device<1>().per_cu;
        case 2: return fused_device<2>().per_cu;
        case 3: return fused_device<3>().per_cu;
        default: return fused_device<4>().per_cu;
    }
}

int pipe_max_chunk(int row_tiles) {
    static_assert(kPipeMaxRowTiles == 3, "the cases below");
    switch (row_tiles) {
        case 1: return max_pipe_chunk<1>();
        case 2: return max_pipe_chunk<2>();
        case 3: return max_pipe_chunk<3>();
        default: return 0;   // not built for more rows
    }
}

int pipe_blocks_per_cu(int row_tiles) {
    switch (row_tiles) {
        case 1: return fused_device<1>().pipe_per_cu;
        case 2: return fused_device<2>().pipe_per_cu;
        case 3: return fused_device<3>().pipe_per_cu;
        default: return fused_device<4>().pipe_per_cu;
    }
}

hipError_t launch_verify_fused(const FusedArgs& a, int n_slots, int row_tiles, hipStream_t stream) {
    switch (row_tiles) {
        case 1: return launch_fused_nrt<1>(a, n_slots, stream);
        case 2: return launch_fused_nrt<2>(a, n_slots, stream);
        case 3: return launch_fused_nrt<3>(a, n_slots, stream);
        default: return launch_fused_nrt<4>(a, n_slots, stream);
    }
}

}  // namespace ssl
