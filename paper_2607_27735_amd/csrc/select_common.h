// select_common.h -- one partition of the Eq. 4 split radix select, for any
// kernel whose workgroups each hold one partition's score bits: the one-kernel
// select, which loads them, and the verify kernel that has just computed them.
// Internal to the library.
//
// A unit's partitions are resident together and exchange what they need
// through the workspace with device-coherent stores and loads, each exchange
// closed by tag words that carry the call tag and the partition's counts (see
// tagged() below):
//   A. every partition publishes its nonzero histogram bins (bin, count),
//      each entry tagged on its own; all of them add the unit's bins and find
//      the bin d1 holding the K_mid-th largest middle score and `need`;
//   B. every partition publishes its bin-d1 candidates (in position order),
//      their count and its count of middle positions above d1;
//   C. every partition gathers the unit's candidates and resolves tau by two
//      10-bit radix passes (the same result in each), then the output offset
//      of every partition and how many of its entries equal to tau it takes
//      (ties go to the lowest positions, i.e. the first partitions);
//   D. every partition emits its own selections at its offset; partition 0
//      also emits the sink and recent ranges and n_idx.
// Every wait is bounded: a partition whose wait gives up reports it on the
// device's status word and leaves without writing indices (the partitions
// waiting on it then give up too), so a broken invariant never hangs and never
// uses counts that were not validated.
#pragma once

#include "device_common.h"
#include "draft_common.h"
#include "launch.h"
#include "verify_common.h"

namespace ssl {
namespace {

constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kRound = 4 * kSelThreads;      // positions per round: 4 per thread
constexpr int kTailCand = 8192;              // candidates the finish kernel caches in LDS
constexpr int kTailWords = 4096;             // bitmask words per emission chunk
constexpr uint32_t kNone = 0xffffffffu;      // "not a middle position" marker

__device__ __forceinline__ uint32_t bin12(uint32_t k) { return (k >> 20) & 2047u; }

struct Geom {
    int T, s_end, r_start, take, parts;
    bool all_mid, simple;
};

__device__ __forceinline__ Geom geom_of(const SelectArgs& a, int b) {
    Geom g;
    g.T = a.ctx[b];
    g.s_end = min(a.k_sink, g.T);
    g.r_start = max(g.T - a.k_recent, g.s_end);
    const int n_mid = g.r_start - g.s_end;
    g.take = min(a.budget - a.k_sink - a.k_recent, n_mid);
    g.all_mid = g.take == n_mid;
    g.simple = g.all_mid || g.take == 0;   // no radix select needed
    g.parts = (g.T + a.part - 1) / a.part;
    return g;
}

// Score bits of position i if it is a middle position, kNone otherwise.  The
// load is clamped into [0, T) so that it is unconditional.
// (The load is unconditional and the result masked, so that the compiler keeps
// the loads of a thread's keys in flight together instead of branching around
// each one and waiting for it.)
__device__ __forceinline__ uint32_t key_of(const float* S, const Geom& g, int i) {
    uint32_t v = __builtin_bit_cast(uint32_t, S[min(i, g.T - 1)]);
    v = v == 0x80000000u ? 0u : v;   // -0 ranks as +0 (equal scores)
    return v | ((i >= g.s_end && i < g.r_start) ? 0u : kNone);
}

// Exclusive prefix sum of one value per thread over the workgroup; *total gets
// the sum.  wave_tot is LDS scratch of kSelWaves words.
__device__ __forceinline__ int block_scan(int v, int* wave_tot, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int incl = wave_incl_scan(v);
    __syncthreads();
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        const int t = wave_tot[w];
        before += w < wave ? t : 0;
        all += t;
    }
    *total = all;
    return before + incl - v;
}

struct Digit {
    int bin, above, count;
};

// In a 1024-bin histogram read from the top bin down, finds the bin where the
// running count first reaches `remaining` (1 <= remaining <= the total), the
// count strictly above that bin and the bin's own count.  Thread t holds the
// four bins 1020-4t .. 1023-4t (one conflict-free 16-byte LDS read); every
// thread gets the result.  It synchronises the workgroup (sh: 3 ints of LDS).
__device__ __forceinline__ Digit find_digit_block(const uint32_t* h, int remaining, int* sh,
                                                  int* wave_tot) {
    const int tid = threadIdx.x;
    const uint4 w = *reinterpret_cast<const uint4*>(h + 1020 - 4 * tid);
    const int c[4] = {(int)w.w, (int)w.z, (int)w.y, (int)w.x};   // descending bins
    const int sum = c[0] + c[1] + c[2] + c[3];
    int total;
    int above = block_scan(sum, wave_tot, &total);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (above < remaining && remaining <= above + c[q]) {
            sh[0] = 1023 - 4 * tid - q;
            sh[1] = above;
            sh[2] = c[q];
        }
        above += c[q];
    }
    __syncthreads();
    Digit d;
    d.bin = sh[0] & 1023;
    d.above = sh[1];
    d.count = sh[2];
    __syncthreads();
    return d;
}


// Sink, then every middle position or none, then recent: ranges.
__device__ __forceinline__ void emit_ranges(const SelectArgs& a, int u, const Geom& g) {
    const int b = u / a.n_kv_heads;
    const int tid = threadIdx.x;
    int32_t* out = a.idx + (size_t)u * a.budget;
    const int n = g.all_mid ? g.T : g.s_end + (g.T - g.r_start);
    for (int x = tid; x < n; x += kSelThreads)
        if (x < a.budget) out[x] = (g.all_mid || x < g.s_end) ? x : g.r_start + (x - g.s_end);
    if (u - b * a.n_kv_heads == 0 && tid == 0) a.n_idx[b] = n;
}


// A count travels in its tag word: the low 48 bits of the exchange tag above
// a 16-bit count (successive calls on a workspace use different exchange
// tags, so a stale or uninitialised word matches only by accident), and the
// wait that finds the word valid has the count without another load.
__device__ __forceinline__ uint64_t tagged(uint64_t call_tag, uint32_t count) {
    return (call_tag << 16) | count;
}
// the counts carried: histogram entries (<= 2048), candidates and middle
// positions above d1 of one partition (<= its length)
static_assert(kSelectMaxRounds * kRound <= 0xffff, "a partition's counts must fit 16 bits");

// A published histogram entry carries its own tag, so that a reader can load
// the entries in the same round trip as the tag word that gives their count:
// the low 39 bits of the exchange tag above the bin (11 bits) and its count
// (14 bits).
constexpr int kBinPayloadBits = 25;
constexpr uint64_t kBinTagMask = (1ull << (64 - kBinPayloadBits)) - 1ull;
__device__ __forceinline__ uint64_t bin_entry(uint64_t call_tag, uint32_t bin, uint32_t count) {
    return ((call_tag & kBinTagMask) << kBinPayloadBits) | ((uint64_t)bin << 14) | count;
}
static_assert(kSelectMaxRounds * kRound < (1 << 14), "a bin count must fit 14 bits");
static_assert(2048 * 2 <= kHistSlotWords, "a partition's bin entries must fit its slot");

// Wave 0 polls until the words tag[q*stride] (and tag[q*stride + 1] when c1
// is given), q < n, all carry the call tag, then writes their counts to c0[q]
// (and c1[q]); after spin_limit polls it gives up and sets *failed instead.
// The caller synchronises the workgroup afterwards.
__device__ __forceinline__ void wait_counts(const uint64_t* tag, int n, int stride, uint64_t call_tag,
                                            uint32_t* c0, uint32_t* c1, int spin_limit,
                                            int* failed) {
    if ((threadIdx.x >> 6) != 0) return;
    const int lane = threadIdx.x & 63;
    const uint64_t want = call_tag & 0xFFFFFFFFFFFFull;
    constexpr int kPer = kMaxSelectParts / kWave;
    uint64_t v0[kPer], v1[kPer];
    int spins = 0;
    bool all_in;
    // (every lane loads, lanes past n re-reading the last words: no branch
    // around the loads, so that they are in flight together)
    const int nj = (n + kWave - 1) / kWave;   // wave-uniform
    do {
        bool in = true;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            if (j < nj) {
                const size_t q = (size_t)min(lane + j * kWave, n - 1) * stride;
                v0[j] = ld_dev64(tag + q);
                v1[j] = c1 ? ld_dev64(tag + q + 1) : want << 16;
            }
        }
#pragma unroll
        for (int j = 0; j < kPer; ++j)
            if (j < nj) in &= (v0[j] >> 16) == want && (v1[j] >> 16) == want;
        all_in = __all(in);
        if (!all_in) __builtin_amdgcn_s_sleep(1);
    } while (!all_in && ++spins < spin_limit);
    if (!all_in) {
        if (lane == 0) *failed = 1;
        return;
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int q = lane + j * kWave;
        if (q < n) {
            c0[q] = (uint32_t)(v0[j] & 0xffffu);
            if (c1) c1[q] = (uint32_t)(v1[j] & 0xffffu);
        }
    }
}

constexpr int kTags = kSelectTagWords;   // tag words per partition: histogram entries, candidates,
                                         // middle above d1, draft partial

// Output columns 4 d4 .. 4 d4 + 3 of head row `row` (x = row * 32 + d4) of KV
// head c of sequence b: the merged sum over its total.
__device__ __forceinline__ void draft_out(const SelectDraft& d, int b, int c, int x, const f32x4& acc, float Lx) {
    const int row = x >> 5, d4 = x & 31;
    const f32x4 o = acc * (1.0f / Lx);
    const size_t base = ((size_t)b * d.n_q_heads + c * d.group + row) * kHeadDim + 4 * d4;
    if (d.out_fp32) {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(d.out) + base) = o;
    } else {
        const uint2 pk = make_uint2(pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3]));
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(d.out) + base) = pk;
    }
}

constexpr int kSelectMergeBatch = 16;   // draft partials merged per round trip

// Folds the draft partials of partitions p0 .. p0 + kSelectMergeBatch - 1
// (those below P) into (Mx, Lx, acc) for head row `row`, columns 4 d4 ..
// 4 d4 + 3: partition 0's own from the LDS park (its four waves), the others'
// from their published slots (loaded together, one round trip).
__device__ __forceinline__ void absorb_partials(int p0, int P, int row, int d4, const float* part0,
                                                const float* park, const float2* gml, float& Mx,
                                                float& Lx, f32x4& acc) {
    constexpr int kStride = kSelectDraftStride;
    float2 ml[kSelectMergeBatch];
    f32x4 o[kSelectMergeBatch];
#pragma unroll
    for (int uu = 0; uu < kSelectMergeBatch; ++uu) {
        const int pp = p0 + uu;
        if (pp == 0) {
            ml[uu] = gml[row];
            f32x4 ov = *reinterpret_cast<const f32x4*>(park + row * kStride + 4 + 4 * d4);
#pragma unroll
            for (int w = 1; w < kSelWaves; ++w)
                ov += *reinterpret_cast<const f32x4*>(park + (w * 16 + row) * kStride + 4 + 4 * d4);
            o[uu] = ov;
        } else if (pp < P) {
            const float* dp = part0 + ((size_t)pp * 16 + row) * kStride;
            ml[uu] = __builtin_bit_cast(float2, ld_dev64(reinterpret_cast<const uint64_t*>(dp)));
            const uint64_t* po = reinterpret_cast<const uint64_t*>(dp + 4) + 2 * d4;
            const float2 lo = __builtin_bit_cast(float2, ld_dev64(po));
            const float2 hi = __builtin_bit_cast(float2, ld_dev64(po + 1));
            o[uu] = f32x4{lo.x, lo.y, hi.x, hi.y};
        } else {
            ml[uu] = make_float2(-INFINITY, 0.f);
            o[uu] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }
    float Mn = Mx;
#pragma unroll
    for (int uu = 0; uu < kSelectMergeBatch; ++uu) Mn = fmaxf(Mn, ml[uu].x);
    const float alpha = Mx == -INFINITY ? 0.f : fast_exp2(Mx - Mn);
    Lx *= alpha;
    acc *= alpha;
#pragma unroll
    for (int uu = 0; uu < kSelectMergeBatch; ++uu) {
        const float wgt = ml[uu].x == -INFINITY ? 0.f : fast_exp2(ml[uu].x - Mn);
        Lx += ml[uu].y * wgt;
        acc += o[uu] * wgt;
    }
    Mx = Mn;
}

// The first draft step (Eq. 5) over the rows partition p selected, run by the
// select kernel so that no second launch reads the index set back.  Entries
// e < n_mid are the partition's selected middle positions (rows_l[e], or
// mid_base + e when its whole range is selected); then s_len sink positions
// and n_rec recent ones (partition 0 only).  Each wave attends over tiles of
// 32 entries (two-deep gather ring); the four waves merge through LDS; every
// partition but 0 publishes its partial per query head with device-coherent
// stores and then a tag, and partition 0 waits for those tags (bounded),
// merges the partials in partition order and writes the output.  Called by
// every thread of the workgroup; returns whether partition 0 completed (the
// caller then advances the exchange epoch).
// (Inlined: a call would take the address of the launch arguments, which the
// compiler then copies to scratch memory for the whole kernel.)
__device__ __forceinline__ bool select_draft_tail(const SelectArgs& a, const Geom& g, int u, int p,
                                                  int n_mid, int mid_base, int s_len, int n_rec,
                                                  const uint32_t* rows_l, float* park, float2* wml,
                                                  float2* gml, float2* xfer, int* wait_failed,
                                                  uint64_t* tag, uint64_t want, uint64_t pub) {
    using dc::kTile;
    const SelectDraft& d = a.d;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m16 = lane & 15, G = lane >> 4;
    const int b = u / a.n_kv_heads, c = u - b * a.n_kv_heads;
    const int gq = d.group;
    const int n = n_mid + s_len + n_rec;
    const size_t cache_off = ((size_t)b * d.n_kv_real + c / d.kv_div) * a.max_ctx * kHeadDim;
    const dc::RowSource src{d.k + cache_off, d.v + cache_off, nullptr, nullptr};
    auto row_of = [&](int e) -> uint32_t {
        e = min(e, n - 1);
        if (e < n_mid) return mid_base >= 0 ? (uint32_t)(mid_base + e) : rows_l[e];
        e -= n_mid;
        return e < s_len ? (uint32_t)e : (uint32_t)(g.r_start + e - s_len);
    };
    u32x4 qop[4];
    if (m16 < gq) {
        const uint16_t* qp = d.q + ((size_t)b * d.n_q_heads + c * gq + m16) * kHeadDim + 8 * G;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qop[kb] = ld_u32x4(qp + 32 * kb);
    } else {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qop[kb] = u32x4{0u, 0u, 0u, 0u};
    }
    float M = -INFINITY, L = 0.f;
    f32x4 oacc[8];
#pragma unroll
    for (int jd = 0; jd < 8; ++jd) oacc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int ntile = (n + kTile - 1) / kTile;
    vc::tile_pipeline<2, dc::Gathered>(
        wave, ntile, kSelWaves,
        [&](dc::Gathered& t, int tile) {
            dc::gather_tile<false>(row_of(tile * kTile + (lane & 31)), 0, src, m16, G, t);
        },
        [&](const dc::Gathered& t, int tile) {
            dc::draft_tile(d.scale_log2, qop, t, tile * kTile, n, G, M, L, oacc);
        });
    L += shfl_xor_f(L, 16);
    L += shfl_xor_f(L, 32);

    // the four waves, merged in a fixed order: (max, sum) per head in gml, the
    // waves' P.V scaled to that max parked in LDS ([wave][head][stride])
    constexpr int kStride = kSelectDraftStride;
    if (G == 0) wml[wave * 16 + m16] = make_float2(M, L);
    __syncthreads();
    if (tid < 16) {
        float Mx = -INFINITY, Lx = 0.f;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) Mx = fmaxf(Mx, wml[w * 16 + tid].x);
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) {
            const float2 v = wml[w * 16 + tid];
            Lx += v.x == -INFINITY ? 0.f : v.y * fast_exp2(v.x - Mx);
        }
        gml[tid] = make_float2(Mx, Lx);
    }
    {
        float Mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) Mx = fmaxf(Mx, wml[w * 16 + m16].x);
        const float f = M == -INFINITY ? 0.f : fast_exp2(M - Mx);
        float* dst = park + (wave * 16 + m16) * kStride + 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int cc = 32 * G + 8 * i;
            *reinterpret_cast<f32x4*>(dst + cc) = f32x4{oacc[0][i], oacc[1][i], oacc[2][i], oacc[3][i]} * f;
            *reinterpret_cast<f32x4*>(dst + cc + 4) = f32x4{oacc[4][i], oacc[5][i], oacc[6][i], oacc[7][i]} * f;
        }
    }
    __syncthreads();

    const int P = g.parts;
    float* part0 = d.part + (size_t)u * a.parts * 16 * kStride;   // [P][16][kStride]
    if (p != 0) {   // publish the partition's partial and its tag, then leave
        float* dp = part0 + (size_t)p * 16 * kStride;
        for (int x = tid; x < gq * (kHeadDim / 2); x += kSelThreads) {
            const int row = x / (kHeadDim / 2), c2 = x - row * (kHeadDim / 2);
            float2 o = *reinterpret_cast<const float2*>(park + row * kStride + 4 + 2 * c2);
#pragma unroll
            for (int w = 1; w < kSelWaves; ++w) {
                const float2 v = *reinterpret_cast<const float2*>(park + (w * 16 + row) * kStride + 4 + 2 * c2);
                o.x += v.x;
                o.y += v.y;
            }
            st_dev64(reinterpret_cast<uint64_t*>(dp + row * kStride + 4) + c2, __builtin_bit_cast(uint64_t, o));
        }
        if (tid < gq)
            st_dev64(reinterpret_cast<uint64_t*>(dp + tid * kStride), __builtin_bit_cast(uint64_t, gml[tid]));
        wait_stores_done();
        __syncthreads();
        if (tid == 0) st_dev64(tag + (size_t)p * kTags + 3, pub);
        return false;
    }
    // partition 0: the others never wait for it, so their tags arrive
    if (wave == 0) {
        int spins = 0;
        bool all_in;
        do {
            bool in = true;
            for (int pp = 1 + lane; pp < P; pp += kWave) in &= ld_dev64(tag + (size_t)pp * kTags + 3) == want;
            all_in = __all(in);
            if (!all_in) __builtin_amdgcn_s_sleep(1);
        } while (!all_in && ++spins < a.xc.spin_limit);
        if (lane == 0) *wait_failed = !all_in;
    }
    __syncthreads();
    if (*wait_failed) {
        if (tid == 0) exchange_gave_up(a.xc, kStatusSelect, a.epoch ? a.epoch + u : nullptr);
        return false;
    }
    // Every head row's output sums P partials; thread (row, d4) takes
    // columns 4 d4 .. 4 d4 + 3, kSelectMergeBatch partitions per round trip.
    // When there are more partitions than one batch and the rows fit in half
    // the workgroup, the halves take alternate batches at once and half 1
    // hands its sum to half 0 through LDS (xfer): one round trip fewer.
    const int cols = gq * (kHeadDim / 4);
    if (P > kSelectMergeBatch && 2 * cols <= kSelThreads) {
        const int half = tid / (kSelThreads / 2), x = tid % (kSelThreads / 2);
        float Mx = -INFINITY, Lx = 0.f;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        if (x < cols)
            for (int p0 = half * kSelectMergeBatch; p0 < P; p0 += 2 * kSelectMergeBatch)
                absorb_partials(p0, P, x >> 5, x & 31, part0, park, gml, Mx, Lx, acc);
        if (half == 1 && x < cols) {
            xfer[x] = make_float2(Mx, Lx);
            reinterpret_cast<f32x4*>(xfer + kSelThreads / 2)[x] = acc;
        }
        __syncthreads();
        if (half == 0 && x < cols) {
            const float2 ml = xfer[x];
            const f32x4 o = reinterpret_cast<const f32x4*>(xfer + kSelThreads / 2)[x];
            const float Mn = fmaxf(Mx, ml.x);
            const float w0 = Mx == -INFINITY ? 0.f : fast_exp2(Mx - Mn);
            const float w1 = ml.x == -INFINITY ? 0.f : fast_exp2(ml.x - Mn);
            draft_out(d, b, c, x, acc * w0 + o * w1, Lx * w0 + ml.y * w1);
        }
        return true;
    }
    for (int x = tid; x < cols; x += kSelThreads) {
        float Mx = -INFINITY, Lx = 0.f;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int p0 = 0; p0 < P; p0 += kSelectMergeBatch)
            absorb_partials(p0, P, x >> 5, x & 31, part0, park, gml, Mx, Lx, acc);
        draft_out(d, b, c, x, acc, Lx);
    }
    return true;
}

// The LDS of one partition's select (and draft step): static in the select
// kernel, carved from the verify kernel's stash once that is free.
struct __attribute__((aligned(16))) SelLds {
    uint32_t hist[2048];             // read as uint4
    uint32_t h2[1024];
    uint32_t h3[1024];
    uint2 cand_lds[kTailCand];       // later: the draft's park
    uint16_t cand_p[kTailCand];      // later: the draft's rows
    uint32_t n_def[kMaxSelectParts], n_above[kMaxSelectParts], n_tie[kMaxSelectParts];
    uint32_t n_cnt[kMaxSelectParts];   // candidates per partition
    int offs[kMaxSelectParts + 1];
    int wave_tot[kSelWaves];
    int def_w[kSelWaves];
    int sh[4];
    int sh_d[3];
    int n_eq;                        // candidates sharing tau's top 22 bits
    int wait_failed;
    float2 d_wml[kSelWaves * 16], d_gml[16];
};

static_assert(sizeof(SelLds::h2) >= (kSelThreads / 2) * (sizeof(float2) + sizeof(f32x4)),
              "the draft merge's half-to-half exchange fits h2 (free by then)");

// Clears the partition's counters and histograms its keys (bins of the top 12
// score bits).  Synchronises the workgroup before and after the adds.
template <int NR>
__device__ __forceinline__ void select_local_hist(const uint32_t (&keys)[4 * NR], SelLds& L) {
    const int tid = threadIdx.x;
    for (int x = tid; x < 2048; x += kSelThreads) L.hist[x] = 0u;
    for (int x = tid; x < 1024; x += kSelThreads) {
        L.h2[x] = 0u;
        L.h3[x] = 0u;
    }
    if (tid < kMaxSelectParts) {
        L.n_above[tid] = 0u;
        L.n_tie[tid] = 0u;
    }
    if (tid == 0) {
        L.n_eq = 0;
        L.wait_failed = 0;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4 * NR; ++j)
        if (keys[j] != kNone) atomicAdd(&L.hist[bin12(keys[j])], 1u);
    __syncthreads();
}

// Units where every middle position is selected, or none (g.simple): ranges,
// no radix select; with kDraft the draft step over those ranges.  Returns
// whether partition 0 completed an exchange (its caller then advances the
// unit's epoch).
template <bool kDraft>
__device__ __forceinline__ bool select_simple(const SelectArgs& a, const Geom& g, int p, int u,
                                              SelLds& L, uint64_t want) {
    if (p == 0) emit_ranges(a, u, g);
    if constexpr (kDraft) {
        if (threadIdx.x == 0) L.wait_failed = 0;
        __syncthreads();
        uint64_t* tag = a.tag + (size_t)u * a.parts * kTags;
        const int lo = p * a.part, hi = min(lo + a.part, g.T);
        const bool all = g.all_mid;
        return select_draft_tail(a, g, u, p, all ? hi - lo : 0, all ? lo : -1,
                                 !all && p == 0 ? g.s_end : 0, !all && p == 0 ? g.T - g.r_start : 0,
                                 reinterpret_cast<uint32_t*>(L.cand_p),
                                 reinterpret_cast<float*>(L.cand_lds), L.d_wml, L.d_gml,
                                 reinterpret_cast<float2*>(L.h2), &L.wait_failed, tag, want,
                                 want ^ a.xc.tag_flip);
    }
    return false;
}

// Phases A-D of partition p of unit u (not g.simple) over its keys: the score
// bits of positions p*part + r*kRound + wave*256 + e*64 + lane in
// keys[4r + e], kNone where a position is not a middle one (or lies past the
// partition).  select_local_hist must have run on the same keys; `want` is
// the unit's exchange tag of this call, whose epoch the caller has checked.
// With kDraft the first draft step over the partition's selections follows.
// mid() runs, on every thread, once the partition's histogram bins are out
// and before it waits for the others' (work off the exchange's path; it may
// not touch the select's LDS).  Returns whether partition 0 completed (its
// caller then advances the unit's epoch); a partition whose wait gave up has
// reported it and returns false.
struct NoMid {
    __device__ void operator()() const {}
};
template <int NR, bool kDraft, typename Mid = NoMid>
__device__ __forceinline__ bool select_partition(const SelectArgs& a, const Geom& g, int p, int u,
                                                 const uint32_t (&keys)[4 * NR], SelLds& L,
                                                 uint64_t want, Mid&& mid = Mid{}) {
    static_assert(!kDraft || NR * kRound <= 4096, "the draft step's row list holds 4096 entries");
    const int b = u / a.n_kv_heads;
    const int c_head = u - b * a.n_kv_heads;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t up0 = (size_t)u * a.parts;
    const int P = g.parts;
    uint64_t* tag = a.tag + up0 * kTags;      // [P][kTags]
    const uint64_t pub = want ^ a.xc.tag_flip;   // what this partition publishes
    uint32_t* const hist = L.hist;
    uint32_t* const h2 = L.h2;
    uint32_t* const h3 = L.h3;
    int* const wave_tot = L.wave_tot;
    int* const def_w = L.def_w;
    int* const sh = L.sh;
    int* const sh_d = L.sh_d;
    int* const offs = L.offs;
    uint32_t* const n_def = L.n_def;
    uint32_t* const n_above = L.n_above;
    uint32_t* const n_tie = L.n_tie;
    uint32_t* const n_cnt = L.n_cnt;
    int& n_eq = L.n_eq;
    uint2* const cand_lds = L.cand_lds;
    uint16_t* const cand_p = L.cand_p;
    int& wait_failed = L.wait_failed;
    float* const d_park = reinterpret_cast<float*>(L.cand_lds);
    uint32_t* const d_rows = reinterpret_cast<uint32_t*>(L.cand_p);
    (void)d_park;
    // a wait gave up: report it and leave (workgroup-uniform: called after a
    // barrier)
    auto give_up = [&]() {
        if (tid == 0) exchange_gave_up(a.xc, kStatusSelect, a.epoch ? a.epoch + u : nullptr);
    };

    // ---- A. nonzero histogram bins -----------------------------------------
    {
        // thread t: bins 8t .. 8t+7
        const uint4 h0 = *reinterpret_cast<const uint4*>(hist + 8 * tid);
        const uint4 h1 = *reinterpret_cast<const uint4*>(hist + 8 * tid + 4);
        const uint32_t hv[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
        int nz = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) nz += hv[q] != 0u;
        int n_entries;
        int slot = block_scan(nz, wave_tot, &n_entries);
        uint64_t* dst = reinterpret_cast<uint64_t*>(a.hist + (up0 + p) * kHistSlotWords);
#pragma unroll
        for (int q = 0; q < 8; ++q)
            if (hv[q] != 0u) st_dev64(dst + slot++, bin_entry(pub, 8 * tid + q, hv[q]));
        // (no wait for the entry stores: every entry carries the call tag)
        if (tid == 0) st_dev64(tag + (size_t)p * kTags + 0, tagged(pub, (uint32_t)n_entries));
    }
    mid();
    __syncthreads();
    for (int x = tid; x < 2048; x += kSelThreads) hist[x] = 0u;   // now the unit's histogram
    __syncthreads();
    {
        // wave w adds partitions w, w+4, ...: for eight partitions at once it
        // polls their tag words and, in the same round trip, their first 64
        // entries until the words and every entry below the count carry the
        // call tag; then any entries past the first 64 the same way
        const uint64_t want48 = want & 0xFFFFFFFFFFFFull;
        const uint64_t etag = want & kBinTagMask;
        bool gave_up = false;
        for (int p0 = wave; p0 < P && !gave_up; p0 += 4 * 8) {
            int n[8];
            uint64_t v[8];
            const uint64_t* ent[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                ent[j] = reinterpret_cast<const uint64_t*>(a.hist + (up0 + min(p0 + 4 * j, P - 1)) * kHistSlotWords);
            int spins = 0;
            bool all_in;
            do {
                uint64_t tw[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    tw[j] = ld_dev64(tag + (size_t)min(p0 + 4 * j, P - 1) * kTags);
                    v[j] = ld_dev64(ent[j] + lane);
                }
                bool in = true;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    n[j] = (int)(tw[j] & 0xffffu);
                    in &= (tw[j] >> 16) == want48 && (lane >= n[j] || (v[j] >> kBinPayloadBits) == etag);
                }
                all_in = __all(in);
                if (!all_in) __builtin_amdgcn_s_sleep(1);
            } while (!all_in && ++spins < a.xc.spin_limit);
            if (!all_in) {   // wave-uniform
                gave_up = true;
                break;
            }
            bool more = false;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                if (p0 + 4 * j < P && lane < n[j]) atomicAdd(&hist[(v[j] >> 14) & 2047u], (uint32_t)(v[j] & 0x3fffu));
                more |= p0 + 4 * j < P && n[j] > kWave;
            }
            for (int e0 = kWave; more; e0 += kWave) {   // wave-uniform
                spins = 0;
                do {
#pragma unroll
                    for (int j = 0; j < 8; ++j) v[j] = ld_dev64(ent[j] + min(e0 + lane, kHistSlotWords / 2 - 1));
                    bool in = true;
#pragma unroll
                    for (int j = 0; j < 8; ++j) in &= e0 + lane >= n[j] || (v[j] >> kBinPayloadBits) == etag;
                    all_in = __all(in);
                    if (!all_in) __builtin_amdgcn_s_sleep(1);
                } while (!all_in && ++spins < a.xc.spin_limit);
                if (!all_in) {
                    gave_up = true;
                    break;
                }
                more = false;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (p0 + 4 * j < P && e0 + lane < n[j])
                        atomicAdd(&hist[(v[j] >> 14) & 2047u], (uint32_t)(v[j] & 0x3fffu));
                    more |= p0 + 4 * j < P && n[j] > e0 + kWave;
                }
            }
        }
        if (gave_up && lane == 0) wait_failed = 1;
    }
    __syncthreads();
    if (wait_failed) {
        give_up();
        return false;
    }
    {
        // thread t: bins 2047-8t down to 2040-8t
        const uint4 h0 = *reinterpret_cast<const uint4*>(hist + 2040 - 8 * tid);
        const uint4 h1 = *reinterpret_cast<const uint4*>(hist + 2044 - 8 * tid);
        const uint32_t hv[8] = {h1.w, h1.z, h1.y, h1.x, h0.w, h0.z, h0.y, h0.x};   // descending
        int sum = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) sum += (int)hv[q];
        int total;
        int above = block_scan(sum, wave_tot, &total);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (above < g.take && g.take <= above + (int)hv[q]) {
                sh[0] = 2047 - 8 * tid - q;
                sh[1] = g.take - above;
            }
            above += (int)hv[q];
        }
    }
    __syncthreads();
    const uint32_t d1 = (uint32_t)sh[0] & 2047u;
    int need = sh[1];

    // ---- B. candidates, counts -----------------------------------------------
    const uint64_t lt = (1ull << lane) - 1ull;
    uint2* seg = a.seg + (up0 + p) * a.part;
    int run = 0, my_def = 0;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int base = p * a.part + r * kRound + wave * 256;
        uint64_t defb[4], candb[4];
        int n_w = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t k = keys[4 * r + e];
            const bool mid = k != kNone;
            const uint32_t dg = bin12(k);
            defb[e] = __ballot(mid && dg > d1);
            candb[e] = __ballot(mid && dg == d1);
            n_w += __builtin_popcountll(candb[e]);
            my_def += __builtin_popcountll(defb[e]);
        }
        int round_total;
        int slot = run + block_scan(lane == 0 ? n_w : 0, wave_tot, &round_total);
        slot = __builtin_amdgcn_readlane(slot, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if ((candb[e] >> lane) & 1ull) {
                const uint32_t pos = (uint32_t)(base + e * 64 + lane);
                st_dev64(reinterpret_cast<uint64_t*>(seg + slot + __builtin_popcountll(candb[e] & lt)),
                         (uint64_t)keys[4 * r + e] | ((uint64_t)pos << 32));
            }
            slot += __builtin_popcountll(candb[e]);
        }
        run += round_total;
    }
    // my_def is per wave (ballots are wave-uniform): add the waves
    if (lane == 0) def_w[wave] = my_def;
    __syncthreads();
    wait_stores_done();
    __syncthreads();
    if (tid == 0) {
        int nd = 0;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) nd += def_w[w];
        st_dev64(tag + (size_t)p * kTags + 1, tagged(pub, (uint32_t)run));
        st_dev64(tag + (size_t)p * kTags + 2, tagged(pub, (uint32_t)nd));
    }
    wait_counts(tag + 1, P, kTags, want, n_cnt, n_def, a.xc.spin_limit, &wait_failed);
    __syncthreads();
    if (wait_failed) {
        give_up();
        return false;
    }

    // ---- C. every partition resolves tau ------------------------------------
    const int my_cnt = tid < P ? (int)n_cnt[tid] : 0;
    int nc;
    {
        const int o = block_scan(my_cnt, wave_tot, &nc);
        if (tid < P) offs[tid] = o;
        if (tid == 0) offs[P] = nc;
        __syncthreads();
    }
    const bool cached = nc <= kTailCand;
    auto part_of = [&](int x) -> int {   // last partition whose offset is <= x
        int lo = 0;
#pragma unroll
        for (int step = kMaxSelectParts / 2; step >= 1; step >>= 1)
            lo += (lo + step < P && offs[lo + step] <= x) ? step : 0;
        return lo;
    };
    auto load_cand = [&](int pp, int j) -> uint2 {
        const uint64_t v = ld_dev64(reinterpret_cast<const uint64_t*>(a.seg + (up0 + pp) * a.part + j));
        return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
    };
    auto cand = [&](int x) -> uint2 {
        if (cached) return cand_lds[x];
        const int pp = part_of(x);
        return load_cand(pp, x - offs[pp]);
    };
    if (cached) {
        // wave w copies partitions w, w+4, ...: the first 128 entries of eight
        // partitions in flight at once, then any remainder
        for (int p0 = wave; p0 < P; p0 += 4 * 8) {
            int n[8], o[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int pp = p0 + 4 * j;
                o[j] = pp < P ? offs[pp] : 0;
                n[j] = pp < P ? offs[pp + 1] - o[j] : 0;
            }
            for (int e0 = 0; ; e0 += 2 * kWave) {
                bool more = false;
                uint2 v[16];
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int pp = p0 + 4 * (j & 7), e = e0 + (j >> 3) * kWave + lane;
                    v[j] = e < n[j & 7] ? load_cand(pp, e) : make_uint2(0u, 0u);
                }
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int e = e0 + (j >> 3) * kWave + lane;
                    if (e < n[j & 7]) {
                        const int x = o[j & 7] + e;
                        cand_lds[x] = v[j];
                        cand_p[x] = (uint16_t)(p0 + 4 * (j & 7));
                        atomicAdd(&h2[(v[j].x >> 10) & 1023u], 1u);
                    }
                    more |= e0 + 2 * kWave < n[j & 7];
                }
                if (!more) break;   // wave-uniform: n[] and e0 are
            }
        }
    } else {
        for (int x = tid; x < nc; x += kSelThreads) atomicAdd(&h2[(cand(x).x >> 10) & 1023u], 1u);
    }
    __syncthreads();
    const Digit dg2 = find_digit_block(h2, need, sh_d, wave_tot);
    need -= dg2.above;
    const uint32_t prefix = (d1 << 20) | ((uint32_t)dg2.bin << 10);
    // Pass 3 (bits 9..0) over the candidates with that 22-bit prefix.  The
    // candidates above the prefix are counted for their partition now; those
    // with it are listed as (partition, low 10 bits) in the free histogram
    // array for the final counts.
    uint32_t* eq_list = hist;
    for (int x = tid; x < nc; x += kSelThreads) {
        const uint32_t k = cand(x).x;
        const uint32_t top = k & 0xfffffc00u;
        if (top >= prefix) {
            const int pp = cached ? (int)cand_p[x] : part_of(x);
            if (top > prefix) {
                atomicAdd(&n_above[pp], 1u);
            } else {
                atomicAdd(&h3[k & 1023u], 1u);
                const int slot = atomicAdd(&n_eq, 1);
                if (slot < 2048) eq_list[slot] = ((uint32_t)pp << 10) | (k & 1023u);
            }
        }
    }
    __syncthreads();
    const Digit dg3 = find_digit_block(h3, need, sh_d, wave_tot);
    need -= dg3.above;                       // entries equal to tau to take
    const uint32_t tau = prefix | (uint32_t)dg3.bin;
    const int neq = n_eq;
    if (neq <= 2048) {
        for (int x = tid; x < neq; x += kSelThreads) {
            const uint32_t e = eq_list[x], lo = e & 1023u;
            if (lo >= (uint32_t)dg3.bin) atomicAdd(lo > (uint32_t)dg3.bin ? &n_above[e >> 10] : &n_tie[e >> 10], 1u);
        }
    } else {
        for (int x = tid; x < nc; x += kSelThreads) {
            const uint32_t k = cand(x).x;
            if ((k & 0xfffffc00u) == prefix && k >= tau) {
                const int pp = cached ? (int)cand_p[x] : part_of(x);
                atomicAdd(k > tau ? &n_above[pp] : &n_tie[pp], 1u);
            }
        }
    }
    __syncthreads();
    // ties go to the first partitions; offsets follow the sink (one wave
    // scans up to 64 partitions, the workgroup more)
    if (P <= kWave) {
        if (wave == 0) {
            const int nt = lane < P ? (int)n_tie[lane] : 0;
            const int tie_before = wave_incl_scan(nt) - nt;
            const int take_t = min(max(need - tie_before, 0), nt);
            const int out_t = lane < P ? (int)n_def[lane] + (int)n_above[lane] + take_t : 0;
            const int incl = wave_incl_scan(out_t);
            if (lane == p) {
                sh[2] = g.s_end + incl - out_t;
                sh[3] = take_t;
            }
            if (lane == kWave - 1) sh[0] = incl;
        }
    } else {
        const int nt = tid < P ? (int)n_tie[tid] : 0;
        int tie_total;
        const int tie_before = block_scan(nt, wave_tot, &tie_total);
        const int take_t = min(max(need - tie_before, 0), nt);
        const int out_t = tid < P ? (int)n_def[tid] + (int)n_above[tid] + take_t : 0;
        int all_out;
        const int off_t = g.s_end + block_scan(out_t, wave_tot, &all_out);
        if (tid == p) {
            sh[2] = off_t;
            sh[3] = take_t;
        }
        if (tid == 0) sh[0] = all_out;
    }
    __syncthreads();
    const int offset = sh[2], take = sh[3], total_mid = sh[0];

    // ---- D. this partition's selections at its offset ------------------------
    // Straight from ballots over the keys: a selected key at position x goes
    // to offset + (selected non-ties before x) + min(ties before x, take); a
    // tie is selected while its rank among the partition's ties is < take.
    // One block scan per round carries both counts (packed, 16 bits each).
    int32_t* out = a.idx + (size_t)u * a.budget;
    int run_a = 0, run_t = 0;   // non-ties selected and ties, before this round (uniform)
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int base = p * a.part + r * kRound + wave * 256;
        uint64_t ab[4], tb[4];
        int na = 0, nt = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t k = keys[4 * r + e];
            const bool mid = k != kNone;
            const uint32_t dg = bin12(k);
            ab[e] = __ballot(mid && (dg > d1 || (dg == d1 && k > tau)));
            tb[e] = __ballot(mid && dg == d1 && k == tau);
            na += __builtin_popcountll(ab[e]);
            nt += __builtin_popcountll(tb[e]);
        }
        int round_tot;
        int pre = block_scan(lane == 0 ? (na << 16) | nt : 0, wave_tot, &round_tot);
        pre = __builtin_amdgcn_readlane(pre, 0);
        int ca = run_a + (pre >> 16), ct = run_t + (pre & 0xffff);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int xa = ca + __builtin_popcountll(ab[e] & lt);
            const int xt = ct + __builtin_popcountll(tb[e] & lt);
            int pos = -1;
            if ((ab[e] >> lane) & 1ull) pos = offset + xa + min(xt, take);
            else if (((tb[e] >> lane) & 1ull) && xt < take) pos = offset + xa + xt;
            if (pos >= 0 && pos < a.budget) out[pos] = base + e * 64 + lane;
            if (kDraft && pos >= 0) d_rows[pos - offset] = (uint32_t)(base + e * 64 + lane);
            ca += __builtin_popcountll(ab[e]);
            ct += __builtin_popcountll(tb[e]);
        }
        run_a += round_tot >> 16;
        run_t += round_tot & 0xffff;
    }
    if (p == 0) {
        // sink, recent and the count
        for (int x = tid; x < g.s_end; x += kSelThreads)
            if (x < a.budget) out[x] = x;
        const int n_recent = g.T - g.r_start;
        const int rbase = g.s_end + total_mid;
        for (int x = tid; x < n_recent; x += kSelThreads)
            if (rbase + x < a.budget) out[rbase + x] = g.r_start + x;
        if (c_head == 0 && tid == 0) a.n_idx[b] = rbase + n_recent;
    }
    if constexpr (kDraft) {
        // this partition's middle selections: the non-ties and its first ties
        const int n_mid = run_a + min(run_t, take);
        __syncthreads();   // the row list and the free candidate cache
        return select_draft_tail(a, g, u, p, n_mid, -1, p == 0 ? g.s_end : 0,
                                 p == 0 ? g.T - g.r_start : 0, d_rows, d_park, L.d_wml, L.d_gml,
                                 reinterpret_cast<float2*>(L.h2), &wait_failed, tag, want, pub);
    }
    return p == 0;
}

}  // namespace
}  // namespace ssl
