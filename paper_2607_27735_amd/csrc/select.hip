// select.hip -- Eq. 4 recallable index sets by a split radix select.
//
// Scores are non-negative fp32, so their bit patterns order like their
// values.  Each (sequence, KV head) unit is cut into partitions of `part`
// positions, one 256-thread workgroup per partition, so that a handful of
// units still spreads over the whole chip.  Two schedules:
//
// One kernel (calls of at most kSelectFuseMaxGroups partitions whose units'
// partitions fit on the device at once, select_fused_kernel):
// the partitions of a unit are resident together and exchange nonzero
// histogram bins, then bin-d1 candidates through the workspace; every
// partition then resolves the exact threshold and emits its own selections
// (see the comment above that kernel).
//
// Three kernels (larger calls), the kernel boundaries being the only
// synchronisation between workgroups:
// hist:   each partition histograms the top 12 bits of its middle scores
//         (2048 fine bins, plus 64 coarse bins of 32) into its own slot of
//         the workspace: no atomics on global memory, nothing to clear.
// mark:   every partition sums the coarse and then the fine slot histograms
//         of its unit and finds the bin d1 holding the K_mid-th largest middle
//         score.  It writes its words of the unit's bitmask of middle
//         positions above bin d1 and appends its bin-d1 positions, in
//         position order, to its own candidate segment.
// finish: one workgroup per unit runs two 10-bit radix passes over the
//         candidates for the exact threshold tau and `need`, the number of
//         entries equal to tau that still fit; it marks the candidates above
//         tau and the first `need` ties (lowest positions) and emits sink,
//         middle selections (by a block scan of per-thread popcounts) and
//         recent in ascending order.
#include "select_common.h"


namespace ssl {
namespace {

// ---------------------------------------------------------------------------
// Kernel 1: per-partition histograms.  grid = (parts, units).
// ---------------------------------------------------------------------------
template <int NR>
__global__ __launch_bounds__(kSelThreads) void select_hist_kernel(SelectArgs a) {
    const int p = blockIdx.x, u = blockIdx.y;
    const int b = u / a.n_kv_heads;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const Geom g = geom_of(a, b);
    if (p >= g.parts || g.simple) return;
    const float* S = a.scores + (size_t)u * a.max_ctx;

    __shared__ uint32_t hist[2048];
    uint32_t keys[4 * NR];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            keys[4 * r + e] = key_of(S, g, p * a.part + r * kRound + wave * 256 + e * 64 + lane);
    for (int x = tid; x < 2048; x += kSelThreads) hist[x] = 0u;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4 * NR; ++j)
        if (keys[j] != kNone) atomicAdd(&hist[bin12(keys[j])], 1u);
    __syncthreads();

    const size_t up = (size_t)u * a.parts + p;
    uint4* dst = reinterpret_cast<uint4*>(a.hist + up * kHistSlotWords);
    const uint4* src = reinterpret_cast<const uint4*>(hist);
    dst[tid] = src[tid];
    dst[tid + kSelThreads] = src[tid + kSelThreads];
    // coarse bin t>>2 = fine bins [32*(t>>2), +32): 4 threads of 8 bins each
    uint32_t s = 0u;
#pragma unroll
    for (int q = 0; q < 8; ++q) s += hist[8 * tid + q];
    s += (uint32_t)__shfl_xor((int)s, 1, kWave);
    s += (uint32_t)__shfl_xor((int)s, 2, kWave);
    if ((tid & 3) == 0) a.coarse[up * 64 + (tid >> 2)] = s;
}

// ---------------------------------------------------------------------------
// The finish of one unit (separate kernel): exact threshold, ties and ordered
// emission from the bitmask, counts and candidates of the mark kernel.
// ---------------------------------------------------------------------------

__device__ void finish_unit(const SelectArgs& a, int u, const Geom& g, uint32_t d1, int need) {
    const int b = u / a.n_kv_heads;
    const int c_head = u - b * a.n_kv_heads;
    const int tid = threadIdx.x;
    const size_t up0 = (size_t)u * a.parts;
    const uint32_t* mask = a.mask + (size_t)u * (a.parts * (a.part / 32));

    __shared__ int sh_d[3];
    __shared__ int wave_tot[kSelWaves];
    __shared__ __attribute__((aligned(16))) uint32_t h2[1024];   // read as uint4
    __shared__ __attribute__((aligned(16))) uint32_t h3[1024];
    __shared__ int offs[kMaxSelectParts + 1];
    __shared__ uint2 cand_lds[kTailCand];
    __shared__ uint32_t lmask[kTailWords];

    // All first-round loads at once: the first bitmask chunk and the
    // partition candidate counts.
    constexpr int kWordsPerThread = kTailWords / kSelThreads;
    const int n_words = (g.T + 31) >> 5;
    uint32_t mw[kWordsPerThread];
#pragma unroll
    for (int j = 0; j < kWordsPerThread; ++j) {
        const int x = tid + j * kSelThreads;
        mw[j] = x < n_words ? mask[x] : 0u;
    }
    const int per_p = (g.parts + kSelThreads - 1) / kSelThreads;
    const int q0 = min(g.parts, tid * per_p), q1 = min(g.parts, q0 + per_p);
    int my_cnt = 0;
    for (int q = q0; q < q1; ++q) my_cnt += (int)a.cnt[up0 + q];
    for (int x = tid; x < 1024; x += kSelThreads) {
        h2[x] = 0u;
        h3[x] = 0u;
    }
#pragma unroll
    for (int j = 0; j < kWordsPerThread; ++j) lmask[tid + j * kSelThreads] = mw[j];

    // Candidate offsets: partition pp owns [offs[pp], offs[pp+1]) of the
    // concatenated list, which is in position order.
    {
        int nc_all;
        int o = block_scan(my_cnt, wave_tot, &nc_all);
        for (int q = q0; q < q1; ++q) {
            offs[q] = o;
            o += (int)a.cnt[up0 + q];
        }
        if (tid == 0) offs[g.parts] = nc_all;
        __syncthreads();
    }
    const int nc = offs[g.parts];
    const bool cached = nc <= kTailCand;
    auto cand_global = [&](int x) -> uint2 {
        int lo = 0;   // last partition whose offset is <= x (fixed steps, unrolled)
#pragma unroll
        for (int step = kMaxSelectParts / 2; step >= 1; step >>= 1)
            lo += (lo + step < g.parts && offs[lo + step] <= x) ? step : 0;
        return a.seg[(up0 + lo) * a.part + (x - offs[lo])];
    };
    auto cand = [&](int x) -> uint2 { return cached ? cand_lds[x] : cand_global(x); };

    uint32_t tau = 0u;
    bool all_ties = true;   // every entry equal to tau is taken
    {
        // Pass 2 (bits 19..10) while gathering: every candidate is in bin d1.
        constexpr int U = 8;   // loads in flight per thread
        for (int x0 = tid; x0 < nc; x0 += U * kSelThreads) {
            uint2 v[U];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int x = x0 + j * kSelThreads;
                v[j] = x < nc ? cand_global(x) : make_uint2(0u, 0u);
            }
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int x = x0 + j * kSelThreads;
                if (x < nc) {
                    if (cached) cand_lds[x] = v[j];
                    atomicAdd(&h2[(v[j].x >> 10) & 1023u], 1u);
                }
            }
        }
        __syncthreads();
        const Digit dg2 = find_digit_block(h2, need, sh_d, wave_tot);
        need -= dg2.above;
        const uint32_t prefix = (d1 << 20) | ((uint32_t)dg2.bin << 10);
        // Pass 3 (bits 9..0) over the candidates with that 22-bit prefix.
        for (int x = tid; x < nc; x += kSelThreads) {
            const uint32_t k = cand(x).x;
            if ((k & 0xfffffc00u) == prefix) atomicAdd(&h3[k & 1023u], 1u);
        }
        __syncthreads();
        const Digit dg3 = find_digit_block(h3, need, sh_d, wave_tot);
        need -= dg3.above;
        tau = prefix | (uint32_t)dg3.bin;
        all_ties = need == dg3.count;
    }
    // Mark the candidates above tau and the chosen ties.  Ties are ranked
    // only when some of them stay out: thread t then takes the contiguous
    // slice [x0, x1) of the (position-ordered) list.
    const int per = (nc + kSelThreads - 1) / kSelThreads;
    const int x0 = min(nc, tid * per), x1 = min(nc, x0 + per);
    int tie_base = 0;
    if (!all_ties) {
        int nt = 0;
        for (int x = x0; x < x1; ++x) nt += cand(x).x == tau;
        int tie_total;
        tie_base = block_scan(nt, wave_tot, &tie_total);
    }
    // Sink, then the middle selections in position order, then the recent
    // span: the bitmask holds middle positions only.
    int32_t* out = a.idx + (size_t)u * a.budget;
    for (int x = tid; x < g.s_end; x += kSelThreads)
        if (x < a.budget) out[x] = x;
    int emitted = g.s_end;
    for (int cw = 0; cw < n_words; cw += kTailWords) {
        const int nw = min(kTailWords, n_words - cw);
        if (cw > 0) {
            __syncthreads();
            for (int x = tid; x < nw; x += kSelThreads) lmask[x] = mask[cw + x];
            __syncthreads();
        }
        if (all_ties) {
            for (int x = tid; x < nc; x += kSelThreads) {
                const uint2 kp = cand(x);
                const int w = (int)(kp.y >> 5) - cw;
                if (kp.x >= tau && w >= 0 && w < nw) atomicOr(&lmask[w], 1u << (kp.y & 31u));
            }
        } else {
            int rank = tie_base;
            for (int x = x0; x < x1; ++x) {
                const uint2 kp = cand(x);
                bool sel = kp.x > tau;
                if (kp.x == tau) {
                    sel = rank < need;
                    ++rank;
                }
                const int w = (int)(kp.y >> 5) - cw;
                if (sel && w >= 0 && w < nw) atomicOr(&lmask[w], 1u << (kp.y & 31u));
            }
        }
        __syncthreads();
        // thread t owns words [w0, w1); their set bits, four words at a time,
        // lowest first, without a branch per bit
        const int wpt = (nw + kSelThreads - 1) / kSelThreads;
        const int w0 = min(nw, tid * wpt), w1 = min(nw, w0 + wpt);
        int cnt = 0;
        for (int w = w0; w < w1; ++w) cnt += __builtin_popcount(lmask[w]);
        int chunk_total;
        int pos = emitted + block_scan(cnt, wave_tot, &chunk_total);
        for (int w = w0; w < w1; w += 4) {
            uint32_t m[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) m[i] = w + i < w1 ? lmask[w + i] : 0u;
            uint64_t lo = (uint64_t)m[0] | ((uint64_t)m[1] << 32);
            uint64_t hi = (uint64_t)m[2] | ((uint64_t)m[3] << 32);
            const int n4 = __builtin_popcountll(lo) + __builtin_popcountll(hi);
            const int base = (cw + w) * 32;
            for (int k = 0; k < n4; ++k) {
                const bool use_lo = lo != 0ull;
                const uint64_t cur = use_lo ? lo : hi;
                const int bit = __builtin_ctzll(cur) + (use_lo ? 0 : 64);
                const uint64_t nxt = cur & (cur - 1ull);
                lo = use_lo ? nxt : lo;
                hi = use_lo ? hi : nxt;
                if (pos < a.budget) out[pos] = base + bit;
                ++pos;
            }
        }
        emitted += chunk_total;
    }
    const int n_recent = g.T - g.r_start;
    for (int x = tid; x < n_recent; x += kSelThreads)
        if (emitted + x < a.budget) out[emitted + x] = g.r_start + x;
    if (c_head == 0 && tid == 0) a.n_idx[b] = emitted + n_recent;
}

__global__ __launch_bounds__(kSelThreads) void select_finish_kernel(SelectArgs a) {
    const int u = blockIdx.x;
    const Geom g = geom_of(a, u / a.n_kv_heads);
    if (g.simple) {
        emit_ranges(a, u, g);
        return;
    }
    finish_unit(a, u, g, a.thr[2 * u], (int)a.thr[2 * u + 1]);
}

// ---------------------------------------------------------------------------
// Kernel 2: threshold bin, bitmask words and candidate segments.
// grid = (parts, units).
// ---------------------------------------------------------------------------
template <int NR>
__global__ __launch_bounds__(kSelThreads) void select_mark_kernel(SelectArgs a) {
    const int p = blockIdx.x, u = blockIdx.y;
    const int b = u / a.n_kv_heads;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const Geom g = geom_of(a, b);
    if (p >= g.parts || g.simple) return;   // the finish kernel emits ranges then
    const float* S = a.scores + (size_t)u * a.max_ctx;
    const size_t up0 = (size_t)u * a.parts;   // first slot of this unit
    uint32_t* mask = a.mask + (size_t)u * (a.parts * (a.part / 32));

    __shared__ uint32_t red[256];
    __shared__ int wave_tot[kSelWaves];
    __shared__ int sh[4];

    // Issue the score loads first; the threshold search below hides them.
    uint32_t keys[4 * NR];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            keys[4 * r + e] = key_of(S, g, p * a.part + r * kRound + wave * 256 + e * 64 + lane);

    // ---- bin d1 and the count still needed from it ------------------------
    uint32_t d1 = 0u;
    int need = 0;
    {
        {   // coarse totals: thread t sums coarse bin t&63 over partitions q, q+4, ...
            const int cb = tid & 63, q = tid >> 6;
            uint32_t s = 0u;
            for (int p0 = q; p0 < g.parts; p0 += 4 * 8) {
                uint32_t v[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int pp = p0 + 4 * j;
                    v[j] = pp < g.parts ? a.coarse[(up0 + pp) * 64 + cb] : 0u;
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) s += v[j];
            }
            red[q * 64 + cb] = s;
        }
        __syncthreads();
        if (wave == 0) {
            const int cb = 63 - lane;   // descending
            const int tot = (int)(red[cb] + red[64 + cb] + red[128 + cb] + red[192 + cb]);
            const int incl = wave_incl_scan(tot);
            const int above = incl - tot;
            if (above < g.take && g.take <= incl) {
                sh[0] = cb;
                sh[1] = above;
            }
        }
        __syncthreads();
        const int dc = sh[0] & 63, above_c = sh[1];   // (mask: malformed scores stay in bounds)
        {   // fine totals of coarse bin dc: thread t sums fine bin t&31 over partitions q, q+8, ...
            const int fb = tid & 31, q = tid >> 5;
            uint32_t s = 0u;
            for (int p0 = q; p0 < g.parts; p0 += 8 * 4) {
                uint32_t v[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int pp = p0 + 8 * j;
                    v[j] = pp < g.parts ? a.hist[(up0 + pp) * kHistSlotWords + dc * 32 + fb] : 0u;
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) s += v[j];
            }
            red[q * 32 + fb] = s;
        }
        __syncthreads();
        if (wave == 0) {
            const int fb = 31 - (lane & 31);
            int tot = 0;
#pragma unroll
            for (int q = 0; q < 8; ++q) tot += (int)red[q * 32 + fb];
            tot = lane < 32 ? tot : 0;
            const int incl = wave_incl_scan(tot);
            const int above = above_c + incl - tot;
            if (lane < 32 && above < g.take && g.take <= above + tot) {
                sh[2] = dc * 32 + fb;
                sh[3] = g.take - above;
            }
        }
        __syncthreads();
        d1 = (uint32_t)sh[2];
        need = sh[3];
    }

    // ---- bitmask words and bin-d1 candidates of this partition -------------
    const uint64_t lt = (1ull << lane) - 1ull;
    uint2* seg = a.seg + (up0 + p) * a.part;
    int run = 0;   // candidates of this partition so far (uniform)
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
            const bool def = mid && dg > d1;
            const bool cand = mid && dg == d1;
            defb[e] = __ballot(def);
            candb[e] = __ballot(cand);
            n_w += __builtin_popcountll(candb[e]);
        }
        if (lane < 8) {
            const uint64_t m = lane < 2 ? defb[0] : lane < 4 ? defb[1] : lane < 6 ? defb[2] : defb[3];
            mask[base / 32 + lane] = (lane & 1) ? (uint32_t)(m >> 32) : (uint32_t)m;
        }
        {
            int round_total;
            int slot = run + block_scan(lane == 0 ? n_w : 0, wave_tot, &round_total);
            slot = __builtin_amdgcn_readlane(slot, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if ((candb[e] >> lane) & 1ull)
                    seg[slot + __builtin_popcountll(candb[e] & lt)] =
                        make_uint2(keys[4 * r + e], (uint32_t)(base + e * 64 + lane));
                slot += __builtin_popcountll(candb[e]);
            }
            run += round_total;
        }
    }
    if (tid == 0) {
        a.cnt[up0 + p] = (uint32_t)run;
        if (p == 0) {
            a.thr[2 * u] = d1;
            a.thr[2 * u + 1] = (uint32_t)need;
        }
    }
}

// ---------------------------------------------------------------------------
// One kernel for calls of at most kSelectFuseMaxGroups partition workgroups:
// the partitions of one unit are resident together (workgroups are
// dispatched in index order and a unit's partitions are consecutive, so when
// the lowest unfinished unit waits, every workgroup ahead of its partitions
// has finished) and run select_partition (select_common.h) on the scores they
// load.
// ---------------------------------------------------------------------------
template <int NR, bool kDraft>
__global__ __launch_bounds__(kSelThreads) void select_fused_kernel(SelectArgs a) {
    const int p = blockIdx.x, u = blockIdx.y;
    const int b = u / a.n_kv_heads;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const Geom g = geom_of(a, b);
    if (p >= g.parts) return;
    __shared__ SelLds L;

    if (g.simple) {
        if (!kDraft) {   // ranges only: no exchange
            if (p == 0) emit_ranges(a, u, g);
            return;
        }
        // every middle position or none: ranges, no list
        const uint64_t epv = scalar_here(a.epoch ? ld_dev64(a.epoch + u) : 0ull);
        if (epoch_is_dirty(epv)) {
            if (tid == 0) exchange_gave_up(a.xc, kStatusSelect, a.epoch ? a.epoch + u : nullptr);
            return;
        }
        const bool done = select_simple<kDraft>(a, g, p, u, L, exchange_tag(a.call_tag, epv));
        if (done && a.epoch && tid == 0) epoch_advance(a.epoch + u);
        return;
    }
    const float* S = a.scores + (size_t)u * a.max_ctx;

    uint32_t keys[4 * NR];
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            keys[4 * r + e] = key_of(S, g, p * a.part + r * kRound + wave * 256 + e * 64 + lane);
    // The unit's exchange epoch (exchange_tag), loaded with the scores so that
    // the wait for them covers its round trip (the tag is formed only after
    // that wait); partition 0 advances it at its end, when every partition has
    // published, and so has read it.
    const uint64_t ep = a.epoch ? ld_dev64(a.epoch + u) : 0ull;
    select_local_hist<NR>(keys, L);
    const uint64_t epv = scalar_here(ep);
    if (epoch_is_dirty(epv)) {   // an earlier captured call on this workspace gave up
        if (tid == 0) exchange_gave_up(a.xc, kStatusSelect, a.epoch ? a.epoch + u : nullptr);
        return;
    }
    const bool done = select_partition<NR, kDraft>(a, g, p, u, keys, L, exchange_tag(a.call_tag, epv));
    // every partition has published, so has read the epoch; advanced last,
    // after the kernel's final wait for loads
    if (done && a.epoch && tid == 0) epoch_advance(a.epoch + u);
}

// One kernel when the caller chose it (a.fused); otherwise histogram, mark and
// finish kernels.
template <int NR>
void launch_nr(const SelectArgs& a, int n_units, hipStream_t stream) {
    const dim3 grid(a.parts, n_units), block(kSelThreads);
    if (a.fused) {
        if constexpr (NR <= 4) {
            if (a.with_draft) {
                hipLaunchKernelGGL((select_fused_kernel<NR, true>), grid, block, 0, stream, a);
                return;
            }
        }
        hipLaunchKernelGGL((select_fused_kernel<NR, false>), grid, block, 0, stream, a);
    } else {
        hipLaunchKernelGGL(select_hist_kernel<NR>, grid, block, 0, stream, a);
        hipLaunchKernelGGL(select_mark_kernel<NR>, grid, block, 0, stream, a);
        hipLaunchKernelGGL(select_finish_kernel, dim3(n_units), block, 0, stream, a);
    }
}

}  // namespace

int select_part_len(int max_t) {
    int nr = 1;
    while (nr < kSelectMaxRounds && (long long)nr * kRound * kSelectTargetParts < max_t) nr <<= 1;
    return nr * kRound;
}

template <int NR>
int blocks_per_cu_nr() {
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, select_fused_kernel<NR, false>, kSelThreads, 0) !=
        hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return blocks;
}

int select_blocks_per_cu(int part) {
    switch (part / kRound) {
        case 1: return blocks_per_cu_nr<1>();
        case 2: return blocks_per_cu_nr<2>();
        case 4: return blocks_per_cu_nr<4>();
        default: return blocks_per_cu_nr<8>();
    }
}

hipError_t launch_select(const SelectArgs& a, int n_units, hipStream_t stream) {
    switch (a.part / kRound) {
        case 1: launch_nr<1>(a, n_units, stream); break;
        case 2: launch_nr<2>(a, n_units, stream); break;
        case 4: launch_nr<4>(a, n_units, stream); break;
        case 8: launch_nr<8>(a, n_units, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace ssl
