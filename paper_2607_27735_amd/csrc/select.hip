// select.hip -- Eq. 4 recallable index sets by radix select.
//
// One 1024-thread workgroup per (sequence, KV head).  Scores are non-negative
// fp32, so their bit patterns order like their values.  Wave w owns the
// contiguous positions [w*span, (w+1)*span) and lane l the positions
// w*span + l + 64j; for contexts up to 64K each lane keeps its scores in
// registers, so the data is read from memory once.
//
// 1. Pass 1 histograms the top 12 bits of the middle scores (LDS) and finds
//    the bin d1 holding the K_mid-th largest score.
// 2. One sweep over the scores marks, in an LDS bitmask of positions, the
//    sink, the recent span and every middle position whose top bits exceed
//    d1 (a 64-lane ballot is exactly two bitmask words), and appends the
//    positions inside bin d1 to an LDS candidate list.
// 3. Passes 2 and 3 (10 + 10 bits) run over the candidates only and give the
//    exact threshold tau and `need`, the number of entries equal to tau that
//    still fit; candidates above tau are marked, and ties are marked lowest
//    position first, so the set is unique.
// 4. The set is emitted in ascending order from the bitmask with one block
//    scan of per-thread popcounts.
//
// If bin d1 holds more candidates than the LDS list (massive ties), or the
// context exceeds the bitmask, the same three radix passes run over all
// middle scores and the set is emitted by an ordered two-pass ballot
// compaction instead.
#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kRegPerLane = 64;           // register-resident scores per lane (T <= 65536)
constexpr int kCandCap = 4096;            // LDS candidate list
constexpr int kSegCap = kCandCap / kSelWaves;   // per-wave segment of the list
constexpr int kMaskWords = 8192;          // LDS position bitmask: T <= 262144
constexpr uint32_t kNone = 0xffffffffu;   // "not a middle position" marker

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// Block-wide search of a histogram read from its top bin down: finds the bin
// where the running count from the top first reaches `remaining` and the count
// strictly above it, and publishes both through LDS.
template <int NBINS>
__device__ __forceinline__ void find_digit(const uint32_t* hist, int remaining, uint32_t* sh_digit,
                                           int32_t* sh_above, uint32_t* wave_tot) {
    constexpr int PER = NBINS >= kSelThreads ? NBINS / kSelThreads : 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Thread t covers bins NBINS-1-PER*t .. NBINS-PER*(t+1) (descending).
    uint32_t h[PER];
    uint32_t sum = 0u;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int bin = NBINS - 1 - PER * tid - q;
        h[q] = bin >= 0 ? hist[bin] : 0u;
        sum += h[q];
    }
    uint32_t incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up((int)incl, off, kWave);
        if (lane >= off) incl += v;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    uint32_t before = 0u;
    for (int w = 0; w < wave; ++w) before += wave_tot[w];
    uint32_t above = before + incl - sum;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const int bin = NBINS - 1 - PER * tid - q;
        if (bin >= 0 && (int)above < remaining && remaining <= (int)(above + h[q])) {
            *sh_digit = (uint32_t)bin;
            *sh_above = (int32_t)above;
        }
        above += h[q];
    }
    __syncthreads();
}

// Exclusive prefix sum of one value per thread over the block; *total gets
// the sum.  Uses wave_tot as scratch.
__device__ __forceinline__ int block_exclusive_scan(int v, uint32_t* wave_tot, int* total) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int u = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += u;
    }
    __syncthreads();
    if (lane == 63) wave_tot[wave] = (uint32_t)incl;
    __syncthreads();
    int before = 0, all = 0;
    for (int w = 0; w < kSelWaves; ++w) {
        const int t = (int)wave_tot[w];
        if (w < wave) before += t;
        all += t;
    }
    *total = all;
    return before + incl - v;
}

// NJ > 0: every lane keeps exactly NJ scores in registers (T <= 1024 * NJ);
// NJ == 0: scores are re-read from memory in each sweep.
template <int NJ>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectArgs a) {
    constexpr bool REG = NJ > 0;
    const int unit = blockIdx.x;
    const int b = unit / a.n_kv_heads;
    const int c = unit - b * a.n_kv_heads;
    const int T = a.ctx[b];
    const float* S = a.scores + (size_t)unit * a.max_ctx;
    int32_t* out = a.idx + (size_t)unit * a.budget;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    const int s_end = min(a.k_sink, T);
    const int r_start = max(T - a.k_recent, s_end);
    const int n_mid = r_start - s_end;
    const int k_mid = a.budget - a.k_sink - a.k_recent;
    const int take = min(k_mid, n_mid);
    const bool all_mid = take == n_mid;

    const int span = REG ? NJ * kWave
                         : ((T + kSelWaves - 1) / kSelWaves + kWave - 1) / kWave * kWave;
    const int lo = wave * span;
    const int hi = min(lo + span, T);
    const int nj = span / kWave;

    __shared__ uint32_t hist[2048];
    __shared__ uint32_t mask[kMaskWords];
    __shared__ uint32_t cand_key[kCandCap];
    __shared__ int32_t cand_pos[kCandCap];
    __shared__ uint32_t wave_tot[kSelWaves];
    __shared__ uint32_t sh_digit;
    __shared__ int32_t sh_above;
    __shared__ int32_t seg_count[kSelWaves];
    __shared__ int32_t sh_overflow;
    __shared__ int32_t w_nontie[kSelWaves], w_ties[kSelWaves];

    // Key of the element at (wave, lane, j): its score bits if it is a middle
    // position, kNone otherwise (sink, recent, beyond T).
    // The load itself is unconditional (clamped to a valid position) so that
    // all of a lane's loads issue back to back.
    uint32_t vals[REG ? NJ : 1];
    auto load_key = [&](int j) -> uint32_t {
        const int i = lo + kWave * j + lane;
        const uint32_t v = __builtin_bit_cast(uint32_t, S[min(i, T - 1)]);
        return (i < hi && i >= s_end && i < r_start) ? v : kNone;
    };
    if (REG) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) vals[j] = load_key(j);
    }
    // Applies f(j, key) to every element of this lane in j order.
    auto for_each = [&](auto&& f) {
        if (REG) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) f(j, vals[j]);
        } else {
            for (int j = 0; j < nj; ++j) f(j, load_key(j));
        }
    };

    const bool use_mask = T <= kMaskWords * 32;
    uint32_t tau = kNone;   // nothing from the middle span unless selection runs
    int need = 0;
    uint32_t d1 = 0u;
    const bool simple = all_mid || take == 0;   // no radix select needed
    bool fast = use_mask;                       // candidate list + bitmask path

    if (!simple) {
        // Pass 1: bits 31..20 (the sign bit is 0: 11 significant bits).
        for (int x = tid; x < 2048; x += kSelThreads) hist[x] = 0u;
        __syncthreads();
        for_each([&](int, uint32_t k) {
            atomicAdd(&hist[(k >> 20) & 2047u], k != kNone ? 1u : 0u);
        });
        __syncthreads();
        find_digit<2048>(hist, take, &sh_digit, &sh_above, wave_tot);
        d1 = sh_digit;
        need = take - sh_above;               // entries still needed from bin d1
        fast = fast && hist[d1] <= (uint32_t)kCandCap;
        __syncthreads();
    }

    if (use_mask && (fast || simple)) {
        // ---- bitmask path -------------------------------------------------
        // sink, recent, and middle positions above bin d1 (or every middle
        // position when all fit); 64 consecutive positions are two words.
        // Candidates (bin d1) go to this wave's segment of the list.
        int run = 0;
        for_each([&](int j, uint32_t k) {
            const int i = lo + kWave * j + lane;
            const bool valid = i < hi;
            const bool edge = valid && (i < s_end || i >= r_start);
            const bool mid = k != kNone;
            const uint32_t dg = (k >> 20) & 2047u;
            const bool def = edge || (mid && (simple ? all_mid : dg > d1));
            const bool cand = !simple && mid && dg == d1;
            const uint64_t m = ballot(def);
            const int w0 = (lo + kWave * j) >> 5;
            if (lane < 2 && w0 + lane < kMaskWords)
                mask[w0 + lane] = lane == 0 ? (uint32_t)m : (uint32_t)(m >> 32);
            const uint64_t cm = ballot(cand);
            const int slot = run + (int)lanes_below(cm);
            if (cand && slot < kSegCap) {
                cand_key[wave * kSegCap + slot] = k;
                cand_pos[wave * kSegCap + slot] = i;
            }
            run += __builtin_popcountll(cm);
        });
        if (tid == 0) sh_overflow = 0;
        __syncthreads();
        if (lane == 0) {
            seg_count[wave] = min(run, kSegCap);
            if (run > kSegCap) sh_overflow = 1;
        }
        __syncthreads();
        fast = !simple && !sh_overflow;
    }
    if (use_mask && (fast || simple)) {
        if (!simple) {
            // candidate x lives at segment x / kSegCap, offset x % kSegCap
            auto cand_ok = [&](int x) { return (x % kSegCap) < seg_count[x / kSegCap]; };
            const int nc = kCandCap;
            // passes 2 and 3 over the candidates (all share the top 12 bits)
            uint32_t prefix = d1 << 20;
#pragma unroll
            for (int pass = 0; pass < 2; ++pass) {
                const int shift = pass == 0 ? 10 : 0;
                const uint32_t pmask = pass == 0 ? 0xfff00000u : 0xfffffc00u;
                hist[tid] = 0u;
                __syncthreads();
                for (int x = tid; x < nc; x += kSelThreads) {
                    const uint32_t k = cand_key[x];
                    if (cand_ok(x) && (k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 1023u], 1u);
                }
                __syncthreads();
                find_digit<1024>(hist, need, &sh_digit, &sh_above, wave_tot);
                prefix |= sh_digit << shift;
                need -= sh_above;
                __syncthreads();
            }
            tau = prefix;
            const int n_ties = (int)hist[tau & 1023u];
            __syncthreads();
            // mark candidates above tau, and the `need` lowest-position ties
            for (int x = tid; x < nc; x += kSelThreads) {
                if (!cand_ok(x)) continue;
                const uint32_t k = cand_key[x];
                bool sel = k > tau;
                if (k == tau) {
                    if (need >= n_ties) {
                        sel = true;
                    } else {
                        const int p = cand_pos[x];
                        int rank = 0;
                        for (int y = 0; y < nc; ++y)
                            rank += (cand_ok(y) && cand_key[y] == tau && cand_pos[y] < p);
                        sel = rank < need;
                    }
                }
                if (sel) {
                    const int p = cand_pos[x];
                    atomicOr(&mask[p >> 5], 1u << (p & 31));
                }
            }
            __syncthreads();
        }
        // ---- ordered emission from the bitmask ------------------------------
        const int n_words = (T + 31) >> 5;
        const int wpt = (n_words + kSelThreads - 1) / kSelThreads;
        const int w_lo = min(tid * wpt, n_words), w_hi = min(w_lo + wpt, n_words);
        int cnt = 0;
        for (int w = w_lo; w < w_hi; ++w) cnt += __builtin_popcount(mask[w]);
        int total = 0;
        int pos = block_exclusive_scan(cnt, wave_tot, &total);
        for (int w = w_lo; w < w_hi; ++w) {
            uint32_t m = mask[w];
            while (m) {
                const int bit = __builtin_ctz(m);
                m &= m - 1u;
                if (pos < a.budget) out[pos] = w * 32 + bit;
                ++pos;
            }
        }
        if (c == 0 && tid == 0) a.n_idx[b] = total;
        return;
    }

    // ---- general path: radix over all middle scores, ordered compaction ----
    if (!simple) {
        uint32_t prefix = d1 << 20;
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
            const int shift = pass == 0 ? 10 : 0;
            const uint32_t pmask = pass == 0 ? 0xfff00000u : 0xfffffc00u;
            hist[tid] = 0u;
            __syncthreads();
            for_each([&](int, uint32_t k) {
                if (k != kNone && (k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 1023u], 1u);
            });
            __syncthreads();
            find_digit<1024>(hist, need, &sh_digit, &sh_above, wave_tot);
            prefix |= sh_digit << shift;
            need -= sh_above;
            __syncthreads();
        }
        tau = prefix;
    }
    auto classify = [&](int j, uint32_t k, bool& edge, bool& gt, bool& tie) {
        const int i = lo + kWave * j + lane;
        edge = i < hi && (i < s_end || i >= r_start);
        const bool mid = k != kNone;
        gt = mid && (all_mid || (take > 0 && k > tau));
        tie = mid && !all_mid && take > 0 && k == tau;
    };
    int nontie = 0, ties = 0;
    for_each([&](int j, uint32_t k) {
        bool edge, gt, tie;
        classify(j, k, edge, gt, tie);
        nontie += __builtin_popcountll(ballot(edge || gt));
        ties += __builtin_popcountll(ballot(tie));
    });
    if (lane == 0) { w_nontie[wave] = nontie; w_ties[wave] = ties; }
    __syncthreads();
    int out_base = 0, tie_base = 0;
    for (int w = 0; w < wave; ++w) {
        out_base += w_nontie[w] + min(max(need - tie_base, 0), w_ties[w]);
        tie_base += w_ties[w];
    }
    int tie_run = 0, out_run = 0;
    for_each([&](int j, uint32_t k) {
        bool edge, gt, tie;
        classify(j, k, edge, gt, tie);
        const uint64_t tmask = ballot(tie);
        const bool take_tie = tie && (tie_base + tie_run + (int)lanes_below(tmask)) < need;
        const bool sel = edge || gt || take_tie;
        const uint64_t smask = ballot(sel);
        const int pos = out_base + out_run + (int)lanes_below(smask);
        if (sel && pos < a.budget) out[pos] = lo + kWave * j + lane;
        tie_run += __builtin_popcountll(tmask);
        out_run += __builtin_popcountll(smask);
    });
    if (c == 0 && tid == 0) {
        int total = 0, tb = 0;
        for (int w = 0; w < kSelWaves; ++w) {
            total += w_nontie[w] + min(max(need - tb, 0), w_ties[w]);
            tb += w_ties[w];
        }
        a.n_idx[b] = total;
    }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, int n_units, hipStream_t stream) {
    int max_t = 0;
    for (int b = 0; b < a.batch; ++b) max_t = max(max_t, a.ctx[b]);
    const dim3 grid(n_units), block(kSelThreads);
    if (max_t <= kSelThreads * 16)
        hipLaunchKernelGGL(select_kernel<16>, grid, block, 0, stream, a);
    else if (max_t <= kSelThreads * 32)
        hipLaunchKernelGGL(select_kernel<32>, grid, block, 0, stream, a);
    else if (max_t <= kSelThreads * kRegPerLane)
        hipLaunchKernelGGL(select_kernel<kRegPerLane>, grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL(select_kernel<0>, grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace ssl
