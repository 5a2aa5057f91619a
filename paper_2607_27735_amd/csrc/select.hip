// select.hip -- Eq. 4 recallable index sets by radix select.
//
// One 1024-thread workgroup per (sequence, KV head).  Scores are non-negative
// fp32, so their bit patterns order like their values; the K_mid-th largest
// middle score is found exactly by four MSB-first 8-bit radix passes over the
// bit patterns (histograms in LDS, equal digits inside a wave aggregated with
// ballots before the LDS atomics).  Its value tau and the number `need` of
// entries equal to tau that still fit follow from the histograms.
//
// The index set is then emitted in ascending position order by a two-pass
// stream compaction: every wave owns a contiguous position range; pass A
// counts, per wave, the non-tie selections and the tau ties; a 16-entry scan
// gives each wave its output offset and its first tie rank; pass B writes.
// Ties are taken lowest position first, so the set is unique.
#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// Histogram add with the lanes of a wave that share a digit merged first: a
// few leader rounds take the common digits, the rest use plain LDS atomics.
__device__ __forceinline__ void wave_hist_add(uint32_t* hist, uint32_t digit, bool active) {
    uint64_t act = ballot(active);
#pragma unroll
    for (int round = 0; round < 4; ++round) {
        if (act == 0) break;
        const int leader = __builtin_ctzll(act);
        const uint32_t d0 = __shfl((int)digit, leader, kWave);
        const uint64_t same = ballot(active && digit == d0);
        if ((threadIdx.x & 63) == leader) atomicAdd(&hist[d0], (uint32_t)__builtin_popcountll(same));
        if (digit == d0) active = false;
        act &= ~same;
    }
    if (active) atomicAdd(&hist[digit], 1u);
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectArgs a) {
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

    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh_prefix;
    __shared__ int32_t sh_remaining;
    __shared__ int32_t w_nontie[kSelWaves], w_ties[kSelWaves];

    // Middle positions strictly above tau are taken, plus the first `need`
    // (in position order) equal to tau.  With no middle budget nothing is.
    uint32_t tau = 0xffffffffu;
    int need = 0;
    if (!all_mid && take > 0) {
        uint32_t prefix = 0u, pmask = 0u;
        int remaining = take;
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            if (tid < 256) hist[tid] = 0u;
            __syncthreads();
            for (int base = s_end; base < r_start; base += kSelThreads) {
                const int i = base + tid;
                const bool valid = i < r_start;
                const uint32_t key = valid ? __builtin_bit_cast(uint32_t, S[i]) : 0u;
                const bool active = valid && (key & pmask) == prefix;
                wave_hist_add(hist, (key >> shift) & 255u, active);
            }
            __syncthreads();
            if (wave == 0) {
                // Lane l holds digits 255-4l .. 252-4l (descending); scan the
                // lane sums to get the count strictly above each digit.
                uint32_t h[4], sum = 0u;
#pragma unroll
                for (int q = 0; q < 4; ++q) { h[q] = hist[255 - 4 * lane - q]; sum += h[q]; }
                uint32_t incl = sum;
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const uint32_t v = __shfl_up((int)incl, off, kWave);
                    if (lane >= off) incl += v;
                }
                uint32_t above = incl - sum;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if ((int)above < remaining && remaining <= (int)(above + h[q])) {
                        sh_prefix = prefix | ((uint32_t)(255 - 4 * lane - q) << shift);
                        sh_remaining = remaining - (int)above;
                    }
                    above += h[q];
                }
            }
            __syncthreads();
            prefix = sh_prefix;
            remaining = sh_remaining;
            pmask |= 255u << shift;
            __syncthreads();
        }
        tau = prefix;
        need = remaining;
    }

    // Ordered compaction.  Wave w owns positions [w*span, min((w+1)*span, T)).
    const int span = ((T + kSelWaves - 1) / kSelWaves + kWave - 1) / kWave * kWave;
    const int lo = wave * span;
    const int hi = min(lo + span, T);
    int nontie = 0, ties = 0;
    for (int base = lo; base < hi; base += kWave) {
        const int i = base + lane;
        const bool valid = i < hi;
        const bool edge = valid && (i < s_end || i >= r_start);
        const bool mid = valid && !edge;
        bool gt = mid, tie = false;
        if (!all_mid && mid) {
            const uint32_t key = __builtin_bit_cast(uint32_t, S[i]);
            gt = key > tau;
            tie = key == tau;
        }
        nontie += __builtin_popcountll(ballot(edge || gt));
        ties += __builtin_popcountll(ballot(tie));
    }
    if (lane == 0) { w_nontie[wave] = nontie; w_ties[wave] = ties; }
    __syncthreads();
    int out_base = 0, tie_base = 0;
    for (int w = 0; w < wave; ++w) {
        const int taken = min(max(need - tie_base, 0), w_ties[w]);
        out_base += w_nontie[w] + taken;
        tie_base += w_ties[w];
    }
    int tie_run = 0, out_run = 0;
    for (int base = lo; base < hi; base += kWave) {
        const int i = base + lane;
        const bool valid = i < hi;
        const bool edge = valid && (i < s_end || i >= r_start);
        const bool mid = valid && !edge;
        bool gt = mid, tie = false;
        if (!all_mid && mid) {
            const uint32_t key = __builtin_bit_cast(uint32_t, S[i]);
            gt = key > tau;
            tie = key == tau;
        }
        const uint64_t tmask = ballot(tie);
        const bool take_tie = tie && (tie_base + tie_run + (int)lanes_below(tmask)) < need;
        const bool sel = edge || gt || take_tie;
        const uint64_t smask = ballot(sel);
        const int pos = out_base + out_run + (int)lanes_below(smask);
        if (sel && pos < a.budget) out[pos] = i;
        tie_run += __builtin_popcountll(tmask);
        out_run += __builtin_popcountll(smask);
    }
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
    hipLaunchKernelGGL(select_kernel, dim3(n_units), dim3(kSelThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ssl
