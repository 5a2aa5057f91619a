// select.hip -- Eq. 4 recallable index sets by radix select.
//
// One 1024-thread workgroup per (sequence, KV head).  Scores are non-negative
// fp32, so their bit patterns order like their values.  Wave w owns the
// contiguous positions [w*span, (w+1)*span) and lane l the positions
// w*span + l + 64j; for contexts up to 64K each lane keeps its scores in
// registers, so the data is read from memory once.
//
// The K_mid-th largest middle score tau is found exactly by an MSB-first
// radix select over the bit patterns in three passes (12 + 10 + 10 bits,
// histograms in LDS); the histograms also give `need`, how many middle
// entries equal to tau still fit.
//
// The index set is then emitted in ascending position order by an ordered
// stream compaction: pass A counts, per wave, the non-tie selections and the
// tau ties; a 16-entry scan gives each wave its output offset and its first
// tie rank; pass B writes.  Ties are taken lowest position first, so the set
// is unique.
#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kRegPerLane = 64;          // register-resident scores per lane (T <= 65536)
constexpr uint32_t kNone = 0xffffffffu;  // "not a middle position" marker

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

template <bool REG>
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

    const int span = ((T + kSelWaves - 1) / kSelWaves + kWave - 1) / kWave * kWave;
    const int lo = wave * span;
    const int hi = min(lo + span, T);
    const int nj = span / kWave;

    __shared__ uint32_t hist[2048];
    __shared__ uint32_t wave_tot[kSelWaves];
    __shared__ uint32_t sh_digit;
    __shared__ int32_t sh_above;
    __shared__ int32_t w_nontie[kSelWaves], w_ties[kSelWaves];

    // Key of the element at (wave, lane, j): its score bits if it is a middle
    // position, kNone otherwise (sink, recent, beyond T).
    uint32_t vals[REG ? kRegPerLane : 1];
    auto load_key = [&](int j) -> uint32_t {
        const int i = lo + kWave * j + lane;
        return (i < hi && i >= s_end && i < r_start) ? __builtin_bit_cast(uint32_t, S[i]) : kNone;
    };
    if (REG) {
#pragma unroll
        for (int j = 0; j < kRegPerLane; ++j) vals[j] = j < nj ? load_key(j) : kNone;
    }

    uint32_t tau = kNone;   // nothing from the middle span unless selection runs
    int need = 0;
    if (!all_mid && take > 0) {
        // Pass 1: bits 31..20 (the sign bit is 0: 11 significant bits).
        for (int x = tid; x < 2048; x += kSelThreads) hist[x] = 0u;
        __syncthreads();
        if (REG) {
#pragma unroll
            for (int j = 0; j < kRegPerLane; ++j)
                if (vals[j] != kNone) atomicAdd(&hist[(vals[j] >> 20) & 2047u], 1u);
        } else {
            for (int j = 0; j < nj; ++j) {
                const uint32_t k = load_key(j);
                if (k != kNone) atomicAdd(&hist[(k >> 20) & 2047u], 1u);
            }
        }
        __syncthreads();
        find_digit<2048>(hist, take, &sh_digit, &sh_above, wave_tot);
        uint32_t prefix = sh_digit << 20;
        int remaining = take - sh_above;
        __syncthreads();
        // Passes 2 and 3: bits 19..10, then 9..0, among keys matching the prefix.
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
            const int shift = pass == 0 ? 10 : 0;
            const uint32_t pmask = pass == 0 ? 0xfff00000u : 0xfffffc00u;
            hist[tid] = 0u;
            __syncthreads();
            if (REG) {
#pragma unroll
                for (int j = 0; j < kRegPerLane; ++j)
                    if (vals[j] != kNone && (vals[j] & pmask) == prefix)
                        atomicAdd(&hist[(vals[j] >> shift) & 1023u], 1u);
            } else {
                for (int j = 0; j < nj; ++j) {
                    const uint32_t k = load_key(j);
                    if (k != kNone && (k & pmask) == prefix)
                        atomicAdd(&hist[(k >> shift) & 1023u], 1u);
                }
            }
            __syncthreads();
            find_digit<1024>(hist, remaining, &sh_digit, &sh_above, wave_tot);
            prefix |= sh_digit << shift;
            remaining -= sh_above;
            __syncthreads();
        }
        tau = prefix;
        need = remaining;
    }

    // Ordered compaction.  Pass A: per-wave counts.
    int nontie = 0, ties = 0;
    auto classify = [&](int j, uint32_t k, bool& edge, bool& gt, bool& tie) {
        const int i = lo + kWave * j + lane;
        edge = i < hi && (i < s_end || i >= r_start);
        const bool mid = k != kNone;
        gt = mid && (all_mid || k > tau);
        tie = mid && !all_mid && k == tau;
    };
    if (REG) {
#pragma unroll
        for (int j = 0; j < kRegPerLane; ++j) {
            if (j < nj) {   // uniform across the block
                bool edge, gt, tie;
                classify(j, vals[j], edge, gt, tie);
                nontie += __builtin_popcountll(ballot(edge || gt));
                ties += __builtin_popcountll(ballot(tie));
            }
        }
    } else {
        for (int j = 0; j < nj; ++j) {
            bool edge, gt, tie;
            classify(j, load_key(j), edge, gt, tie);
            nontie += __builtin_popcountll(ballot(edge || gt));
            ties += __builtin_popcountll(ballot(tie));
        }
    }
    if (lane == 0) { w_nontie[wave] = nontie; w_ties[wave] = ties; }
    __syncthreads();
    int out_base = 0, tie_base = 0;
    for (int w = 0; w < wave; ++w) {
        out_base += w_nontie[w] + min(max(need - tie_base, 0), w_ties[w]);
        tie_base += w_ties[w];
    }
    // Pass B: write positions in order.
    int tie_run = 0, out_run = 0;
    auto emit = [&](int j, uint32_t k) {
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
    };
    if (REG) {
#pragma unroll
        for (int j = 0; j < kRegPerLane; ++j)
            if (j < nj) emit(j, vals[j]);
    } else {
        for (int j = 0; j < nj; ++j) emit(j, load_key(j));
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
    int max_t = 0;
    for (int b = 0; b < a.batch; ++b) max_t = max(max_t, a.ctx[b]);
    if (max_t <= kSelWaves * kWave * kRegPerLane)
        hipLaunchKernelGGL(select_kernel<true>, dim3(n_units), dim3(kSelThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(select_kernel<false>, dim3(n_units), dim3(kSelThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ssl
