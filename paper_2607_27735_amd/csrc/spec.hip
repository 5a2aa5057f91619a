// spec.hip -- speculative sampling: the verification rule that keeps the
// target model's output distribution (Sec. 1 and Sec. 2.1 rely on it).
//
// At temperature tau, p_j = softmax(target row j / tau) and q_j =
// softmax(drafter row j / tau).  Drafted token x_j passes when
// u_j q_j(x_j) < p_j(x_j); after the first failure (position m) the next
// token is drawn by inversion from max(0, p_m - q_m), after k passes from p_k.
// Five small launches, the kernel boundaries their only synchronisation:
//   stats:  per (row, chunk of 8192 logits) the max of x / tau and the sum of
//           e^(x / tau - max), for the target rows 0..k and drafter rows 0..k-1;
//   rows:   per row, the chunks merged in a fixed order (one wave);
//   decide: per sequence, lane j tests drafted token j; m = the first failure;
//   mass:   per (sequence, chunk) the mass of the distribution drawn from
//           (residual and plain target), summed in a fixed order;
//   sample: per sequence, the chunk where the cumulative mass passes
//           u * total, then a scan of that chunk in index order.
// Everything is fp32.  The chunk masses and the in-chunk scan add in
// different orders; when rounding leaves the scan short of the target, the
// chunk's last element with mass is drawn.
#include "device_common.h"
#include "launch.h"
#include "logit_common.h"

namespace ssl {
namespace {

using lc::kLog2e;
using lc::kThreads;
constexpr int kWaves = kThreads / kWave;

// Row r of sequence b in the row tables: target rows 0..max_k, then drafter
// rows 0..max_k-1.
__device__ __forceinline__ const char* row_base(const SpecArgs& a, int b, int r, bool f32) {
    const size_t esz = f32 ? 4 : 2;
    if (r <= a.max_k)
        return static_cast<const char*>(a.tlogits) + ((size_t)b * (a.max_k + 1) + r) * a.row_stride * esz;
    return static_cast<const char*>(a.dlogits) + ((size_t)b * a.max_k + (r - a.max_k - 1)) * a.row_stride * esz;
}

__device__ __forceinline__ bool row_needed(const SpecArgs& a, int b, int r) {
    const int k = a.k_len[b];
    return r <= a.max_k ? r <= k : (r - a.max_k - 1) < k;
}

__device__ __forceinline__ float2 ms_merge(float2 p, float2 q) {
    const float m = fmaxf(p.x, q.x);
    if (m == -INFINITY) return make_float2(-INFINITY, 0.f);
    return make_float2(m, p.y * fast_exp2((p.x - m) * kLog2e) + q.y * fast_exp2((q.x - m) * kLog2e));
}

__device__ __forceinline__ float2 wave_ms(float2 v) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1)
        v = ms_merge(v, make_float2(__shfl_xor(v.x, o, kWave), __shfl_xor(v.y, o, kWave)));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// v of the lane the DPP control selects (0 where there is none).
template <int kCtrl, int kRows>
__device__ __forceinline__ float dpp_f(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), kCtrl,
                                                                 kRows, 0xf, false));
}

// Inclusive scan of one float per lane over the wave (fixed order).
__device__ __forceinline__ float wave_incl_scan_f(float x) {
    x += dpp_f<0x111, 0xf>(x);   // row_shr:1
    x += dpp_f<0x112, 0xf>(x);   // row_shr:2
    x += dpp_f<0x114, 0xf>(x);   // row_shr:4
    x += dpp_f<0x118, 0xf>(x);   // row_shr:8
    x += dpp_f<0x142, 0xa>(x);   // row_bcast:15 -> rows 1, 3
    x += dpp_f<0x143, 0xc>(x);   // row_bcast:31 -> rows 2, 3
    return x;
}

// ---- stats: grid (n_chunks, batch * (2 max_k + 1)) ----------------------------
template <bool kF32>
__global__ __launch_bounds__(kThreads) void spec_stats_kernel(SpecArgs a) {
    const int chunk = blockIdx.x, rows = 2 * a.max_k + 1;
    const int b = blockIdx.y / rows, r = blockIdx.y - b * rows;
    if (!row_needed(a, b, r)) return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float x[32];
    lc::load_chunk<kF32>(row_base(a, b, r, kF32), a.vocab, chunk, tid, x);
    float m = -INFINITY;
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        x[q] *= a.inv_tau;
        m = fmaxf(m, x[q]);
    }
    float s = 0.f;
    if (m != -INFINITY) {
#pragma unroll
        for (int q = 0; q < 32; ++q) s += fast_exp2((x[q] - m) * kLog2e);
    }
    __shared__ float2 wv[kWaves];
    const float2 v = wave_ms(make_float2(m, s));
    if (lane == 0) wv[wave] = v;
    __syncthreads();
    if (tid == 0) {
        float2 t = wv[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) t = ms_merge(t, wv[w]);
        a.chunk_ms[((size_t)b * rows + r) * a.n_chunks + chunk] = t;
    }
}

// ---- rows: one wave per (sequence, row) -------------------------------------------
__global__ __launch_bounds__(kWave) void spec_rows_kernel(SpecArgs a) {
    const int rows = 2 * a.max_k + 1;
    const int b = blockIdx.x / rows, r = blockIdx.x - b * rows;
    if (!row_needed(a, b, r)) return;
    const int lane = threadIdx.x;
    const size_t base = ((size_t)b * rows + r) * a.n_chunks;
    const float2 v = lane < a.n_chunks ? a.chunk_ms[base + lane] : make_float2(-INFINITY, 0.f);
    const float2 t = wave_ms(v);
    if (lane == 0) a.row_ms[(size_t)b * rows + r] = t;
}

// p(x) for a row with merged (max, sum) ms at scaled logit y = x / tau.
__device__ __forceinline__ float prob(float y, float2 ms) {
    return fast_exp2((y - ms.x) * kLog2e) / ms.y;
}

template <bool kF32>
__device__ __forceinline__ float logit_at(const char* row, int i) {
    if (kF32) return reinterpret_cast<const float*>(row)[i];
    return bf16_lo((uint32_t)reinterpret_cast<const uint16_t*>(row)[i]);
}

// ---- decide: one wave per sequence ---------------------------------------------------
template <bool kF32>
__global__ __launch_bounds__(kWave) void spec_decide_kernel(SpecArgs a) {
    const int b = blockIdx.x, lane = threadIdx.x;
    const int k = a.k_len[b], rows = 2 * a.max_k + 1;
    bool pass = true;
    if (lane < k) {
        const int x = min(max(a.draft[(size_t)b * a.max_k + lane], 0), a.vocab - 1);
        const float2 mt = a.row_ms[(size_t)b * rows + lane];
        const float2 md = a.row_ms[(size_t)b * rows + a.max_k + 1 + lane];
        const float p = prob(logit_at<kF32>(row_base(a, b, lane, kF32), x) * a.inv_tau, mt);
        const float q = prob(logit_at<kF32>(row_base(a, b, a.max_k + 1 + lane, kF32), x) * a.inv_tau, md);
        pass = a.u_acc[(size_t)b * a.max_k + lane] * q < p;
    }
    const uint64_t fail = __ballot(!pass);
    const int m = fail ? __builtin_ctzll(fail) : k;
    if (lane == 0) {
        a.n_accepted[b] = m;
        a.pick[b] = m;
    }
}

// The weights of thread tid's 32 elements of chunk `chunk`: with a residual
// (m < k), max(0, p_m - q_m) in w and p_m in pw; else p_k in both.
template <bool kF32>
__device__ __forceinline__ void chunk_weights(const SpecArgs& a, int b, int m, int chunk, int tid,
                                              float2 mt, float2 md, float (&w)[32], float (&pw)[32]) {
    const bool resid = m < a.k_len[b];
    float xt[32];
    lc::load_chunk<kF32>(row_base(a, b, m, kF32), a.vocab, chunk, tid, xt);
#pragma unroll
    for (int q = 0; q < 32; ++q) pw[q] = xt[q] == -INFINITY ? 0.f : prob(xt[q] * a.inv_tau, mt);
    if (resid) {
        float xd[32];
        lc::load_chunk<kF32>(row_base(a, b, a.max_k + 1 + m, kF32), a.vocab, chunk, tid, xd);
#pragma unroll
        for (int q = 0; q < 32; ++q)
            w[q] = fmaxf(pw[q] - (xd[q] == -INFINITY ? 0.f : prob(xd[q] * a.inv_tau, md)), 0.f);
    } else {
#pragma unroll
        for (int q = 0; q < 32; ++q) w[q] = pw[q];
    }
}

// ---- mass: grid (n_chunks, batch) -----------------------------------------------------
template <bool kF32>
__global__ __launch_bounds__(kThreads) void spec_mass_kernel(SpecArgs a) {
    const int chunk = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, rows = 2 * a.max_k + 1;
    const int m = a.pick[b];
    const float2 mt = a.row_ms[(size_t)b * rows + m];
    const float2 md = a.row_ms[(size_t)b * rows + a.max_k + 1 + min(m, a.max_k - 1)];
    float w[32], pw[32];
    chunk_weights<kF32>(a, b, m, chunk, tid, mt, md, w, pw);
    float s = 0.f, sp = 0.f;
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        s += w[q];
        sp += pw[q];
    }
    s = wave_sum(s);
    sp = wave_sum(sp);
    __shared__ float2 wv[kWaves];
    if (lane == 0) wv[wave] = make_float2(s, sp);
    __syncthreads();
    if (tid == 0) {
        float2 t = wv[0];
#pragma unroll
        for (int v = 1; v < kWaves; ++v) {
            t.x += wv[v].x;
            t.y += wv[v].y;
        }
        a.mass[(size_t)b * a.n_chunks + chunk] = t;
    }
}

// ---- sample: one workgroup per sequence -------------------------------------------------
template <bool kF32>
__global__ __launch_bounds__(kThreads) void spec_sample_kernel(SpecArgs a) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, rows = 2 * a.max_k + 1;
    const int m = a.pick[b];
    const float2 mt = a.row_ms[(size_t)b * rows + m];
    const float2 md = a.row_ms[(size_t)b * rows + a.max_k + 1 + min(m, a.max_k - 1)];
    __shared__ int sh_chunk, sh_use_p, sh_found, sh_last;
    __shared__ float sh_target;
    __shared__ float wtot[kWaves];
    if (tid == 0) {
        // the residual when it has mass, else the plain target row; the chunk
        // where the cumulative mass (chunk order) passes u * total
        float tot = 0.f, totp = 0.f;
        for (int c = 0; c < a.n_chunks; ++c) {
            const float2 v = a.mass[(size_t)b * a.n_chunks + c];
            tot += v.x;
            totp += v.y;
        }
        const bool use_p = !(tot > 0.f);
        const float total = use_p ? totp : tot;
        const float target = a.u_smp[b] * total;
        float run = 0.f;
        int cstar = -1, last = 0;
        for (int c = 0; c < a.n_chunks; ++c) {
            const float2 v = a.mass[(size_t)b * a.n_chunks + c];
            const float mc = use_p ? v.y : v.x;
            if (mc > 0.f) last = c;
            if (cstar < 0 && run + mc > target) cstar = c;
            if (cstar < 0) run += mc;
        }
        if (cstar < 0) {   // rounding left the cumulative mass short: the last chunk with mass
            cstar = last;
            run = 0.f;
            for (int c = 0; c < last; ++c) {
                const float2 v = a.mass[(size_t)b * a.n_chunks + c];
                run += use_p ? v.y : v.x;
            }
        }
        sh_chunk = cstar;
        sh_use_p = use_p ? 1 : 0;
        sh_target = target - run;
        sh_found = 0x7fffffff;
        sh_last = -1;
    }
    __syncthreads();
    const int chunk = sh_chunk;
    const float target = sh_target;
    float w[32], pw[32];
    chunk_weights<kF32>(a, b, m, chunk, tid, mt, md, w, pw);
    if (sh_use_p) {
#pragma unroll
        for (int q = 0; q < 32; ++q) w[q] = pw[q];
    }
    // scan in index order: load j of every thread, thread by thread, then its
    // elements in order
    constexpr int per = lc::per_load<kF32>();
    constexpr int nl = lc::loads<kF32>();
    float carry = 0.f;
    int last = -1;
#pragma unroll
    for (int j = 0; j < nl; ++j) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < per; ++e) {
            s += w[j * per + e];
            if (w[j * per + e] > 0.f) last = lc::elem<kF32>(chunk, j * per + e, tid);
        }
        const float incl = wave_incl_scan_f(s);
        if (lane == kWave - 1) wtot[wave] = incl;
        __syncthreads();
        float before = carry, all = carry;
#pragma unroll
        for (int v = 0; v < kWaves; ++v) {
            before += v < wave ? wtot[v] : 0.f;
            all += wtot[v];
        }
        float run = before + incl - s;
        int cand = 0x7fffffff;
#pragma unroll
        for (int e = 0; e < per; ++e) {
            run += w[j * per + e];
            if (cand == 0x7fffffff && run > target) cand = lc::elem<kF32>(chunk, j * per + e, tid);
        }
        if (cand != 0x7fffffff) atomicMin(&sh_found, cand);
        __syncthreads();
        carry = all;
        if (sh_found != 0x7fffffff) break;   // uniform: read after the barrier
    }
    if (last >= 0) atomicMax(&sh_last, last);
    __syncthreads();
    if (tid == 0) a.next_token[b] = sh_found != 0x7fffffff ? sh_found : max(sh_last, 0);
}

}  // namespace

hipError_t launch_spec_accept(const SpecArgs& a, int batch, bool f32, hipStream_t stream) {
    const int rows = 2 * a.max_k + 1;
    const dim3 block(kThreads);
    if (f32)
        hipLaunchKernelGGL(spec_stats_kernel<true>, dim3(a.n_chunks, batch * rows), block, 0, stream, a);
    else
        hipLaunchKernelGGL(spec_stats_kernel<false>, dim3(a.n_chunks, batch * rows), block, 0, stream, a);
    hipLaunchKernelGGL(spec_rows_kernel, dim3(batch * rows), dim3(kWave), 0, stream, a);
    if (f32) {
        hipLaunchKernelGGL(spec_decide_kernel<true>, dim3(batch), dim3(kWave), 0, stream, a);
        hipLaunchKernelGGL(spec_mass_kernel<true>, dim3(a.n_chunks, batch), block, 0, stream, a);
        hipLaunchKernelGGL(spec_sample_kernel<true>, dim3(batch), block, 0, stream, a);
    } else {
        hipLaunchKernelGGL(spec_decide_kernel<false>, dim3(batch), dim3(kWave), 0, stream, a);
        hipLaunchKernelGGL(spec_mass_kernel<false>, dim3(a.n_chunks, batch), block, 0, stream, a);
        hipLaunchKernelGGL(spec_sample_kernel<false>, dim3(batch), block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace ssl
