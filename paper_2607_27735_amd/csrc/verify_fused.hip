// verify_fused.hip -- single-sweep verify attention with fused Eq. 3 scores.
//
// The Eq. 3 score of a key needs the final normalizer of every verify row,
// which no split of the context knows while it streams.  When every work item
// of the call fits on the GPU at once, one sweep suffices:
//
//   1. each workgroup streams its chunk of K and V once, runs an online
//      softmax per verify row (P.V on the MFMA, as in the two-sweep kernel)
//      and keeps the scaled logits of its chunk in LDS;
//   2. it publishes its partial output and (running max, sum) per row, then
//      waits at a per-(sequence, KV head) arrival counter until every chunk of
//      that head has published (agent-scope release/acquire);
//   3. from the merged (max, sum) of all chunks it forms the exact
//      probabilities of its own keys from the LDS logits and writes their
//      scores, and it combines one share of the head's output rows.
//
// The launch is cooperative, so all workgroups are co-resident and the wait
// always ends; it is additionally bounded, so a broken invariant cannot hang
// the GPU (the results would then be wrong, never a fault).
#include "verify_common.h"

namespace ssl {
namespace {

using namespace vc;

constexpr int kStashPad = 4;          // floats of padding per stashed row
constexpr int kSpinLimit = 1 << 22;   // bounded wait (far above any real wait)
constexpr int kCombGroups = kThreads / 32;

template <int NRT>
constexpr int static_lds_bytes() {
    return NRT * 16 * kHeadDim * 4          // red
           + kWaves * NRT * 16 * 8          // wml
           + kRowCap * 8                    // row_ml
           + kRowCap * 4                    // row_lse
           + kWaves * kRowCap * 8           // lse_part
           + kCombGroups * 32 * 16          // comb
           + 64;
}

__device__ __forceinline__ float safe_max(float m) { return m == -INFINITY ? 0.f : m; }

// One 32-key tile: logits to the LDS stash, online softmax, P.V.
template <int NRT>
__device__ __forceinline__ void fused_tile(const VerifyArgs& a, const Rows<NRT>& r,
                                           const KVTile& tl, int key0, int kl0, float* stash,
                                           int stride, int m16, int G, float (&M)[NRT],
                                           float (&L)[NRT], f32x4 (&oacc)[8][NRT]) {
    f32x4 acc[2][NRT];
    qk_tile<NRT>(tl.k, r, acc);
    float p[2][NRT][4];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        float y[8];
        float mt = -INFINITY;
        float* srow = stash + (rt * 16 + m16) * stride + kl0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int t = e >> 2, i = e & 3;
            const int key = key0 + 16 * t + G + 4 * i;
            y[e] = key <= r.plim[rt] ? acc[t][rt][i] * a.scale_log2 : -INFINITY;
            srow[16 * t + G + 4 * i] = y[e];
            mt = fmaxf(mt, y[e]);
        }
        mt = fmaxf(mt, shfl_xor_f(mt, 16));
        mt = fmaxf(mt, shfl_xor_f(mt, 32));
        const float Mn = safe_max(fmaxf(M[rt], mt));
        const float alpha = fast_exp2(M[rt] - Mn);
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            p[e >> 2][rt][e & 3] = fast_exp2(y[e] - Mn);
            sum += p[e >> 2][rt][e & 3];
        }
        L[rt] = L[rt] * alpha + sum;
        M[rt] = fmaxf(M[rt], mt);
#pragma unroll
        for (int jd = 0; jd < 8; ++jd) oacc[jd][rt] *= alpha;
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

template <int NRT>
__global__ __launch_bounds__(kThreads) void verify_fused_kernel(FusedArgs fa) {
    const VerifyArgs& a = fa.v;
    const FusedTable& ft = fa.ft;
    extern __shared__ float stash[];            // [NRT*16][chunk + pad]
    __shared__ f32x4 red[NRT * 16][kHeadDim / 4];
    __shared__ float2 wml[kWaves][NRT * 16];
    __shared__ float2 row_ml[kRowCap];
    __shared__ float row_lse[kRowCap];
    __shared__ float2 lse_part[kWaves][kRowCap];
    __shared__ f32x4 comb[kCombGroups][32];

    const int slot = blockIdx.x;
    int u = 0;
    while (u + 1 < ft.n_units && slot >= ft.slot_start[u + 1]) ++u;
    const int unit = ft.unit[u];
    const int b = unit / a.n_kv_heads, c = unit - b * a.n_kv_heads;
    const int slot0 = ft.slot_start[u];
    const int nchunk = ft.slot_start[u + 1] - slot0;
    const int s = slot - slot0;
    const int T = a.seq.ctx[b], nq = a.seq.qlen[b];
    const int R = nq * a.group;
    const int chunk = ft.chunk;
    const int key_begin = s * chunk, key_end = min(key_begin + chunk, T);
    const int stride = chunk + kStashPad;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m16 = lane & 15, G = lane >> 4;

    Rows<NRT> r;
    load_rows<NRT>(a, b, c, T, nq, m16, G, r);
    const size_t cache_off = (size_t)unit * a.max_ctx * kHeadDim;
    const uint16_t* kbase = a.k + cache_off;
    const uint16_t* vbase = a.v + cache_off;

    // ---- 1. the sweep ------------------------------------------------------
    float M[NRT], L[NRT];
    f32x4 oacc[8][NRT];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        M[rt] = -INFINITY;
        L[rt] = 0.f;
#pragma unroll
        for (int jd = 0; jd < 8; ++jd) oacc[jd][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int ntile = (key_end - key_begin + kTile - 1) / kTile;
    tile_pipeline<(NRT <= 2 ? 3 : 2), KVTile>(
        wave, ntile, kWaves,
        [&](KVTile& bf, int t) {
            load_k(kbase, key_begin + t * kTile, T, m16, G, bf.k);
            load_v(vbase, key_begin + t * kTile, T, m16, G, bf.v);
        },
        [&](const KVTile& bf, int t) {
            fused_tile<NRT>(a, r, bf, key_begin + t * kTile, t * kTile, stash, stride, m16, G, M,
                            L, oacc);
        });

    // ---- 2. publish the item's partial output and row statistics ----------
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        L[rt] += shfl_xor_f(L[rt], 16);
        L[rt] += shfl_xor_f(L[rt], 32);
        if (G == 0) wml[wave][rt * 16 + m16] = make_float2(M[rt], L[rt]);
    }
    __syncthreads();
    // rescale every wave's output to the workgroup's row maximum, then add
    // the waves in a fixed order
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        float Mw = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) Mw = fmaxf(Mw, wml[w][rt * 16 + m16].x);
        const float f = fast_exp2(M[rt] - safe_max(Mw));
#pragma unroll
        for (int jd = 0; jd < 8; ++jd) oacc[jd][rt] *= f;
    }
    for (int w = 0; w < kWaves; ++w) {
        if (wave == w) {
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = rt * 16 + m16;
                    const int c4 = (32 * G + 8 * i) / 4;
                    f32x4 w0 = {oacc[0][rt][i], oacc[1][rt][i], oacc[2][rt][i], oacc[3][rt][i]};
                    f32x4 w1 = {oacc[4][rt][i], oacc[5][rt][i], oacc[6][rt][i], oacc[7][rt][i]};
                    if (w == 0) {
                        red[row][c4] = w0;
                        red[row][c4 + 1] = w1;
                    } else {
                        red[row][c4] += w0;
                        red[row][c4 + 1] += w1;
                    }
                }
        }
        __syncthreads();
    }
    f32x4* po = reinterpret_cast<f32x4*>(a.part_o + (size_t)slot * kRowCap * kHeadDim);
    for (int x = tid; x < R * (kHeadDim / 4); x += kThreads) po[x] = red[x >> 5][x & 31];
    if (tid < R) {
        float Mw = -INFINITY, Lw = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) Mw = fmaxf(Mw, wml[w][tid].x);
#pragma unroll
        for (int w = 0; w < kWaves; ++w) Lw += wml[w][tid].y * fast_exp2(wml[w][tid].x - safe_max(Mw));
        a.part_ml[(size_t)slot * kRowCap + tid] = make_float2(Mw, Lw);
    }

    // ---- arrival barrier of this (sequence, KV head) -----------------------
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (tid == 0) {
        __hip_atomic_fetch_add(&fa.arrive[u], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int spins = 0;
        while (__hip_atomic_load(&fa.arrive[u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
                   (uint32_t)nchunk &&
               ++spins < kSpinLimit)
            __builtin_amdgcn_s_sleep(1);
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");

    // ---- 3a. exact row statistics over every chunk of the head -------------
    {
        const int rr = tid & (kRowCap - 1), ph = tid >> 6;
        float Mx = -INFINITY, Lx = 0.f;
        if (rr < R) {
            for (int s0 = ph; s0 < nchunk; s0 += 8 * kWaves) {
                float2 v[8];
#pragma unroll
                for (int uu = 0; uu < 8; ++uu) {
                    const int s2 = s0 + uu * kWaves;
                    v[uu] = s2 < nchunk ? a.part_ml[(size_t)(slot0 + s2) * kRowCap + rr]
                                        : make_float2(-INFINITY, 0.f);
                }
#pragma unroll
                for (int uu = 0; uu < 8; ++uu) ml_merge(Mx, Lx, v[uu].x, v[uu].y);
            }
        }
        lse_part[ph][rr] = make_float2(Mx, Lx);
    }
    __syncthreads();
    if (tid < kRowCap) {
        float Mx = -INFINITY, Lx = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) ml_merge(Mx, Lx, lse_part[w][tid].x, lse_part[w][tid].y);
        row_ml[tid] = make_float2(Mx, Lx);
        row_lse[tid] = Lx > 0.f ? Mx + fast_log2(Lx) : INFINITY;
    }
    __syncthreads();

    // ---- 3b. scores of this chunk's keys from the stashed logits -----------
    {
        const int wn = min(a.window, nq);
        const int r0 = (nq - wn) * a.group;   // first window row
        float* srow = a.scores + (size_t)unit * a.max_ctx;
        for (int kl = tid; kl < key_end - key_begin; kl += kThreads) {
            float sc = 0.f;
            for (int row = r0; row < R; ++row) sc += fast_exp2(stash[row * stride + kl] - row_lse[row]);
            srow[key_begin + kl] = sc;
        }
    }

    // ---- 3c. combine this item's share of the head's output rows ------------
    const int d4 = tid & 31, sg = tid >> 5;
    const f32x4* pall = reinterpret_cast<const f32x4*>(a.part_o);
    for (int row = s; row < R; row += nchunk) {
        const float Mr = safe_max(row_ml[row].x);
        const float inv = 1.0f / row_ml[row].y;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int s0 = sg; s0 < nchunk; s0 += 8 * kCombGroups) {
            f32x4 v[8];
            float wgt[8];
#pragma unroll
            for (int uu = 0; uu < 8; ++uu) {
                const int s2 = s0 + uu * kCombGroups;
                const bool ok = s2 < nchunk;
                const size_t sl = (size_t)(slot0 + (ok ? s2 : 0)) * kRowCap + row;
                v[uu] = ok ? pall[sl * (kHeadDim / 4) + d4] : f32x4{0.f, 0.f, 0.f, 0.f};
                wgt[uu] = ok ? fast_exp2(a.part_ml[sl].x - Mr) : 0.f;
            }
#pragma unroll
            for (int uu = 0; uu < 8; ++uu) acc += v[uu] * wgt[uu];
        }
        comb[sg][d4] = acc;
        __syncthreads();
        if (sg == 0) {
            f32x4 o = comb[0][d4];
#pragma unroll
            for (int gq = 1; gq < kCombGroups; ++gq) o += comb[gq][d4];
            o *= inv;
            const int j = row / a.group;
            const int h = c * a.group + (row - j * a.group);
            const size_t base = (((size_t)b * a.max_q + j) * a.n_q_heads + h) * kHeadDim + 4 * d4;
            if (a.out_fp32) {
                *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + base) = o;
            } else {
                uint2 pk = make_uint2(pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3]));
                *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + base) = pk;
            }
        }
        __syncthreads();
    }
}

__global__ void zero_u32_kernel(uint32_t* p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

template <int NRT>
hipError_t launch_fused_nrt(const FusedArgs& a, int n_slots, hipStream_t stream) {
    const size_t dyn = (size_t)NRT * 16 * (a.ft.chunk + kStashPad) * sizeof(float);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(verify_fused_kernel<NRT>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(zero_u32_kernel, dim3(1), dim3(256), 0, stream, a.arrive, a.ft.n_units);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    FusedArgs local = a;
    void* args[] = {&local};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(verify_fused_kernel<NRT>),
                                      dim3(n_slots), dim3(kThreads), args, (unsigned)dyn, stream);
}

}  // namespace

int fused_max_chunk(int row_tiles) {
    constexpr int kLds = 160 * 1024;
    int stat = 0;
    switch (row_tiles) {
        case 1: stat = static_lds_bytes<1>(); break;
        case 2: stat = static_lds_bytes<2>(); break;
        case 3: stat = static_lds_bytes<3>(); break;
        default: stat = static_lds_bytes<4>(); break;
    }
    const int floats_per_row = (kLds - stat - 1024) / (int)sizeof(float) / (16 * row_tiles);
    return (floats_per_row - kStashPad) / 128 * 128;
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
