// verify.hip -- dense verification attention with fused importance scores.
//
// Computes, for every verify row of every sequence, softmax attention over the
// whole dense cache (Sec. 3.1) and, from the same probabilities, the Eq. 3
// importance of every cached key: the probability mass it receives from the
// last min(W, q) verify rows of all query heads sharing its KV head.
//
// The scores need each row's *global* normalizer, which a split-K pass only
// knows after every split has finished.  The work is therefore two sweeps over
// the context, both split-K over (sequence, KV head, key chunk) work items:
//
//   verify_stats  reads K only; per item and row it returns the running
//                 maximum and sum of 2^y (y = logit * log2 e);
//   verify_main   merges those into the exact log-sum-exp of each row, then
//                 reads K and V once more and forms the final probabilities
//                 P = 2^(y - lse) directly: the key's score is a plain sum of
//                 P over rows (written straight to `scores`, no later pass),
//                 and the item's contribution to the output is sum P * V,
//                 which needs no rescaling when items are added;
//   verify_combine adds the per-item outputs of each row.
//
// Both sweeps run the K.Q^T product on the bf16 MFMA (the k+1 verify rows of
// all query heads of a KV head, 12..64 rows, form a genuine 16-row-tiled
// contraction); P.V runs on the MFMA as O^T = V^T P^T so that every row's
// softmax state and output stay in the lane that owns the row.
#include "verify_common.h"

namespace ssl {
namespace {

using namespace vc;


// ---------------------------------------------------------------------------
// Sweep 1: per-item row statistics from K only.
// ---------------------------------------------------------------------------
template <int NRT>
__device__ __forceinline__ void stats_tile(const VerifyArgs& a, const Rows<NRT>& r,
                                           const u32x4 (&kr)[2][4], int key0, int G,
                                           float (&M)[NRT], float (&L)[NRT]) {
    f32x4 acc[2][NRT];
    qk_tile<NRT>(kr, r, acc);
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        float y[8];
        float mt = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int t = e >> 2, i = e & 3;
            const int key = key0 + 16 * t + G + 4 * i;
            y[e] = key <= r.plim[rt] ? acc[t][rt][i] * a.scale_log2 : -INFINITY;
            mt = fmaxf(mt, y[e]);
        }
        const float Mn = fmaxf(M[rt], mt);
        if (Mn != -INFINITY) {
            float sum = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) sum += fast_exp2(y[e] - Mn);
            L[rt] = L[rt] * fast_exp2(M[rt] - Mn) + sum;
            M[rt] = Mn;
        }
    }
}

template <int NRT, bool kPaged>
__global__ __launch_bounds__(kThreads) void verify_stats_kernel(VerifyArgs a) {
    const Item it = decode_item<true>(a, a.seq, blockIdx.x, a.chunk);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m16 = lane & 15, G = lane >> 4;
    Rows<NRT> r;
    load_rows<NRT>(a, it.b, it.c, it.T, it.nq, it.qoff, it.qfull, m16, G, r);
    const uint16_t* kbase = a.k + (size_t)it.unit * a.max_ctx * kHeadDim;

    float M[NRT], L[NRT];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) { M[rt] = -INFINITY; L[rt] = 0.f; }

    const int ntile = (it.key_end - it.key_begin + kTile - 1) / kTile;
    const int pages = kPaged ? wave_pages(a, it.b, it.key_begin, ntile, wave, lane) : 0;
    tile_pipeline<4, KTile>(
        wave, ntile, kWaves,
        [&](KTile& b, int t) {
            const int key0 = it.key_begin + t * kTile;
            if constexpr (kPaged)
                load_k<false>(a.k + paged_row(a, tile_page(pages, t, wave), it.c, key0) * kHeadDim,
                              0, it.T - key0, m16, G, b.k);
            else
                load_k<false>(kbase, key0, it.T, m16, G, b.k);
        },
        [&](const KTile& b, int t) {
            stats_tile<NRT>(a, r, b.k, it.key_begin + t * kTile, G, M, L);
        });
    // Merge the four lane groups (they saw disjoint keys of the same rows).
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        ml_merge(M[rt], L[rt], shfl_xor_f(M[rt], 16), shfl_xor_f(L[rt], 16));
        ml_merge(M[rt], L[rt], shfl_xor_f(M[rt], 32), shfl_xor_f(L[rt], 32));
    }
    __shared__ float2 wml[kWaves][NRT * 16];
    if (G == 0) {
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) wml[wave][rt * 16 + m16] = make_float2(M[rt], L[rt]);
    }
    __syncthreads();
    if (threadIdx.x < NRT * 16) {
        float Mx = -INFINITY, Lx = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) ml_merge(Mx, Lx, wml[w][threadIdx.x].x, wml[w][threadIdx.x].y);
        a.part_ml[(size_t)blockIdx.x * kRowCap + threadIdx.x] = make_float2(Mx, Lx);
    }
}

// ---------------------------------------------------------------------------
// Sweep 2: exact probabilities -> scores and per-item P.V.
// ---------------------------------------------------------------------------
template <int NRT, bool kPerHead>
__device__ __forceinline__ void main_tile(const VerifyArgs& a, const Rows<NRT>& r,
                                          const float (&lse)[NRT], const u32x4 (&kr)[2][4],
                                          const u32x4 (&vr)[8], int key0, int key_end,
                                          float* srow, int m16, int G,
                                          f32x4 (&oacc)[8][NRT]) {
    f32x4 acc[2][NRT];
    qk_tile<NRT>(kr, r, acc);

    float p[2][NRT][4];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = key0 + 16 * t + G + 4 * i;
                p[t][rt][i] = key <= r.plim[rt] ? fast_exp2(acc[t][rt][i] * a.scale_log2 - lse[rt])
                                                : 0.f;
            }

    // One index set per query head (the group divides 16, so head hh owns the
    // lanes m16 = hh mod group of every row tile): lane m16 < group sums its
    // head's window rows for the lane group's eight keys and writes them.
    if constexpr (kPerHead) {
        float hs[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int t = e >> 2, i = e & 3;
            float s = 0.f;
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) s += r.inwin[rt] ? p[t][rt][i] : 0.f;
            for (int o = 8; o >= a.group; o >>= 1) s += __shfl_xor(s, o, kWave);
            hs[e] = s;
        }
        if (m16 < a.group) {
            float* hrow = srow + (size_t)m16 * a.max_ctx;   // srow: head c * group of this sequence
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int key = key0 + 16 * (e >> 2) + G + 4 * (e & 3);
                if (key < key_end) hrow[key] = a.score_add ? hrow[key] + hs[e] : hs[e];
            }
        }
    } else {
    // Scores: sum of P over the window rows; rows live on the 16 lanes of the
    // DPP row and on the row tiles.
    float sp[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int t = e >> 2, i = e & 3;
        float s = 0.f;
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) s += r.inwin[rt] ? p[t][rt][i] : 0.f;
        sp[e] = row16_sum(s);
    }
    if (m16 < 8) {
        float val = sp[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) val = (m16 == e) ? sp[e] : val;
        const int key = key0 + 16 * (m16 >> 2) + G + 4 * (m16 & 3);
        if (key < key_end) srow[key] = a.score_add ? srow[key] + val : val;
    }
    }

    // O^T += V^T P^T.  B operand: slot e = 4t + i of P^T for the lane's row.
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
        for (int sp2 = 0; sp2 < 4; ++sp2) {
            const uint32_t x = vr[2 * sp2][jd >> 1], y = vr[2 * sp2 + 1][jd >> 1];
            av[sp2] = (jd & 1) ? perm_hi(x, y) : perm_lo(x, y);
        }
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) oacc[jd][rt] = mfma_bf16(av, pb[rt], oacc[jd][rt]);
    }
}

template <int NRT, bool kPaged, bool kPerHead>
__global__ __launch_bounds__(kThreads) void verify_main_kernel(VerifyArgs a) {
    const Item it = decode_item<true>(a, a.seq, blockIdx.x, a.chunk);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m16 = lane & 15, G = lane >> 4;

    Rows<NRT> r;
    load_rows<NRT>(a, it.b, it.c, it.T, it.nq, it.qoff, it.qfull, m16, G, r);
    const size_t cache_off = (size_t)it.unit * a.max_ctx * kHeadDim;
    const uint16_t* kbase = a.k + cache_off;
    const uint16_t* vbase = a.v + cache_off;
    // (per-head scores: the row of the group's first query head)
    float* srow = a.scores + (a.per_head ? ((size_t)it.b * a.n_q_heads + it.c * a.group) * a.max_ctx
                                         : (size_t)it.unit * a.max_ctx);
    const int ntile = (it.key_end - it.key_begin + kTile - 1) / kTile;
    const int pages = kPaged ? wave_pages(a, it.b, it.key_begin, ntile, wave, lane) : 0;

    // Row log-sum-exp from the statistics of every item of this (sequence, KV
    // head), computed while the first K/V tiles are loading: thread t merges
    // row t % 64 over the items t / 64, t / 64 + 4, ... (all of its loads in
    // flight together), then the four partial states of each row are merged
    // in a fixed order.
    __shared__ float2 lse_part[kWaves][kRowCap];
    __shared__ float lse_row[kRowCap];
    float lse[NRT];
    auto row_lse = [&] {
        const int R = it.nq * a.group;
        const int rr = threadIdx.x & (kRowCap - 1), ph = threadIdx.x >> 6;
        float M = -INFINITY, L = 0.f;
        if (rr < R) {
            for (int s0 = ph; s0 < it.nchunk; s0 += 8 * kWaves) {
                float2 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int s2 = s0 + u * kWaves;
                    v[u] = s2 < it.nchunk ? a.part_ml[(size_t)(it.item0 + s2) * kRowCap + rr]
                                          : make_float2(-INFINITY, 0.f);
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) ml_merge(M, L, v[u].x, v[u].y);
            }
        }
        lse_part[ph][rr] = make_float2(M, L);
        __syncthreads();
        if (threadIdx.x < kRowCap) {
            float Mx = -INFINITY, Lx = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w)
                ml_merge(Mx, Lx, lse_part[w][threadIdx.x].x, lse_part[w][threadIdx.x].y);
            lse_row[threadIdx.x] = Lx > 0.f ? Mx + fast_log2(Lx) : INFINITY;
        }
        __syncthreads();
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) lse[rt] = lse_row[rt * 16 + m16];
    };

    f32x4 oacc[8][NRT];
#pragma unroll
    for (int jd = 0; jd < 8; ++jd)
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) oacc[jd][rt] = f32x4{0.f, 0.f, 0.f, 0.f};

    tile_pipeline<(NRT <= 2 ? 3 : 2), KVTile>(
        wave, ntile, kWaves,
        [&](KVTile& b, int t) {
            load_kv_tile<kPaged, true>(a, kbase, vbase, kPaged ? tile_page(pages, t, wave) : 0, it.c,
                                       it.key_begin + t * kTile, it.T, m16, G, b);
        },
        [&](const KVTile& b, int t) {
            main_tile<NRT, kPerHead>(a, r, lse, b.k, b.v, it.key_begin + t * kTile, it.key_end, srow, m16,
                           G, oacc);
        },
        row_lse);

    // Sum the four waves' partial outputs in LDS (fixed order), then write the
    // item's rows.  oacc[jd][rt][i] is row rt*16+m16, head-dim 32G + 8i + jd.
    __shared__ f32x4 red[NRT * 16][kHeadDim / 4];
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
    const int R = it.nq * a.group;
    f32x4* po = reinterpret_cast<f32x4*>(a.part_o + (size_t)blockIdx.x * kRowCap * kHeadDim);
    for (int x = threadIdx.x; x < R * (kHeadDim / 4); x += kThreads) po[x] = red[x >> 5][x & 31];
}

// ---------------------------------------------------------------------------
// Combine: out row = sum over the items of its (sequence, KV head).
// 256 threads per row: thread t sums head-dim quad t % 32 over the items
// t / 32, t / 32 + 8, ... with all its loads in flight at once; the eight
// partial sums are then added in a fixed order.
// ---------------------------------------------------------------------------
constexpr int kCombineThreads = 256;
constexpr int kCombineGroups = kCombineThreads / 32;

__global__ __launch_bounds__(kCombineThreads) void verify_combine_kernel(VerifyArgs a) {
    const SeqTable& st = a.seq;
    const int gr = blockIdx.x;
    int bt = 0;
    while (bt + 1 < st.n_seq && gr >= st.row_start[bt + 1]) ++bt;
    const int b = a.sid[bt];
    const int R = st.qlen[bt] * a.group;
    const int local = gr - st.row_start[bt];
    const int c = local / R;
    const int row = local - c * R;
    const int nchunk = (st.ctx[bt] + a.chunk - 1) / a.chunk;
    const int item0 = st.item_start[bt] + c * nchunk;
    const int d4 = threadIdx.x & 31, sg = threadIdx.x >> 5;
    const f32x4* po = reinterpret_cast<const f32x4*>(a.part_o);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = sg; s0 < nchunk; s0 += 8 * kCombineGroups) {
        f32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int s = s0 + u * kCombineGroups;
            v[u] = s < nchunk ? po[((size_t)(item0 + s) * kRowCap + row) * (kHeadDim / 4) + d4]
                              : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += v[u];
    }
    __shared__ f32x4 red[kCombineGroups][32];
    red[sg][d4] = acc;
    __syncthreads();
    if (sg != 0) return;
    f32x4 o = red[0][d4];
#pragma unroll
    for (int gq = 1; gq < kCombineGroups; ++gq) o += red[gq][d4];
    const int jl = row / a.group;
    const int h = c * a.group + (row - jl * a.group);
    const int j = a.qoff[bt] + jl;
    const size_t base = (((size_t)b * a.max_q + j) * a.n_q_heads + h) * kHeadDim + 4 * d4;
    if (a.out_fp32) {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + base) = o;
    } else {
        uint2 pk = make_uint2(pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3]));
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + base) = pk;
    }
}

template <int NRT>
hipError_t launch_verify_nrt(const VerifyArgs& a, int n_items, int n_rows_total,
                             hipStream_t stream) {
    const dim3 grid(n_items), block(kThreads);
    if (a.block_table) {
        hipLaunchKernelGGL((verify_stats_kernel<NRT, true>), grid, block, 0, stream, a);
        if (a.per_head)
            hipLaunchKernelGGL((verify_main_kernel<NRT, true, true>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((verify_main_kernel<NRT, true, false>), grid, block, 0, stream, a);
    } else {
        hipLaunchKernelGGL((verify_stats_kernel<NRT, false>), grid, block, 0, stream, a);
        if (a.per_head)
            hipLaunchKernelGGL((verify_main_kernel<NRT, false, true>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((verify_main_kernel<NRT, false, false>), grid, block, 0, stream, a);
    }
    hipLaunchKernelGGL(verify_combine_kernel, dim3(n_rows_total), dim3(kCombineThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_verify_combine(const VerifyArgs& a, int n_rows_total, hipStream_t stream) {
    hipLaunchKernelGGL(verify_combine_kernel, dim3(n_rows_total), dim3(kCombineThreads), 0, stream,
                       a);
    return hipGetLastError();
}

hipError_t launch_verify(const VerifyArgs& a, int n_items, int n_rows_total, int row_tiles,
                         hipStream_t stream) {
    switch (row_tiles) {
        case 1: return launch_verify_nrt<1>(a, n_items, n_rows_total, stream);
        case 2: return launch_verify_nrt<2>(a, n_items, n_rows_total, stream);
        case 3: return launch_verify_nrt<3>(a, n_items, n_rows_total, stream);
        default: return launch_verify_nrt<4>(a, n_items, n_rows_total, stream);
    }
}

}  // namespace ssl
