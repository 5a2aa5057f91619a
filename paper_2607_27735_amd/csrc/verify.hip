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
#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace {

constexpr int kThreads = 256;  // 4 waves
constexpr int kWaves = 4;
constexpr int kTile = 32;      // keys per wave step
constexpr int kRowCap = 64;    // rows per item slot in the workspace

// Tile-local key assigned to A row m of a 16-key half tile.  The accumulator
// rows lane group G receives are 4G + i, which then hold keys G + 4i: the same
// keys lane group G loads as full 256-byte rows for the V^T operand.
__device__ __forceinline__ int a_row_key(int m) { return (m >> 2) + 4 * (m & 3); }

struct Item {
    int b, c, s, nchunk, T, nq, key_begin, key_end, unit, item0;
};

__device__ __forceinline__ Item decode_item(const SeqTable& st, int item, int n_kv, int chunk) {
    Item it;
    int b = 0;
    while (b + 1 < st.n_seq && item >= st.item_start[b + 1]) ++b;
    it.b = b;
    it.T = st.ctx[b];
    it.nq = st.qlen[b];
    it.nchunk = (it.T + chunk - 1) / chunk;
    const int local = item - st.item_start[b];
    it.c = local / it.nchunk;
    it.s = local - it.c * it.nchunk;
    it.key_begin = it.s * chunk;
    it.key_end = min(it.key_begin + chunk, it.T);
    it.unit = b * n_kv + it.c;
    it.item0 = st.item_start[b] + it.c * it.nchunk;
    return it;
}

// The verify rows a lane owns: row rt*16 + (lane & 15) of each row tile.
template <int NRT>
struct Rows {
    int plim[NRT];      // last key the row may see; -1 for padding rows
    bool inwin[NRT];    // row contributes to the scores
    u32x4 q[NRT][4];    // B operand (Q^T): row's head-dim slice per 32-wide k-block
};

template <int NRT>
__device__ __forceinline__ void load_rows(const VerifyArgs& a, const Item& it, int m16, int G,
                                          Rows<NRT>& r) {
    const int g = a.group;
    const int R = it.nq * g;
    const int wn = min(a.window, it.nq);
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) {
        const int row = rt * 16 + m16;
        if (row < R) {
            const int j = row / g;
            const int hh = row - j * g;
            r.plim[rt] = it.T - it.nq + j;
            r.inwin[rt] = j >= it.nq - wn;
            const uint16_t* qp = a.q + (((size_t)it.b * a.max_q + j) * a.n_q_heads + it.c * g + hh) *
                                           kHeadDim + 8 * G;
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
__device__ __forceinline__ void load_k(const uint16_t* kbase, int key0, int T, int m16, int G,
                                       u32x4 (&kr)[2][4]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int key = min(key0 + 16 * t + a_row_key(m16), T - 1);
        const uint16_t* p = kbase + (size_t)key * kHeadDim + 8 * G;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) kr[t][kb] = ld_u32x4(p + 32 * kb);
    }
}

// V rows of a 32-key tile: slot e = 4t + i is key 16t + G + 4i, and lane
// (m16, G) holds its head-dim elements 8*m16 .. +8; one load instruction
// covers four whole consecutive rows.
__device__ __forceinline__ void load_v(const uint16_t* vbase, int key0, int T, int m16, int G,
                                       u32x4 (&vr)[8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int key = min(key0 + 16 * (e >> 2) + G + 4 * (e & 3), T - 1);
        vr[e] = ld_u32x4(vbase + (size_t)key * kHeadDim + 8 * m16);
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

template <int NRT>
__global__ __launch_bounds__(kThreads) void verify_stats_kernel(VerifyArgs a) {
    const Item it = decode_item(a.seq, blockIdx.x, a.n_kv_heads, a.chunk);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m16 = lane & 15, G = lane >> 4;
    Rows<NRT> r;
    load_rows<NRT>(a, it, m16, G, r);
    const uint16_t* kbase = a.k + (size_t)it.unit * a.max_ctx * kHeadDim;

    float M[NRT], L[NRT];
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt) { M[rt] = -INFINITY; L[rt] = 0.f; }

    const int ntile = (it.key_end - it.key_begin + kTile - 1) / kTile;
    int tt = wave;
    if (tt < ntile) {
        u32x4 ka[2][4], kb_[2][4];
        load_k(kbase, it.key_begin + tt * kTile, it.T, m16, G, ka);
        for (;;) {
            int tn = tt + kWaves < ntile ? tt + kWaves : tt;
            load_k(kbase, it.key_begin + tn * kTile, it.T, m16, G, kb_);
            stats_tile<NRT>(a, r, ka, it.key_begin + tt * kTile, G, M, L);
            tt += kWaves;
            if (tt >= ntile) break;
            tn = tt + kWaves < ntile ? tt + kWaves : tt;
            load_k(kbase, it.key_begin + tn * kTile, it.T, m16, G, ka);
            stats_tile<NRT>(a, r, kb_, it.key_begin + tt * kTile, G, M, L);
            tt += kWaves;
            if (tt >= ntile) break;
        }
    }
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
template <int NRT>
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
        if (key < key_end) srow[key] = val;
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

template <int NRT>
__global__ __launch_bounds__(kThreads) void verify_main_kernel(VerifyArgs a) {
    const Item it = decode_item(a.seq, blockIdx.x, a.n_kv_heads, a.chunk);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m16 = lane & 15, G = lane >> 4;

    // Row log-sum-exp from every item of this (sequence, KV head): lane group
    // G merges items G, G+4, ... and the groups are merged by shuffles.
    float lse[NRT];
    {
        float M[NRT], L[NRT];
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) { M[rt] = -INFINITY; L[rt] = 0.f; }
        for (int s2 = G; s2 < it.nchunk; s2 += 4) {
            const float2* pm = a.part_ml + (size_t)(it.item0 + s2) * kRowCap + m16;
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) {
                const float2 ml = pm[rt * 16];
                ml_merge(M[rt], L[rt], ml.x, ml.y);
            }
        }
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) {
            ml_merge(M[rt], L[rt], shfl_xor_f(M[rt], 16), shfl_xor_f(L[rt], 16));
            ml_merge(M[rt], L[rt], shfl_xor_f(M[rt], 32), shfl_xor_f(L[rt], 32));
            lse[rt] = L[rt] > 0.f ? M[rt] + fast_log2(L[rt]) : INFINITY;
        }
    }

    Rows<NRT> r;
    load_rows<NRT>(a, it, m16, G, r);
    const size_t cache_off = (size_t)it.unit * a.max_ctx * kHeadDim;
    const uint16_t* kbase = a.k + cache_off;
    const uint16_t* vbase = a.v + cache_off;
    float* srow = a.scores + (size_t)it.unit * a.max_ctx;

    f32x4 oacc[8][NRT];
#pragma unroll
    for (int jd = 0; jd < 8; ++jd)
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) oacc[jd][rt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int ntile = (it.key_end - it.key_begin + kTile - 1) / kTile;
    int tt = wave;
    if (tt < ntile) {
        u32x4 ka[2][4], kb_[2][4], va[8], vb[8];
        load_k(kbase, it.key_begin + tt * kTile, it.T, m16, G, ka);
        load_v(vbase, it.key_begin + tt * kTile, it.T, m16, G, va);
        for (;;) {
            int tn = tt + kWaves < ntile ? tt + kWaves : tt;
            load_k(kbase, it.key_begin + tn * kTile, it.T, m16, G, kb_);
            load_v(vbase, it.key_begin + tn * kTile, it.T, m16, G, vb);
            main_tile<NRT>(a, r, lse, ka, va, it.key_begin + tt * kTile, it.key_end, srow, m16, G,
                           oacc);
            tt += kWaves;
            if (tt >= ntile) break;
            tn = tt + kWaves < ntile ? tt + kWaves : tt;
            load_k(kbase, it.key_begin + tn * kTile, it.T, m16, G, ka);
            load_v(vbase, it.key_begin + tn * kTile, it.T, m16, G, va);
            main_tile<NRT>(a, r, lse, kb_, vb, it.key_begin + tt * kTile, it.key_end, srow, m16, G,
                           oacc);
            tt += kWaves;
            if (tt >= ntile) break;
        }
    }

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
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kHeadDim) void verify_combine_kernel(VerifyArgs a) {
    const SeqTable& st = a.seq;
    const int gr = blockIdx.x;
    int b = 0;
    while (b + 1 < st.n_seq && gr >= st.row_start[b + 1]) ++b;
    const int R = st.qlen[b] * a.group;
    const int local = gr - st.row_start[b];
    const int c = local / R;
    const int row = local - c * R;
    const int nchunk = (st.ctx[b] + a.chunk - 1) / a.chunk;
    const int item0 = st.item_start[b] + c * nchunk;
    const int d = threadIdx.x;
    float acc = 0.f;
    for (int s = 0; s < nchunk; ++s)
        acc += a.part_o[((size_t)(item0 + s) * kRowCap + row) * kHeadDim + d];
    const int j = row / a.group;
    const int h = c * a.group + (row - j * a.group);
    const size_t o = (((size_t)b * a.max_q + j) * a.n_q_heads + h) * kHeadDim + d;
    if (a.out_fp32)
        reinterpret_cast<float*>(a.out)[o] = acc;
    else
        reinterpret_cast<__bf16*>(a.out)[o] = (__bf16)acc;
}

template <int NRT>
hipError_t launch_verify_nrt(const VerifyArgs& a, int n_items, int n_rows_total,
                             hipStream_t stream) {
    hipLaunchKernelGGL(verify_stats_kernel<NRT>, dim3(n_items), dim3(kThreads), 0, stream, a);
    hipLaunchKernelGGL(verify_main_kernel<NRT>, dim3(n_items), dim3(kThreads), 0, stream, a);
    hipLaunchKernelGGL(verify_combine_kernel, dim3(n_rows_total), dim3(kHeadDim), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

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
