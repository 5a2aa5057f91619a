// draft.hip -- draft-step attention over the gathered sparse view (Eq. 5).
//
// The gather is fused: K/V rows named by the index set are read in place from
// the dense cache, never copied.  Work items are (sequence, KV head, chunk of
// the index list), one wave each; the wave keeps an online softmax per query
// head of the group (up to 16 heads = one MFMA row tile) and writes its
// unnormalized partial output with the running (max, sum).  A combine kernel
// merges the partials of each query head.
//
// The MFMA layouts are the verify kernel's: K.Q^T on the bf16 MFMA with the
// keys as A rows, O^T = V^T P^T so a head's softmax state and output stay in
// the lane that owns the head; V is loaded as whole 256-byte rows per lane
// group and transposed in registers with byte permutes.
#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace {

constexpr int kTile = 32;
constexpr int kRowCap = 16;

__device__ __forceinline__ int a_row_key(int m) { return (m >> 2) + 4 * (m & 3); }

struct DItem {
    int b, c, n, nchunk, key_begin, key_end, unit, item0;
};

__device__ __forceinline__ DItem decode_ditem(const SeqTable& st, int item, int n_kv, int chunk) {
    DItem it;
    int b = 0;
    while (b + 1 < st.n_seq && item >= st.item_start[b + 1]) ++b;
    it.b = b;
    it.n = st.ctx[b];
    it.nchunk = (it.n + chunk - 1) / chunk;
    const int local = item - st.item_start[b];
    it.c = local / it.nchunk;
    const int s = local - it.c * it.nchunk;
    it.key_begin = s * chunk;
    it.key_end = min(it.key_begin + chunk, it.n);
    it.unit = b * n_kv + it.c;
    it.item0 = st.item_start[b] + it.c * it.nchunk;
    return it;
}

struct Gathered {
    u32x4 k[2][4];
    u32x4 v[8];
};

// Gathers the K and V rows of the 32-key tile starting at chunk position p0.
// Lane l of the wave holds the cache row of chunk position l in `my_row`;
// the rows each lane needs are fetched from their owners by lane shuffles.
__device__ __forceinline__ void gather_tile(int my_row, int p0, const uint16_t* kbase,
                                            const uint16_t* vbase, int m16, int G, Gathered& t) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int row = __shfl(my_row, p0 + 16 * h + a_row_key(m16), kWave);
        const uint16_t* p = kbase + (size_t)row * kHeadDim + 8 * G;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) t.k[h][kb] = ld_u32x4(p + 32 * kb);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int row = __shfl(my_row, p0 + 16 * (e >> 2) + G + 4 * (e & 3), kWave);
        t.v[e] = ld_u32x4(vbase + (size_t)row * kHeadDim + 8 * m16);
    }
}

__device__ __forceinline__ void draft_tile(const DraftArgs& a, const u32x4 (&qop)[4],
                                           const Gathered& t, int pos0, int pos_end, int G,
                                           float& M, float& L, f32x4 (&oacc)[8]) {
    f32x4 acc[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) s = mfma_bf16(t.k[h][kb], qop[kb], s);
        acc[h] = s;
    }
    float y[8];
    float mt = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int h = e >> 2, i = e & 3;
        const int pos = pos0 + 16 * h + G + 4 * i;
        y[e] = pos < pos_end ? acc[h][i] * a.scale_log2 : -INFINITY;
        mt = fmaxf(mt, y[e]);
    }
    mt = fmaxf(mt, shfl_xor_f(mt, 16));
    mt = fmaxf(mt, shfl_xor_f(mt, 32));
    const float Mn = fmaxf(M, mt);
    const float alpha = fast_exp2(M - Mn);   // M = -inf on the first tile: alpha = 0
    float p[8], sum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        p[e] = fast_exp2(y[e] - Mn);
        sum += p[e];
    }
    L = L * alpha + sum;
    M = Mn;
#pragma unroll
    for (int jd = 0; jd < 8; ++jd) oacc[jd] *= alpha;

    u32x4 pb;
    pb[0] = pack_bf16(p[0], p[1]);
    pb[1] = pack_bf16(p[2], p[3]);
    pb[2] = pack_bf16(p[4], p[5]);
    pb[3] = pack_bf16(p[6], p[7]);
#pragma unroll
    for (int jd = 0; jd < 8; ++jd) {
        u32x4 av;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            const uint32_t x = t.v[2 * s2][jd >> 1], yv = t.v[2 * s2 + 1][jd >> 1];
            av[s2] = (jd & 1) ? perm_hi(x, yv) : perm_lo(x, yv);
        }
        oacc[jd] = mfma_bf16(av, pb, oacc[jd]);
    }
}

__global__ __launch_bounds__(kWave) void draft_kernel(DraftArgs a) {
    const DItem it = decode_ditem(a.seq, blockIdx.x, a.n_kv_heads, a.chunk);
    const int lane = threadIdx.x;
    const int m16 = lane & 15, G = lane >> 4;
    const int g = a.group;

    u32x4 qop[4];
    if (m16 < g) {
        const uint16_t* qp = a.q + ((size_t)it.b * a.n_q_heads + it.c * g + m16) * kHeadDim + 8 * G;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qop[kb] = ld_u32x4(qp + 32 * kb);
    } else {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qop[kb] = u32x4{0u, 0u, 0u, 0u};
    }
    const size_t cache_off = (size_t)it.unit * a.max_ctx * kHeadDim;
    const uint16_t* kbase = a.k + cache_off;
    const uint16_t* vbase = a.v + cache_off;
    const int32_t* ib = a.idx + (size_t)it.unit * a.budget;
    const int last = it.n - 1;

    float M = -INFINITY, L = 0.f;
    f32x4 oacc[8];
#pragma unroll
    for (int jd = 0; jd < 8; ++jd) oacc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};

    // One chunk is two 32-key tiles: lane l loads the cache row of chunk
    // position l once, then every K/V row of both tiles is requested at once.
    const int my_row = min(max(ib[min(it.key_begin + lane, last)], 0), a.max_ctx - 1);
    Gathered ta, tb;
    gather_tile(my_row, 0, kbase, vbase, m16, G, ta);
    gather_tile(my_row, kTile, kbase, vbase, m16, G, tb);
    draft_tile(a, qop, ta, it.key_begin, it.key_end, G, M, L, oacc);
    if (it.key_begin + kTile < it.key_end)
        draft_tile(a, qop, tb, it.key_begin + kTile, it.key_end, G, M, L, oacc);
    L += shfl_xor_f(L, 16);
    L += shfl_xor_f(L, 32);

    const size_t item = blockIdx.x;
    if (G == 0) a.part_ml[item * kRowCap + m16] = make_float2(M, L);
    f32x4* po = reinterpret_cast<f32x4*>(a.part_o + (item * kRowCap + m16) * kHeadDim);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c4 = (32 * G + 8 * i) / 4;
        po[c4] = f32x4{oacc[0][i], oacc[1][i], oacc[2][i], oacc[3][i]};
        po[c4 + 1] = f32x4{oacc[4][i], oacc[5][i], oacc[6][i], oacc[7][i]};
    }
}

// Combine of one query head's partials.  256 threads: thread t handles
// head-dim quad t % 32 for the items t / 32, t / 32 + 8, ..., merging them
// online; the eight partial states are then merged in a fixed order.
constexpr int kCombineThreads = 256;
constexpr int kCombineGroups = kCombineThreads / 32;

__global__ __launch_bounds__(kCombineThreads) void draft_combine_kernel(DraftArgs a) {
    const SeqTable& st = a.seq;
    const int bh = blockIdx.x;
    const int b = bh / a.n_q_heads;
    const int h = bh - b * a.n_q_heads;
    const int c = h / a.group;
    const int row = h - c * a.group;
    const int nchunk = (st.ctx[b] + a.chunk - 1) / a.chunk;
    const int item0 = st.item_start[b] + c * nchunk;
    const int d4 = threadIdx.x & 31, sg = threadIdx.x >> 5;
    const f32x4* po = reinterpret_cast<const f32x4*>(a.part_o);
    float M = -INFINITY, L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = sg; s0 < nchunk; s0 += 8 * kCombineGroups) {
        float2 ml[8];
        f32x4 o[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int s = s0 + u * kCombineGroups;
            const bool ok = s < nchunk;
            const size_t slot = (size_t)(item0 + (ok ? s : 0)) * kRowCap + row;
            ml[u] = ok ? a.part_ml[slot] : make_float2(-INFINITY, 0.f);
            o[u] = ok ? po[slot * (kHeadDim / 4) + d4] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        float Mn = M;
#pragma unroll
        for (int u = 0; u < 8; ++u) Mn = fmaxf(Mn, ml[u].x);
        const float alpha = fast_exp2(M - Mn);   // M = -inf at first: 0
        L *= alpha;
        acc *= alpha;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const float wgt = fast_exp2(ml[u].x - Mn);   // empty slots: 0
            L += ml[u].y * wgt;
            acc += o[u] * wgt;
        }
        M = Mn;
    }
    __shared__ f32x4 racc[kCombineGroups][32];
    __shared__ float2 rml[kCombineGroups][32];
    racc[sg][d4] = acc;
    rml[sg][d4] = make_float2(M, L);
    __syncthreads();
    if (sg != 0) return;
    float Mx = -INFINITY;
#pragma unroll
    for (int gq = 0; gq < kCombineGroups; ++gq) Mx = fmaxf(Mx, rml[gq][d4].x);
    float Lx = 0.f;
    f32x4 ox = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int gq = 0; gq < kCombineGroups; ++gq) {
        const float2 m = rml[gq][d4];
        const float wgt = m.x == -INFINITY ? 0.f : fast_exp2(m.x - Mx);
        Lx += m.y * wgt;
        ox += racc[gq][d4] * wgt;
    }
    ox *= 1.0f / Lx;
    const size_t base = ((size_t)b * a.n_q_heads + h) * kHeadDim + 4 * d4;
    if (a.out_fp32) {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + base) = ox;
    } else {
        uint2 pk = make_uint2(pack_bf16(ox[0], ox[1]), pack_bf16(ox[2], ox[3]));
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + base) = pk;
    }
}

}  // namespace

hipError_t launch_draft(const DraftArgs& a, int n_items, int n_rows_total, hipStream_t stream) {
    hipLaunchKernelGGL(draft_kernel, dim3(n_items), dim3(kWave), 0, stream, a);
    hipLaunchKernelGGL(draft_combine_kernel, dim3(n_rows_total), dim3(kCombineThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ssl
