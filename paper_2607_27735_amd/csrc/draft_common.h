// draft_common.h -- the gather and attention math of one 32-entry draft tile,
// shared by the draft kernels and the select kernel's draft step.  Internal to
// the library.
//
// The MFMA layouts are the verify kernel's: K.Q^T on the bf16 MFMA with the
// keys as A rows and the query heads (up to 16) as B columns, O^T = V^T P^T so
// a head's softmax state and output stay in the lane that owns the head; V is
// loaded as whole 256-byte rows per lane group and transposed in registers
// with byte permutes.
#pragma once

#include "device_common.h"

namespace ssl {
namespace dc {

constexpr int kTile = 32;

// Tile-local key assigned to A row m of a 16-key half tile (see verify).
__device__ __forceinline__ int a_row_key(int m) { return (m >> 2) + 4 * (m & 3); }

struct Gathered {
    u32x4 k[2][4];
    u32x4 v[8];
};

// Where the rows of the entries live: the dense cache of the unit, and (draft
// round steps) the unit's materialized rows.  A row id with kSelBit set is a
// row of the materialized copy.
constexpr uint32_t kSelBit = 0x80000000u;
struct RowSource {
    const uint16_t* k;
    const uint16_t* v;
    const uint16_t* k_sel;
    const uint16_t* v_sel;
};

template <bool kRound>
__device__ __forceinline__ const uint16_t* row_ptr(const uint16_t* cache, const uint16_t* sel,
                                                   uint32_t row) {
    if (!kRound) return cache + (size_t)row * kHeadDim;
    return (row & kSelBit) ? sel + (size_t)(row & ~kSelBit) * kHeadDim
                           : cache + (size_t)row * kHeadDim;
}

// Gathers the K and V rows of the 32-key tile starting at chunk position p0.
// Lane l of the wave holds the row id of chunk position l in `my_row`; the
// rows each lane needs are fetched from their owners by lane shuffles.
template <bool kRound>
__device__ __forceinline__ void gather_tile(uint32_t my_row, int p0, const RowSource& src,
                                            int m16, int G, Gathered& t) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t row = __shfl(my_row, p0 + 16 * h + a_row_key(m16), kWave);
        const uint16_t* p = row_ptr<kRound>(src.k, src.k_sel, row) + 8 * G;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) t.k[h][kb] = ld_u32x4(p + 32 * kb);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t row = __shfl(my_row, p0 + 16 * (e >> 2) + G + 4 * (e & 3), kWave);
        t.v[e] = ld_u32x4(row_ptr<kRound>(src.v, src.v_sel, row) + 8 * m16);
    }
}

__device__ __forceinline__ void draft_tile(float scale_log2, const u32x4 (&qop)[4],
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
        y[e] = pos < pos_end ? acc[h][i] * scale_log2 : -INFINITY;
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


}  // namespace dc
}  // namespace ssl
