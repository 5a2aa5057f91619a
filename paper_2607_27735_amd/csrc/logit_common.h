// logit_common.h -- reading one chunk of a logit row, shared by the token
// statistics and the speculative-sampling kernels.  Internal to the library.
#pragma once

#include "device_common.h"
#include "launch.h"

namespace ssl {
namespace lc {

constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;

// Logits per 16-byte load and loads per thread (32 logits per thread).
template <bool kF32>
constexpr int per_load() { return kF32 ? 4 : 8; }
template <bool kF32>
constexpr int loads() { return 32 / per_load<kF32>(); }

// The row index of x[q] as load_chunk fills it: thread tid's loads j cover
// consecutive 16-byte blocks kThreads apart, so x[q] is element
// (blk0 + (q / per) * kThreads + tid) * per + q % per of the row.
template <bool kF32>
__device__ __forceinline__ int elem(int chunk, int q, int tid) {
    constexpr int per = per_load<kF32>();
    const int blk0 = chunk * (kLogitChunk / per);
    return (blk0 + (q / per) * kThreads + tid) * per + q % per;
}

// The 32 logits of thread tid in chunk `chunk` of the row at `row_base`
// (bf16 or fp32), all loads in flight together; loads are clamped into the
// row's last 16-byte block and elements at or past vocab read as -inf.
template <bool kF32>
__device__ __forceinline__ void load_chunk(const void* row_base, int vocab, int chunk, int tid,
                                           float (&x)[32]) {
    constexpr int per = per_load<kF32>();
    constexpr int nl = loads<kF32>();
    const int last_blk = (vocab - 1) / per;
    const int blk0 = chunk * (kLogitChunk / per);
    const char* base = static_cast<const char*>(row_base);
    uint4 raw[nl];
#pragma unroll
    for (int j = 0; j < nl; ++j) {
        const int blk = min(blk0 + j * kThreads + tid, last_blk);
        raw[j] = *reinterpret_cast<const uint4*>(base + (size_t)blk * 16);
    }
#pragma unroll
    for (int j = 0; j < nl; ++j) {
        const uint32_t w[4] = {raw[j].x, raw[j].y, raw[j].z, raw[j].w};
#pragma unroll
        for (int e = 0; e < per; ++e) {
            const int i = (blk0 + j * kThreads + tid) * per + e;
            const float v = kF32 ? __builtin_bit_cast(float, w[e])
                                 : ((e & 1) ? bf16_hi(w[e >> 1]) : bf16_lo(w[e >> 1]));
            x[j * per + e] = i < vocab ? v : -INFINITY;
        }
    }
}

}  // namespace lc
}  // namespace ssl
