// device_common.h -- CDNA4 (gfx950) building blocks shared by the kernels.
//
// Wave64 throughout.  Matrix products use the gfx950 bf16 MFMA
// v_mfma_f32_16x16x32_bf16: A is 16(M) x 32(K), B is 32(K) x 16(N), fp32
// 16x16 accumulator.  Lane l supplies A row (l & 15) and B column (l & 15),
// each as 8 consecutive K elements starting at 8 * (l >> 4); it receives
// accumulator column (l & 15), rows 4 * (l >> 4) + 0..3.  Because a lane's
// 8 K elements only need to agree between A and B, the kernels are free to
// map K slots to keys or to head-dim elements in whatever order makes their
// global loads contiguous.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"

namespace ssl {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;
constexpr int kMaxBatch = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Two fp32 values -> packed bf16 pair (round to nearest even), lo in bits 0-15.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2 v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xffff0000u); }

// Low halves of x and y packed as (x.lo, y.lo); high halves as (x.hi, y.hi).
__device__ __forceinline__ uint32_t perm_lo(uint32_t x, uint32_t y) {
    return __builtin_amdgcn_perm(y, x, 0x05040100u);
}
__device__ __forceinline__ uint32_t perm_hi(uint32_t x, uint32_t y) {
    return __builtin_amdgcn_perm(y, x, 0x07060302u);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Row rotation inside each 16-lane DPP row.
template <int N>
__device__ __forceinline__ float row_ror(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
        0, __builtin_bit_cast(int, x), 0x120 + N, 0xf, 0xf, false));
}

// Sum over the 16 lanes of a DPP row; every lane of the row gets the total.
__device__ __forceinline__ float row16_sum(float x) {
    x += row_ror<8>(x);
    x += row_ror<4>(x);
    x += row_ror<2>(x);
    x += row_ror<1>(x);
    return x;
}

// Inclusive prefix sum over the 64 lanes of a wave: shifts within rows of 16
// lanes, then the row broadcasts of lanes 15 and 31 (DPP, no LDS traffic).
__device__ __forceinline__ int wave_incl_scan(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15 -> rows 1, 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31 -> rows 2, 3
    return x;
}

// Device-coherent accesses (agent scope, relaxed atomics): the stores write
// through and the loads read past the per-XCD L2, so a few words published by
// one workgroup reach another without an L2 writeback.  After
// wait_stores_done() every store the wave issued has completed.
__device__ __forceinline__ void st_dev(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev32(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_dev32(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev64(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_dev64(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_dev2(const float2* p) {
    const float* f = reinterpret_cast<const float*>(p);
    return make_float2(ld_dev(f), ld_dev(f + 1));
}
// The tag that workgroups of one cross-workgroup exchange publish and wait
// for: the host's call tag (a process-wide sequence with a random start) plus
// the exchange group's epoch, a workspace word that the group's finisher
// advances by one once every member has read it.  The epoch makes replays of a
// launch captured in a graph, whose call tag is fixed, use a new tag each
// time (eager launches, whose call tags already differ, pass no epoch words
// and skip both the load and the advance); the odd factor keeps 2^39 consecutive epochs distinct in the low 39
// bits that the shortest tags keep, and makes an epoch word that other data
// overwrote line up with a stale tag only by accident.
__device__ __forceinline__ uint64_t exchange_tag(uint64_t call_tag, uint64_t epoch) {
    return call_tag + epoch * 0x9E3779B97F4A7C15ull;
}

// A bounded wait gave up (one thread per workgroup calls this): the device's
// status word gets the kernel family's bit and, for a call under graph
// capture, the group's epoch word the mark kEpochDirty, so that every later
// captured call on the workspace gives up at once instead of matching tags
// that members of the failed call published late.  (When the group's
// finisher did complete, every member had read the epoch, and its advance may
// overwrite the mark: then no stale tag can match.)
__device__ __forceinline__ void exchange_gave_up(const Exchange& xc, uint32_t bit,
                                                 uint64_t* epoch_word) {
    __hip_atomic_fetch_or(xc.status, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (epoch_word) st_dev64(epoch_word, kEpochDirty);
}

// The group's finisher advances the epoch once every member has read it.
__device__ __forceinline__ void epoch_advance(uint64_t* epoch_word) {
    __hip_atomic_fetch_add(epoch_word, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool epoch_is_dirty(uint64_t epoch) { return epoch == kEpochDirty; }

// The wave-uniform 64-bit value v, moved to scalar registers here.  A uniform
// value loaded from memory is otherwise moved right where it is loaded, and
// the move waits for the load there; called where the value is first needed,
// after a wait that already covers the load, the move costs nothing.
__device__ __forceinline__ uint64_t scalar_here(uint64_t v) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    asm volatile("" : "+v"(lo), "+v"(hi));
    lo = __builtin_amdgcn_readfirstlane(lo);
    hi = __builtin_amdgcn_readfirstlane(hi);
    return ((uint64_t)hi << 32) | lo;
}

// (the signal fences keep the compiler from moving memory accesses across it)
__device__ __forceinline__ void wait_stores_done() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ float shfl_xor_f(float x, int mask) {
    return __shfl_xor(x, mask, kWave);
}

// Merge of two online-softmax summaries in the log2 domain: (M, L) absorbs
// (m, l), where L = sum 2^(y - M).  Empty summaries carry M = -inf, L = 0.
__device__ __forceinline__ void ml_merge(float& M, float& L, float m, float l) {
    const float Mn = fmaxf(M, m);
    if (Mn == -INFINITY) return;
    L = L * fast_exp2(M - Mn) + l * fast_exp2(m - Mn);
    M = Mn;
}

__device__ __forceinline__ u32x4 ld_u32x4(const uint16_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
}
// The same load with the non-temporal hint, for K/V cache rows that are read
// once per call: it streams measurably faster than the default policy.
__device__ __forceinline__ u32x4 ld_stream_u32x4(const uint16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

}  // namespace ssl
