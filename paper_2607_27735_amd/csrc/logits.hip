// logits.hip -- token statistics of logit rows, around the decode hot path.
//
// Sec. 3.3 feeds the length controller with the entropy H_i of the drafter's
// output distribution for every drafted token; the verification stage of
// Sec. 2.1 keeps the drafted tokens the target model agrees with.  Both read
// vocabulary-sized logit rows once, so this is a bandwidth-bound row
// reduction: per row, the largest logit (lowest index on ties), and with
// p = softmax(x) the entropy -sum p ln p = ln S + M - T / S, where
// M = max x, S = sum e^(x - M), T = sum x e^(x - M).
//
// A row is cut into chunks of kChunk logits, one 256-thread workgroup each
// (32 logits per thread, 16-byte loads all in flight together), so that even
// the handful of rows of one decode step spread over many CUs.  A chunk's
// (M, S, T, argmax) is merged over lanes by shuffles and over waves through
// LDS in a fixed order.  Every chunk but the row's last publishes it with
// device-coherent stores, then its 64-bit call tag, and leaves; the last
// chunk's workgroup waits for the others (they have lower workgroup indices,
// were dispatched first and never wait; the wait is also bounded) and merges
// the chunks in order.  The greedy acceptance then runs as one small
// workgroup per sequence over the rows' argmax.
#include "device_common.h"
#include "launch.h"
#include "logit_common.h"

namespace ssl {
namespace {

constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Running statistics of a set of logits: max, sum e^(x - max), sum x e^(x - max)
// and the lowest index holding the max.
struct Stat {
    float m, s, t;
    int a;
};

__device__ __forceinline__ Stat merge(const Stat& p, const Stat& q) {
    const float m = fmaxf(p.m, q.m);
    if (m == -INFINITY) return p;   // both empty
    const float fp = fast_exp2((p.m - m) * kLog2e), fq = fast_exp2((q.m - m) * kLog2e);
    Stat r;
    r.m = m;
    r.s = p.s * fp + q.s * fq;
    r.t = p.t * fp + q.t * fq;
    r.a = (p.m > q.m || (p.m == q.m && p.a < q.a)) ? p.a : q.a;
    return r;
}

__device__ __forceinline__ Stat shfl_xor_stat(const Stat& x, int mask) {
    Stat r;
    r.m = __shfl_xor(x.m, mask, kWave);
    r.s = __shfl_xor(x.s, mask, kWave);
    r.t = __shfl_xor(x.t, mask, kWave);
    r.a = __shfl_xor(x.a, mask, kWave);
    return r;
}

__device__ __forceinline__ Stat wave_merge(Stat x) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) x = merge(x, shfl_xor_stat(x, o));
    return x;
}

// The (max, sum, sum x e, argmax) of thread tid's 32 logits of chunk `chunk`
// of a row (lc::load_chunk's layout).
template <bool kF32>
__device__ __forceinline__ Stat chunk_stat(const LogitArgs& a, int row, int chunk, int tid) {
    const char* base = static_cast<const char*>(a.logits) +
                       (size_t)row * a.row_stride * (kF32 ? 4 : 2);
    float x[32];
    lc::load_chunk<kF32>(base, a.vocab, chunk, tid, x);
    Stat st;
    st.m = -INFINITY;
    st.a = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        const int i = lc::elem<kF32>(chunk, q, tid);
        if (x[q] > st.m) {   // elements in increasing index order: the first max stays
            st.m = x[q];
            st.a = i;
        }
    }
    st.s = 0.f;
    st.t = 0.f;
    if (st.m != -INFINITY) {
#pragma unroll
        for (int q = 0; q < 32; ++q) {
            const float e = fast_exp2((x[q] - st.m) * kLog2e);   // 0 for masked elements
            st.s += e;
            st.t += x[q] == -INFINITY ? 0.f : x[q] * e;
        }
    }
    return st;
}

__device__ __forceinline__ void write_row(const LogitArgs& a, int row, const Stat& st) {
    if (a.entropy) a.entropy[row] = fast_log2(st.s) * kLn2 + st.m - st.t / st.s;
    if (a.argmax) a.argmax[row] = st.a;
}

template <bool kF32>
__global__ __launch_bounds__(kThreads) void logit_stats_kernel(LogitArgs a) {
    const int row = blockIdx.x / a.n_chunks, chunk = blockIdx.x - row * a.n_chunks;
    if (a.rows_per_seq > 0) {   // acceptance: rows past a sequence's k + 1 are not needed
        const int b = row / a.rows_per_seq, j = row - b * a.rows_per_seq;
        if (j > a.k_len[b]) return;
    }
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // The row's exchange epoch (exchange_tag), loaded before the logits so that
    // the wait for them covers its round trip; the last chunk advances it at
    // its end, when every other chunk has published, and so has read it.
    const uint64_t ep = a.epoch ? ld_dev64(a.epoch + row) : 0ull;
    __shared__ Stat ws[kThreads / kWave];
    Stat st = wave_merge(chunk_stat<kF32>(a, row, chunk, tid));
    if (lane == 0) ws[wave] = st;
    __syncthreads();
    if (wave != 0) return;
    st = ws[0];
#pragma unroll
    for (int w = 1; w < kThreads / kWave; ++w) st = merge(st, ws[w]);
    if (a.n_chunks == 1) {
        if (lane == 0) write_row(a, row, st);
        return;
    }
    const size_t slot = (size_t)row * a.n_chunks;
    const uint64_t epv = scalar_here(ep);
    const uint64_t want = exchange_tag(a.call_tag, epv);
    if (epoch_is_dirty(epv)) {   // an earlier captured call on this workspace gave up
        if (lane == 0) exchange_gave_up(a.xc, kStatusLogits, nullptr);
        return;
    }
    if (chunk + 1 < a.n_chunks) {   // publish and leave
        if (lane == 0) {
            st_dev64(reinterpret_cast<uint64_t*>(a.part + 4 * (slot + chunk)),
                     __builtin_bit_cast(uint64_t, make_float2(st.m, st.s)));
            st_dev64(reinterpret_cast<uint64_t*>(a.part + 4 * (slot + chunk)) + 1,
                     __builtin_bit_cast(uint64_t, make_float2(st.t, __builtin_bit_cast(float, st.a))));
            wait_stores_done();
            st_dev64(a.tag + slot + chunk, want ^ a.xc.tag_flip);
        }
        return;
    }
    // the row's last chunk: wait for the others, then merge all in chunk order
    // (lane c holds chunk c; the shuffle tree's order is fixed); if the bounded
    // wait gives up, the status word says so and the row is not written
    int spins = 0;
    bool all_in;
    const int c = min(lane, a.n_chunks - 2);
    do {
        all_in = __all(lane >= a.n_chunks - 1 || ld_dev64(a.tag + slot + c) == want);
        if (!all_in) __builtin_amdgcn_s_sleep(1);
    } while (!all_in && ++spins < a.xc.spin_limit);
    if (!all_in) {
        if (lane == 0) exchange_gave_up(a.xc, kStatusLogits, a.epoch ? a.epoch + row : nullptr);
        return;
    }
    Stat mine;
    const float2 ms = __builtin_bit_cast(float2, ld_dev64(reinterpret_cast<const uint64_t*>(a.part + 4 * (slot + c))));
    const float2 ta = __builtin_bit_cast(float2, ld_dev64(reinterpret_cast<const uint64_t*>(a.part + 4 * (slot + c)) + 1));
    mine.m = ms.x;
    mine.s = ms.y;
    mine.t = ta.x;
    mine.a = __builtin_bit_cast(int, ta.y);
    if (lane == a.n_chunks - 1) mine = st;
    if (lane >= a.n_chunks) {
        mine.m = -INFINITY;
        mine.s = 0.f;
        mine.t = 0.f;
        mine.a = 0x7fffffff;
    }
    mine = wave_merge(mine);
    if (lane == 0) {
        write_row(a, row, mine);
        if (a.epoch) epoch_advance(a.epoch + row);   // every other chunk has read it
    }
}

// Greedy acceptance: one wave per sequence over the argmax of its k + 1 rows.
__global__ __launch_bounds__(kWave) void greedy_accept_kernel(AcceptArgs a) {
    const int b = blockIdx.x, lane = threadIdx.x;
    const int k = a.k_len[b];
    const int* t = a.argmax + (size_t)b * (a.max_k + 1);
    const int tj = t[min(lane, k)];
    const bool agree = lane >= k || a.draft[(size_t)b * a.max_k + lane] == tj;
    const uint64_t bad = __ballot(!agree);
    const int m = bad ? __builtin_ctzll(bad) : k;
    const int next = __shfl(tj, m, kWave);
    if (lane == 0) {
        a.n_accepted[b] = m;
        a.next_token[b] = next;
    }
}

}  // namespace

hipError_t launch_logit_stats(const LogitArgs& a, bool f32, hipStream_t stream) {
    const dim3 grid(a.n_rows * a.n_chunks);
    if (f32)
        hipLaunchKernelGGL(logit_stats_kernel<true>, grid, dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(logit_stats_kernel<false>, grid, dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_greedy_accept(const AcceptArgs& a, int batch, hipStream_t stream) {
    hipLaunchKernelGGL(greedy_accept_kernel, dim3(batch), dim3(kWave), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ssl
