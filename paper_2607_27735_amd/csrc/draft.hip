// draft.hip -- draft-step attention over the gathered sparse view (Eq. 5).
//
// The gather is fused: K/V rows named by the index set are read in place from
// the dense cache, never copied.  A workgroup takes 128 consecutive entries of
// one (sequence, KV head)'s index list, one wave per 32; each wave keeps an
// online softmax per query head of the group (up to 16 heads = one MFMA row
// tile).  The four waves are merged through LDS into one partial output with
// its (max, sum) per head.  Every workgroup but the one of the unit's last
// chunk publishes that partial with device-coherent stores, then its 64-bit
// call tag, and leaves; the last chunk's workgroup waits for the other tags
// of its (sequence, KV head), merges all partials in chunk order (its own
// from LDS) and writes the output.
//
// A draft round (Sec. 3.1: k tokens drafted one after another over this view)
// runs the same kernel per step with entries that name either a fixed row (sink
// or TopK: through the index list, or from a compact copy made once per round
// by draft_materialize_kernel) or a row of the recent window, which has slid to
// end at the newest drafted token and is read straight from the cache.
//
// The tile math (gather, MFMA layouts, online softmax) is in draft_common.h.
#include "device_common.h"
#include "launch.h"
#include "draft_common.h"
#include "verify_common.h"

namespace ssl {
namespace {

using dc::Gathered;
using dc::RowSource;
using dc::draft_tile;
using dc::gather_tile;
using dc::kSelBit;
using dc::kTile;
constexpr int kRowCap = 16;
constexpr int kDraftWaves = 4;
constexpr int kDraftThreads = kDraftWaves * kWave;
constexpr int kParkStride = kHeadDim + 4;      // floats per parked head row
constexpr int kMergeBatch = 16;                // partials loaded at once by the merging workgroup

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

// Where an entry's row comes from: the index list (Eq. 5), or a draft-round
// step whose fixed rows come through the index list or from the materialized
// copy, and whose window rows are consecutive cache rows; each from the dense
// cache or through the block table of a paged one.
constexpr int kPlain = 0, kRoundIdx = 1, kRoundSel = 2, kPlainPaged = 3, kRoundIdxPaged = 4,
              kRoundSelPaged = 5;
constexpr bool mode_paged(int m) { return m == kPlainPaged || m == kRoundIdxPaged || m == kRoundSelPaged; }
constexpr bool mode_round(int m) { return m == kRoundIdx || m == kRoundSel || m == kRoundIdxPaged || m == kRoundSelPaged; }
constexpr bool mode_sel(int m) { return m == kRoundSel || m == kRoundSelPaged; }

// Row r of cache head kvc of sequence b: dense, an offset from the unit's
// base; paged, a row of the page pool (rows numbered over the whole pool).
template <bool kPaged>
__device__ __forceinline__ uint32_t cache_row(const DraftArgs& a, int b, int kvc, int r) {
    if (!kPaged) return (uint32_t)r;
    const int pg = a.block_table[(size_t)b * a.max_blocks + r / a.page_size];
    return (uint32_t)(((size_t)pg * a.n_kv_real + kvc) * a.page_size + r % a.page_size);
}

// TPW tiles of 32 entries per wave (4 * 32 * TPW entries per workgroup): a
// wave finds the rows of all its entries at once (64 per lane map), then
// gathers tile t + 1 while it computes tile t (a two-deep register ring; a
// third buffer measured no faster).  At most 256 registers per lane, so that
// a CU holds two workgroups even at four tiles per wave (the 8B batch-8
// workload's draft: 46.7 -> 25.8 us with both, from 1 tile per wave).
template <int kMode, int TPW>
__global__ __launch_bounds__(kDraftThreads, 2) void draft_kernel(DraftArgs a) {
    const DItem it = decode_ditem(a.seq, blockIdx.x, a.n_kv_heads, a.chunk);
    // (read here, outside the wave-dependent branch below, so that they are
    // scalar loads and not vector loads that the index load waits for)
    const int nf = mode_round(kMode) ? a.n_fixed[it.b] : 0;
    const int win0 = mode_round(kMode) ? a.win0[it.b] : 0;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m16 = lane & 15, G = lane >> 4;
    const int g = a.group;
    // The unit's exchange epoch (exchange_tag), loaded first so that the
    // waits for the index loads cover its round trip; the last chunk advances
    // it at its end, when every other chunk has published, and so has read it.
    const uint64_t ep = a.epoch ? ld_dev64(a.epoch + it.unit) : 0ull;

    __shared__ int wait_failed;
    __shared__ float2 wml[kDraftWaves][kRowCap];
    __shared__ float2 gml[kRowCap];
    __shared__ float park[kDraftWaves][kRowCap][kParkStride];

    // ---- one wave: 32 * TPW entries of the index list -----------------------
    const int wbeg = it.key_begin + wave * kTile * TPW;
    const int wend = min(wbeg + kTile * TPW, it.key_end);
    float M = -INFINITY, L = 0.f;
    f32x4 oacc[8];
#pragma unroll
    for (int jd = 0; jd < 8; ++jd) oacc[jd] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (wbeg < wend) {
        u32x4 qop[4];
        if (m16 < g) {
            const uint16_t* qp =
                a.q + ((size_t)it.b * a.n_q_heads + it.c * g + m16) * kHeadDim + 8 * G;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) qop[kb] = ld_u32x4(qp + 32 * kb);
        } else {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) qop[kb] = u32x4{0u, 0u, 0u, 0u};
        }
        // (paged: rows are numbered over the whole page pool; per-head units
        // read the rows of cache head it.c / kv_div)
        const int kvc = it.c / a.kv_div;
        const size_t cache_off = mode_paged(kMode)
            ? 0 : ((size_t)it.b * a.n_kv_real + kvc) * a.max_ctx * kHeadDim;
        const size_t sel_off = (size_t)it.unit * a.budget * kHeadDim;
        const RowSource src{a.k + cache_off, a.v + cache_off, a.k_sel + sel_off, a.v_sel + sel_off};
        const int last = it.n - 1;
        // Lane l of map j finds the row of entry 64 j + l once; every K/V row
        // of a tile is then requested at once.
        constexpr int kMaps = (TPW + 1) / 2;
        int32_t raw[kMaps];
#pragma unroll
        for (int j = 0; j < kMaps; ++j) {   // all index loads in flight together
            const int e = min(wbeg + 64 * j + lane, last);
            raw[j] = !mode_sel(kMode) ? a.idx[(size_t)it.unit * a.budget + e] : 0;
        }
        uint32_t my_row[kMaps];
#pragma unroll
        for (int j = 0; j < kMaps; ++j) {
            const int e = min(wbeg + 64 * j + lane, last);
            constexpr bool kPg = mode_paged(kMode);
            if (!mode_round(kMode)) {
                my_row[j] = cache_row<kPg>(a, it.b, kvc, min(max(raw[j], 0), a.max_ctx - 1));
            } else {
                // (the index load does not wait for n_fixed: entry e < budget is
                // in bounds, and its value is used only when e < n_fixed)
                const int r = e < nf ? min(max(raw[j], 0), a.max_ctx - 1)
                                     : min(max(win0 + e - nf, 0), a.max_ctx - 1);
                my_row[j] = (mode_sel(kMode) && e < nf) ? (uint32_t)e | kSelBit
                                                        : cache_row<kPg>(a, it.b, kvc, r);
            }
        }
        const int ntile = (wend - wbeg + kTile - 1) / kTile;   // wave-uniform
        vc::tile_pipeline<2, Gathered>(
            0, ntile, 1,
            [&](Gathered& t, int tile) {
                uint32_t r = my_row[0];
#pragma unroll
                for (int j = 1; j < kMaps; ++j) r = (tile >> 1) == j ? my_row[j] : r;
                gather_tile<mode_sel(kMode)>(r, 32 * (tile & 1), src, m16, G, t);
            },
            [&](const Gathered& t, int tile) {
                draft_tile(a.scale_log2, qop, t, wbeg + kTile * tile, wend, G, M, L, oacc);
            });
        L += shfl_xor_f(L, 16);
        L += shfl_xor_f(L, 32);
    }

    // ---- merge the four waves (fixed order) --------------------------------
    // (every lane takes its head's maximum over the waves straight from wml;
    // the first 16 threads also keep the merged (max, sum))
    if (G == 0) wml[wave][m16] = make_float2(M, L);
    __syncthreads();
    if (tid < kRowCap) {
        float Mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < kDraftWaves; ++w) Mx = fmaxf(Mx, wml[w][tid].x);
        float Lx = 0.f;
#pragma unroll
        for (int w = 0; w < kDraftWaves; ++w)
            Lx += wml[w][tid].x == -INFINITY ? 0.f : wml[w][tid].y * fast_exp2(wml[w][tid].x - Mx);
        gml[tid] = make_float2(Mx, Lx);
    }
    {
        float Mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < kDraftWaves; ++w) Mx = fmaxf(Mx, wml[w][m16].x);
        const float f = M == -INFINITY ? 0.f : fast_exp2(M - Mx);
        float* dst = &park[wave][m16][0];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = 32 * G + 8 * i;
            *reinterpret_cast<f32x4*>(dst + c) =
                f32x4{oacc[0][i], oacc[1][i], oacc[2][i], oacc[3][i]} * f;
            *reinterpret_cast<f32x4*>(dst + c + 4) =
                f32x4{oacc[4][i], oacc[5][i], oacc[6][i], oacc[7][i]} * f;
        }
    }
    __syncthreads();

    // ---- every chunk but the unit's last publishes its partial and leaves ----
    const size_t wg = blockIdx.x;
    const bool finisher = it.key_begin + a.chunk >= it.n;   // the unit's last chunk
    const uint64_t epv = scalar_here(ep);
    const uint64_t want = exchange_tag(a.call_tag, epv);
    if (epoch_is_dirty(epv)) {   // an earlier captured call on this workspace gave up
        if (tid == 0) exchange_gave_up(a.xc, kStatusDraft, nullptr);
        return;
    }
    if (!finisher) {
        for (int x = tid; x < g * (kHeadDim / 2); x += kDraftThreads) {
            const int row = x / (kHeadDim / 2), c2 = x - row * (kHeadDim / 2);
            float2 o = *reinterpret_cast<const float2*>(&park[0][row][2 * c2]);
#pragma unroll
            for (int w = 1; w < kDraftWaves; ++w) {
                const float2 v = *reinterpret_cast<const float2*>(&park[w][row][2 * c2]);
                o.x += v.x;
                o.y += v.y;
            }
            st_dev64(reinterpret_cast<uint64_t*>(a.part_o + (wg * kRowCap + row) * kHeadDim) + c2,
                     __builtin_bit_cast(uint64_t, o));
        }
        if (tid < g)
            st_dev64(reinterpret_cast<uint64_t*>(a.part_ml + wg * kRowCap + tid),
                     __builtin_bit_cast(uint64_t, gml[tid]));
        wait_stores_done();
        __syncthreads();
        if (tid == 0) st_dev64(a.tag + wg, want ^ a.xc.tag_flip);
        return;
    }
    // The last chunk waits for the others: they have lower workgroup indices,
    // so they were dispatched first, and they never wait.  The wait is also
    // bounded: if it gives up, the status word says so and no output is written.
    if (wave == 0) {
        int spins = 0;
        bool all_in;
        do {
            bool in = true;
            for (int j = lane; j < it.nchunk - 1; j += kWave) in &= ld_dev64(a.tag + it.item0 + j) == want;
            all_in = __all(in);
            if (!all_in) __builtin_amdgcn_s_sleep(1);
        } while (!all_in && ++spins < a.xc.spin_limit);
        if (lane == 0) wait_failed = !all_in;
    }
    __syncthreads();
    if (wait_failed) {
        if (tid == 0) exchange_gave_up(a.xc, kStatusDraft, a.epoch ? a.epoch + it.unit : nullptr);
        return;
    }

    // ---- merge the partials of every head, in chunk order ---------------------
    for (int x = tid; x < g * (kHeadDim / 4); x += kDraftThreads) {
        const int row = x >> 5, d4 = x & 31;
        float Mx = -INFINITY, Lx = 0.f;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int j0 = 0; j0 < it.nchunk; j0 += kMergeBatch) {
            float2 ml[kMergeBatch];
            f32x4 o[kMergeBatch];
#pragma unroll
            for (int uu = 0; uu < kMergeBatch; ++uu) {
                const int j = j0 + uu;
                if (j + 1 < it.nchunk) {
                    const size_t slot = (size_t)(it.item0 + j) * kRowCap + row;
                    ml[uu] = __builtin_bit_cast(float2, ld_dev64(reinterpret_cast<const uint64_t*>(a.part_ml + slot)));
                    const uint64_t* po = reinterpret_cast<const uint64_t*>(a.part_o + slot * kHeadDim) + 2 * d4;
                    const float2 flo = __builtin_bit_cast(float2, ld_dev64(po));
                    const float2 fhi = __builtin_bit_cast(float2, ld_dev64(po + 1));
                    o[uu] = f32x4{flo.x, flo.y, fhi.x, fhi.y};
                } else if (j + 1 == it.nchunk) {   // this workgroup's own partial
                    ml[uu] = gml[row];
                    f32x4 ov = *reinterpret_cast<const f32x4*>(&park[0][row][4 * d4]);
#pragma unroll
                    for (int w = 1; w < kDraftWaves; ++w) ov += *reinterpret_cast<const f32x4*>(&park[w][row][4 * d4]);
                    o[uu] = ov;
                } else {
                    ml[uu] = make_float2(-INFINITY, 0.f);
                    o[uu] = f32x4{0.f, 0.f, 0.f, 0.f};
                }
            }
            float Mn = Mx;
#pragma unroll
            for (int uu = 0; uu < kMergeBatch; ++uu) Mn = fmaxf(Mn, ml[uu].x);
            const float alpha = Mx == -INFINITY ? 0.f : fast_exp2(Mx - Mn);
            Lx *= alpha;
            acc *= alpha;
#pragma unroll
            for (int uu = 0; uu < kMergeBatch; ++uu) {
                const float wgt = ml[uu].x == -INFINITY ? 0.f : fast_exp2(ml[uu].x - Mn);
                Lx += ml[uu].y * wgt;
                acc += o[uu] * wgt;
            }
            Mx = Mn;
        }
        acc *= 1.0f / Lx;
        const int h = it.c * g + row;
        const size_t base = ((size_t)it.b * a.n_q_heads + h) * kHeadDim + 4 * d4;
        if (a.out_fp32) {
            *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + base) = acc;
        } else {
            uint2 pk = make_uint2(pack_bf16(acc[0], acc[1]), pack_bf16(acc[2], acc[3]));
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + base) = pk;
        }
    }
    // every other chunk has published, so has read the epoch; advanced last,
    // after the workgroup's final wait for loads
    if (a.epoch && tid == 0 && it.nchunk > 1) epoch_advance(a.epoch + it.unit);
}

// Materialization for a draft round: workgroup (x, u) copies rows
// 32x .. 32x + 31 of unit u's sink and TopK entries (the first n_fixed[b]
// entries of its index list) from the cache (dense, or paged through the
// block table) to k_sel/v_sel (a unit per query head reads the rows of its KV
// head).  Thread t moves 16 bytes of two rows of K and of V, all four loads
// in flight together.
constexpr int kMatRows = 32;
template <bool kPaged>
__global__ __launch_bounds__(kDraftThreads) void draft_materialize_kernel(DraftArgs a) {
    const int u = blockIdx.y, b = u / a.n_kv_heads;
    const int nf = a.n_fixed[b];
    const int q = threadIdx.x & 15, r = threadIdx.x >> 4;   // 16 rows per pass
    const int32_t* ib = a.idx + (size_t)u * a.budget;
    const int kvc = (u - b * a.n_kv_heads) / a.kv_div;
    const size_t cache_off = kPaged ? 0 : ((size_t)b * a.n_kv_real + kvc) * a.max_ctx * kHeadDim;
    const size_t sel_off = (size_t)u * a.budget * kHeadDim;
    int e[2];
    u32x4 kk[2], vv[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        e[j] = blockIdx.x * kMatRows + 16 * j + r;
        const int row = cache_row<kPaged>(a, b, kvc, min(max(ib[min(e[j], max(nf - 1, 0))], 0), a.max_ctx - 1));
        kk[j] = ld_u32x4(a.k + cache_off + (size_t)row * kHeadDim + 8 * q);
        vv[j] = ld_u32x4(a.v + cache_off + (size_t)row * kHeadDim + 8 * q);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        if (e[j] < nf) {
            *reinterpret_cast<u32x4*>(a.k_sel + sel_off + (size_t)e[j] * kHeadDim + 8 * q) = kk[j];
            *reinterpret_cast<u32x4*>(a.v_sel + sel_off + (size_t)e[j] * kHeadDim + 8 * q) = vv[j];
        }
    }
}

template <int kMode>
void launch_mode(const DraftArgs& a, int n_items, hipStream_t stream) {
    switch (a.chunk / (kDraftWaves * kTile)) {
        case 4:
            hipLaunchKernelGGL((draft_kernel<kMode, 4>), dim3(n_items), dim3(kDraftThreads), 0, stream, a);
            break;
        case 2:
            hipLaunchKernelGGL((draft_kernel<kMode, 2>), dim3(n_items), dim3(kDraftThreads), 0, stream, a);
            break;
        default:
            hipLaunchKernelGGL((draft_kernel<kMode, 1>), dim3(n_items), dim3(kDraftThreads), 0, stream, a);
            break;
    }
}

}  // namespace

int draft_chunk_for(int64_t entries, int n_cu) {
    // the most tiles per wave that still leave a workgroup per CU
    for (int tpw = 4; tpw > 1; tpw >>= 1)
        if (entries / ((int64_t)kDraftWaves * kTile * tpw) >= (int64_t)n_cu)
            return kDraftWaves * kTile * tpw;
    return kDraftWaves * kTile;
}

hipError_t launch_draft(const DraftArgs& a, int n_items, hipStream_t stream) {
    if (a.block_table)
        launch_mode<kPlainPaged>(a, n_items, stream);
    else
        launch_mode<kPlain>(a, n_items, stream);
    return hipGetLastError();
}

hipError_t launch_draft_step(const DraftArgs& a, int n_items, hipStream_t stream) {
    if (a.block_table) {
        if (a.k_sel)
            launch_mode<kRoundSelPaged>(a, n_items, stream);
        else
            launch_mode<kRoundIdxPaged>(a, n_items, stream);
    } else {
        if (a.k_sel)
            launch_mode<kRoundSel>(a, n_items, stream);
        else
            launch_mode<kRoundIdx>(a, n_items, stream);
    }
    return hipGetLastError();
}

hipError_t launch_draft_materialize(const DraftArgs& a, int max_fixed, int n_units,
                                    hipStream_t stream) {
    const int blocks = (max_fixed + kMatRows - 1) / kMatRows;
    if (blocks < 1 || n_units < 1) return hipSuccess;
    if (a.block_table)
        hipLaunchKernelGGL(draft_materialize_kernel<true>, dim3(blocks, n_units),
                           dim3(kDraftThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(draft_materialize_kernel<false>, dim3(blocks, n_units),
                           dim3(kDraftThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ssl
