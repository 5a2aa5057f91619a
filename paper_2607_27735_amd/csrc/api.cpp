// api.cpp -- the C ABI: argument validation, work decomposition, launches.
//
// Every check runs on the host before the first HIP call, so a rejected call
// leaves the device untouched and is testable without a GPU.
#include <math.h>
#include <string.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>

#include "../../include/sparsespec_l.h"
#include "launch.h"

using namespace ssl;

static_assert((uint32_t)SSL_EXCHANGE_VERIFY == kStatusVerify &&
                  (uint32_t)SSL_EXCHANGE_SELECT == kStatusSelect &&
                  (uint32_t)SSL_EXCHANGE_DRAFT == kStatusDraft &&
                  (uint32_t)SSL_EXCHANGE_LOGITS == kStatusLogits,
              "status bits of the ABI and the kernels agree");

namespace {

constexpr size_t kAlign = 256;
constexpr int kVerifyRowCap = 64;
constexpr int kDraftRowCap = 16;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// The HIP error behind this thread's last SSL_ERR_HIP (ssl_last_hip_error).
thread_local hipError_t t_last_hip = hipSuccess;

// SSL_OK for hipSuccess; otherwise records e and returns SSL_ERR_HIP.
int hip_rc(hipError_t e) {
    if (e == hipSuccess) return SSL_OK;
    t_last_hip = e;
    return SSL_ERR_HIP;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int check_shape(const ssl_shape* s) {
    if (!s) return SSL_ERR_NULL;
    if (s->batch < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->max_ctx < 1 || s->max_q < 1)
        return SSL_ERR_SHAPE;
    if (s->n_q_heads % s->n_kv_heads != 0) return SSL_ERR_SHAPE;
    if (s->head_dim != 128) return SSL_ERR_UNSUPPORTED;
    if (s->batch > kTableBatch) return SSL_ERR_UNSUPPORTED;
    return SSL_OK;
}

int check_budget(const ssl_params* p) {
    if (!p) return SSL_ERR_NULL;
    if (p->budget < 1 || p->k_sink < 0 || p->k_recent < 0) return SSL_ERR_BUDGET;
    if ((int64_t)p->k_sink + p->k_recent > p->budget) return SSL_ERR_BUDGET;
    if (p->per_head != 0 && p->per_head != 1) return SSL_ERR_SHAPE;
    return SSL_OK;
}

// One index set per query head: select and draft work on units (sequence,
// query head), each reading the cache rows of KV head h / group.
ssl_shape unit_shape(const ssl_shape* s, const ssl_params* p) {
    ssl_shape u = *s;
    if (p->per_head) u.n_kv_heads = s->n_q_heads;
    return u;
}

// Verify work decomposition.  Two-sweep items are (sequence, KV head, key
// chunk); the one-sweep schedule uses the same kind of items ("slots"), all
// resident at once.  The workspace holds per-item row statistics and partial
// outputs for whichever schedule needs more, plus the one-sweep tags.
constexpr int kFusedMaxSlotsPerUnit = 128;

// A 64-bit mixing function (the 64-bit finaliser of Appleby's MurmurHash3).
uint64_t mix64(uint64_t x) {
    x ^= x >> 33;
    x *= 0xff51afd7ed558ccdull;
    x ^= x >> 33;
    x *= 0xc4ceb9fe1a85ec53ull;
    x ^= x >> 33;
    return x;
}

// One-sweep publication tags: a process-wide sequence whose start mixes the
// clock and the process id, so that tags differ between calls and, with
// overwhelming probability, from whatever a workspace held before.
uint64_t next_call_tag() {
    static std::atomic<uint64_t> seq{mix64(
        (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count() ^
        ((uint64_t)getpid() << 32))};
    return seq.fetch_add(1, std::memory_order_relaxed) + 1;
}

// The workspace's exchange epochs (its first kEpochWords words, one per
// exchange group), passed to the kernels only when the launch is being
// captured into a graph: every replay of a captured launch repeats its call
// tag, and the epochs give each replay a new exchange tag.  Eager launches
// have a new call tag each and skip the epochs' load and advance.  If the
// query fails, its error is cleared and the epochs are used.  A captured call
// with more exchange groups than epoch words is refused.
int epochs_if_captured(hipStream_t stream, void* ws, int64_t n_groups, uint64_t** epochs) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &st) != hipSuccess) {
        (void)hipGetLastError();
        st = hipStreamCaptureStatusActive;
    }
    *epochs = nullptr;
    if (st == hipStreamCaptureStatusNone) return SSL_OK;
    if (n_groups > kEpochWords) return SSL_ERR_UNSUPPORTED;
    *epochs = static_cast<uint64_t*>(ws);
    return SSL_OK;
}

// Process-wide settings: the CU count plans assume (0: the device's own), and
// the test hook that makes every exchange wait give up.
std::atomic<int32_t> g_cu_budget{0};
std::atomic<int32_t> g_spin_limit{0};      // 0: kDefaultSpinLimit
std::atomic<uint64_t> g_tag_flip{0};

// What an exchanging kernel needs besides its data (the device's status word
// is looked up once per device).
int make_exchange(Exchange* xc) {
    uint32_t* word = nullptr;
    if (const int hip_st = hip_rc(exchange_status_word(&word))) return hip_st;
    xc->status = word;
    xc->tag_flip = g_tag_flip.load(std::memory_order_relaxed);
    const int32_t lim = g_spin_limit.load(std::memory_order_relaxed);
    xc->spin_limit = lim > 0 ? lim : kDefaultSpinLimit;
    return SSL_OK;
}

// Compute units the plans may count on: the caller's budget if one is set,
// else the current device's count (read once per device), else 256 (the
// MI355X's count) when no device can be queried.
constexpr int kDefaultCUs = 256;
int device_cus() {
    const int32_t budget = g_cu_budget.load(std::memory_order_relaxed);
    if (budget > 0) return budget;
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cus[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return kDefaultCUs;
    }
    const bool cached = dev >= 0 && dev < kMaxDevices;
    int n = cached ? cus[dev].load(std::memory_order_relaxed) : 0;
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) {
            (void)hipGetLastError();
            return kDefaultCUs;
        }
        if (cached) cus[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Exchange groups whose members must all be resident at once get at most half
// of what the device holds (blocks_per_cu workgroups on each CU; 1 when the
// device cannot be queried), which leaves room for an uneven spread of the
// group over the chip's dies.
int64_t resident_group_cap(int blocks_per_cu) {
    return std::max<int64_t>(1, (int64_t)device_cus() * std::max(blocks_per_cu, 1) / 2);
}

struct VerifyPlan {
    int chunk, n_items, n_rows, row_tiles;
    int block_pos;   // verify positions per launch (row blocks); >= every q_len when one block
    bool fused_ok;
    int fused_chunk, fused_slots;
    bool one_round;  // the one-workgroup-per-chunk one sweep runs in one round of workgroups
    bool pipe;       // one sweep by the persistent kernel: fused_slots chunks over pipe_grid workgroups
    int pipe_grid;
    size_t ml_off, o_off, bytes;
    SeqTable seq;
    SeqTable fseq;   // the one-sweep slots as items
};

int plan_verify(const ssl_shape* s, const ssl_params* p, const int32_t* ctx, const int32_t* ql,
                VerifyPlan* plan) {
    int rc = check_shape(s);
    if (rc) return rc;
    if (!p) return SSL_ERR_NULL;
    if (!ctx || !ql) return SSL_ERR_NULL;
    if (s->max_q > 64) return SSL_ERR_SHAPE;
    if (p->window < 1 || !(p->sm_scale > 0.f) || !isfinite(p->sm_scale)) return SSL_ERR_SHAPE;
    if (p->verify_mode < SSL_VERIFY_AUTO || p->verify_mode > SSL_VERIFY_ONE_SWEEP)
        return SSL_ERR_SHAPE;
    const int g = s->n_q_heads / s->n_kv_heads;
    int64_t total_keys = 0;
    int max_rows = 0;
    for (int b = 0; b < s->batch; ++b) {
        if (ql[b] < 1 || ql[b] > ctx[b] || ctx[b] > s->max_ctx || ql[b] > s->max_q)
            return SSL_ERR_SHAPE;
        max_rows = std::max(max_rows, ql[b] * g);
        total_keys += (int64_t)ctx[b] * s->n_kv_heads;
    }
    // More rows per KV head than one launch holds (e.g. Eq. 3 over the last
    // W = 16 prompt positions of a group of 8): the two-sweep schedule runs
    // once per block of positions, the scores of later blocks added.
    if (g > kVerifyRowCap) return SSL_ERR_UNSUPPORTED;
    plan->block_pos = kVerifyRowCap / g;
    if (max_rows > kVerifyRowCap) {
        if (p->verify_mode == SSL_VERIFY_ONE_SWEEP) return SSL_ERR_UNSUPPORTED;
        max_rows = plan->block_pos * g;
    } else {
        plan->block_pos = s->max_q;
    }
    plan->row_tiles = (max_rows + 15) / 16;

    // Two-sweep chunk: the power of two in [128, 65536] that minimises
    // rounds * (chunk + 256), a round being one item per CU: each round of
    // workgroups costs the CUs a drain and a ramp, about 256 keys' streaming
    // (at 131K and the 70B shape, one round of 4096- / 8192-key items took
    // 140 / 265 us against 154 / 316 us for two and four rounds of 2048).
    const int64_t n_cu = device_cus();
    int chunk = 128;
    {
        int64_t best = -1;
        for (int64_t c = 128; c <= 65536; c *= 2) {
            int64_t n = 0;
            for (int b = 0; b < s->batch; ++b) n += (int64_t)s->n_kv_heads * ((ctx[b] + c - 1) / c);
            const int64_t cost = (n + n_cu - 1) / n_cu * (c + 256);
            if (best < 0 || cost < best) {
                best = cost;
                chunk = (int)c;
            }
        }
    }
    memset(&plan->seq, 0, sizeof plan->seq);
    plan->seq.n_seq = s->batch;
    int64_t items = 0, rows = 0;
    for (int b = 0; b < s->batch; ++b) {
        plan->seq.item_start[b] = (int32_t)items;
        plan->seq.row_start[b] = (int32_t)rows;
        plan->seq.ctx[b] = ctx[b];
        plan->seq.qlen[b] = ql[b];
        items += (int64_t)s->n_kv_heads * ((ctx[b] + chunk - 1) / chunk);
        rows += (int64_t)s->n_kv_heads * std::min(ql[b], plan->block_pos) * g;
    }
    if (items > (1 << 30) || rows > (1 << 30)) return SSL_ERR_UNSUPPORTED;
    plan->seq.item_start[s->batch] = (int32_t)items;
    plan->seq.row_start[s->batch] = (int32_t)rows;
    plan->chunk = chunk;
    plan->n_items = (int)items;
    plan->n_rows = (int)rows;

    // One-sweep: chunks (multiples of 128 keys, at most what the LDS logit
    // stash holds) of about one slot per CU over the whole call, but never
    // more slots per (sequence, KV head) than can be resident together: at
    // most kFusedMaxSlotsPerUnit, and at most half of what the device's CUs
    // hold at once.
    plan->fused_ok = false;
    plan->fused_slots = 0;
    plan->fused_chunk = 0;
    const int cap = fused_max_chunk(plan->row_tiles);
    const int64_t max_slots =
        std::min<int64_t>(kFusedMaxSlotsPerUnit, resident_group_cap(fused_blocks_per_cu(plan->row_tiles)));
    int max_ctx = 0;
    for (int b = 0; b < s->batch; ++b) max_ctx = std::max(max_ctx, ctx[b]);
    const int64_t per_unit_min = ((int64_t)max_ctx + max_slots - 1) / max_slots;
    const int64_t spread = (total_keys + n_cu - 1) / n_cu;
    int64_t fc = std::max(per_unit_min, spread);
    fc = std::max<int64_t>(128, (fc + 127) / 128 * 128);
    if (fc > cap) fc = cap / 128 * 128;
    if (plan->block_pos >= s->max_q && fc >= 128 && ((int64_t)max_ctx + fc - 1) / fc <= max_slots) {
        int64_t slots = 0;
        plan->fseq = plan->seq;
        for (int b = 0; b < s->batch; ++b) {
            plan->fseq.item_start[b] = (int32_t)slots;
            slots += (int64_t)s->n_kv_heads * ((ctx[b] + fc - 1) / fc);
        }
        if (slots <= (1 << 30)) {
            plan->fseq.item_start[s->batch] = (int32_t)slots;
            plan->fused_ok = true;
            plan->fused_chunk = (int)fc;
            plan->fused_slots = (int)slots;
        }
    }
    // Persistent one sweep, where the chunks above would take more than one
    // round of workgroups (or do not fit at all) and a KV head has at most 48
    // rows: a grid of what the device holds at once (the whole grid must be
    // resident), each workgroup taking every grid-th chunk of a 16-bit stash
    // size, a unit's chunks within two consecutive rounds (at most one grid
    // of them) and at most kPipeMaxChunksPerUnit of them (every chunk's finish
    // loads each chunk's statistics and its rows' partials in passes of 32
    // chunks, one round trip each: at 103 and 256 chunks per unit the call
    // measured slower than two sweeps).  The chunk is the one that minimises
    // rounds * (chunk + 96): a round costs about 96 keys' streaming besides
    // its own keys.
    constexpr int64_t kPipeMaxChunksPerUnit = 64;
    plan->pipe = false;
    plan->pipe_grid = 0;
    const int64_t resident1 = n_cu * std::max(fused_blocks_per_cu(plan->row_tiles), 1);
    const bool one_round = plan->fused_ok && plan->fused_slots <= resident1;
    plan->one_round = one_round;
    // (pipe_max_chunk is 0 where the persistent kernel is not built: > 48 rows)
    if (!one_round && plan->block_pos >= s->max_q) {
        const int64_t grid_cap = n_cu * std::max(pipe_blocks_per_cu(plan->row_tiles), 1);
        int64_t best_cost = -1, best_chunk = 0, best_tasks = 0;
        for (int64_t pc = pipe_max_chunk(plan->row_tiles); pc >= 128; pc -= 128) {
            int64_t tasks = 0;
            for (int b = 0; b < s->batch; ++b) tasks += (int64_t)s->n_kv_heads * ((ctx[b] + pc - 1) / pc);
            const int64_t grid = std::min(tasks, grid_cap);
            const int64_t per_unit = (max_ctx + pc - 1) / pc;
            if (per_unit > grid || per_unit > kPipeMaxChunksPerUnit || tasks > (1 << 30)) continue;
            const int64_t cost = (tasks + grid - 1) / grid * (pc + 96);
            if (best_cost < 0 || cost < best_cost) {
                best_cost = cost;
                best_chunk = pc;
                best_tasks = tasks;
            }
        }
        if (best_cost >= 0) {
            plan->fseq = plan->seq;
            int64_t slots = 0;
            for (int b = 0; b < s->batch; ++b) {
                plan->fseq.item_start[b] = (int32_t)slots;
                slots += (int64_t)s->n_kv_heads * ((ctx[b] + best_chunk - 1) / best_chunk);
            }
            plan->fseq.item_start[s->batch] = (int32_t)slots;
            plan->fused_ok = true;
            plan->fused_chunk = (int)best_chunk;
            plan->fused_slots = (int)best_tasks;
            plan->pipe = true;
            plan->pipe_grid = (int)std::min(best_tasks, grid_cap);
        }
    }
    if (p->verify_mode == SSL_VERIFY_ONE_SWEEP && !plan->fused_ok) return SSL_ERR_UNSUPPORTED;
    const size_t slots_max = (size_t)std::max(plan->n_items, plan->fused_slots);
    // per item and row: (max, sum), each word tagged in the one-sweep schedule
    plan->ml_off = kEpochBytes;
    plan->o_off = plan->ml_off + align_up(slots_max * kVerifyRowCap * sizeof(uint64_t) * 2);
    plan->bytes = plan->o_off + align_up(slots_max * kVerifyRowCap * 128 * sizeof(float));
    return SSL_OK;
}

// AUTO takes one sweep where it fits and a KV head has at most 32 verify rows,
// or more when it runs in one round of workgroups or (up to 48 rows) in the
// persistent form; over several rounds at 33-64 rows (one wave per SIMD,
// logits of every row in LDS) the one-workgroup-per-chunk kernel waits
// across rounds and two sweeps are faster (70B shape: 457 vs 336 us), while
// in one round it wins (44 rows at 16K: 26.1 vs 36.5 us; 48 rows at 8K: 21.8
// vs 29.6 us; 64 rows at 8K: 25.2 vs 34.0 us).
bool use_one_sweep(const VerifyPlan& plan, const ssl_params* p) {
    if (!plan.fused_ok || p->verify_mode == SSL_VERIFY_TWO_SWEEP) return false;
    return p->verify_mode == SSL_VERIFY_ONE_SWEEP || plan.row_tiles <= 2 || plan.pipe || plan.one_round;
}

struct DraftPlan {
    int chunk, n_items, n_rows, n_units;
    size_t ml_off, o_off, tag_off, bytes;
    SeqTable seq;
};

int plan_draft(const ssl_shape* s, const ssl_params* p, const int32_t* n_idx, DraftPlan* plan) {
    int rc = check_shape(s);
    if (rc) return rc;
    rc = check_budget(p);
    if (rc) return rc;
    if (!n_idx) return SSL_ERR_NULL;
    if (!(p->sm_scale > 0.f) || !isfinite(p->sm_scale)) return SSL_ERR_SHAPE;
    const int g = s->n_q_heads / s->n_kv_heads;
    if (g > kDraftRowCap) return SSL_ERR_UNSUPPORTED;
    memset(&plan->seq, 0, sizeof plan->seq);
    plan->seq.n_seq = s->batch;
    int64_t entries = 0;
    for (int b = 0; b < s->batch; ++b) {
        if (n_idx[b] < 1 || n_idx[b] > p->budget) return SSL_ERR_SHAPE;
        entries += (int64_t)n_idx[b] * s->n_kv_heads;
    }
    const int chunk = draft_chunk_for(entries, device_cus());
    int64_t items = 0;
    for (int b = 0; b < s->batch; ++b) {
        plan->seq.item_start[b] = (int32_t)items;
        plan->seq.ctx[b] = n_idx[b];
        items += (int64_t)s->n_kv_heads * ((n_idx[b] + chunk - 1) / chunk);
    }
    if (items > (1 << 30)) return SSL_ERR_UNSUPPORTED;
    plan->seq.item_start[s->batch] = (int32_t)items;
    plan->chunk = chunk;
    plan->n_items = (int)items;
    plan->n_rows = s->batch * s->n_q_heads;
    plan->n_units = s->batch * s->n_kv_heads;
    plan->ml_off = kEpochBytes;
    plan->o_off = plan->ml_off + align_up((size_t)items * kDraftRowCap * sizeof(float) * 2);
    plan->tag_off = plan->o_off + align_up((size_t)items * kDraftRowCap * 128 * sizeof(float));
    plan->bytes = plan->tag_off + align_up((size_t)items * sizeof(uint64_t));
    return SSL_OK;
}

// A draft-round step over the index set built at T = ctx[b]: the sink and
// TopK entries (n_fixed of them) stay, the recent window slides to end at
// cur[b].  Entry counts per sequence go to the plan's seq table.
struct StepPlan {
    DraftPlan d;
    int32_t n_fixed[kTableBatch];
    int32_t win0[kTableBatch];
    int max_fixed;
};

int plan_draft_step(const ssl_shape* s, const ssl_params* p, const int32_t* ctx,
                    const int32_t* cur, StepPlan* plan) {
    int rc = check_shape(s);
    if (rc) return rc;
    rc = check_budget(p);
    if (rc) return rc;
    if (!ctx || !cur) return SSL_ERR_NULL;
    int32_t n_step[kTableBatch];
    plan->max_fixed = 0;
    for (int b = 0; b < s->batch; ++b) {
        const int32_t T = ctx[b], c = cur[b];
        if (T < 1 || c < T || c > s->max_ctx || (int64_t)c - T > p->k_recent) return SSL_ERR_SHAPE;
        const int32_t n = ssl_index_count(T, p->k_sink, p->k_recent, p->budget);
        const int32_t s_end = std::min(p->k_sink, T);
        const int32_t r_T = std::max(T - p->k_recent, s_end);
        plan->n_fixed[b] = n - (T - r_T);
        plan->win0[b] = std::max(r_T, c - p->k_recent);
        n_step[b] = plan->n_fixed[b] + (c - plan->win0[b]);
        plan->max_fixed = std::max(plan->max_fixed, plan->n_fixed[b]);
    }
    return plan_draft(s, p, n_step, &plan->d);
}

int check_select(const ssl_shape* s, const ssl_params* p, const int32_t* ctx) {
    int rc = check_shape(s);
    if (rc) return rc;
    rc = check_budget(p);
    if (rc) return rc;
    if (!ctx) return SSL_ERR_NULL;
    for (int b = 0; b < s->batch; ++b)
        if (ctx[b] < 1 || ctx[b] > s->max_ctx) return SSL_ERR_SHAPE;
    return SSL_OK;
}

// Select workspace: per-partition histograms, candidate segments and the
// position bitmask of every unit, sized for the longest context of the call.
struct SelectPlan {
    int part, parts;
    bool fused;
    size_t hist_off, coarse_off, cnt_off, thr_off, mask_off, seg_off, tag_off, bytes;
};

int plan_select(const ssl_shape* s, const int32_t* ctx, SelectPlan* plan) {
    int max_t = 0;
    for (int b = 0; b < s->batch; ++b) max_t = ctx[b] > max_t ? ctx[b] : max_t;
    plan->part = ssl::select_part_len(max_t);
    plan->parts = (max_t + plan->part - 1) / plan->part;
    if (plan->parts > ssl::kMaxSelectParts) return SSL_ERR_UNSUPPORTED;
    const size_t slots = (size_t)s->batch * s->n_kv_heads * plan->parts;
    const size_t units = (size_t)s->batch * s->n_kv_heads;
    // one kernel when the call is small and a unit's partitions can all be
    // resident at once
    plan->fused = slots <= (size_t)kSelectFuseMaxGroups &&
                  plan->parts <= resident_group_cap(select_blocks_per_cu(plan->part));
    plan->hist_off = kEpochBytes;
    plan->coarse_off = plan->hist_off + align_up(slots * kHistSlotWords * sizeof(uint32_t));
    plan->cnt_off = plan->coarse_off + align_up(slots * 64 * sizeof(uint32_t));
    plan->thr_off = plan->cnt_off + align_up(slots * sizeof(uint32_t));
    plan->mask_off = plan->thr_off + align_up(units * 2 * sizeof(uint32_t));
    plan->seg_off = plan->mask_off + align_up(slots * (plan->part / 32) * sizeof(uint32_t));
    plan->tag_off = plan->seg_off + align_up(slots * plan->part * 2 * sizeof(uint32_t));
    plan->bytes = plan->tag_off + align_up(slots * kSelectTagWords * sizeof(uint64_t));
    return SSL_OK;
}

int check_workspace(const void* ws, size_t have, size_t need) {
    if (need == 0) return SSL_OK;
    if (!ws || have < need) return SSL_ERR_WORKSPACE;
    if (!aligned(ws, 16)) return SSL_ERR_ALIGN;
    return SSL_OK;
}

}  // namespace

extern "C" {

const char* ssl_status_string(int status) {
    switch (status) {
        case SSL_OK: return "ok";
        case SSL_ERR_NULL: return "a required pointer is NULL";
        case SSL_ERR_SHAPE: return "inconsistent shape, length or parameter";
        case SSL_ERR_UNSUPPORTED: return "request outside the supported limits";
        case SSL_ERR_BUDGET: return "invalid budget: need budget >= 1, k_sink, k_recent >= 0, k_sink + k_recent <= budget";
        case SSL_ERR_ALIGN: return "device pointer is not suitably aligned";
        case SSL_ERR_WORKSPACE: return "workspace missing or too small";
        case SSL_ERR_HIP: return "a HIP call failed (ssl_last_hip_error names it)";
        default: return "unknown status";
    }
}

#ifndef SSL_BUILD_ID
#define SSL_BUILD_ID "unknown"
#endif

const char* ssl_build_id(void) { return SSL_BUILD_ID; }

int ssl_exchange_status(hipStream_t stream, uint32_t* flags_out) {
    if (!flags_out) return SSL_ERR_NULL;
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (const int hip_st = hip_rc(hipStreamIsCapturing(stream, &st))) {
        (void)hipGetLastError();
        return hip_st;
    }
    if (st != hipStreamCaptureStatusNone) return SSL_ERR_UNSUPPORTED;
    return hip_rc(take_exchange_status(stream, flags_out));
}

const char* ssl_last_hip_error(void) { return hipGetErrorName(t_last_hip); }

int ssl_set_cu_budget(int32_t n_cu) {
    if (n_cu < 0) return SSL_ERR_SHAPE;
    g_cu_budget.store(n_cu, std::memory_order_relaxed);
    return SSL_OK;
}

int ssl_test_exchange_faults(int32_t spin_limit, int32_t mismatch_tags) {
    if (spin_limit < 0 || (mismatch_tags != 0 && mismatch_tags != 1)) return SSL_ERR_SHAPE;
    g_spin_limit.store(spin_limit, std::memory_order_relaxed);
    g_tag_flip.store(mismatch_tags ? 0x5A5A5A5A5A5A5A5Aull : 0ull, std::memory_order_relaxed);
    return SSL_OK;
}

int32_t ssl_index_count(int32_t T, int32_t k_sink, int32_t k_recent, int32_t budget) {
    if (budget < 1 || k_sink < 0 || k_recent < 0 || (int64_t)k_sink + k_recent > budget)
        return SSL_ERR_BUDGET;
    if (T < 1) return SSL_ERR_SHAPE;
    const int32_t k_mid = budget - k_sink - k_recent;
    const int32_t s_end = std::min(k_sink, T);
    const int32_t r_start = std::max(T - k_recent, s_end);
    return s_end + std::min(k_mid, r_start - s_end) + (T - r_start);
}

int ssl_verify_workspace(const ssl_shape* shape, const ssl_params* params,
                         const int32_t* ctx_len_host, const int32_t* q_len_host, size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    VerifyPlan plan;
    const int rc = plan_verify(shape, params, ctx_len_host, q_len_host, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

int ssl_verify_plan(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                    const int32_t* q_len_host, int32_t* schedule_out, int32_t* chunk_out,
                    int32_t* items_out) {
    if (!schedule_out || !chunk_out || !items_out) return SSL_ERR_NULL;
    VerifyPlan plan;
    const int rc = plan_verify(shape, params, ctx_len_host, q_len_host, &plan);
    if (rc) return rc;
    const bool one = use_one_sweep(plan, params);
    *schedule_out = !one ? SSL_VERIFY_TWO_SWEEP : plan.pipe ? SSL_VERIFY_ONE_SWEEP_PERSISTENT : SSL_VERIFY_ONE_SWEEP;
    *chunk_out = one ? plan.fused_chunk : plan.chunk;
    *items_out = one ? plan.fused_slots : plan.n_items;
    return SSL_OK;
}

}  // extern "C"

namespace {

// Paged cache arguments: page_size a multiple of 32, every context within
// max_blocks pages.
int check_paged(const ssl_shape* s, const int32_t* ctx, const int32_t* block_table,
                int32_t page_size, int32_t max_blocks) {
    if (!block_table) return SSL_ERR_NULL;
    if (!aligned(block_table, 4)) return SSL_ERR_ALIGN;
    if (page_size < 32 || page_size % 32 != 0 || max_blocks < 1) return SSL_ERR_SHAPE;
    for (int b = 0; b < s->batch; ++b)
        if ((int64_t)ctx[b] > (int64_t)page_size * max_blocks) return SSL_ERR_SHAPE;
    return SSL_OK;
}

int verify_call(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                const int32_t* q_len_host, const void* q, const void* k_cache,
                const void* v_cache, const int32_t* block_table, int32_t page_size,
                int32_t max_blocks, void* out, float* scores, void* workspace,
                size_t workspace_bytes, hipStream_t stream, const StaticScratch* scratch = nullptr) {
    VerifyPlan plan;
    int rc = plan_verify(shape, params, ctx_len_host, q_len_host, &plan);
    if (rc) return rc;
    if (block_table || page_size || max_blocks) {
        rc = check_paged(shape, ctx_len_host, block_table, page_size, max_blocks);
        if (rc) return rc;
    }
    if (!q || !k_cache || !v_cache || !out || !scores) return SSL_ERR_NULL;
    if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
        !aligned(scores, 4))
        return SSL_ERR_ALIGN;
    if (scratch) {
        // the library's static scratch: refuse what it cannot hold, then (the
        // arguments all checked) look up its address on this device
        if (plan.bytes > scratch->bytes) return SSL_ERR_WORKSPACE;
        if (const int hip_st = hip_rc(scratch->address(&workspace))) return hip_st;
        workspace_bytes = scratch->bytes;
    }
    rc = check_workspace(workspace, workspace_bytes, plan.bytes);
    if (rc) return rc;

    VerifyArgs a = {};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k_cache);
    a.v = static_cast<const uint16_t*>(v_cache);
    a.part_ml = reinterpret_cast<float2*>(static_cast<char*>(workspace) + plan.ml_off);
    a.part_o = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.o_off);
    a.scores = scores;
    a.out = out;
    a.n_q_heads = shape->n_q_heads;
    a.n_kv_heads = shape->n_kv_heads;
    a.group = shape->n_q_heads / shape->n_kv_heads;
    a.max_ctx = shape->max_ctx;
    a.max_q = shape->max_q;
    a.window = params->window;
    a.chunk = plan.chunk;
    a.out_fp32 = params->out_fp32 ? 1 : 0;
    a.scale_log2 = params->sm_scale * 1.4426950408889634f;
    a.seq = plan.seq;
    a.block_table = block_table;
    a.page_size = page_size;
    a.max_blocks = max_blocks;
    a.per_head = params->per_head;
    for (int b = 0; b < shape->batch; ++b) {   // one block: every sequence, all its rows
        a.sid[b] = b;
        a.qoff[b] = 0;
        a.qfull[b] = q_len_host[b];
    }
    a.score_add = 0;
    if (params->per_head && !use_one_sweep(plan, params)) {
        // two sweeps sum a head's rows across the 16 lanes of a row tile
        const int g = a.group;
        if (g > 16 || (g & (g - 1)) != 0) return SSL_ERR_UNSUPPORTED;
    }
    if (use_one_sweep(plan, params)) {
        FusedArgs fa = {};
        fa.v = a;
        fa.v.chunk = plan.fused_chunk;
        fa.v.seq = plan.fseq;
        rc = epochs_if_captured(stream, workspace, (int64_t)shape->batch * shape->n_kv_heads, &fa.epoch);
        if (rc) return rc;
        rc = make_exchange(&fa.xc);
        if (rc) return rc;
        fa.call_tag = next_call_tag();
        // An eager call on the static scratch, which no caller can clear,
        // re-arms its units' epochs with a value unrelated to earlier epochs,
        // lifting the mark a captured call that gave up may have left there.
        fa.heal = scratch && !fa.epoch ? static_cast<uint64_t*>(workspace) : nullptr;
        fa.heal_value = mix64(fa.call_tag);
        fa.n_tasks = plan.pipe ? plan.fused_slots : 0;
        return hip_rc(launch_verify_fused(fa, plan.pipe ? plan.pipe_grid : plan.fused_slots, plan.row_tiles,
                                          stream));
    }
    if (plan.block_pos >= shape->max_q)
        return hip_rc(launch_verify(a, plan.n_items, plan.n_rows, plan.row_tiles, stream));
    // Row blocks, the last positions of every sequence first (that block has
    // all sequences, so it writes every score; later blocks add theirs).  A
    // block's table holds only the sequences that still have positions.
    int max_q = 0;
    for (int b = 0; b < shape->batch; ++b) max_q = std::max(max_q, q_len_host[b]);
    const int P = plan.block_pos, g = a.group;
    for (int k = 0; k * P < max_q; ++k) {
        VerifyArgs blk = a;
        memset(&blk.seq, 0, sizeof blk.seq);
        int n = 0;
        int64_t items = 0, rows = 0;
        for (int b = 0; b < shape->batch; ++b) {
            const int j_end = q_len_host[b] - k * P;
            if (j_end <= 0) continue;
            const int j0 = std::max(0, j_end - P);
            blk.seq.item_start[n] = (int32_t)items;
            blk.seq.row_start[n] = (int32_t)rows;
            blk.seq.ctx[n] = ctx_len_host[b];
            blk.seq.qlen[n] = j_end - j0;
            blk.sid[n] = b;
            blk.qoff[n] = j0;
            blk.qfull[n] = q_len_host[b];
            items += (int64_t)shape->n_kv_heads * ((ctx_len_host[b] + plan.chunk - 1) / plan.chunk);
            rows += (int64_t)shape->n_kv_heads * (j_end - j0) * g;
            ++n;
        }
        blk.seq.n_seq = n;
        blk.seq.item_start[n] = (int32_t)items;
        blk.seq.row_start[n] = (int32_t)rows;
        blk.score_add = k > 0 ? 1 : 0;
        if (const int hip_st = hip_rc(launch_verify(blk, (int)items, (int)rows, plan.row_tiles, stream))) return hip_st;
    }
    return SSL_OK;
}

}  // namespace

namespace ssl {

int verify_attn_static_scratch(const ssl_shape* shape, const ssl_params* params,
                               const int32_t* ctx_len_host, const int32_t* q_len_host,
                               const void* q, const void* k_cache, const void* v_cache, void* out,
                               float* scores, const StaticScratch& scratch, hipStream_t stream) {
    return verify_call(shape, params, ctx_len_host, q_len_host, q, k_cache, v_cache, nullptr, 0, 0,
                       out, scores, nullptr, 0, stream, &scratch);
}

}  // namespace ssl

namespace {

// The first draft step that ssl_select_draft hands to the select kernel.
struct DraftInputs {
    const void* q_draft;
    const void* k_cache;
    const void* v_cache;
    void* out;
};

// Whether select's one-kernel schedule also runs the first draft step: the
// kernel's row list holds 4096 entries (partitions of at most 4096 positions)
// and the draft tile holds 16 query heads.
bool select_draft_fused(const SelectPlan& plan, int group) {
    return plan.fused && plan.part <= 4096 && group <= 16;
}

size_t select_draft_part_bytes(const SelectPlan& plan, int64_t units) {
    return align_up((size_t)units * plan.parts * 16 * kSelectDraftStride * sizeof(float));
}

int select_call(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                const float* scores, int32_t* idx, int32_t* n_idx, void* workspace,
                size_t workspace_bytes, hipStream_t stream, const DraftInputs* draft) {
    int rc = check_select(shape, params, ctx_len_host);
    if (rc) return rc;
    if (!scores || !idx || !n_idx) return SSL_ERR_NULL;
    if (!aligned(scores, 4) || !aligned(idx, 4) || !aligned(n_idx, 4)) return SSL_ERR_ALIGN;
    const ssl_shape us = unit_shape(shape, params);
    SelectPlan plan;
    rc = plan_select(&us, ctx_len_host, &plan);
    if (rc) return rc;
    const int64_t units = (int64_t)shape->batch * us.n_kv_heads;
    const size_t need = plan.bytes + (draft ? select_draft_part_bytes(plan, units) : 0);
    rc = check_workspace(workspace, workspace_bytes, need);
    if (rc) return rc;
    char* ws = static_cast<char*>(workspace);
    SelectArgs a;
    memset(&a, 0, sizeof a);
    a.scores = scores;
    a.idx = idx;
    a.n_idx = n_idx;
    a.hist = reinterpret_cast<uint32_t*>(ws + plan.hist_off);
    a.coarse = reinterpret_cast<uint32_t*>(ws + plan.coarse_off);
    a.cnt = reinterpret_cast<uint32_t*>(ws + plan.cnt_off);
    a.thr = reinterpret_cast<uint32_t*>(ws + plan.thr_off);
    a.mask = reinterpret_cast<uint32_t*>(ws + plan.mask_off);
    a.seg = reinterpret_cast<uint2*>(ws + plan.seg_off);
    a.tag = reinterpret_cast<uint64_t*>(ws + plan.tag_off);
    if (plan.fused) {   // the three-kernel schedule exchanges nothing inside a kernel
        rc = epochs_if_captured(stream, ws, units, &a.epoch);
        if (rc) return rc;
    }
    rc = make_exchange(&a.xc);
    if (rc) return rc;
    a.call_tag = next_call_tag();
    a.fused = plan.fused ? 1 : 0;
    a.part = plan.part;
    a.parts = plan.parts;
    a.n_kv_heads = us.n_kv_heads;
    a.max_ctx = shape->max_ctx;
    a.k_sink = params->k_sink;
    a.k_recent = params->k_recent;
    a.budget = params->budget;
    a.batch = shape->batch;
    for (int b = 0; b < shape->batch; ++b) a.ctx[b] = ctx_len_host[b];
    if (draft) {
        a.with_draft = 1;
        a.d.q = static_cast<const uint16_t*>(draft->q_draft);
        a.d.k = static_cast<const uint16_t*>(draft->k_cache);
        a.d.v = static_cast<const uint16_t*>(draft->v_cache);
        a.d.out = draft->out;
        a.d.part = reinterpret_cast<float*>(ws + plan.bytes);
        a.d.n_q_heads = shape->n_q_heads;
        a.d.group = us.n_q_heads / us.n_kv_heads;
        a.d.kv_div = shape->n_kv_heads == us.n_kv_heads ? 1 : shape->n_q_heads / shape->n_kv_heads;
        a.d.n_kv_real = shape->n_kv_heads;
        a.d.out_fp32 = params->out_fp32 ? 1 : 0;
        a.d.scale_log2 = params->sm_scale * 1.4426950408889634f;
    }
    return hip_rc(launch_select(a, (int)units, stream));
}

}  // namespace

extern "C" {

int ssl_verify_attn(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                    const int32_t* q_len_host, const void* q, const void* k_cache,
                    const void* v_cache, void* out, float* scores, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
    return verify_call(shape, params, ctx_len_host, q_len_host, q, k_cache, v_cache, nullptr, 0, 0,
                       out, scores, workspace, workspace_bytes, stream);
}

int ssl_verify_attn_paged(const ssl_shape* shape, const ssl_params* params,
                          const int32_t* ctx_len_host, const int32_t* q_len_host, const void* q,
                          const void* k_pages, const void* v_pages, const int32_t* block_table,
                          int32_t page_size, int32_t max_blocks, void* out, float* scores,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!block_table) return SSL_ERR_NULL;
    return verify_call(shape, params, ctx_len_host, q_len_host, q, k_pages, v_pages, block_table,
                       page_size, max_blocks, out, scores, workspace, workspace_bytes, stream);
}

int ssl_select_workspace(const ssl_shape* shape, const ssl_params* params,
                         const int32_t* ctx_len_host, size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    int rc = check_select(shape, params, ctx_len_host);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);
    SelectPlan plan;
    rc = plan_select(&us, ctx_len_host, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

int ssl_select_plan(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                    int32_t* one_kernel_out, int32_t* part_out, int32_t* parts_out) {
    if (!one_kernel_out || !part_out || !parts_out) return SSL_ERR_NULL;
    int rc = check_select(shape, params, ctx_len_host);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);
    SelectPlan plan;
    rc = plan_select(&us, ctx_len_host, &plan);
    if (rc) return rc;
    *one_kernel_out = plan.fused ? 1 : 0;
    *part_out = plan.part;
    *parts_out = plan.parts;
    return SSL_OK;
}

int ssl_select_topb(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                    const float* scores, int32_t* idx, int32_t* n_idx, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
    return select_call(shape, params, ctx_len_host, scores, idx, n_idx, workspace, workspace_bytes,
                       stream, nullptr);
}

int ssl_draft_workspace(const ssl_shape* shape, const ssl_params* params,
                        const int32_t* n_idx_host, size_t* bytes_out) {
    if (!bytes_out || !shape || !params) return SSL_ERR_NULL;
    int rc = check_budget(params);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);
    DraftPlan plan;
    rc = plan_draft(&us, params, n_idx_host, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

}  // extern "C"

namespace {

// A paged cache for the draft calls (none when block_table is NULL): every
// row they read is below max_ctx, so the pages must cover max_ctx keys.
int check_draft_pages(const ssl_shape* shape, const int32_t* block_table, int32_t page_size,
                      int32_t max_blocks) {
    if (!block_table) return SSL_OK;
    if (!aligned(block_table, 4)) return SSL_ERR_ALIGN;
    if (page_size < 32 || page_size % 32 != 0 || max_blocks < 1 ||
        (int64_t)page_size * max_blocks < shape->max_ctx)
        return SSL_ERR_SHAPE;
    return SSL_OK;
}

int draft_call(const ssl_shape* shape, const ssl_params* params, const int32_t* n_idx_host,
               const void* q_draft, const void* k_cache, const void* v_cache,
               const int32_t* block_table, int32_t page_size, int32_t max_blocks,
               const int32_t* idx, void* out, void* workspace, size_t workspace_bytes,
               hipStream_t stream) {
    if (!shape || !params) return SSL_ERR_NULL;
    int rc = check_budget(params);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);
    DraftPlan plan;
    rc = plan_draft(&us, params, n_idx_host, &plan);
    if (rc) return rc;
    rc = check_draft_pages(shape, block_table, page_size, max_blocks);
    if (rc) return rc;
    if (!q_draft || !k_cache || !v_cache || !idx || !out) return SSL_ERR_NULL;
    if (!aligned(q_draft, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
        !aligned(out, 16) || !aligned(idx, 4))
        return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, plan.bytes);
    if (rc) return rc;
    DraftArgs a = {};
    a.q = static_cast<const uint16_t*>(q_draft);
    a.k = static_cast<const uint16_t*>(k_cache);
    a.v = static_cast<const uint16_t*>(v_cache);
    a.idx = idx;
    a.part_ml = reinterpret_cast<float2*>(static_cast<char*>(workspace) + plan.ml_off);
    a.part_o = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.o_off);
    a.tag = reinterpret_cast<uint64_t*>(static_cast<char*>(workspace) + plan.tag_off);
    rc = epochs_if_captured(stream, workspace, plan.n_units, &a.epoch);
    if (rc) return rc;
    rc = make_exchange(&a.xc);
    if (rc) return rc;
    a.call_tag = next_call_tag();
    a.out = out;
    a.n_q_heads = shape->n_q_heads;
    a.n_kv_heads = us.n_kv_heads;
    a.group = us.n_q_heads / us.n_kv_heads;
    a.kv_div = shape->n_kv_heads == us.n_kv_heads ? 1 : shape->n_q_heads / shape->n_kv_heads;
    a.n_kv_real = shape->n_kv_heads;
    a.max_ctx = shape->max_ctx;
    a.budget = params->budget;
    a.chunk = plan.chunk;
    a.out_fp32 = params->out_fp32 ? 1 : 0;
    a.scale_log2 = params->sm_scale * 1.4426950408889634f;
    a.seq = plan.seq;
    a.block_table = block_table;
    a.page_size = page_size;
    a.max_blocks = max_blocks;
    return hip_rc(launch_draft(a, plan.n_items, stream));
}

}  // namespace

extern "C" {

int ssl_draft_attn(const ssl_shape* shape, const ssl_params* params, const int32_t* n_idx_host,
                   const void* q_draft, const void* k_cache, const void* v_cache,
                   const int32_t* idx, void* out, void* workspace, size_t workspace_bytes,
                   hipStream_t stream) {
    return draft_call(shape, params, n_idx_host, q_draft, k_cache, v_cache, nullptr, 0, 0, idx,
                      out, workspace, workspace_bytes, stream);
}

int ssl_draft_attn_paged(const ssl_shape* shape, const ssl_params* params,
                         const int32_t* n_idx_host, const void* q_draft, const void* k_pages,
                         const void* v_pages, const int32_t* block_table, int32_t page_size,
                         int32_t max_blocks, const int32_t* idx, void* out, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
    if (!block_table) return SSL_ERR_NULL;
    return draft_call(shape, params, n_idx_host, q_draft, k_pages, v_pages, block_table, page_size,
                      max_blocks, idx, out, workspace, workspace_bytes, stream);
}

// select + the first draft step: the draft's entries per sequence (Eq. 4's
// count at T = ctx_len), and whether the select kernel runs the draft itself.
namespace {
int select_draft_plan(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx,
                      SelectPlan* plan, bool* fused, int32_t* n_idx_host, size_t* bytes) {
    int rc = check_select(shape, params, ctx);
    if (rc) return rc;
    if (!(params->sm_scale > 0.f) || !isfinite(params->sm_scale)) return SSL_ERR_SHAPE;
    const ssl_shape us = unit_shape(shape, params);
    rc = plan_select(&us, ctx, plan);
    if (rc) return rc;
    for (int b = 0; b < shape->batch; ++b)
        n_idx_host[b] = ssl_index_count(ctx[b], params->k_sink, params->k_recent, params->budget);
    DraftPlan dp;
    rc = plan_draft(&us, params, n_idx_host, &dp);
    if (rc) return rc;
    *fused = select_draft_fused(*plan, us.n_q_heads / us.n_kv_heads);
    *bytes = *fused ? plan->bytes + select_draft_part_bytes(*plan, (int64_t)shape->batch * us.n_kv_heads)
                    : std::max(plan->bytes, dp.bytes);
    return SSL_OK;
}
}  // namespace

int ssl_select_draft_workspace(const ssl_shape* shape, const ssl_params* params,
                               const int32_t* ctx_len_host, size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    SelectPlan plan;
    bool fused = false;
    int32_t n_idx_host[kTableBatch];
    return select_draft_plan(shape, params, ctx_len_host, &plan, &fused, n_idx_host, bytes_out);
}

int ssl_select_draft(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                     const float* scores, int32_t* idx, int32_t* n_idx, const void* q_draft,
                     const void* k_cache, const void* v_cache, void* out, void* workspace,
                     size_t workspace_bytes, hipStream_t stream) {
    SelectPlan plan;
    bool fused = false;
    int32_t n_idx_host[kTableBatch];
    size_t need = 0;
    int rc = select_draft_plan(shape, params, ctx_len_host, &plan, &fused, n_idx_host, &need);
    if (rc) return rc;
    if (!scores || !idx || !n_idx || !q_draft || !k_cache || !v_cache || !out) return SSL_ERR_NULL;
    if (!aligned(scores, 4) || !aligned(idx, 4) || !aligned(n_idx, 4) || !aligned(q_draft, 16) ||
        !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16))
        return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, need);
    if (rc) return rc;
    if (fused) {
        const DraftInputs d{q_draft, k_cache, v_cache, out};
        return select_call(shape, params, ctx_len_host, scores, idx, n_idx, workspace,
                           workspace_bytes, stream, &d);
    }
    rc = select_call(shape, params, ctx_len_host, scores, idx, n_idx, workspace, workspace_bytes,
                     stream, nullptr);
    if (rc) return rc;
    return draft_call(shape, params, n_idx_host, q_draft, k_cache, v_cache, nullptr, 0, 0, idx, out,
                      workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {

// The whole decode step: one kernel where verify takes one sweep (then every
// chunk workgroup of a unit is also a select partition and drafts over its
// selections), else verify, then select_draft, on one workspace.
struct DecodePlan {
    VerifyPlan v;
    bool one_kernel;
    int parts;   // chunks of the longest context: the select arrays' partition stride
    size_t hist_off, seg_off, tag_off, part_off, bytes;
};

int plan_decode(const ssl_shape* s, const ssl_params* p, const int32_t* ctx, const int32_t* ql,
                DecodePlan* plan) {
    int rc = plan_verify(s, p, ctx, ql, &plan->v);
    if (rc) return rc;
    ssl_shape ds = *s;
    ds.max_q = 1;
    SelectPlan sp;
    bool sd_fused = false;
    int32_t n_idx_host[kTableBatch];
    size_t sd_bytes = 0;
    rc = select_draft_plan(&ds, p, ctx, &sp, &sd_fused, n_idx_host, &sd_bytes);
    if (rc) return rc;
    // One kernel only when every chunk workgroup of the call is resident at
    // once (with more, later units wait behind earlier units' select and
    // draft exchanges instead of streaming: measured far slower) and chunks
    // hold at least kStepMinChunk keys (smaller chunks make many small select
    // partitions, whose exchanges measured slower than select's own).
    constexpr int kStepMinChunk = 512;
    const int g = s->n_q_heads / s->n_kv_heads;
    const int64_t resident = (int64_t)device_cus() * std::max(fused_blocks_per_cu(plan->v.row_tiles), 1);
    plan->one_kernel = use_one_sweep(plan->v, p) && !plan->v.pipe && !p->per_head && g <= 16 &&
                       plan->v.fused_slots <= resident && plan->v.fused_chunk >= kStepMinChunk;
    if (!plan->one_kernel) {
        plan->parts = 0;
        plan->hist_off = plan->seg_off = plan->tag_off = plan->part_off = 0;
        plan->bytes = std::max(plan->v.bytes, sd_bytes);
        return SSL_OK;
    }
    const int chunk = plan->v.fused_chunk;
    int max_t = 0;
    for (int b = 0; b < s->batch; ++b) max_t = std::max(max_t, ctx[b]);
    plan->parts = (max_t + chunk - 1) / chunk;
    const size_t slots = (size_t)s->batch * s->n_kv_heads * plan->parts;
    plan->hist_off = align_up(plan->v.bytes);
    plan->seg_off = plan->hist_off + align_up(slots * kHistSlotWords * sizeof(uint32_t));
    plan->tag_off = plan->seg_off + align_up(slots * chunk * 2 * sizeof(uint32_t));
    plan->part_off = plan->tag_off + align_up(slots * kSelectTagWords * sizeof(uint64_t));
    plan->bytes = plan->part_off + align_up(slots * 16 * kSelectDraftStride * sizeof(float));
    return SSL_OK;
}

}  // namespace

extern "C" {

int ssl_decode_step_workspace(const ssl_shape* shape, const ssl_params* params,
                              const int32_t* ctx_len_host, const int32_t* q_len_host,
                              size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    DecodePlan plan;
    const int rc = plan_decode(shape, params, ctx_len_host, q_len_host, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

int ssl_decode_step_plan(const ssl_shape* shape, const ssl_params* params,
                         const int32_t* ctx_len_host, const int32_t* q_len_host,
                         int32_t* one_kernel_out) {
    if (!one_kernel_out) return SSL_ERR_NULL;
    DecodePlan plan;
    const int rc = plan_decode(shape, params, ctx_len_host, q_len_host, &plan);
    if (rc) return rc;
    *one_kernel_out = plan.one_kernel ? 1 : 0;
    return SSL_OK;
}

int ssl_decode_step(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                    const int32_t* q_len_host, const void* q, const void* k_cache,
                    const void* v_cache, void* out, float* scores, int32_t* idx, int32_t* n_idx,
                    const void* q_draft, void* draft_out, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    DecodePlan plan;
    int rc = plan_decode(shape, params, ctx_len_host, q_len_host, &plan);
    if (rc) return rc;
    if (!q || !k_cache || !v_cache || !out || !scores || !idx || !n_idx || !q_draft || !draft_out)
        return SSL_ERR_NULL;
    if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) ||
        !aligned(scores, 4) || !aligned(idx, 4) || !aligned(n_idx, 4) || !aligned(q_draft, 16) ||
        !aligned(draft_out, 16))
        return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, plan.bytes);
    if (rc) return rc;
    ssl_shape ds = *shape;
    ds.max_q = 1;
    if (!plan.one_kernel) {
        rc = verify_call(shape, params, ctx_len_host, q_len_host, q, k_cache, v_cache, nullptr, 0, 0,
                         out, scores, workspace, workspace_bytes, stream);
        if (rc) return rc;
        return ssl_select_draft(&ds, params, ctx_len_host, scores, idx, n_idx, q_draft, k_cache,
                                v_cache, draft_out, workspace, workspace_bytes, stream);
    }
    char* ws = static_cast<char*>(workspace);
    const VerifyPlan& vp = plan.v;
    FusedArgs fa = {};
    VerifyArgs& a = fa.v;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k_cache);
    a.v = static_cast<const uint16_t*>(v_cache);
    a.part_ml = reinterpret_cast<float2*>(ws + vp.ml_off);
    a.part_o = reinterpret_cast<float*>(ws + vp.o_off);
    a.scores = scores;
    a.out = out;
    a.n_q_heads = shape->n_q_heads;
    a.n_kv_heads = shape->n_kv_heads;
    a.group = shape->n_q_heads / shape->n_kv_heads;
    a.max_ctx = shape->max_ctx;
    a.max_q = shape->max_q;
    a.window = params->window;
    a.chunk = vp.fused_chunk;
    a.out_fp32 = params->out_fp32 ? 1 : 0;
    a.scale_log2 = params->sm_scale * 1.4426950408889634f;
    a.seq = vp.fseq;
    for (int b = 0; b < shape->batch; ++b) {
        a.sid[b] = b;
        a.qfull[b] = q_len_host[b];
    }
    const int64_t units = (int64_t)shape->batch * shape->n_kv_heads;
    rc = epochs_if_captured(stream, workspace, units, &fa.epoch);
    if (rc) return rc;
    rc = make_exchange(&fa.xc);
    if (rc) return rc;
    fa.call_tag = next_call_tag();
    fa.step = 1;
    SelectArgs& sa = fa.sel;
    sa.idx = idx;
    sa.n_idx = n_idx;
    sa.hist = reinterpret_cast<uint32_t*>(ws + plan.hist_off);
    sa.seg = reinterpret_cast<uint2*>(ws + plan.seg_off);
    sa.tag = reinterpret_cast<uint64_t*>(ws + plan.tag_off);
    sa.epoch = fa.epoch;
    sa.call_tag = fa.call_tag;
    sa.xc = fa.xc;
    sa.fused = 1;
    sa.with_draft = 1;
    sa.d.q = static_cast<const uint16_t*>(q_draft);
    sa.d.k = a.k;
    sa.d.v = a.v;
    sa.d.out = draft_out;
    sa.d.part = reinterpret_cast<float*>(ws + plan.part_off);
    sa.d.n_q_heads = shape->n_q_heads;
    sa.d.group = a.group;
    sa.d.kv_div = 1;
    sa.d.n_kv_real = shape->n_kv_heads;
    sa.d.out_fp32 = a.out_fp32;
    sa.d.scale_log2 = a.scale_log2;
    sa.n_kv_heads = shape->n_kv_heads;
    sa.max_ctx = shape->max_ctx;
    sa.k_sink = params->k_sink;
    sa.k_recent = params->k_recent;
    sa.budget = params->budget;
    sa.batch = shape->batch;
    sa.part = vp.fused_chunk;
    sa.parts = plan.parts;
    for (int b = 0; b < shape->batch; ++b) sa.ctx[b] = ctx_len_host[b];
    return hip_rc(launch_verify_fused(fa, vp.fused_slots, vp.row_tiles, stream));
}

}  // extern "C"

namespace {

int materialize_call(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                     const void* k_cache, const void* v_cache, const int32_t* block_table,
                     int32_t page_size, int32_t max_blocks, const int32_t* idx, void* k_sel,
                     void* v_sel, hipStream_t stream) {
    if (!shape || !params) return SSL_ERR_NULL;
    int rc = check_budget(params);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);   // per_head: one unit per query head
    StepPlan plan;
    rc = plan_draft_step(&us, params, ctx_len_host, ctx_len_host, &plan);
    if (rc) return rc;
    rc = check_draft_pages(shape, block_table, page_size, max_blocks);
    if (rc) return rc;
    if (!k_cache || !v_cache || !idx || !k_sel || !v_sel) return SSL_ERR_NULL;
    if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(k_sel, 16) ||
        !aligned(v_sel, 16) || !aligned(idx, 4))
        return SSL_ERR_ALIGN;
    DraftArgs a = {};
    a.k = static_cast<const uint16_t*>(k_cache);
    a.v = static_cast<const uint16_t*>(v_cache);
    a.idx = idx;
    a.k_sel = static_cast<uint16_t*>(k_sel);
    a.v_sel = static_cast<uint16_t*>(v_sel);
    a.n_kv_heads = us.n_kv_heads;
    a.kv_div = shape->n_kv_heads == us.n_kv_heads ? 1 : shape->n_q_heads / shape->n_kv_heads;
    a.n_kv_real = shape->n_kv_heads;
    a.max_ctx = shape->max_ctx;
    a.budget = params->budget;
    a.block_table = block_table;
    a.page_size = page_size;
    a.max_blocks = max_blocks;
    for (int b = 0; b < shape->batch; ++b) a.n_fixed[b] = plan.n_fixed[b];
    return hip_rc(launch_draft_materialize(a, plan.max_fixed, shape->batch * us.n_kv_heads, stream));
}

}  // namespace

extern "C" {

int ssl_draft_materialize(const ssl_shape* shape, const ssl_params* params,
                          const int32_t* ctx_len_host, const void* k_cache, const void* v_cache,
                          const int32_t* idx, void* k_sel, void* v_sel, hipStream_t stream) {
    return materialize_call(shape, params, ctx_len_host, k_cache, v_cache, nullptr, 0, 0, idx,
                            k_sel, v_sel, stream);
}

int ssl_draft_materialize_paged(const ssl_shape* shape, const ssl_params* params,
                                const int32_t* ctx_len_host, const void* k_pages,
                                const void* v_pages, const int32_t* block_table, int32_t page_size,
                                int32_t max_blocks, const int32_t* idx, void* k_sel, void* v_sel,
                                hipStream_t stream) {
    if (!block_table) return SSL_ERR_NULL;
    return materialize_call(shape, params, ctx_len_host, k_pages, v_pages, block_table, page_size,
                            max_blocks, idx, k_sel, v_sel, stream);
}

int ssl_draft_step_workspace(const ssl_shape* shape, const ssl_params* params,
                             const int32_t* ctx_len_host, const int32_t* cur_len_host,
                             size_t* bytes_out) {
    if (!bytes_out || !shape || !params) return SSL_ERR_NULL;
    int rc = check_budget(params);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);
    StepPlan plan;
    rc = plan_draft_step(&us, params, ctx_len_host, cur_len_host, &plan);
    if (rc) return rc;
    *bytes_out = plan.d.bytes;
    return SSL_OK;
}

}  // extern "C"

namespace {

int draft_step_call(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                    const int32_t* cur_len_host, const void* q_draft, const void* k_cache,
                    const void* v_cache, const int32_t* block_table, int32_t page_size,
                    int32_t max_blocks, const int32_t* idx, const void* k_sel, const void* v_sel,
                    void* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!shape || !params) return SSL_ERR_NULL;
    int rc = check_budget(params);
    if (rc) return rc;
    const ssl_shape us = unit_shape(shape, params);   // per_head: one unit per query head
    StepPlan plan;
    rc = plan_draft_step(&us, params, ctx_len_host, cur_len_host, &plan);
    if (rc) return rc;
    if (!(params->sm_scale > 0.f) || !isfinite(params->sm_scale)) return SSL_ERR_SHAPE;
    rc = check_draft_pages(shape, block_table, page_size, max_blocks);
    if (rc) return rc;
    const bool sel = k_sel || v_sel;
    if (!q_draft || !k_cache || !v_cache || !out) return SSL_ERR_NULL;
    if (sel ? (!k_sel || !v_sel) : !idx) return SSL_ERR_NULL;
    if (!aligned(q_draft, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
        !aligned(out, 16) || (sel && (!aligned(k_sel, 16) || !aligned(v_sel, 16))) ||
        (!sel && !aligned(idx, 4)))
        return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, plan.d.bytes);
    if (rc) return rc;
    DraftArgs a = {};
    a.q = static_cast<const uint16_t*>(q_draft);
    a.k = static_cast<const uint16_t*>(k_cache);
    a.v = static_cast<const uint16_t*>(v_cache);
    a.idx = sel ? nullptr : idx;
    a.k_sel = sel ? const_cast<uint16_t*>(static_cast<const uint16_t*>(k_sel)) : nullptr;   // read only here
    a.v_sel = sel ? const_cast<uint16_t*>(static_cast<const uint16_t*>(v_sel)) : nullptr;
    a.part_ml = reinterpret_cast<float2*>(static_cast<char*>(workspace) + plan.d.ml_off);
    a.part_o = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.d.o_off);
    a.tag = reinterpret_cast<uint64_t*>(static_cast<char*>(workspace) + plan.d.tag_off);
    rc = epochs_if_captured(stream, workspace, plan.d.n_units, &a.epoch);
    if (rc) return rc;
    rc = make_exchange(&a.xc);
    if (rc) return rc;
    a.call_tag = next_call_tag();
    a.out = out;
    a.n_q_heads = shape->n_q_heads;
    a.n_kv_heads = us.n_kv_heads;
    a.group = us.n_q_heads / us.n_kv_heads;
    a.kv_div = shape->n_kv_heads == us.n_kv_heads ? 1 : shape->n_q_heads / shape->n_kv_heads;
    a.n_kv_real = shape->n_kv_heads;
    a.max_ctx = shape->max_ctx;
    a.budget = params->budget;
    a.chunk = plan.d.chunk;
    a.out_fp32 = params->out_fp32 ? 1 : 0;
    a.scale_log2 = params->sm_scale * 1.4426950408889634f;
    a.seq = plan.d.seq;
    a.block_table = block_table;
    a.page_size = page_size;
    a.max_blocks = max_blocks;
    for (int b = 0; b < shape->batch; ++b) {
        a.n_fixed[b] = plan.n_fixed[b];
        a.win0[b] = plan.win0[b];
    }
    return hip_rc(launch_draft_step(a, plan.d.n_items, stream));
}

}  // namespace

extern "C" {

int ssl_draft_step(const ssl_shape* shape, const ssl_params* params, const int32_t* ctx_len_host,
                   const int32_t* cur_len_host, const void* q_draft, const void* k_cache,
                   const void* v_cache, const int32_t* idx, const void* k_sel, const void* v_sel,
                   void* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return draft_step_call(shape, params, ctx_len_host, cur_len_host, q_draft, k_cache, v_cache,
                           nullptr, 0, 0, idx, k_sel, v_sel, out, workspace, workspace_bytes,
                           stream);
}

int ssl_draft_step_paged(const ssl_shape* shape, const ssl_params* params,
                         const int32_t* ctx_len_host, const int32_t* cur_len_host,
                         const void* q_draft, const void* k_pages, const void* v_pages,
                         const int32_t* block_table, int32_t page_size, int32_t max_blocks,
                         const int32_t* idx, const void* k_sel, const void* v_sel, void* out,
                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!block_table) return SSL_ERR_NULL;
    return draft_step_call(shape, params, ctx_len_host, cur_len_host, q_draft, k_pages, v_pages,
                           block_table, page_size, max_blocks, idx, k_sel, v_sel, out, workspace,
                           workspace_bytes, stream);
}

// ---- token statistics of logit rows ----------------------------------------

struct LogitPlan {
    int n_chunks;
    size_t part_off, tag_off, argmax_off, bytes;
};

int plan_logits(int32_t n_rows, int32_t vocab, LogitPlan* plan) {
    if (n_rows < 1 || vocab < 1) return SSL_ERR_SHAPE;
    if (vocab > kLogitChunk * kLogitMaxChunks) return SSL_ERR_UNSUPPORTED;
    if ((int64_t)n_rows * ((vocab + kLogitChunk - 1) / kLogitChunk) > (1 << 30))
        return SSL_ERR_UNSUPPORTED;
    plan->n_chunks = (vocab + kLogitChunk - 1) / kLogitChunk;
    const size_t slots = (size_t)n_rows * plan->n_chunks;
    plan->part_off = kEpochBytes;
    plan->tag_off = plan->part_off + align_up(slots * 4 * sizeof(float));
    plan->argmax_off = plan->tag_off + align_up(slots * sizeof(uint64_t));
    plan->bytes = plan->argmax_off + align_up((size_t)n_rows * sizeof(int32_t));
    return SSL_OK;
}

int check_logits(const void* logits, int32_t dtype, int32_t vocab, int32_t row_stride) {
    if (dtype != SSL_DT_BF16 && dtype != SSL_DT_F32) return SSL_ERR_SHAPE;
    if (row_stride < vocab) return SSL_ERR_SHAPE;
    if (!logits) return SSL_ERR_NULL;
    const int64_t row_bytes = (int64_t)row_stride * (dtype == SSL_DT_F32 ? 4 : 2);
    if (!aligned(logits, 16) || row_bytes % 16 != 0) return SSL_ERR_ALIGN;
    return SSL_OK;
}

int ssl_logit_stats_workspace(int32_t n_rows, int32_t vocab, size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    LogitPlan plan;
    const int rc = plan_logits(n_rows, vocab, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

int ssl_logit_stats(const void* logits, int32_t dtype, int32_t n_rows, int32_t vocab,
                    int32_t row_stride, float* entropy, int32_t* argmax, void* workspace,
                    size_t workspace_bytes, hipStream_t stream) {
    LogitPlan plan;
    int rc = plan_logits(n_rows, vocab, &plan);
    if (rc) return rc;
    rc = check_logits(logits, dtype, vocab, row_stride);
    if (rc) return rc;
    if (!entropy && !argmax) return SSL_ERR_NULL;
    if ((entropy && !aligned(entropy, 4)) || (argmax && !aligned(argmax, 4))) return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, plan.bytes);
    if (rc) return rc;
    LogitArgs a = {};
    a.logits = logits;
    a.n_rows = n_rows;
    a.vocab = vocab;
    a.row_stride = row_stride;
    a.n_chunks = plan.n_chunks;
    a.entropy = entropy;
    a.argmax = argmax;
    a.part = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.part_off);
    a.tag = reinterpret_cast<uint64_t*>(static_cast<char*>(workspace) + plan.tag_off);
    rc = epochs_if_captured(stream, workspace, n_rows, &a.epoch);
    if (rc) return rc;
    rc = make_exchange(&a.xc);
    if (rc) return rc;
    a.call_tag = next_call_tag();
    a.rows_per_seq = 0;
    return hip_rc(launch_logit_stats(a, dtype == SSL_DT_F32, stream));
}

int ssl_greedy_accept_workspace(int32_t batch, int32_t max_k, int32_t vocab, size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    if (batch < 1 || max_k < 0) return SSL_ERR_SHAPE;
    if (batch > kTableBatch || max_k > kAcceptMaxK) return SSL_ERR_UNSUPPORTED;
    LogitPlan plan;
    const int rc = plan_logits(batch * (max_k + 1), vocab, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

int ssl_greedy_accept(const void* logits, int32_t dtype, int32_t batch, int32_t max_k,
                      const int32_t* k_len_host, int32_t vocab, int32_t row_stride,
                      const int32_t* draft_tokens, int32_t* n_accepted, int32_t* next_token,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (batch < 1 || max_k < 0) return SSL_ERR_SHAPE;
    if (batch > kTableBatch || max_k > kAcceptMaxK) return SSL_ERR_UNSUPPORTED;
    LogitPlan plan;
    int rc = plan_logits(batch * (max_k + 1), vocab, &plan);
    if (rc) return rc;
    rc = check_logits(logits, dtype, vocab, row_stride);
    if (rc) return rc;
    if (!k_len_host || !n_accepted || !next_token || (max_k > 0 && !draft_tokens))
        return SSL_ERR_NULL;
    for (int b = 0; b < batch; ++b)
        if (k_len_host[b] < 0 || k_len_host[b] > max_k) return SSL_ERR_SHAPE;
    if (!aligned(n_accepted, 4) || !aligned(next_token, 4) ||
        (draft_tokens && !aligned(draft_tokens, 4)))
        return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, plan.bytes);
    if (rc) return rc;
    char* ws = static_cast<char*>(workspace);
    LogitArgs a = {};
    a.logits = logits;
    a.n_rows = batch * (max_k + 1);
    a.vocab = vocab;
    a.row_stride = row_stride;
    a.n_chunks = plan.n_chunks;
    a.entropy = nullptr;
    a.argmax = reinterpret_cast<int32_t*>(ws + plan.argmax_off);
    a.part = reinterpret_cast<float*>(ws + plan.part_off);
    a.tag = reinterpret_cast<uint64_t*>(ws + plan.tag_off);
    rc = epochs_if_captured(stream, ws, a.n_rows, &a.epoch);
    if (rc) return rc;
    rc = make_exchange(&a.xc);
    if (rc) return rc;
    a.call_tag = next_call_tag();
    a.rows_per_seq = max_k + 1;
    for (int b = 0; b < batch; ++b) a.k_len[b] = k_len_host[b];
    if (const int hip_st = hip_rc(launch_logit_stats(a, dtype == SSL_DT_F32, stream))) return hip_st;
    AcceptArgs c = {};
    c.argmax = a.argmax;
    c.draft = draft_tokens;
    c.n_accepted = n_accepted;
    c.next_token = next_token;
    c.max_k = max_k;
    for (int b = 0; b < batch; ++b) c.k_len[b] = k_len_host[b];
    return hip_rc(launch_greedy_accept(c, batch, stream));
}

}  // extern "C"

namespace {

// Speculative sampling workspace: chunk and row statistics of the 2 max_k + 1
// rows of every sequence, the picked positions and the chunk masses.
struct SpecPlan {
    int n_chunks;
    size_t chunk_off, row_off, pick_off, mass_off, bytes;
};

int plan_spec(int32_t batch, int32_t max_k, int32_t vocab, SpecPlan* plan) {
    if (batch < 1 || max_k < 0 || vocab < 1) return SSL_ERR_SHAPE;
    if (batch > kTableBatch || max_k > kAcceptMaxK) return SSL_ERR_UNSUPPORTED;
    if (vocab > kLogitChunk * kLogitMaxChunks) return SSL_ERR_UNSUPPORTED;
    plan->n_chunks = (vocab + kLogitChunk - 1) / kLogitChunk;
    const size_t rows = (size_t)batch * (2 * max_k + 1);
    plan->chunk_off = kEpochBytes;
    plan->row_off = plan->chunk_off + align_up(rows * plan->n_chunks * sizeof(float2));
    plan->pick_off = plan->row_off + align_up(rows * sizeof(float2));
    plan->mass_off = plan->pick_off + align_up((size_t)batch * sizeof(int32_t));
    plan->bytes = plan->mass_off + align_up((size_t)batch * plan->n_chunks * sizeof(float2));
    return SSL_OK;
}

}  // namespace

extern "C" {

int ssl_spec_accept_workspace(int32_t batch, int32_t max_k, int32_t vocab, size_t* bytes_out) {
    if (!bytes_out) return SSL_ERR_NULL;
    SpecPlan plan;
    const int rc = plan_spec(batch, max_k, vocab, &plan);
    if (rc) return rc;
    *bytes_out = plan.bytes;
    return SSL_OK;
}

int ssl_spec_accept(const void* target_logits, const void* draft_logits, int32_t dtype,
                    int32_t batch, int32_t max_k, const int32_t* k_len_host, int32_t vocab,
                    int32_t row_stride, const int32_t* draft_tokens, float temperature,
                    const float* u_accept, const float* u_sample, int32_t* n_accepted,
                    int32_t* next_token, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    SpecPlan plan;
    int rc = plan_spec(batch, max_k, vocab, &plan);
    if (rc) return rc;
    if (!(temperature > 0.f) || !isfinite(temperature) || !isfinite(1.0f / temperature))
        return SSL_ERR_SHAPE;
    rc = check_logits(target_logits, dtype, vocab, row_stride);
    if (rc) return rc;
    if (max_k > 0) {
        rc = check_logits(draft_logits, dtype, vocab, row_stride);
        if (rc) return rc;
    }
    if (!k_len_host || !u_sample || !n_accepted || !next_token ||
        (max_k > 0 && (!draft_tokens || !u_accept)))
        return SSL_ERR_NULL;
    for (int b = 0; b < batch; ++b)
        if (k_len_host[b] < 0 || k_len_host[b] > max_k) return SSL_ERR_SHAPE;
    if (!aligned(u_sample, 4) || !aligned(n_accepted, 4) || !aligned(next_token, 4) ||
        (draft_tokens && !aligned(draft_tokens, 4)) || (u_accept && !aligned(u_accept, 4)))
        return SSL_ERR_ALIGN;
    rc = check_workspace(workspace, workspace_bytes, plan.bytes);
    if (rc) return rc;
    char* ws = static_cast<char*>(workspace);
    SpecArgs a = {};
    a.tlogits = target_logits;
    a.dlogits = draft_logits;
    a.vocab = vocab;
    a.row_stride = row_stride;
    a.n_chunks = plan.n_chunks;
    a.max_k = max_k;
    a.inv_tau = 1.0f / temperature;
    a.draft = draft_tokens;
    a.u_acc = u_accept;
    a.u_smp = u_sample;
    a.n_accepted = n_accepted;
    a.next_token = next_token;
    a.chunk_ms = reinterpret_cast<float2*>(ws + plan.chunk_off);
    a.row_ms = reinterpret_cast<float2*>(ws + plan.row_off);
    a.pick = reinterpret_cast<int32_t*>(ws + plan.pick_off);
    a.mass = reinterpret_cast<float2*>(ws + plan.mass_off);
    for (int b = 0; b < batch; ++b) a.k_len[b] = k_len_host[b];
    return hip_rc(launch_spec_accept(a, batch, dtype == SSL_DT_F32, stream));
}

}  // extern "C"
