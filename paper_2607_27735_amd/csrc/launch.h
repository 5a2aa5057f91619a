// launch.h -- argument blocks and launchers shared by the ABI layer (api.cpp)
// and the kernel translation units.  Everything here is internal.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssl {

constexpr int kTableBatch = 64;   // per-sequence tables travel as kernel arguments

// Every workspace layout starts with kEpochWords 64-bit exchange epochs, one
// per exchange group (KV-head unit, logit row) of a call made under graph
// capture: calls that share a workspace then share these words, which every
// call only ever advances, and no call keeps other data there.
constexpr int kEpochWords = 8192;
constexpr size_t kEpochBytes = (size_t)kEpochWords * sizeof(uint64_t);
// Stored in an epoch word when an exchange of its group gave up: every later
// captured call on that workspace gives up at once (and says so) until the
// caller clears the workspace.  A whole 64-bit value, not a bit, so that a
// workspace's initial contents look marked only by a 2^-64 accident.
constexpr uint64_t kEpochDirty = 0xD1A7E5C0FFEE5EEDull;

// The device's exchange status word: one bit per kernel family whose bounded
// cross-workgroup wait gave up (its results are then unspecified).
enum : uint32_t {
    kStatusVerify = 1u,   // one-sweep verify
    kStatusSelect = 2u,   // one-kernel select
    kStatusDraft = 4u,    // draft and draft-round steps
    kStatusLogits = 8u    // logit statistics and acceptance
};

// What every exchanging kernel needs beyond its data: where to report a wait
// that gave up, how long to wait, and (tests only) a mask XORed into every tag
// it publishes, so that no wait can succeed.
struct Exchange {
    uint32_t* status;       // the device's status word
    uint64_t tag_flip;      // 0 except when testing the give-up path
    int32_t spin_limit;     // polls before a wait gives up
};
constexpr int32_t kDefaultSpinLimit = 1 << 20;

// The current device's status word (its address is looked up once per device).
hipError_t exchange_status_word(uint32_t** word);
// Reads and clears the current device's status word in stream order, then
// waits for the stream.
hipError_t take_exchange_status(hipStream_t stream, uint32_t* flags);

// Per-sequence table, passed by value.  Work items of sequence b are
// [item_start[b], item_start[b + 1]); rows of the combine kernel likewise
// [row_start[b], row_start[b + 1]).
struct SeqTable {
    int32_t n_seq;
    int32_t item_start[kTableBatch + 1];
    int32_t row_start[kTableBatch + 1];
    int32_t ctx[kTableBatch];     // verify: context length; draft: index count
    int32_t qlen[kTableBatch];    // verify rows (verify only)
};

struct VerifyArgs {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    float2* part_ml;    // [n_items][64]  per-split (max, sum) in the log2 domain (two
                        // sweeps; the one-sweep kernel keeps a tagged word pair per row)
    float* part_o;      // [n_items][64][128] per-split sum of P * V
    float* scores;      // [batch][n_kv][max_ctx]
    void* out;          // [batch][max_q][n_q][128]
    int32_t n_q_heads, n_kv_heads, group, max_ctx, max_q, window, chunk, out_fp32;
    float scale_log2;   // sm_scale * log2(e)
    SeqTable seq;
    // Paged cache (block_table non-null): k and v are page pools
    // [n_pages][n_kv][page_size][128], and key t of sequence b is row
    // t % page_size of page block_table[b * max_blocks + t / page_size].
    const int32_t* block_table;
    int32_t page_size, max_blocks;
    // 1: scores per query head, [batch][n_q][max_ctx] (Eq. 3 for each head of
    // the group on its own); 0: per KV head, summed over the group.
    int32_t per_head;
    // Row blocks (a KV head with more verify rows than one launch holds runs
    // one launch per block of positions).  Per entry of seq: the sequence it
    // is (sid), the first of its verify positions in this block (qoff; the
    // block's count is seq.qlen) and its verify positions in all (qfull), so
    // that causal limits and the Eq. 3 window are those of the whole call.
    // One block: sid = b, qoff = 0, qfull = qlen.
    int32_t sid[kTableBatch];
    int32_t qoff[kTableBatch];
    int32_t qfull[kTableBatch];
    int32_t score_add;   // 1: add this block's scores to those already written
};

// Select splits each (sequence, KV head) unit into partitions of `part`
// positions (a multiple of 1024, at most kSelectMaxRounds * 1024); `parts` is
// the partition stride of the workspace arrays (partitions of the longest
// sequence), at most kSelectMaxParts.
constexpr int kSelectMaxRounds = 8;
constexpr int kSelectTargetParts = 32;
constexpr int kMaxSelectParts = 256;
// 32-bit words per partition in SelectArgs::hist: a dense 2048-bin histogram
// (three-kernel path) or up to 2048 tagged 64-bit bin entries (one kernel).
constexpr int kHistSlotWords = 4096;
// 64-bit tag words per partition in SelectArgs::tag.
constexpr int kSelectTagWords = 4;

// The first draft step over the index sets, run by the one-kernel select
// (Eq. 5 with the rows each partition selected): per unit, query heads
// [c*group, (c+1)*group) of q, rows of cache head c / kv_div.
struct SelectDraft {
    const uint16_t* q;      // [batch][n_q][128]
    const uint16_t* k;      // [batch][n_kv_real][max_ctx][128]
    const uint16_t* v;
    void* out;              // [batch][n_q][128]
    float* part;            // [units][parts][16][132] per partition and head: max, sum, 2 spare, P.V
    int32_t n_q_heads, group, kv_div, n_kv_real, out_fp32;
    float scale_log2;
};
constexpr int kSelectDraftStride = 132;   // floats per (partition, head) partial

struct SelectArgs {
    const float* scores;
    int32_t* idx;
    int32_t* n_idx;
    uint32_t* hist;     // [units][parts][kHistSlotWords] histogram of each partition's top 11 score bits
    uint32_t* coarse;   // [units][parts][64]   the same in bins of 32
    uint32_t* cnt;      // [units][parts]       candidates of each partition
    uint32_t* thr;      // [units][2]           threshold bin d1 and the count needed from it
    uint32_t* mask;     // [units][parts * part / 32] position bitmask
    uint2* seg;         // [units][parts][part] candidate (score bits, position)
    uint64_t* tag;      // [units][parts][kSelectTagWords] publication tags (no initialisation needed)
    uint64_t* epoch;    // [units] exchange epochs (any initial value), or null
    uint64_t call_tag;  // this call's tag: unique within the process (see exchange_tag)
    Exchange xc;
    int32_t fused;      // 1: one kernel (the partitions of a unit exchange while resident)
    int32_t with_draft; // 1: the one kernel also runs the first draft step (d)
    SelectDraft d;
    int32_t n_kv_heads, max_ctx, k_sink, k_recent, budget, batch, part, parts;
    int32_t ctx[kTableBatch];
};

struct DraftArgs {
    const uint16_t* q;      // [batch][n_q][128]
    const uint16_t* k;
    const uint16_t* v;
    const int32_t* idx;     // [batch][n_kv][budget]
    float2* part_ml;        // [n_items][16]       per-workgroup (max, sum) per head
    float* part_o;          // [n_items][16][128]  per-workgroup partial outputs
    uint64_t* tag;          // [n_items] publication tags (no initialisation needed)
    uint64_t* epoch;        // [units] exchange epochs (any initial value), or null
    uint64_t call_tag;      // this call's tag: unique within the process (see exchange_tag)
    Exchange xc;
    void* out;              // [batch][n_q][128]
    int32_t n_q_heads, n_kv_heads, group, max_ctx, budget, chunk, out_fp32;
    float scale_log2;
    SeqTable seq;           // ctx[] holds the entry count per sequence
    // Draft-round step only: entry e < n_fixed[b] is cache row idx[e], or,
    // when k_sel is set, row e of k_sel/v_sel ([batch][n_kv][budget][128], the
    // materialized sink and TopK rows); entry e >= n_fixed[b] is cache row
    // win0[b] + e - n_fixed[b].
    uint16_t* k_sel;        // written by the materialization, read by the steps
    uint16_t* v_sel;
    int32_t n_fixed[kTableBatch];
    int32_t win0[kTableBatch];
    // Paged cache, as in VerifyArgs (plain draft only).
    const int32_t* block_table;
    int32_t page_size, max_blocks;
    // Units are (sequence, head u) with n_kv_heads heads; their K/V rows are
    // those of cache head u / kv_div of n_kv_real (one index set per query
    // head: n_kv_heads = n_q, group 1, kv_div = the GQA group).
    int32_t kv_div, n_kv_real;
};

// Single-sweep verify: the slots (items of v.seq / v.chunk) of one KV-head
// unit must be resident at once.
struct FusedArgs {
    VerifyArgs v;           // part_ml ([slot][64] tagged (max, sum) word pairs) / part_o by slot
    uint64_t* epoch;        // [units] exchange epochs (any initial value), or null
    uint64_t call_tag;      // this call's tag: unique within the process (see exchange_tag)
    Exchange xc;
    // Eager calls on the library's static scratch: epoch words of the call's
    // units to set to heal_value + unit at the end (null otherwise).
    uint64_t* heal;
    uint64_t heal_value;
    // Persistent schedule: n_tasks chunks (work items) over a grid of at most
    // n_tasks workgroups, all resident at once, each taking every grid-th
    // chunk; 0: one workgroup per chunk.
    int32_t n_tasks;
    // Whole decode step (step = 1): after its outputs and scores, each
    // workgroup runs the one-kernel select as partition s (the chunk) of its
    // unit over the scores it has just computed, and then the first draft
    // step over its selections (sel.part = chunk, sel.parts = the most chunks
    // of a unit, sel.with_draft = 1; same call tag, epochs and status word).
    int32_t step;
    SelectArgs sel;
};

// The library's static device scratch (the no-allocation entry point): its
// size, and how to find its address on the current device.
struct StaticScratch {
    size_t bytes;
    hipError_t (*address)(void** ptr);
};


// Launchers return hipSuccess or the error of the launch.
hipError_t launch_verify(const VerifyArgs& a, int n_items, int n_rows_total, int row_tiles,
                         hipStream_t stream);
// Launches the single-sweep kernel over n_slots workgroups (it adds the
// chunks of each row itself; with a.step it also selects and drafts), or,
// with a.n_tasks > 0, the persistent one over a grid of n_slots workgroups.
// Returns the launch error.
hipError_t launch_verify_fused(const FusedArgs& a, int n_slots, int row_tiles, hipStream_t stream);
// The combine kernel alone: out[row] = sum of the row's normalised partials.
hipError_t launch_verify_combine(const VerifyArgs& a, int n_rows_total, hipStream_t stream);
// Largest key chunk the single-sweep kernel can hold in LDS for row_tiles.
int fused_max_chunk(int row_tiles);
// Workgroups of the single-sweep kernel (row_tiles, at its largest LDS use)
// and of the one-kernel select (partition length part) that one CU of the
// current device holds at once; 0 if the device cannot be queried.
int fused_blocks_per_cu(int row_tiles);
int select_blocks_per_cu(int part);
// The persistent single-sweep kernel (FusedArgs.n_tasks > 0): the largest key
// chunk its two 16-bit stash buffers hold (0 for row_tiles it is not built
// for), and its workgroups per CU.
int pipe_max_chunk(int row_tiles);
int pipe_blocks_per_cu(int row_tiles);
// Partition length for the longest context max_t: the smallest multiple of
// 1024 (in powers of two, at most kSelectMaxRounds * 1024) that keeps a unit at
// <= kSelectTargetParts partitions.
int select_part_len(int max_t);
// a.fused chooses the schedule (the caller checks that a unit's partitions fit
// on the device at once).
hipError_t launch_select(const SelectArgs& a, int n_units, hipStream_t stream);
// Calls of at most this many partition workgroups may run as one kernel.
constexpr int kSelectFuseMaxGroups = 256;
// Index entries per draft workgroup for a call of `entries` entries (all
// units) on n_cu CUs: 128, 256 or 512 (32, 64 or 128 per wave).
int draft_chunk_for(int64_t entries, int n_cu);
// One workgroup per `chunk` index entries; no combine kernel.
hipError_t launch_draft(const DraftArgs& a, int n_items, hipStream_t stream);
// Draft round: copy the sink and TopK rows (n_fixed per sequence) of every
// (sequence, KV head) to k_sel/v_sel; then any number of steps over them and
// the slid recent window.
hipError_t launch_draft_materialize(const DraftArgs& a, int max_fixed, int n_units,
                                    hipStream_t stream);
hipError_t launch_draft_step(const DraftArgs& a, int n_items, hipStream_t stream);

// Token statistics of logit rows (entropy, argmax) and greedy acceptance.
constexpr int kLogitChunk = 8192;        // logits per workgroup
constexpr int kLogitMaxChunks = 64;      // chunks per row: vocab <= 524288
constexpr int kAcceptMaxK = 63;          // drafted tokens per sequence (one wave)

struct LogitArgs {
    const void* logits;     // [n_rows][row_stride] bf16 or fp32
    int32_t n_rows, vocab, row_stride, n_chunks;
    float* entropy;         // [n_rows] nats, or null
    int32_t* argmax;        // [n_rows], or null
    float* part;            // [n_rows][n_chunks][4] chunk statistics
    uint64_t* tag;          // [n_rows][n_chunks] publication tags (no initialisation needed)
    uint64_t* epoch;        // [n_rows] exchange epochs (any initial value), or null
    uint64_t call_tag;
    Exchange xc;
    int32_t rows_per_seq;   // acceptance: max_k + 1 (rows past k_len[b] + 1 skipped); else 0
    int32_t k_len[kTableBatch];
};

struct AcceptArgs {
    const int32_t* argmax;  // [batch][max_k + 1]
    const int32_t* draft;   // [batch][max_k]
    int32_t* n_accepted;    // [batch]
    int32_t* next_token;    // [batch]
    int32_t max_k;
    int32_t k_len[kTableBatch];
};

hipError_t launch_logit_stats(const LogitArgs& a, bool f32, hipStream_t stream);
hipError_t launch_greedy_accept(const AcceptArgs& a, int batch, hipStream_t stream);

// Speculative sampling.  Rows of sequence b: target rows 0..max_k of tlogits
// ([batch][max_k + 1][row_stride]) and drafter rows 0..max_k-1 of dlogits
// ([batch][max_k][row_stride]); in the tables below they are rows
// 0..2 max_k of the sequence (drafter row j at max_k + 1 + j).
struct SpecArgs {
    const void* tlogits;
    const void* dlogits;
    int32_t vocab, row_stride, n_chunks, max_k;
    float inv_tau;           // 1 / temperature
    const int32_t* draft;    // [batch][max_k]
    const float* u_acc;      // [batch][max_k] uniforms in [0, 1)
    const float* u_smp;      // [batch]
    int32_t* n_accepted;     // [batch]
    int32_t* next_token;     // [batch]
    float2* chunk_ms;        // [batch][2 max_k + 1][n_chunks] (max, sum) of x / tau per chunk
    float2* row_ms;          // [batch][2 max_k + 1] the same per row
    int32_t* pick;           // [batch] the first failing position (or k)
    float2* mass;            // [batch][n_chunks] (residual, target) mass per chunk
    int32_t k_len[kTableBatch];
};
hipError_t launch_spec_accept(const SpecArgs& a, int batch, bool f32, hipStream_t stream);

}  // namespace ssl
