// launch.h -- argument blocks and launchers shared by the ABI layer (api.cpp)
// and the kernel translation units.  Everything here is internal.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssl {

constexpr int kTableBatch = 64;   // per-sequence tables travel as kernel arguments

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
    float2* part_ml;    // [n_items][64]  per-split (max, sum) in the log2 domain
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
    uint64_t* tag;      // [units][parts][4] publication tags (no initialisation needed)
    uint64_t* epoch;    // [units] exchange epochs (any initial value), or null
    uint64_t call_tag;  // this call's tag: unique within the process (see exchange_tag)
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
    uint64_t* epoch;        // [n_items] exchange epoch of each unit at its first item, or null
    uint64_t call_tag;      // this call's tag: unique within the process (see exchange_tag)
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
    VerifyArgs v;           // part_ml / part_o indexed by slot
    uint64_t* tag;          // [n_slots] publication tags (no initialisation needed)
    uint64_t* epoch;        // [n_slots] exchange epoch of each unit at its first slot, or null
    uint64_t call_tag;      // this call's tag: unique within the process (see exchange_tag)
};

// Launchers return hipSuccess or the error of the launch.
hipError_t launch_verify(const VerifyArgs& a, int n_items, int n_rows_total, int row_tiles,
                         hipStream_t stream);
// Launches the single-sweep kernel over n_slots workgroups (it adds the
// chunks of each row itself).  Returns the launch error.
hipError_t launch_verify_fused(const FusedArgs& a, int n_slots, int row_tiles, hipStream_t stream);
// The combine kernel alone: out[row] = sum of the row's normalised partials.
hipError_t launch_verify_combine(const VerifyArgs& a, int n_rows_total, hipStream_t stream);
// Largest key chunk the single-sweep kernel can hold in LDS for row_tiles.
int fused_max_chunk(int row_tiles);
// Partition length for the longest context max_t: the smallest multiple of
// 1024 (in powers of two, at most kSelectMaxRounds * 1024) that keeps a unit at
// <= kSelectTargetParts partitions.
int select_part_len(int max_t);
hipError_t launch_select(const SelectArgs& a, int n_units, hipStream_t stream);
// One workgroup per `chunk` (128) index entries; no combine kernel.
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

}  // namespace ssl
