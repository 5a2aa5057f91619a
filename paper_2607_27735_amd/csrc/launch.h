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
};

struct SelectArgs {
    const float* scores;
    int32_t* idx;
    int32_t* n_idx;
    int32_t n_kv_heads, max_ctx, k_sink, k_recent, budget, batch;
    int32_t ctx[kTableBatch];
};

struct DraftArgs {
    const uint16_t* q;      // [batch][n_q][128]
    const uint16_t* k;
    const uint16_t* v;
    const int32_t* idx;     // [batch][n_kv][budget]
    float2* part_ml;        // [n_items][16]
    float* part_o;          // [n_items][16][128]
    void* out;              // [batch][n_q][128]
    int32_t n_q_heads, n_kv_heads, group, max_ctx, budget, chunk, out_fp32;
    float scale_log2;
    SeqTable seq;           // ctx[] holds n_idx per sequence
};

// Single-sweep verify: every work item of the launch is resident at once
// (cooperative launch), items of KV-head unit u are slots
// [slot_start[u], slot_start[u + 1]), each covering `chunk` keys.
constexpr int kFusedMaxUnits = 128;

struct FusedTable {
    int32_t n_units;
    int32_t chunk;
    int32_t unit[kFusedMaxUnits];            // b * n_kv_heads + c
    int32_t slot_start[kFusedMaxUnits + 1];
};

struct FusedArgs {
    VerifyArgs v;           // part_ml / part_o are indexed by slot
    uint32_t* arrive;       // [n_units] arrival counters, zero at launch
    FusedTable ft;
};

// Launchers return hipSuccess or the error of the launch.
hipError_t launch_verify(const VerifyArgs& a, int n_items, int n_rows_total, int row_tiles,
                         hipStream_t stream);
// Zeroes the arrival counters, then launches the single-sweep kernel as a
// cooperative grid of n_slots workgroups.  Returns the launch error (for
// instance when the grid cannot be co-resident; nothing has run then except
// the counter fill).
hipError_t launch_verify_fused(const FusedArgs& a, int n_slots, int row_tiles, hipStream_t stream);
// Largest key chunk the single-sweep kernel can hold in LDS for row_tiles.
int fused_max_chunk(int row_tiles);
hipError_t launch_select(const SelectArgs& a, int n_units, hipStream_t stream);
hipError_t launch_draft(const DraftArgs& a, int n_items, int n_rows_total, hipStream_t stream);

}  // namespace ssl
