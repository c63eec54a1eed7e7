// Internal interface between the C-ABI host layer (api.cpp) and the gfx950 kernels
// (attn_kernels.hip, kv_pages.hip).  Not installed; callers use include/pearl_attn.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/pearl_attn.h"

namespace pearl {

// Thread-local detail message returned by pearl_last_error() (defined in api.cpp).
void clear_error();
pearl_status set_error(pearl_status st, const char* fmt, ...);

constexpr int kPage = 16;            // tokens per KV page
constexpr int kThreads = 512;        // threads per attention workgroup (8 waves of 64)
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerTile = 256;    // q-rows (token x head-in-group) per prefill work item
constexpr int kKeysPerStage = 64;    // keys staged in LDS per prefill step (4 pages)
constexpr int kMinPagesPerSplit = 16;
constexpr int kMaxPagesPerSplit = 512;
// The planner sizes decode splits from the launch's actual pages: about this many decode items
// per compute unit (never fewer pages per split than the host's bound, which sizes the workspace).
constexpr int kDecItemsPerCU = 4;
constexpr int kDecLongSplitPages = 128;
// Compute units assumed when sizing decode splits (MI355X has 256).  A fixed value keeps the
// workspace size a pure function of the shapes; the launch grid uses the device's real count.
constexpr int kPlanComputeUnits = 256;
// Prefill tiles are split along the keys only when the launch has few of them (at most one item
// per compute unit); a split then holds at least kMinSplitKeys keys, and all split items of a
// launch fit in kMaxPreSplitItems partial slots (kRowsPerTile rows each).
constexpr int kMinSplitKeys = 1024;
constexpr int kMaxPreSplitItems = 2 * kPlanComputeUnits;
// Entry encoding of a prefill work item: y = tile | split << 16.
constexpr int kMaxQLen = 1 << 21;        // tiles per sequence < 2^16 (>= 32 tokens per tile)
constexpr int kMaxKvLen = 1 << 25;       // splits per tile < 2^15 (>= 1024 keys per split)

// XCDs (accelerator complex dies) of an MI355X, each with its own L2.
constexpr int kNumXcd = 8;

// Decode batches of up to this many sequences are planned inside the attention kernel (in LDS);
// larger ones go through plan_kernel.
constexpr int kDecPlanMaxSeqs = 1024;

enum Mode : int { kModePrefill = 0, kModeDecode = 1, kModeMixed = 2 };

// Kinds recorded per sequence by the planner.
enum SeqKind : int { kSeqNone = 0, kSeqPrefill = 1, kSeqDecode = 2 };

// Workspace header (int32 words).
enum Hdr : int {
  kHdrCounter = 0,     // dynamic work counter (atomic)
  kHdrNumPre = 1,      // prefill entries
  kHdrNumDec = 2,      // decode split entries
  kHdrError = 3,       // nonzero: a sequence violated the host bounds; nothing is computed
  kHdrNumItems = 4,    // (pre + dec) * H_kv
  kHdrPreSplitKeys = 5,  // keys per prefill split (a multiple of 64); 0 = tiles are not split
  kHdrNumPreJobs = 6,  // prefill tiles with more than one split (merge jobs)
  // word 7: unused
  kHdrPreFirstWG = 8,  // mixed launches: workgroups [0, this) take prefill items first
  kHdrPagesPerSplit = 9,  // pages per decode split chosen by the planner
  kHdrQueues = 16,     // words 16..23: prefill items, one work counter per XCD (atomic)
  kHdrZero = 32,       // words 32..63: a zeroed 128-byte block (source for keys past the end)
  kHdrWords = 64
};

// Per-sequence record written by the planner.
struct SeqInfo {
  int32_t q_start;   // first row of the sequence in q/out
  int32_t q_len;     // new tokens
  int32_t ctx_len;   // cached tokens before the call
  int32_t kind;      // SeqKind | (n_splits << 4) for decode sequences
};

// Offsets (bytes) of the workspace regions; all 256-byte aligned.
struct WsLayout {
  size_t hdr, seqinfo, split_base, entries, part_o, part_ml, pre_jobs, part_pre_o, part_pre_ml, split_cnt, total;
  int64_t max_pre, max_dec;
  int64_t pre_slots;     // partial slots for split prefill items (0: prefill tiles never split)
  int64_t pre_jobs_cap;  // capacity of the prefill merge-job list
};

struct PlanParams {
  int mode;
  int batch;
  int total_q;
  int max_q_len;
  int max_kv_len;
  int bt_stride;
  int num_kv_heads;
  int group;             // G
  int tokens_per_tile;   // kRowsPerTile / G
  int pages_per_split;   // the least pages per decode split (the workspace holds that many splits)
  int64_t max_pre;       // capacity of the prefill entry list
  int64_t max_dec;       // capacity of the decode entry list (and of the partial buffers)
  int64_t pre_slots;     // partial slots for split prefill items
  int64_t pre_jobs_cap;  // capacity of the prefill merge-job list
  int mixed_grid;        // mixed launches: workgroups of the attention grid (0 otherwise)
};

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_table;
  uint16_t* out;
  float* lse;                // may be null
  int32_t* ws_hdr;
  const SeqInfo* seqinfo;
  const int32_t* split_base;
  const int2* entries;
  float* part_o;
  float* part_ml;
  const int4* pre_jobs;      // (sequence, tile, first entry, splits) per split prefill tile
  float* part_pre_o;         // [slot][kRowsPerTile][D] unnormalised partial outputs
  float* part_pre_ml;        // [slot][kRowsPerTile][2] running max (log2 units) and sum
  int32_t* split_cnt;        // [batch][num_kv_heads] splits finished per pair (decode planned in-kernel)
  // fused append and decode (decode planned in-kernel only): the new token's K/V rows
  // [batch][num_kv_heads][D], or null; the pools again, writable
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* k_pool_w;
  uint16_t* v_pool_w;
  int bt_stride;
  int num_pages;
  int num_q_heads;
  int num_kv_heads;
  int group;
  int tokens_per_tile;
  float scale_log2;          // softmax_scale * log2(e)
};

// Arguments of the in-kernel decode plan.
struct DecPlanArgs {
  const int32_t* ctx_lens;
  int batch;
  int max_kv_len;
  int pps_min;           // least pages per split (the host's bound, which sizes the workspace)
  int max_dec;           // partial slots in the workspace
};

WsLayout workspace_layout(int batch, int total_q, int max_kv_len, int num_q_heads,
                          int num_kv_heads, int head_dim, int group, int pages_per_split,
                          bool has_prefill);
int choose_pages_per_split(int batch, int num_kv_heads, int max_kv_len, int num_cu);
int device_num_cu();
// Bytes of the per-device static workspace of pearl_attn_decode_static.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
// Device address of the current device's static workspace (NULL with *err set on failure).  The
// address is taken once per device, on the first call made with that device current.
void* static_scratch(hipError_t* err);
// Workgroups of a full persistent attention grid on the current device (compute units x
// occupancy of the kernel for this head_dim and kinds).
int attention_grid(int head_dim, int kinds);

hipError_t launch_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                            uint16_t* v_pool, const int32_t* block_table, int bt_stride,
                            const int32_t* ctx_lens, const int32_t* cu_q_lens, int batch,
                            int max_q_len, int num_kv_heads, int head_dim, int num_pages,
                            int total_q, hipStream_t stream);

hipError_t launch_kv_pack(const uint16_t* k_pool, const uint16_t* v_pool, uint16_t* k_rows, uint16_t* v_rows,
                          const int32_t* block_table, int bt_stride, const int32_t* ctx_lens,
                          const int32_t* cu_q_lens, int batch, int max_q_len, int num_kv_heads, int head_dim,
                          int num_pages, int total_q, hipStream_t stream);

hipError_t launch_plan(const PlanParams& p, const int32_t* ctx_lens, const int32_t* cu_q_lens,
                       void* workspace, const WsLayout& lay, hipStream_t stream);

// kinds: 1 = prefill tiles only, 2 = decode splits only, 3 = both.
hipError_t launch_attention(const AttnArgs& a, int head_dim, int kinds, int64_t max_items, int max_pre,
                            hipStream_t stream);

hipError_t launch_merge(const AttnArgs& a, int head_dim, int batch, hipStream_t stream);

// Decode planned in-kernel (batch <= kDecPlanMaxSeqs): the zeroing prologue, then the kernel.
hipError_t launch_decode_prologue(const AttnArgs& a, int batch, hipStream_t stream);
hipError_t launch_decode(const AttnArgs& a, const DecPlanArgs& d, int head_dim, int64_t max_items,
                         hipStream_t stream);

// Merge of split prefill tiles; jobs_cap bounds the device-side job count.
hipError_t launch_merge_prefill(const AttnArgs& a, int head_dim, int64_t jobs_cap, hipStream_t stream);

}  // namespace pearl
