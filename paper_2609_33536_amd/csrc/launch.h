// Host-side launchers of the libekv kernels (internal header).  The C ABI in
// api.hip validates arguments and calls these; each launcher only enqueues.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ekv {

struct DecodeArgs {
  const uint16_t* pool;      // [NB][2][Hkv][16][128]
  const uint16_t* q;         // [B][Hq][128]
  const int32_t* seq_lens;   // [B]
  const int32_t* bt;         // [B][max_blocks]
  const uint8_t* tags;       // [B][max_blocks] or null
  const int32_t* bounds;     // [B][2] or null
  float* ws_o;               // [2 grid][G][128] partial outputs, two slots per workgroup
  float* ws_ml;              // [2 grid][G][2]   partial (max, sum)
  uint32_t* counters;        // [2 grid] merge counters (at a cut (seq, KV head)'s piece-0 slot), zero between calls
  void* out;                 // [B][Hq][128]
  int32_t batch, num_kv_heads, num_q_heads, max_blocks;
  int32_t num_blocks;        // pool size: table entries are clamped into it
  int32_t len_cap;           // sequence lengths are clamped to this (max_seq_len)
  int32_t min_chunk;         // fewest pairs a workgroup streams
  int32_t grid;              // workgroups launched (decode_grid of the same arguments; the workspace has 2 grid slots)
  int64_t pairs_max;         // upper bound on the pairs of all (seq, KV head)s
  int32_t out_fp32;
  int32_t slots;             // LDS ring depth per wave (2..4)
  int32_t heavy;             // leading workgroups with longer ranges (set by the launcher)
  int32_t heavy_permille;    // their range length over the mean, x 1000
  float scale_log2;          // softmax scale * log2(e)
  // Fused append (null otherwise): the K / V rows of each sequence's newest
  // token (position seq_lens[s] - 1), [B][Hkv][128] in the pool's element
  // type, replace that token's rows where decode reads them and are written
  // to the pool (pool_out: the same pool, writable).
  const void* k_new;
  const void* v_new;
  void* pool_out;
};

// Most workgroups one decode launch uses (a cap on the resident grid).
constexpr int kMaxDecodeGrid = 4096;

// dtype: 0 bf16, 1 fp16, 3 8-bit.  elastic: false = native path (tags never read).
hipError_t launch_decode(const DecodeArgs& a, int dtype, int group, bool elastic, hipStream_t st);
// The grid launch_decode would use for these arguments (min_chunk, pairs_max
// and slots must be set): the resident workgroups of the kernel instance,
// or fewer for small work.
hipError_t decode_grid(const DecodeArgs& a, int dtype, int group, bool elastic, int* grid);
hipError_t launch_zero_u32(uint32_t* p, size_t n, hipStream_t st);

struct TransitionArgs {
  uint16_t* pool;            // the pool of a single-layer call
  const uint64_t* layers;    // device [num_layers] pool addresses, or null (single layer: pool)
  const int32_t* pairs;      // [n][2] = (s, j)
  const int32_t* new_blocks; // refine: [n]
  int32_t* bt;               // [B][max_blocks]
  uint8_t* tags;             // [B][max_blocks]
  int32_t* freed;            // demote: [n]
  uint8_t* lo;               // demote: lo_out (nullable); refine: lo_in; [n][num_layers][one block]
  int32_t n, num_kv_heads, max_blocks;
  int32_t num_layers;        // 1 for a single-layer call
  int32_t staged;            // refine: pair i's refinement bytes are in block new_blocks[i] (lo unused)
  int32_t elem8;             // 8-bit TARGET / 4-bit BASE pool (else 16-bit / 8-bit)
  int32_t batch;             // rows of bt and tags: pairs outside them are skipped
  int32_t num_blocks;        // pool size: pairs whose blocks lie outside it are skipped
};

hipError_t launch_demote(const TransitionArgs& a, hipStream_t st);
hipError_t launch_refine(const TransitionArgs& a, hipStream_t st);

// Block copies of one launch; the addresses travel in the kernel arguments.
constexpr int kStageMax = 256;
struct StageArgs {
  uint8_t* pool;
  int64_t block_bytes;                  // a multiple of 4096
  const uint8_t* src[kStageMax];        // device-readable address of source i's block bytes
  int32_t dst[kStageMax];               // destination block of source i
  int32_t n;                            // 1..kStageMax
};

hipError_t launch_stage(const StageArgs& a, hipStream_t st);

struct AppendArgs {
  uint16_t* pool;
  const int32_t* slots;
  const uint16_t* k;
  const uint16_t* v;
  int32_t n, num_kv_heads;
  int32_t elem8;             // 1-byte elements
  int32_t num_blocks;        // pool size: slots outside it are skipped
};

hipError_t launch_append(const AppendArgs& a, hipStream_t st);

struct PrefillArgs {
  const uint16_t* pool;
  const uint16_t* q;         // [total][Hq][128]
  const int32_t* cu_q;       // [B+1]
  const int32_t* seq_lens;   // [B]
  const int32_t* bt;
  const uint8_t* tags;
  const int32_t* bounds;
  void* out;                 // [total][Hq][128]
  int32_t batch, num_kv_heads, num_q_heads, max_blocks, max_q_len, out_fp32;
  int32_t num_blocks;        // pool size: table entries are clamped into it
  int32_t total_q;           // rows of q and out: query offsets are clamped into them
  float scale_log2;
};

// dtype: 0 bf16, 1 fp16, 3 8-bit (E5M2 TARGET / 4-bit BASE, FP16 queries).
hipError_t launch_prefill(const PrefillArgs& a, int dtype, int group, bool elastic, hipStream_t st);

struct ValidateBatchArgs {
  const int32_t* seq_lens;   // [B]
  const int32_t* bt;         // [B][max_blocks]
  const uint8_t* tags;       // [B][max_blocks] or null
  const int32_t* bounds;     // [B][2] or null
  int32_t* report;           // [2 * EKV_VIOL_COUNT]
  int32_t batch, max_blocks, num_blocks, max_seq_len, mode;
};

struct ValidateListArgs {
  const int32_t* pairs;      // [n][2]
  const int32_t* new_blocks; // [n] or null
  const int32_t* bt;         // [B][max_blocks]
  const uint8_t* tags;       // [B][max_blocks]
  const int32_t* seq_lens;   // [B] or null
  int32_t* report;           // [2 * EKV_VIOL_COUNT]
  int32_t n, kind, batch, max_blocks, num_blocks;
};

// Both initialise the report, then count into it.
hipError_t launch_validate_batch(const ValidateBatchArgs& a, hipStream_t st);
hipError_t launch_validate_list(const ValidateListArgs& a, hipStream_t st);

}  // namespace ekv
