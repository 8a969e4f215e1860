// Device-side definitions shared by the HIP kernels and the host launch code.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kvp_plan.h"

namespace kvp {

// One run of tokens of one sequence that falls in one logical page (kv_append / kv_gather).
struct PageRun {
  int32_t row;      // block-table row
  int32_t lpage;    // logical page
  int32_t s_lo;     // first slot written / read
  int32_t s_hi;     // one past the last slot
  int64_t src0;     // token index (in the k / v arrays) of slot s_lo
};
static_assert(sizeof(PageRun) == 24, "PageRun is uploaded as raw bytes");

struct AppendArgs {
  const uint16_t* k;        // [T, Hkv, D]
  const uint16_t* v;
  uint16_t* layer;          // pool layer base
  const int32_t* bt;        // [B, maxp]
  const PageRun* runs;
  int n_runs;
  int maxp, Hkv, num_pages;
  int* err;
  int fp8;                  // FP8 pool: quantise with the inverse scales
  float inv_scale_k, inv_scale_v;
};

struct GatherArgs {
  uint16_t* k;              // [T, Hkv, D] out
  uint16_t* v;
  const uint16_t* layer;
  const int32_t* bt;
  const PageRun* runs;
  int n_runs;
  int maxp, Hkv, num_pages;
  int* err;
  int fp8;                  // FP8 pool: dequantise with the scales
  float scale_k, scale_v;
};

struct DecodeArgs {
  const uint16_t* q;        // [B, Hq, D] bf16
  const uint16_t* layer;
  const int32_t* bt;
  int maxp;
  const DecodeItem* items;    // wave path: chunks in segment order
  int n_items;                // wave path: segment count
  const int32_t* seg_off;     // wave path: [segments + 1] chunk offsets
  const DecodeItem* group_items;  // shared-prefix path (LDS-staged, > 16 query columns)
  int n_group_items;
  int n_group_blocks;         // n_group_items * Hkv
  int n_wave_blocks;          // ceil(segments * Hkv / 4): one wave per (segment, KV head)
  const int32_t* members;
  const int32_t* part_base;
  float* part_acc;          // [parts, Hq, D]
  float2* part_ml;          // [parts, Hq] (running max in log2 units, sum of weights)
  void* out;                // [B, Hq, D]
  int out_f32;
  int Hq, Hkv, G, num_pages;
  float scale_log2;         // scale * log2(e) (times the K scale of an FP8 pool)
  float v_scale;            // 1, or the V scale of an FP8 pool (applied to the output)
  int fp8;                  // pages are FP8 E4M3
  int* err;
};

struct MergeArgs {
  const int32_t* merge_info;  // per merged sequence: {seq, first partial index, partial count, 0}
  int n_merge;
  const float* part_acc;
  const float2* part_ml;
  void* out;
  int out_f32;
  int Hq, Hkv;
  int hw;                     // query heads per merge workgroup (set by launch_decode_merge)
};

struct PrefillArgs {
  const uint16_t* q;        // [sum C, Hq, D]
  const uint16_t* layer;
  const int32_t* bt;
  int maxp;
  const PrefillItem* items;
  int n_items;
  const int32_t* ctx_lens;  // device copies
  const int32_t* cu_q;
  const int32_t* part_base; // [B] first partial of each session (split sessions only)
  const int32_t* nsplit;    // [B] key ranges per query row
  float* part_acc;          // [parts, Hq, D] unnormalised accumulators of split tiles
  float2* part_ml;          // [parts, Hq] (running max in log2 units, weight sum)
  void* out;
  int out_f32;
  int Hq, Hkv, G, num_pages;
  float scale_log2;         // scale * log2(e) (times the K scale of an FP8 pool)
  float v_scale;            // 1, or the V scale of an FP8 pool
  int fp8;
  int* err;
};

// One page moved between the pool and the host tier; row / lpage name the block-table entry a restore
// points at the page (ignored when no table is patched).
struct TierItem {
  int32_t page, row, lpage, pad;
};

struct TierArgs {
  unsigned char* layer;     // pool layer base
  unsigned char* host;      // pinned host pages, item i at host + i * page_bytes
  int64_t page_bytes;
  const TierItem* items;    // n items (read from pinned host memory)
  int n;
  int32_t* bt;              // device block tables to patch, or NULL
  int maxp;
};

// Block hashing works on chunks of up to 64 full pages of one sequence.
struct HashChunk {
  int32_t t0;               // first token of the chunk
  int32_t o0;               // first output slot of the chunk
  int32_t n;                // pages in the chunk (1..64)
  int32_t c;                // chunk index within its sequence
  int32_t g0;               // index of the sequence's first chunk in `totals`
  int32_t pad[3];           // lookup: the sequence's chunk count, the sequence, its full pages
};

struct HashArgs {
  const int32_t* tokens;
  const HashChunk* chunks;  // [n_chunks] (pinned host)
  uint64_t seed;
  uint64_t* out;            // [total full pages]; chunk-local chain values between the two passes
  uint64_t* totals;         // [2 * n_chunks] scratch: each chunk's composed map (slope, offset)
};

struct GroupLcpArgs {
  const uint64_t* hashes;
  const int4* seq_info;     // as in HashArgs
  const int32_t* grp_off;   // [num_groups + 1] offsets into members (pinned host)
  const int32_t* members;   // sequence ids of each group's members
  int32_t* shared_pages;    // [num_groups] device output
};

struct TableArgs {
  uint64_t* keys;           // [mask + 1]
  int32_t* vals;            // [mask + 1]
  uint64_t mask;
  const uint64_t* hashes;   // insert / erase: [n]; lookup: per-page hashes laid out as seq_info says
  const int32_t* pages;     // insert / erase: [n]
  int64_t n;
  const HashChunk* chunks;  // lookup: 64-page chunks of the sequences (pinned host)
  int32_t* first_miss;      // lookup scratch: [chunks]
  int32_t* matched;         // lookup: [num_seqs]
  int32_t* out_pages;       // lookup: [total full pages]
  int* err;
};

hipError_t launch_append(const AppendArgs& a, int D, hipStream_t s);
hipError_t launch_gather(const GatherArgs& a, int D, hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
// Copy n bytes from pinned host memory (src) to device memory (dst; 16-byte aligned, like src) with a
// kernel on stream s.
hipError_t launch_copy_from_host(void* dst, const void* src, size_t n, hipStream_t s);
hipError_t launch_decode(const DecodeArgs& a, int D, hipStream_t s);
// Copy n host bytes (n rounded up to 16; dst 16-byte aligned) to device memory on stream s through the
// launch arguments of small kernels: asynchronous, and neither side needs an allocation.
hipError_t launch_put_bytes(void* dst, const void* src, size_t n, hipStream_t s);
hipError_t launch_decode_merge(const MergeArgs& a, int D, hipStream_t s);
hipError_t launch_prefill(const PrefillArgs& a, int D, hipStream_t s);
// One launch of decode wave-path blocks followed by prefill blocks (mixed.hip; the decode's LDS-staged
// prefix blocks are not part of it); the decode block count is padded to a multiple of 8 so each prefill
// item keeps its planned XCD.
hipError_t launch_mixed_step(const DecodeArgs& d, const PrefillArgs& p, int D, bool fp8, hipStream_t s);
int mixed_step_decode_blocks(const DecodeArgs& d);
hipError_t launch_tier(const TierArgs& a, bool restore, hipStream_t s);
hipError_t launch_block_hash(const HashArgs& a, int n_chunks, hipStream_t s);
hipError_t launch_group_lcp(const GroupLcpArgs& a, int n_groups, hipStream_t s);
// op: 0 insert, 1 erase, 2 lookup, 3 clear
hipError_t launch_table(const TableArgs& a, int op, int n_seqs, hipStream_t s);

}  // namespace kvp
