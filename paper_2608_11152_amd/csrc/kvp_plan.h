// Host-side planning for the paged attention kernels: validation of host metadata and the split-KV /
// shared-prefix work lists the kernels consume.  Pure C++ (no HIP), so it builds and tests on a CPU.
#pragma once
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/kvpattn.h"

namespace kvp {

constexpr int kPage = 16;
constexpr int kMaxColsPerWave = 16;   // query columns one wave's MFMA tile holds (members x heads)
constexpr int kMaxColsPerGroup = 64;  // query columns one shared-prefix workgroup holds (4 waves)
constexpr int kMinSegmentPages = 8;   // smallest page count of a decode wave segment
// A wave chunk's start (its item, query fragments and first page ids are dependent reads) in pages of
// streaming: bf16 pages, and FP8 pages (half the bytes, so a start is worth more of them).
constexpr int kChunkStartPages = 3;
constexpr int kChunkStartPagesFp8 = 5;
constexpr int kGroupChunkPages = 16;  // pages per workgroup of the LDS-staged shared-prefix kernel
// Decode waves per call: one round of the waves resident at once on 256 CUs (4 SIMDs x 2 waves each).
// Sweeps of 1024-16384 put the optimum here on the target workloads.
constexpr int kDecodeWaves = 2048;

// One unit of decode work: one KV head of it is processed by one wave (private, <= 16 query columns)
// or one 4-wave workgroup (shared prefix, <= 64 query columns).  Mirrors kvp_plan_decode's 8 ints.
struct DecodeItem {
  int32_t kind;      // 0 = private range of one sequence, 1 = shared prefix of a group (or subgroup)
  int32_t row;       // block-table row the pages are read from
  int32_t page_lo;   // first logical page
  int32_t page_hi;   // one past the last logical page
  int32_t tok_end;   // tokens [0, tok_end) of the row are valid
  int32_t mem_off;   // first entry in the member list (sequence ids owning the query columns)
  int32_t n_mem;     // member count; query columns = n_mem * G
  int32_t slot;      // partial index within each member's list, -1 = write the final output directly
};
static_assert(sizeof(DecodeItem) == 32, "DecodeItem is uploaded as raw bytes");

struct DecodePlan {
  std::vector<DecodeItem> wave_items;   // chunks in segment order (private and <= 16-column prefix)
  std::vector<int32_t> seg_off;         // [segments + 1]: chunks of segment s are seg_off[s]..seg_off[s+1]
  std::vector<DecodeItem> group_items;  // prefix items with 16 < n_mem * G <= 64 (LDS-staged kernel)
  std::vector<int32_t> members;         // member lists referenced by items
  std::vector<int32_t> part_base;       // [B] first partial index of each sequence
  std::vector<int32_t> n_parts;         // [B] partial count of each sequence
  std::vector<int32_t> merge_seqs;      // sequences whose output the merge kernel writes (0 or >= 2 parts)
  int32_t total_parts = 0;
  int32_t pages_per_split = 0;          // pages per wave segment
  int32_t group_reserved_blocks = 0;    // block slots the wave budget leaves to the shared-prefix path
};

// Prefill: one 4-wave workgroup per (session, kv head, 128-row query tile, key range).  The key range is
// a run of 64-key stages [st_lo, st_hi) (st_hi is clamped to the tile's own last stage); a tile whose
// history is split over several workgroups writes one partial softmax state per range, merged per query
// row by log-sum-exp afterwards.
struct PrefillItem {
  int32_t seq;       // session index (block-table row)
  int32_t kvh;       // KV head
  int32_t row0;      // first flattened query row (position * G + head-in-group) of the tile
  int32_t st_lo;     // first 64-key stage of the range (st_lo * 64 <= the session's cached length)
  int32_t st_hi;     // one past the last stage of the range
  int32_t slot;      // partial index of the range within each query row's list, -1 = write the output
  int32_t pad[2];
};
static_assert(sizeof(PrefillItem) == 32, "PrefillItem is uploaded as raw bytes");

struct PrefillPlan {
  std::vector<PrefillItem> items;  // blockIdx order (XCD-aware, empty entries have seq = -1)
  int64_t real_items = 0;
  std::vector<int32_t> nsplit;     // [B] key ranges per query row of each session (1 = not split)
  std::vector<int32_t> part_base;  // [B] first partial of each session (its row r owns part_base + r * nsplit)
  std::vector<int32_t> merge_info; // per merged query row: {row in q / out, first partial, nsplit, 0}
  int32_t total_parts = 0;
};

struct Status {
  int code = KVP_OK;
  std::string msg;
  bool ok() const { return code == KVP_OK; }
};

Status validate_group_prefix(const int32_t* lens, int B, const kvp_group_prefix* gp);
// chunk_start_pages: the start cost a segment's budget charges per chunk (kChunkStartPages for bf16
// pools, kChunkStartPagesFp8 for FP8 pools).
Status plan_decode(const int32_t* seq_lens, int B, int maxp, const kvp_group_prefix* gp, int Hq, int Hkv,
                   DecodePlan* plan, int chunk_start_pages = kChunkStartPages);
Status plan_prefill(const int32_t* ctx_lens, const int32_t* cu_q, int B, int maxp, int Hq, int Hkv,
                    PrefillPlan* plan);
Status check_tables(const int32_t* bt, int maxp, const int32_t* lens, int B, int num_pages,
                    const kvp_group_prefix* gp);

constexpr int kPrefillWaves = 8;                    // waves per prefill workgroup, 32 query rows each
constexpr int kPrefillRows = 32 * kPrefillWaves;    // flattened query rows per prefill workgroup
// A call whose tiles (x their 64-key stages) would not give about this many equal workgroups splits
// tile histories into key ranges: the resident prefill workgroups of 256 CUs (8 waves per CU).
constexpr int kPrefillSplitTarget = 256 * 8 / kPrefillWaves;
constexpr int kPrefillMinSplitStages = 8;  // smallest key range of a split (512 keys)

}  // namespace kvp
