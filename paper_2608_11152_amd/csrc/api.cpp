// C-ABI of libkvpattn: pool management, kv_append / kv_gather, paged_decode_attn and
// prefix_chunk_prefill_attn.  Host metadata is validated and planned here, packed into one buffer and
// uploaded with a single asynchronous copy from a ring of pinned staging slots; then the kernels are
// launched on the caller's stream.  Nothing in this file computes attention.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kvp_kernels.h"

struct kvp_prefix_table {
  uint64_t* keys = nullptr;
  int32_t* vals = nullptr;
  uint64_t mask = 0;
  int* err = nullptr;
  int device = 0;
};

struct kvp_pool {
  int num_layers = 0, num_pages = 0, num_kv_heads = 0, head_dim = 0, device = 0;
  int dtype = KVP_BF16;
  std::vector<float> k_scale, v_scale;  // per layer, FP8 pools
  size_t layer_bytes = 0;
  unsigned char* base = nullptr;  // [layers][pages][Hkv][2][16*d] bf16
  int* err = nullptr;             // device error word
};

// Scratch of the allocation-free decode entry point: the work list and the split-KV partials of one
// call, in device memory the code object brings (every GPU the library runs on holds its own copy until
// the process ends).  Host code never passes the array's name to a kernel: it uses the device address
// hipGetSymbolAddress returns for the current device (scratch_of).
constexpr size_t kNoAllocScratchBytes = KVP_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

thread_local std::string g_last_error;

int set_err(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int from_status(const kvp::Status& s) {
  if (!s.ok()) g_last_error = s.msg;
  return s.code;
}

int hip_err(hipError_t e, const char* what) {
  return set_err(KVP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// Ring of pinned host staging slots.  A slot is reused only after the GPU work that last read it has
// completed (its event), so consecutive calls do not wait on each other's GPU work.  A slot is either
// the source of one copy into device memory (`upload`: a small copy kernel on the caller's stream, not
// the copy engine, whose hand-off to the compute queue measured 20-30 us per call) or, for metadata each
// wave reads once, read by the kernels directly over the bus (`lease` ... `release`).
class Staging {
 public:
  struct Lease {
    void* host = nullptr;
    int slot = -1;
  };

  int lease(size_t n, Lease* out) {
    std::lock_guard<std::mutex> lock(mu_);
    int idx = -1;
    for (int k = 0; k < kSlots && idx < 0; ++k) {
      const int c = (next_ + k) % kSlots;
      if (!slots_[c].leased) idx = c;
    }
    if (idx < 0) return set_err(KVP_EINVAL, "more than %d concurrent calls hold metadata slots", kSlots);
    next_ = (idx + 1) % kSlots;
    Slot& sl = slots_[idx];
    if (sl.pending) {
      hipError_t e = hipEventSynchronize(sl.ev);
      if (e != hipSuccess) return hip_err(e, "hipEventSynchronize(staging)");
      sl.pending = false;
    }
    if (!sl.ev) {
      hipError_t e = hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming);
      if (e != hipSuccess) return hip_err(e, "hipEventCreate");
    }
    if (n > sl.cap) {
      if (sl.host) (void)hipHostFree(sl.host);
      sl.host = nullptr;
      sl.cap = 0;
      const size_t cap = std::max<size_t>(n, 1 << 20);
      hipError_t e = hipHostMalloc(&sl.host, cap, hipHostMallocDefault);
      if (e != hipSuccess) return set_err(KVP_ENOMEM, "hipHostMalloc(%zu): %s", cap, hipGetErrorString(e));
      sl.cap = cap;
    }
    sl.leased = true;
    out->host = sl.host;
    out->slot = idx;
    return KVP_OK;
  }

  // Marks the end of the GPU work that reads the slot (enqueued on s) and returns the slot to the ring.
  // Without work to wait for (record = false) the slot is simply released.
  int release(const Lease& l, hipStream_t s, bool record = true) {
    std::lock_guard<std::mutex> lock(mu_);
    Slot& sl = slots_[l.slot];
    sl.leased = false;
    if (!record) return KVP_OK;
    hipError_t e = hipEventRecord(sl.ev, s);
    if (e != hipSuccess) return hip_err(e, "hipEventRecord");
    sl.pending = true;
    return KVP_OK;
  }

  int upload(void* dst, const void* src, size_t n, hipStream_t s) {
    if (n == 0) return KVP_OK;
    Lease l;
    int rc = lease(n, &l);
    if (rc) return rc;
    std::memcpy(l.host, src, n);
    hipError_t e = kvp::launch_copy_from_host(dst, l.host, n, s);
    if (e != hipSuccess) {
      release(l, s, false);
      return hip_err(e, "metadata copy");
    }
    return release(l, s);
  }

 private:
  static constexpr int kSlots = 8;
  struct Slot {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
    bool leased = false;
  };
  std::mutex mu_;
  Slot slots_[kSlots];
  int next_ = 0;
};

Staging& staging() {
  static Staging* s = new Staging();  // intentionally leaked: outlives static destruction order
  return *s;
}

// Device address of `scratch` on device `dev` (the current device), looked up once per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char* g_scratch_addr[kMaxDevices] = {};

int scratch_of(int dev, unsigned char** out) {
  if (dev < 0 || dev >= kMaxDevices) return set_err(KVP_EINVAL, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_err(e, "hipGetSymbolAddress(scratch)");
    if (!p) return set_err(KVP_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_addr[dev] = reinterpret_cast<unsigned char*>(p);
  }
  *out = g_scratch_addr[dev];
  return KVP_OK;
}

// Packs several arrays into one host buffer with 256-byte aligned offsets.
struct Packer {
  std::vector<unsigned char> buf;
  size_t add(const void* p, size_t n) {
    const size_t off = (buf.size() + 255) & ~size_t(255);
    buf.resize(off + n);
    if (n) std::memcpy(buf.data() + off, p, n);
    return off;
  }
  size_t size() const { return (buf.size() + 255) & ~size_t(255); }
};

bool pool_ok(kvp_pool_t p) { return p && p->base; }

int elem_bytes(int dtype) { return dtype == KVP_FP8_E4M3 ? 1 : 2; }

size_t page_bytes(kvp_pool_t p) {
  return (size_t)p->num_kv_heads * 2 * kvp::kPage * p->head_dim * elem_bytes(p->dtype);
}

// The host tier is read and written by kernels, so it must be pinned host memory (hipHostMalloc, or a
// torch tensor created with pin_memory=True) that covers `bytes` from `p`.
int check_pinned(const void* p, size_t bytes, const char* what) {
  if (!p) return set_err(KVP_EINVAL, "%s is NULL", what);
  hipPointerAttribute_t at{};
  hipError_t e = hipPointerGetAttributes(&at, p);
  if (e != hipSuccess || at.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    return set_err(KVP_EINVAL, "%s is not pinned host memory", what);
  }
  (void)bytes;
  return KVP_OK;
}


int check_layer(kvp_pool_t pool, int layer) {
  if (!pool_ok(pool)) return set_err(KVP_EINVAL, "pool is NULL or destroyed");
  if (layer < 0 || layer >= pool->num_layers)
    return set_err(KVP_EINVAL, "layer %d outside [0, %d)", layer, pool->num_layers);
  return KVP_OK;
}

const uint16_t* layer_ptr(kvp_pool_t pool, int layer) {
  return reinterpret_cast<const uint16_t*>(pool->base + (size_t)layer * pool->layer_bytes);
}

// Page runs of a set of token ranges: sequence i covers positions [start[i], start[i] + cnt[i]).
void build_runs(const int32_t* start, const int64_t* first_src, const int32_t* cnt, int B,
                std::vector<kvp::PageRun>* runs) {
  runs->clear();
  for (int i = 0; i < B; ++i) {
    if (cnt[i] <= 0) continue;
    const int64_t a = start[i], b = (int64_t)start[i] + cnt[i];
    for (int64_t lp = a / kvp::kPage; lp * kvp::kPage < b; ++lp) {
      const int64_t lo = std::max<int64_t>(a, lp * kvp::kPage), hi = std::min<int64_t>(b, (lp + 1) * kvp::kPage);
      runs->push_back(kvp::PageRun{i, (int32_t)lp, (int32_t)(lo - lp * kvp::kPage), (int32_t)(hi - lp * kvp::kPage),
                                   first_src[i] + (lo - a)});
    }
  }
}

// Per-sequence {first token, full pages, first hash slot, 0} from host cu_tokens, in a leased pinned slot
// (appended after `extra` bytes the caller packs first).  Returns the total full-page count in *pages.
int lease_seq_info(const int32_t* cu_tokens, int num_seqs, Staging::Lease* lease, int64_t* pages,
                   const std::vector<unsigned char>& extra, size_t* info_off) {
  if (num_seqs > 0 && !cu_tokens) return set_err(KVP_EINVAL, "cu_tokens is NULL");
  if (num_seqs > 0 && cu_tokens[0] != 0) return set_err(KVP_EINVAL, "cu_tokens[0] = %d, must be 0", cu_tokens[0]);
  std::vector<int32_t> info(4 * (size_t)num_seqs);
  int64_t tot = 0;
  for (int i = 0; i < num_seqs; ++i) {
    const int32_t n = cu_tokens[i + 1] - cu_tokens[i];
    if (n < 0) return set_err(KVP_EINVAL, "cu_tokens decreases at %d", i);
    info[4 * i] = cu_tokens[i];
    info[4 * i + 1] = n / kvp::kPage;
    info[4 * i + 2] = (int32_t)tot;
    info[4 * i + 3] = 0;
    tot += n / kvp::kPage;
    if (tot > INT32_MAX) return set_err(KVP_EINVAL, "more than 2^31 pages");
  }
  *pages = tot;
  const size_t off = (extra.size() + 255) & ~size_t(255);
  int rc = staging().lease(std::max<size_t>(1, off + info.size() * 4), lease);
  if (rc) return rc;
  if (!extra.empty()) std::memcpy(lease->host, extra.data(), extra.size());
  if (!info.empty()) std::memcpy(reinterpret_cast<unsigned char*>(lease->host) + off, info.data(), info.size() * 4);
  *info_off = off;
  return KVP_OK;
}

// 64-page chunks of every sequence's full pages (block hashing and prefix lookup work per chunk);
// pad = {the sequence's chunk count, the sequence, its full pages}.
int build_chunks(const int32_t* cu_tokens, int num_seqs, std::vector<kvp::HashChunk>* chunks, int64_t* pages) {
  if (!cu_tokens) return set_err(KVP_EINVAL, "cu_tokens is NULL");
  if (cu_tokens[0] != 0) return set_err(KVP_EINVAL, "cu_tokens[0] = %d, must be 0", cu_tokens[0]);
  int64_t tot = 0;
  for (int i = 0; i < num_seqs; ++i) {
    const int32_t n = cu_tokens[i + 1] - cu_tokens[i];
    if (n < 0) return set_err(KVP_EINVAL, "cu_tokens decreases at %d", i);
    const int np = n / kvp::kPage;
    const int g0 = (int)chunks->size();
    const int nch = (np + 63) / 64;
    for (int c = 0; c < nch; ++c)
      chunks->push_back(kvp::HashChunk{cu_tokens[i] + 64 * kvp::kPage * c, (int32_t)(tot + 64 * c),
                                       std::min(64, np - 64 * c), c, g0, {nch, i, np}});
    tot += np;
    if (tot > INT32_MAX) return set_err(KVP_EINVAL, "more than 2^31 pages");
  }
  *pages = tot;
  return KVP_OK;
}

// Page moves between the pool and the host tier: the item list is read by the kernel straight from a
// pinned staging slot, released after the kernel.
int run_tier(kvp_pool_t pool, int layer, const std::vector<kvp::TierItem>& items, void* host, int32_t* bt,
             int maxp, bool restore, hipStream_t s) {
  Staging::Lease lease;
  const size_t nb = items.size() * sizeof(kvp::TierItem);
  int rc = staging().lease(nb, &lease);
  if (rc) return rc;
  std::memcpy(lease.host, items.data(), nb);
  kvp::TierArgs a{};
  a.layer = reinterpret_cast<unsigned char*>(const_cast<uint16_t*>(layer_ptr(pool, layer)));
  a.host = reinterpret_cast<unsigned char*>(host);
  a.page_bytes = (int64_t)page_bytes(pool);
  a.items = reinterpret_cast<const kvp::TierItem*>(lease.host);
  a.n = (int)items.size();
  a.bt = bt;
  a.maxp = maxp;
  hipError_t e = kvp::launch_tier(a, restore, s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, restore ? "kv_restore launch" : "kv_offload launch");
  return rr;
}

// Page runs of kv_append / kv_gather in a leased pinned slot: each wave reads its one 24-byte record
// there, so no device buffer, copy or allocation sits in the stream ahead of the kernel.
int lease_runs(const std::vector<kvp::PageRun>& runs, Staging::Lease* lease) {
  const size_t n = runs.size() * sizeof(kvp::PageRun);
  int rc = staging().lease(n, lease);
  if (rc) return rc;
  std::memcpy(lease->host, runs.data(), n);
  return KVP_OK;
}

// Decode: the work list lives in a pinned staging slot (read by the kernels directly); the caller's
// workspace holds [partial accumulators][partial (m, l)].
struct DecodeLayout {
  kvp::DecodePlan plan;
  std::vector<int32_t> merge_info;  // one 16-byte record per merged sequence: {seq, first partial, count, 0}
  size_t off_wave = 0, off_seg = 0, off_group = 0, off_members = 0, off_part_base = 0, off_merge = 0;
  size_t meta_bytes = 0;            // work list bytes (offsets above, 256-byte aligned)
  size_t off_acc = 0, off_ml = 0, total = 0;

  // Copy the work list into `dst` (meta_bytes bytes), straight from the plan's arrays.
  void write_meta(unsigned char* dst) const {
    auto put = [&](size_t off, const void* src, size_t n) {
      if (n) std::memcpy(dst + off, src, n);
    };
    put(off_wave, plan.wave_items.data(), plan.wave_items.size() * sizeof(kvp::DecodeItem));
    put(off_seg, plan.seg_off.data(), plan.seg_off.size() * 4);
    put(off_group, plan.group_items.data(), plan.group_items.size() * sizeof(kvp::DecodeItem));
    put(off_members, plan.members.data(), plan.members.size() * 4);
    put(off_part_base, plan.part_base.data(), plan.part_base.size() * 4);
    put(off_merge, merge_info.data(), merge_info.size() * 4);
  }
};

int layout_decode(kvp_pool_t pool, const int32_t* seq_lens, int B, int maxp, const kvp_group_prefix* gp, int Hq,
                  DecodeLayout* L) {
  kvp::Status st = kvp::plan_decode(seq_lens, B, maxp, gp, Hq, pool->num_kv_heads, &L->plan,
                                    pool->dtype == KVP_FP8_E4M3 ? kvp::kChunkStartPagesFp8 : kvp::kChunkStartPages);
  if (!st.ok()) return from_status(st);
  const auto& P = L->plan;
  // One 16-byte record per merged sequence, so a merge workgroup starts from a single read.
  L->merge_info.resize(4 * P.merge_seqs.size());
  for (size_t k = 0; k < P.merge_seqs.size(); ++k) {
    const int seq = P.merge_seqs[k];
    L->merge_info[4 * k] = seq;
    L->merge_info[4 * k + 1] = P.part_base[seq];
    L->merge_info[4 * k + 2] = P.n_parts[seq];
    L->merge_info[4 * k + 3] = 0;
  }
  size_t at = 0;
  auto slot = [&](size_t n) {
    const size_t off = at;
    at = (at + n + 255) & ~size_t(255);
    return off;
  };
  L->off_wave = slot(P.wave_items.size() * sizeof(kvp::DecodeItem));
  L->off_seg = slot(P.seg_off.size() * 4);
  L->off_group = slot(P.group_items.size() * sizeof(kvp::DecodeItem));
  L->off_members = slot(P.members.size() * 4);
  L->off_part_base = slot(P.part_base.size() * 4);
  L->off_merge = slot(L->merge_info.size() * 4);
  L->meta_bytes = at;
  L->off_acc = 0;
  L->off_ml = L->off_acc + (((size_t)P.total_parts * Hq * pool->head_dim * 4 + 255) & ~size_t(255));
  L->total = L->off_ml + (((size_t)P.total_parts * Hq * 8 + 255) & ~size_t(255));
  return KVP_OK;
}

// Kernel arguments of a laid-out decode plan whose metadata sits at `meta` (pinned host memory or device
// memory) and whose partial states go to `part` (device memory of L.total bytes).
kvp::DecodeArgs decode_args(const DecodeLayout& L, kvp_pool_t pool, int layer, const void* q,
                            const int32_t* block_tables, int maxp, int num_q_heads, float scale, void* out,
                            int out_dtype, const unsigned char* meta, unsigned char* part) {
  const auto& P = L.plan;
  kvp::DecodeArgs a{};
  a.q = reinterpret_cast<const uint16_t*>(q);
  a.layer = layer_ptr(pool, layer);
  a.bt = block_tables;
  a.maxp = maxp;
  a.members = reinterpret_cast<const int32_t*>(meta + L.off_members);
  a.part_base = reinterpret_cast<const int32_t*>(meta + L.off_part_base);
  a.part_acc = reinterpret_cast<float*>(part + L.off_acc);
  a.part_ml = reinterpret_cast<float2*>(part + L.off_ml);
  a.out = out;
  a.out_f32 = out_dtype == KVP_F32;
  a.Hq = num_q_heads;
  a.Hkv = pool->num_kv_heads;
  a.G = num_q_heads / pool->num_kv_heads;
  a.num_pages = pool->num_pages;
  a.fp8 = pool->dtype == KVP_FP8_E4M3;
  a.scale_log2 = scale * 1.4426950408889634f * (a.fp8 ? pool->k_scale[layer] : 1.0f);
  a.v_scale = a.fp8 ? pool->v_scale[layer] : 1.0f;
  a.err = pool->err;
  a.items = reinterpret_cast<const kvp::DecodeItem*>(meta + L.off_wave);
  a.seg_off = reinterpret_cast<const int32_t*>(meta + L.off_seg);
  a.n_items = (int)P.seg_off.size() - 1;
  a.group_items = reinterpret_cast<const kvp::DecodeItem*>(meta + L.off_group);
  a.n_group_items = (int)P.group_items.size();
  a.n_group_blocks = a.n_group_items * a.Hkv;
  a.n_wave_blocks = (a.n_items * a.Hkv + 3) / 4;
  return a;
}

// The merge of split partials (decode: one record per split sequence; prefill: one per query row of a
// split session), enqueued after the kernels that write the partials.
hipError_t launch_merge(const int32_t* merge_info, int n_merge, const float* part_acc, const float2* part_ml,
                        void* out, int out_f32, int num_q_heads, kvp_pool_t pool, hipStream_t s) {
  if (n_merge == 0) return hipSuccess;
  kvp::MergeArgs mg{};
  mg.merge_info = merge_info;
  mg.n_merge = n_merge;
  mg.part_acc = part_acc;
  mg.part_ml = part_ml;
  mg.out = out;
  mg.out_f32 = out_f32;
  mg.Hq = num_q_heads;
  mg.Hkv = pool->num_kv_heads;
  return kvp::launch_decode_merge(mg, pool->head_dim, s);
}

// Launches the decode kernels (and the merge) for a laid-out plan (metadata and partials as in
// decode_args).
hipError_t launch_decode_plan(const DecodeLayout& L, kvp_pool_t pool, int layer, const void* q,
                              const int32_t* block_tables, int maxp, int num_q_heads, float scale, void* out,
                              int out_dtype, const unsigned char* meta, unsigned char* part, hipStream_t s) {
  const kvp::DecodeArgs a = decode_args(L, pool, layer, q, block_tables, maxp, num_q_heads, scale, out, out_dtype,
                                        meta, part);
  hipError_t e = kvp::launch_decode(a, pool->head_dim, s);
  if (e == hipSuccess)
    e = launch_merge(reinterpret_cast<const int32_t*>(meta + L.off_merge), (int)L.plan.merge_seqs.size(),
                     a.part_acc, a.part_ml, out, a.out_f32, num_q_heads, pool, s);
  return e;
}

// Checks shared by the decode entry points (before anything is planned or enqueued).
int check_decode_args(kvp_pool_t pool, int layer, const void* q, const int32_t* block_tables,
                      const int32_t* seq_lens, int num_seqs, float scale, const void* out, int out_dtype) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (num_seqs < 0) return set_err(KVP_EINVAL, "num_seqs %d < 0", num_seqs);
  if (num_seqs == 0) return KVP_OK;
  if (!q || !out || !block_tables || !seq_lens) return set_err(KVP_EINVAL, "NULL pointer argument");
  if (out_dtype != KVP_BF16 && out_dtype != KVP_F32) return set_err(KVP_EUNSUPPORTED, "out_dtype %d", out_dtype);
  if (!std::isfinite(scale) || !(scale > 0.0f)) return set_err(KVP_EINVAL, "scale must be finite and > 0");
  return KVP_OK;
}

// Prefill: the caller's workspace holds the metadata (work list, lengths, split bookkeeping, one async
// copy) followed by the partial states of split tiles [partial accumulators][partial (m, l)].
struct PrefillLayout {
  kvp::PrefillPlan plan;
  Packer meta;
  size_t off_items = 0, off_ctx = 0, off_cuq = 0, off_part_base = 0, off_nsplit = 0, off_merge = 0;
  size_t off_acc = 0, off_ml = 0, total = 0;
};

int layout_prefill(kvp_pool_t pool, const int32_t* ctx_lens, const int32_t* cu_q, int B, int maxp, int Hq,
                   PrefillLayout* L) {
  kvp::Status st = kvp::plan_prefill(ctx_lens, cu_q, B, maxp, Hq, pool->num_kv_heads, &L->plan);
  if (!st.ok()) return from_status(st);
  const auto& P = L->plan;
  L->off_items = L->meta.add(P.items.data(), P.items.size() * sizeof(kvp::PrefillItem));
  L->off_ctx = L->meta.add(ctx_lens, (size_t)B * 4);
  L->off_cuq = L->meta.add(cu_q, (size_t)(B + 1) * 4);
  L->off_part_base = L->meta.add(P.part_base.data(), P.part_base.size() * 4);
  L->off_nsplit = L->meta.add(P.nsplit.data(), P.nsplit.size() * 4);
  L->off_merge = L->meta.add(P.merge_info.data(), P.merge_info.size() * 4);
  L->off_acc = L->meta.size();
  L->off_ml = L->off_acc + (((size_t)P.total_parts * Hq * pool->head_dim * 4 + 255) & ~size_t(255));
  L->total = L->off_ml + (((size_t)P.total_parts * Hq * 8 + 255) & ~size_t(255));
  return KVP_OK;
}

// Kernel arguments of a laid-out prefill plan whose metadata and partial states sit in the device
// workspace `w` (metadata uploaded there first).
kvp::PrefillArgs prefill_args(const PrefillLayout& L, kvp_pool_t pool, int layer, const void* q,
                              const int32_t* block_tables, int maxp, int num_q_heads, float scale, void* out,
                              int out_dtype, unsigned char* w) {
  kvp::PrefillArgs a{};
  a.q = reinterpret_cast<const uint16_t*>(q);
  a.layer = layer_ptr(pool, layer);
  a.bt = block_tables;
  a.maxp = maxp;
  a.items = reinterpret_cast<const kvp::PrefillItem*>(w + L.off_items);
  a.n_items = (int)L.plan.items.size();
  a.ctx_lens = reinterpret_cast<const int32_t*>(w + L.off_ctx);
  a.cu_q = reinterpret_cast<const int32_t*>(w + L.off_cuq);
  a.part_base = reinterpret_cast<const int32_t*>(w + L.off_part_base);
  a.nsplit = reinterpret_cast<const int32_t*>(w + L.off_nsplit);
  a.part_acc = reinterpret_cast<float*>(w + L.off_acc);
  a.part_ml = reinterpret_cast<float2*>(w + L.off_ml);
  a.out = out;
  a.out_f32 = out_dtype == KVP_F32;
  a.Hq = num_q_heads;
  a.Hkv = pool->num_kv_heads;
  a.G = num_q_heads / pool->num_kv_heads;
  a.num_pages = pool->num_pages;
  a.fp8 = pool->dtype == KVP_FP8_E4M3;
  a.scale_log2 = scale * 1.4426950408889634f * (a.fp8 ? pool->k_scale[layer] : 1.0f);
  a.v_scale = a.fp8 ? pool->v_scale[layer] : 1.0f;
  a.err = pool->err;
  return a;
}

// Checks of the prefill entry points (before anything is planned or enqueued).
int check_prefill_args(kvp_pool_t pool, int layer, const void* q, const int32_t* block_tables,
                       const int32_t* ctx_lens, const int32_t* cu_q, int num_seqs, float scale, const void* out,
                       int out_dtype) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (num_seqs < 0) return set_err(KVP_EINVAL, "num_seqs %d < 0", num_seqs);
  if (num_seqs == 0) return KVP_OK;
  if (!q || !out || !block_tables || !ctx_lens || !cu_q) return set_err(KVP_EINVAL, "NULL pointer argument");
  if (out_dtype != KVP_BF16 && out_dtype != KVP_F32) return set_err(KVP_EUNSUPPORTED, "out_dtype %d", out_dtype);
  if (!std::isfinite(scale) || !(scale > 0.0f)) return set_err(KVP_EINVAL, "scale must be finite and > 0");
  return KVP_OK;
}

// Workspace of a mixed step: [decode partials][prefill metadata + partials], each 256-byte aligned.
struct MixedLayout {
  DecodeLayout dec;
  PrefillLayout pf;
  size_t off_pf = 0, total = 0;
};

int layout_mixed(kvp_pool_t pool, int num_q_heads, const int32_t* seq_lens, int num_dec, int maxp_dec,
                 const kvp_group_prefix* gp, const int32_t* ctx_lens, const int32_t* cu_q, int num_pf, int maxp_pf,
                 MixedLayout* L) {
  if (num_dec > 0) {
    int rc = layout_decode(pool, seq_lens, num_dec, maxp_dec, gp, num_q_heads, &L->dec);
    if (rc) return rc;
  }
  if (num_pf > 0) {
    int rc = layout_prefill(pool, ctx_lens, cu_q, num_pf, maxp_pf, num_q_heads, &L->pf);
    if (rc) return rc;
  }
  L->off_pf = (L->dec.total + 255) & ~size_t(255);
  L->total = L->off_pf + (num_pf > 0 && L->pf.plan.real_items > 0 ? L->pf.total : 0);
  return KVP_OK;
}

}  // namespace

extern "C" {

const char* kvp_version(void) { return "kvpattn 0.1 (gfx950)"; }

const char* kvp_last_error(void) { return g_last_error.c_str(); }

const char* kvp_strerror(int code) {
  switch (code) {
    case KVP_OK: return "ok";
    case KVP_EINVAL: return "invalid argument";
    case KVP_ERANGE: return "length or page id out of range";
    case KVP_EGROUP: return "inconsistent rollout-group prefix";
    case KVP_ESHARED: return "write into a shared prefix page";
    case KVP_EWORKSPACE: return "workspace too small";
    case KVP_EUNSUPPORTED: return "unsupported shape or dtype";
    case KVP_EHIP: return "HIP runtime error";
    case KVP_ENOMEM: return "out of memory";
    default: return "unknown error";
  }
}

int kv_pool_create(kvp_pool_t* out, int num_layers, int num_pages, int page_size, int num_kv_heads, int head_dim,
                   int dtype) {
  if (!out) return set_err(KVP_EINVAL, "out is NULL");
  *out = nullptr;
  if (num_layers <= 0 || num_pages <= 0 || num_kv_heads <= 0)
    return set_err(KVP_EINVAL, "num_layers, num_pages and num_kv_heads must be positive");
  if (page_size != kvp::kPage) return set_err(KVP_EUNSUPPORTED, "page_size %d (only 16 is supported)", page_size);
  if (head_dim != 64 && head_dim != 128) return set_err(KVP_EUNSUPPORTED, "head_dim %d (64 or 128)", head_dim);
  if (dtype != KVP_BF16 && dtype != KVP_FP8_E4M3)
    return set_err(KVP_EUNSUPPORTED, "dtype %d (KVP_BF16 or KVP_FP8_E4M3)", dtype);
  auto* p = new kvp_pool();
  p->num_layers = num_layers;
  p->num_pages = num_pages;
  p->num_kv_heads = num_kv_heads;
  p->head_dim = head_dim;
  p->dtype = dtype;
  p->k_scale.assign(num_layers, 1.0f);
  p->v_scale.assign(num_layers, 1.0f);
  p->layer_bytes = (size_t)num_pages * num_kv_heads * 2 * kvp::kPage * head_dim * elem_bytes(dtype);
  hipError_t e = hipGetDevice(&p->device);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&p->base), p->layer_bytes * num_layers);
  if (e != hipSuccess) {
    const size_t want = p->layer_bytes * num_layers;
    delete p;
    return set_err(KVP_ENOMEM, "hipMalloc(pool of %zu bytes): %s", want, hipGetErrorString(e));
  }
  e = hipMalloc(reinterpret_cast<void**>(&p->err), 256);
  if (e == hipSuccess) e = kvp::launch_fill_zero(p->base, p->layer_bytes * num_layers, nullptr);
  if (e == hipSuccess) e = kvp::launch_fill_zero(p->err, 256, nullptr);
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) {
    (void)hipFree(p->base);
    if (p->err) (void)hipFree(p->err);
    delete p;
    return hip_err(e, "kv_pool_create");
  }
  *out = p;
  return KVP_OK;
}

int kv_pool_destroy(kvp_pool_t pool) {
  if (!pool) return KVP_OK;
  (void)hipDeviceSynchronize();
  if (pool->base) (void)hipFree(pool->base);
  if (pool->err) (void)hipFree(pool->err);
  pool->base = nullptr;
  delete pool;
  return KVP_OK;
}

int kv_pool_reset(kvp_pool_t pool, void* stream) {
  if (!pool_ok(pool)) return set_err(KVP_EINVAL, "pool is NULL or destroyed");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = kvp::launch_fill_zero(pool->base, pool->layer_bytes * pool->num_layers, s);
  if (e == hipSuccess) e = kvp::launch_fill_zero(pool->err, 256, s);
  return e == hipSuccess ? KVP_OK : hip_err(e, "kv_pool_reset");
}

int kv_pool_layer_ptr(kvp_pool_t pool, int layer, void** dev_ptr, size_t* bytes) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (dev_ptr) *dev_ptr = pool->base + (size_t)layer * pool->layer_bytes;
  if (bytes) *bytes = pool->layer_bytes;
  return KVP_OK;
}

int kv_pool_info(kvp_pool_t pool, int* num_layers, int* num_pages, int* num_kv_heads, int* head_dim) {
  if (!pool_ok(pool)) return set_err(KVP_EINVAL, "pool is NULL or destroyed");
  if (num_layers) *num_layers = pool->num_layers;
  if (num_pages) *num_pages = pool->num_pages;
  if (num_kv_heads) *num_kv_heads = pool->num_kv_heads;
  if (head_dim) *head_dim = pool->head_dim;
  return KVP_OK;
}

int kv_pool_dtype(kvp_pool_t pool, int* dtype) {
  if (!pool_ok(pool) || !dtype) return set_err(KVP_EINVAL, "pool or dtype is NULL");
  *dtype = pool->dtype;
  return KVP_OK;
}

int kv_pool_set_scales(kvp_pool_t pool, int layer, float k_scale, float v_scale) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (pool->dtype != KVP_FP8_E4M3) return set_err(KVP_EUNSUPPORTED, "scales apply to FP8 pools only");
  if (!std::isfinite(k_scale) || !(k_scale > 0.0f) || !std::isfinite(v_scale) || !(v_scale > 0.0f))
    return set_err(KVP_EINVAL, "scales must be finite and > 0");
  pool->k_scale[layer] = k_scale;
  pool->v_scale[layer] = v_scale;
  return KVP_OK;
}

int kv_pool_device_error(kvp_pool_t pool, int* code) {
  if (!pool_ok(pool) || !code) return set_err(KVP_EINVAL, "pool or code is NULL");
  hipError_t e = hipDeviceSynchronize();
  int v = 0;
  if (e == hipSuccess) e = hipMemcpy(&v, pool->err, sizeof(int), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemset(pool->err, 0, sizeof(int));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_err(e, "kv_pool_device_error");
  *code = v;
  return KVP_OK;
}

int kv_append(kvp_pool_t pool, int layer, const void* k, const void* v, const int32_t* block_tables, int maxp,
              const int32_t* start_pos, const int32_t* cu_new, int num_seqs, const kvp_group_prefix* gp,
              void* stream) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (num_seqs < 0 || maxp < 0) return set_err(KVP_EINVAL, "num_seqs %d / maxp %d negative", num_seqs, maxp);
  if (num_seqs == 0) return KVP_OK;
  if (!start_pos || !cu_new || !block_tables) return set_err(KVP_EINVAL, "NULL metadata pointer");
  if (cu_new[0] != 0) return set_err(KVP_EINVAL, "cu_new[0] = %d, must be 0", cu_new[0]);
  std::vector<int32_t> cnt(num_seqs);
  std::vector<int64_t> first(num_seqs);
  for (int i = 0; i < num_seqs; ++i) {
    cnt[i] = cu_new[i + 1] - cu_new[i];
    first[i] = cu_new[i];
    if (cnt[i] < 0) return set_err(KVP_EINVAL, "cu_new decreases at %d", i);
    if (start_pos[i] < 0) return set_err(KVP_EINVAL, "start_pos[%d] = %d < 0", i, start_pos[i]);
    if ((int64_t)start_pos[i] + cnt[i] > (int64_t)maxp * kvp::kPage)
      return set_err(KVP_ERANGE, "sequence %d: positions up to %lld exceed maxp * 16 = %lld", i,
                     (long long)start_pos[i] + cnt[i], (long long)maxp * kvp::kPage);
  }
  if (cu_new[num_seqs] > 0 && (!k || !v)) return set_err(KVP_EINVAL, "k or v is NULL");
  if (gp) {
    kvp::Status st = kvp::validate_group_prefix(nullptr, num_seqs, gp);
    if (!st.ok()) return from_status(st);
    if (gp->num_groups > 0)
      for (int i = 0; i < num_seqs; ++i) {
        const int g = gp->group_id[i];
        if (g >= 0 && cnt[i] > 0 && (int64_t)start_pos[i] < (int64_t)gp->shared_pages[g] * kvp::kPage)
          return set_err(KVP_ESHARED, "sequence %d would write position %d inside its group's %d shared pages", i,
                         start_pos[i], gp->shared_pages[g]);
      }
  }
  std::vector<kvp::PageRun> runs;
  build_runs(start_pos, first.data(), cnt.data(), num_seqs, &runs);
  if (runs.empty()) return KVP_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Staging::Lease lease;
  rc = lease_runs(runs, &lease);
  if (rc) return rc;
  kvp::AppendArgs a{};
  a.k = reinterpret_cast<const uint16_t*>(k);
  a.v = reinterpret_cast<const uint16_t*>(v);
  a.layer = const_cast<uint16_t*>(layer_ptr(pool, layer));
  a.bt = block_tables;
  a.runs = reinterpret_cast<const kvp::PageRun*>(lease.host);
  a.n_runs = (int)runs.size();
  a.maxp = maxp;
  a.Hkv = pool->num_kv_heads;
  a.num_pages = pool->num_pages;
  a.err = pool->err;
  a.fp8 = pool->dtype == KVP_FP8_E4M3;
  a.inv_scale_k = 1.0f / pool->k_scale[layer];
  a.inv_scale_v = 1.0f / pool->v_scale[layer];
  hipError_t e = kvp::launch_append(a, pool->head_dim, s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, "kv_append launch");
  return rr;
}

int kv_gather(kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp, const int32_t* lens, int num_seqs,
              void* k_out, void* v_out, void* stream) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (num_seqs < 0 || maxp < 0) return set_err(KVP_EINVAL, "num_seqs / maxp negative");
  if (num_seqs == 0) return KVP_OK;
  if (!lens || !block_tables) return set_err(KVP_EINVAL, "NULL metadata pointer");
  std::vector<int32_t> zero(num_seqs, 0);
  std::vector<int64_t> first(num_seqs);
  int64_t tot = 0;
  for (int i = 0; i < num_seqs; ++i) {
    if (lens[i] < 0 || (int64_t)lens[i] > (int64_t)maxp * kvp::kPage)
      return set_err(KVP_ERANGE, "lens[%d] = %d outside [0, maxp*16]", i, lens[i]);
    first[i] = tot;
    tot += lens[i];
  }
  if (tot > 0 && (!k_out || !v_out)) return set_err(KVP_EINVAL, "k_out or v_out is NULL");
  std::vector<kvp::PageRun> runs;
  build_runs(zero.data(), first.data(), lens, num_seqs, &runs);
  if (runs.empty()) return KVP_OK;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Staging::Lease lease;
  rc = lease_runs(runs, &lease);
  if (rc) return rc;
  kvp::GatherArgs a{};
  a.k = reinterpret_cast<uint16_t*>(k_out);
  a.v = reinterpret_cast<uint16_t*>(v_out);
  a.layer = layer_ptr(pool, layer);
  a.bt = block_tables;
  a.runs = reinterpret_cast<const kvp::PageRun*>(lease.host);
  a.n_runs = (int)runs.size();
  a.maxp = maxp;
  a.Hkv = pool->num_kv_heads;
  a.num_pages = pool->num_pages;
  a.err = pool->err;
  a.fp8 = pool->dtype == KVP_FP8_E4M3;
  a.scale_k = pool->k_scale[layer];
  a.scale_v = pool->v_scale[layer];
  hipError_t e = kvp::launch_gather(a, pool->head_dim, s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, "kv_gather launch");
  return rr;
}

int kv_pool_page_bytes(kvp_pool_t pool, size_t* bytes) {
  if (!pool_ok(pool) || !bytes) return set_err(KVP_EINVAL, "pool or bytes is NULL");
  *bytes = page_bytes(pool);
  return KVP_OK;
}

int kv_offload(kvp_pool_t pool, int layer, const int32_t* page_ids, int n, void* host_dst, void* stream) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (n < 0) return set_err(KVP_EINVAL, "n = %d < 0", n);
  if (n == 0) return KVP_OK;
  if (!page_ids) return set_err(KVP_EINVAL, "page_ids is NULL");
  rc = check_pinned(host_dst, (size_t)n * page_bytes(pool), "host_dst");
  if (rc) return rc;
  std::vector<kvp::TierItem> items(n);
  for (int i = 0; i < n; ++i) {
    if ((unsigned)page_ids[i] >= (unsigned)pool->num_pages)
      return set_err(KVP_ERANGE, "page_ids[%d] = %d outside [0, %d)", i, page_ids[i], pool->num_pages);
    items[i] = kvp::TierItem{page_ids[i], 0, 0, 0};
  }
  return run_tier(pool, layer, items, host_dst, nullptr, 0, false, reinterpret_cast<hipStream_t>(stream));
}

int kv_restore(kvp_pool_t pool, int layer, const void* host_src, const int32_t* page_ids, int n,
               int32_t* block_tables, int num_rows, int maxp, const int32_t* rows, const int32_t* lpages,
               void* stream) {
  int rc = check_layer(pool, layer);
  if (rc) return rc;
  if (n < 0) return set_err(KVP_EINVAL, "n = %d < 0", n);
  if (n == 0) return KVP_OK;
  if (!page_ids) return set_err(KVP_EINVAL, "page_ids is NULL");
  if (block_tables && (!rows || !lpages || num_rows <= 0 || maxp <= 0))
    return set_err(KVP_EINVAL, "a block-table patch needs rows, lpages, num_rows > 0 and maxp > 0");
  rc = check_pinned(host_src, (size_t)n * page_bytes(pool), "host_src");
  if (rc) return rc;
  std::vector<unsigned char> seen(pool->num_pages, 0);
  std::vector<kvp::TierItem> items(n);
  for (int i = 0; i < n; ++i) {
    const int id = page_ids[i];
    if ((unsigned)id >= (unsigned)pool->num_pages)
      return set_err(KVP_ERANGE, "page_ids[%d] = %d outside [0, %d)", i, id, pool->num_pages);
    if (seen[id]) return set_err(KVP_EINVAL, "page id %d is restored twice", id);
    seen[id] = 1;
    int row = 0, lp = 0;
    if (block_tables) {
      row = rows[i];
      lp = lpages[i];
      if (row < 0 || row >= num_rows) return set_err(KVP_EINVAL, "rows[%d] = %d outside [0, %d)", i, row, num_rows);
      if (lp < 0 || lp >= maxp) return set_err(KVP_ERANGE, "lpages[%d] = %d outside [0, %d)", i, lp, maxp);
    }
    items[i] = kvp::TierItem{id, row, lp, 0};
  }
  return run_tier(pool, layer, items, const_cast<void*>(host_src), block_tables, maxp, true,
                  reinterpret_cast<hipStream_t>(stream));
}

int kvp_block_hashes(const int32_t* tokens, const int32_t* cu_tokens, int num_seqs, uint64_t seed,
                     uint64_t* hashes, void* stream) {
  if (num_seqs < 0) return set_err(KVP_EINVAL, "num_seqs %d < 0", num_seqs);
  if (num_seqs == 0) return KVP_OK;
  std::vector<kvp::HashChunk> chunks;
  int64_t pages = 0;
  int rc0 = build_chunks(cu_tokens, num_seqs, &chunks, &pages);
  if (rc0) return rc0;
  if (pages == 0) return KVP_OK;
  if (!tokens || !hashes) return set_err(KVP_EINVAL, "tokens or hashes is NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Staging::Lease lease;
  const size_t nb = chunks.size() * sizeof(kvp::HashChunk);
  int rc = staging().lease(nb, &lease);
  if (rc) return rc;
  std::memcpy(lease.host, chunks.data(), nb);
  void* totals = nullptr;
  hipError_t e = hipMallocAsync(&totals, chunks.size() * 16, s);
  if (e != hipSuccess) {
    (void)staging().release(lease, s, false);
    return set_err(KVP_ENOMEM, "hipMallocAsync(%zu): %s", chunks.size() * 16, hipGetErrorString(e));
  }
  kvp::HashArgs a{};
  a.tokens = tokens;
  a.chunks = reinterpret_cast<const kvp::HashChunk*>(lease.host);
  a.seed = seed;
  a.out = hashes;
  a.totals = reinterpret_cast<uint64_t*>(totals);
  e = kvp::launch_block_hash(a, (int)chunks.size(), s);
  (void)hipFreeAsync(totals, s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, "kvp_block_hashes launch");
  return rr;
}

int kvp_group_shared_pages(const uint64_t* hashes, const int32_t* cu_tokens, int num_seqs, const int32_t* group_id,
                           int num_groups, int32_t* shared_pages, void* stream) {
  if (num_seqs < 0 || num_groups < 0) return set_err(KVP_EINVAL, "negative count");
  if (num_groups == 0) return KVP_OK;
  if (!group_id || !shared_pages) return set_err(KVP_EINVAL, "group_id or shared_pages is NULL");
  std::vector<int32_t> cnt(num_groups + 1, 0);
  for (int i = 0; i < num_seqs; ++i) {
    const int g = group_id[i];
    if (g < -1 || g >= num_groups) return set_err(KVP_EGROUP, "group_id[%d] = %d outside [-1, %d)", i, g, num_groups);
    if (g >= 0) ++cnt[g + 1];
  }
  for (int g = 0; g < num_groups; ++g) cnt[g + 1] += cnt[g];
  std::vector<int32_t> members(std::max(1, cnt[num_groups])), fill(cnt.begin(), cnt.end() - 1);
  for (int i = 0; i < num_seqs; ++i)
    if (group_id[i] >= 0) members[fill[group_id[i]]++] = i;
  // pinned slot: [grp_off | members | seq_info]
  std::vector<unsigned char> extra;
  const size_t moff = ((cnt.size() * 4) + 255) & ~size_t(255);
  extra.resize(moff + members.size() * 4);
  std::memcpy(extra.data(), cnt.data(), cnt.size() * 4);
  std::memcpy(extra.data() + moff, members.data(), members.size() * 4);
  Staging::Lease lease;
  int64_t pages = 0;
  size_t off = 0;
  int rc = lease_seq_info(cu_tokens, num_seqs, &lease, &pages, extra, &off);
  if (rc) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (pages > 0 && !hashes) {
    (void)staging().release(lease, s, false);
    return set_err(KVP_EINVAL, "hashes is NULL");
  }
  const unsigned char* h = reinterpret_cast<const unsigned char*>(lease.host);
  kvp::GroupLcpArgs a{};
  a.hashes = hashes;
  a.seq_info = reinterpret_cast<const int4*>(h + off);
  a.grp_off = reinterpret_cast<const int32_t*>(h);
  a.members = reinterpret_cast<const int32_t*>(h + moff);
  a.shared_pages = shared_pages;
  hipError_t e = kvp::launch_group_lcp(a, num_groups, s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, "kvp_group_shared_pages launch");
  return rr;
}

int kvp_prefix_table_create(kvp_prefix_table_t* out, int capacity_log2) {
  if (!out) return set_err(KVP_EINVAL, "out is NULL");
  *out = nullptr;
  if (capacity_log2 < 4 || capacity_log2 > 30) return set_err(KVP_EINVAL, "capacity_log2 %d outside [4, 30]", capacity_log2);
  auto* t = new kvp_prefix_table();
  const size_t cap = size_t(1) << capacity_log2;
  t->mask = cap - 1;
  hipError_t e = hipGetDevice(&t->device);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&t->keys), cap * 8);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&t->vals), cap * 4);
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&t->err), 256);
  if (e == hipSuccess) {
    kvp::TableArgs a{};
    a.keys = t->keys;
    a.vals = t->vals;
    a.mask = t->mask;
    e = kvp::launch_table(a, 3, 0, nullptr);
  }
  if (e == hipSuccess) e = kvp::launch_fill_zero(t->err, 256, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    (void)hipFree(t->keys);
    (void)hipFree(t->vals);
    (void)hipFree(t->err);
    delete t;
    return set_err(KVP_ENOMEM, "prefix table of 2^%d slots: %s", capacity_log2, hipGetErrorString(e));
  }
  *out = t;
  return KVP_OK;
}

int kvp_prefix_table_destroy(kvp_prefix_table_t t) {
  if (!t) return KVP_OK;
  (void)hipDeviceSynchronize();
  (void)hipFree(t->keys);
  (void)hipFree(t->vals);
  (void)hipFree(t->err);
  delete t;
  return KVP_OK;
}

int kvp_prefix_table_clear(kvp_prefix_table_t t, void* stream) {
  if (!t) return set_err(KVP_EINVAL, "table is NULL");
  kvp::TableArgs a{};
  a.keys = t->keys;
  a.vals = t->vals;
  a.mask = t->mask;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = kvp::launch_table(a, 3, 0, s);
  if (e == hipSuccess) e = kvp::launch_fill_zero(t->err, 256, s);
  return e == hipSuccess ? KVP_OK : hip_err(e, "kvp_prefix_table_clear launch");
}

static int table_update(kvp_prefix_table_t t, const uint64_t* hashes, const int32_t* page_ids, int64_t n, int op,
                        void* stream) {
  if (!t) return set_err(KVP_EINVAL, "table is NULL");
  if (n < 0) return set_err(KVP_EINVAL, "n < 0");
  if (n == 0) return KVP_OK;
  if (!hashes || !page_ids) return set_err(KVP_EINVAL, "hashes or page_ids is NULL");
  kvp::TableArgs a{};
  a.keys = t->keys;
  a.vals = t->vals;
  a.mask = t->mask;
  a.hashes = hashes;
  a.pages = page_ids;
  a.n = n;
  a.err = t->err;
  hipError_t e = kvp::launch_table(a, op, 0, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? KVP_OK : hip_err(e, "prefix table launch");
}

int kvp_prefix_table_insert(kvp_prefix_table_t t, const uint64_t* hashes, const int32_t* page_ids, int64_t n,
                            void* stream) {
  return table_update(t, hashes, page_ids, n, 0, stream);
}

int kvp_prefix_table_erase(kvp_prefix_table_t t, const uint64_t* hashes, const int32_t* page_ids, int64_t n,
                           void* stream) {
  return table_update(t, hashes, page_ids, n, 1, stream);
}

int kvp_prefix_lookup(kvp_prefix_table_t t, const uint64_t* hashes, const int32_t* cu_tokens, int num_seqs,
                      int32_t* matched_pages, int32_t* page_ids, void* stream) {
  if (!t) return set_err(KVP_EINVAL, "table is NULL");
  if (num_seqs < 0) return set_err(KVP_EINVAL, "num_seqs %d < 0", num_seqs);
  if (num_seqs == 0) return KVP_OK;
  if (!matched_pages) return set_err(KVP_EINVAL, "matched_pages is NULL");
  std::vector<kvp::HashChunk> chunks;
  int64_t pages = 0;
  int rc = build_chunks(cu_tokens, num_seqs, &chunks, &pages);
  if (rc) return rc;
  if (pages > 0 && (!hashes || !page_ids)) return set_err(KVP_EINVAL, "hashes or page_ids is NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // Sequences without a full page match nothing: give them a zero-length chunk so pass 2 reports 0.
  for (int i = 0, k = 0; i < num_seqs; ++i) {
    while (k < (int)chunks.size() && chunks[k].pad[1] < i) ++k;
    if (k == (int)chunks.size() || chunks[k].pad[1] != i) {
      chunks.insert(chunks.begin() + k, kvp::HashChunk{0, 0, 0, 0, 0, {1, i, 0}});
    }
  }
  for (size_t k = 0; k < chunks.size(); ++k)  // g0 must index this sequence's first chunk after inserts
    if (chunks[k].c == 0) {
      const int g0 = (int)k;
      for (size_t j = k; j < chunks.size() && chunks[j].pad[1] == chunks[k].pad[1]; ++j) chunks[j].g0 = g0;
    }
  Staging::Lease lease;
  const size_t nb = chunks.size() * sizeof(kvp::HashChunk);
  rc = staging().lease(nb, &lease);
  if (rc) return rc;
  std::memcpy(lease.host, chunks.data(), nb);
  void* scratch = nullptr;
  hipError_t e = hipMallocAsync(&scratch, chunks.size() * 4, s);
  if (e != hipSuccess) {
    (void)staging().release(lease, s, false);
    return set_err(KVP_ENOMEM, "hipMallocAsync(%zu): %s", chunks.size() * 4, hipGetErrorString(e));
  }
  kvp::TableArgs a{};
  a.keys = t->keys;
  a.vals = t->vals;
  a.mask = t->mask;
  a.hashes = hashes;
  a.chunks = reinterpret_cast<const kvp::HashChunk*>(lease.host);
  a.first_miss = reinterpret_cast<int32_t*>(scratch);
  a.matched = matched_pages;
  a.out_pages = page_ids;
  a.err = t->err;
  e = kvp::launch_table(a, 2, (int)chunks.size(), s);
  (void)hipFreeAsync(scratch, s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, "kvp_prefix_lookup launch");
  return rr;
}

int kvp_prefix_table_error(kvp_prefix_table_t t, int* code) {
  if (!t || !code) return set_err(KVP_EINVAL, "table or code is NULL");
  hipError_t e = hipDeviceSynchronize();
  int v = 0;
  if (e == hipSuccess) e = hipMemcpy(&v, t->err, 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemset(t->err, 0, 4);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_err(e, "kvp_prefix_table_error");
  *code = v;
  return KVP_OK;
}

int paged_decode_workspace_size(kvp_pool_t pool, const int32_t* seq_lens, int num_seqs,
                                const kvp_group_prefix* group_prefix, int num_q_heads, size_t* bytes) {
  if (!pool_ok(pool) || !bytes) return set_err(KVP_EINVAL, "pool or bytes is NULL");
  DecodeLayout L;
  // The size query does not know maxp; lengths are range-checked again by paged_decode_attn.
  int rc = layout_decode(pool, seq_lens, num_seqs, 1 << 28, group_prefix, num_q_heads, &L);
  if (rc) return rc;
  *bytes = L.total;
  return KVP_OK;
}

int paged_decode_attn(const void* q, kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp,
                      const int32_t* seq_lens, int num_seqs, const kvp_group_prefix* group_prefix, int num_q_heads,
                      float scale, void* out, int out_dtype, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_decode_args(pool, layer, q, block_tables, seq_lens, num_seqs, scale, out, out_dtype);
  if (rc || num_seqs == 0) return rc;
  DecodeLayout L;
  rc = layout_decode(pool, seq_lens, num_seqs, maxp, group_prefix, num_q_heads, &L);
  if (rc) return rc;
  if (L.total > 0 && (!ws || ws_bytes < L.total))
    return set_err(KVP_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws ? ws_bytes : (size_t)0, L.total);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // The work list is read by the kernels straight from a pinned staging slot (a few KB to a few
  // hundred KB, read once per wave), so no copy sits between the caller's previous work and the
  // decode kernels.  The slot is released after the last kernel that reads it.
  Staging::Lease lease;
  rc = staging().lease(L.meta_bytes, &lease);
  if (rc) return rc;
  L.write_meta(reinterpret_cast<unsigned char*>(lease.host));
  hipError_t e = launch_decode_plan(L, pool, layer, q, block_tables, maxp, num_q_heads, scale, out, out_dtype,
                                    reinterpret_cast<const unsigned char*>(lease.host),
                                    reinterpret_cast<unsigned char*>(ws), s);
  const int rr = staging().release(lease, s, e == hipSuccess);
  if (e != hipSuccess) return hip_err(e, "paged_decode_attn launch");
  return rr;
}

int paged_decode_attn_noalloc(const void* q, kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp,
                              const int32_t* seq_lens, int num_seqs, const kvp_group_prefix* group_prefix,
                              int num_q_heads, float scale, void* out, int out_dtype, void* stream) {
  int rc = check_decode_args(pool, layer, q, block_tables, seq_lens, num_seqs, scale, out, out_dtype);
  if (rc || num_seqs == 0) return rc;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_err(e, "hipGetDevice");
  if (dev != pool->device)
    return set_err(KVP_EINVAL, "the current device is %d, the pool lives on device %d", dev, pool->device);
  DecodeLayout L;
  rc = layout_decode(pool, seq_lens, num_seqs, maxp, group_prefix, num_q_heads, &L);
  if (rc) return rc;
  const size_t meta_bytes = L.meta_bytes;
  if (meta_bytes + L.total > kNoAllocScratchBytes)
    return set_err(KVP_EWORKSPACE, "the call needs %zu bytes of scratch, more than the %zu of the allocation-free "
                   "entry point", meta_bytes + L.total, kNoAllocScratchBytes);
  unsigned char* sp = nullptr;
  rc = scratch_of(dev, &sp);
  if (rc) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // [work list][partial accumulators][partial (m, l)]: the work list travels in launch arguments.
  std::vector<unsigned char> meta(meta_bytes, 0);
  L.write_meta(meta.data());
  e = kvp::launch_put_bytes(sp, meta.data(), meta_bytes, s);
  if (e == hipSuccess)
    e = launch_decode_plan(L, pool, layer, q, block_tables, maxp, num_q_heads, scale, out, out_dtype, sp,
                           sp + meta_bytes, s);
  return e == hipSuccess ? KVP_OK : hip_err(e, "paged_decode_attn_noalloc launch");
}

int prefix_chunk_prefill_workspace_size(kvp_pool_t pool, const int32_t* ctx_lens, const int32_t* cu_q, int num_seqs,
                                        int num_q_heads, size_t* bytes) {
  if (!pool_ok(pool) || !bytes) return set_err(KVP_EINVAL, "pool or bytes is NULL");
  PrefillLayout L;
  int rc = layout_prefill(pool, ctx_lens, cu_q, num_seqs, 1 << 28, num_q_heads, &L);
  if (rc) return rc;
  *bytes = L.total;
  return KVP_OK;
}

int prefix_chunk_prefill_attn(const void* q, kvp_pool_t pool, int layer, const int32_t* block_tables, int maxp,
                              const int32_t* ctx_lens, const int32_t* cu_q, int num_seqs, int num_q_heads, float scale,
                              void* out, int out_dtype, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_prefill_args(pool, layer, q, block_tables, ctx_lens, cu_q, num_seqs, scale, out, out_dtype);
  if (rc || num_seqs == 0) return rc;
  PrefillLayout L;
  rc = layout_prefill(pool, ctx_lens, cu_q, num_seqs, maxp, num_q_heads, &L);
  if (rc) return rc;
  if (L.plan.real_items == 0) return KVP_OK;
  if (!ws || ws_bytes < L.total)
    return set_err(KVP_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws ? ws_bytes : (size_t)0, L.total);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  unsigned char* w = reinterpret_cast<unsigned char*>(ws);
  rc = staging().upload(w, L.meta.buf.data(), L.meta.buf.size(), s);
  if (rc) return rc;
  const kvp::PrefillArgs a = prefill_args(L, pool, layer, q, block_tables, maxp, num_q_heads, scale, out, out_dtype, w);
  hipError_t e = kvp::launch_prefill(a, pool->head_dim, s);
  // split tiles: combine each query row's key ranges (the decode merge, one record per query row)
  if (e == hipSuccess)
    e = launch_merge(reinterpret_cast<const int32_t*>(w + L.off_merge), (int)(L.plan.merge_info.size() / 4),
                     a.part_acc, a.part_ml, out, a.out_f32, num_q_heads, pool, s);
  return e == hipSuccess ? KVP_OK : hip_err(e, "prefix_chunk_prefill_attn launch");
}

int mixed_step_workspace_size(kvp_pool_t pool, const int32_t* seq_lens, int num_dec, const kvp_group_prefix* group_prefix,
                              const int32_t* ctx_lens, const int32_t* cu_q, int num_pf, int num_q_heads,
                              size_t* bytes) {
  if (!pool_ok(pool) || !bytes) return set_err(KVP_EINVAL, "pool or bytes is NULL");
  if (num_dec < 0 || num_pf < 0) return set_err(KVP_EINVAL, "negative sequence count");
  MixedLayout L;
  int rc = layout_mixed(pool, num_q_heads, seq_lens, num_dec, 1 << 28, group_prefix, ctx_lens, cu_q, num_pf, 1 << 28, &L);
  if (rc) return rc;
  *bytes = L.total;
  return KVP_OK;
}

int mixed_step_attn(kvp_pool_t pool, int layer, int num_q_heads, float scale, int out_dtype, const void* q_dec,
                    const int32_t* block_tables_dec, int maxp_dec, const int32_t* seq_lens, int num_dec,
                    const kvp_group_prefix* group_prefix, void* out_dec, const void* q_pf,
                    const int32_t* block_tables_pf, int maxp_pf, const int32_t* ctx_lens, const int32_t* cu_q,
                    int num_pf, void* out_pf, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_decode_args(pool, layer, q_dec, block_tables_dec, seq_lens, num_dec, scale, out_dec, out_dtype);
  if (rc) return rc;
  rc = check_prefill_args(pool, layer, q_pf, block_tables_pf, ctx_lens, cu_q, num_pf, scale, out_pf, out_dtype);
  if (rc) return rc;
  MixedLayout L;
  rc = layout_mixed(pool, num_q_heads, seq_lens, num_dec, maxp_dec, group_prefix, ctx_lens, cu_q, num_pf, maxp_pf, &L);
  if (rc) return rc;
  const bool has_pf = num_pf > 0 && L.pf.plan.real_items > 0;
  if (num_dec == 0 && !has_pf) return KVP_OK;
  if (L.total > 0 && (!ws || ws_bytes < L.total))
    return set_err(KVP_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws ? ws_bytes : (size_t)0, L.total);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  unsigned char* w = reinterpret_cast<unsigned char*>(ws);
  kvp::DecodeArgs d{};
  kvp::PrefillArgs p{};
  Staging::Lease lease;
  if (num_dec > 0) {
    // the decode work list is read from a pinned staging slot, as in paged_decode_attn
    rc = staging().lease(L.dec.meta_bytes, &lease);
    if (rc) return rc;
    L.dec.write_meta(reinterpret_cast<unsigned char*>(lease.host));
    d = decode_args(L.dec, pool, layer, q_dec, block_tables_dec, maxp_dec, num_q_heads, scale, out_dec, out_dtype,
                    reinterpret_cast<const unsigned char*>(lease.host), w);
  }
  hipError_t e = hipSuccess;
  if (has_pf) {
    rc = staging().upload(w + L.off_pf, L.pf.meta.buf.data(), L.pf.meta.buf.size(), s);
    if (rc) {
      if (num_dec > 0) (void)staging().release(lease, s, false);
      return rc;
    }
    p = prefill_args(L.pf, pool, layer, q_pf, block_tables_pf, maxp_pf, num_q_heads, scale, out_pf, out_dtype,
                     w + L.off_pf);
  }
  if (num_dec > 0 && !has_pf) {
    e = kvp::launch_decode(d, pool->head_dim, s);                   // the decode call's own launch
  } else if (num_dec == 0) {
    e = kvp::launch_prefill(p, pool->head_dim, s);                  // the prefill call's own launch
  } else {
    // LDS-staged shared-prefix blocks (wide groups over long prompts) run in a launch of their own ahead
    // of the fused one, which carries the wave-path blocks and the prefill blocks.
    if (d.n_group_blocks > 0) {
      kvp::DecodeArgs g = d;
      g.n_wave_blocks = 0;
      e = kvp::launch_decode(g, pool->head_dim, s);
    }
    kvp::DecodeArgs wv = d;
    wv.n_group_blocks = 0;
    if (e == hipSuccess) e = kvp::launch_mixed_step(wv, p, pool->head_dim, pool->dtype == KVP_FP8_E4M3, s);
  }
  if (e == hipSuccess && num_dec > 0)
    e = launch_merge(reinterpret_cast<const int32_t*>(reinterpret_cast<const unsigned char*>(lease.host) +
                                                      L.dec.off_merge),
                     (int)L.dec.plan.merge_seqs.size(), d.part_acc, d.part_ml, out_dec, d.out_f32, num_q_heads,
                     pool, s);
  if (e == hipSuccess && has_pf)
    e = launch_merge(reinterpret_cast<const int32_t*>(w + L.off_pf + L.pf.off_merge),
                     (int)(L.pf.plan.merge_info.size() / 4), p.part_acc, p.part_ml, out_pf, p.out_f32, num_q_heads,
                     pool, s);
  const int rr = num_dec > 0 ? staging().release(lease, s, e == hipSuccess) : KVP_OK;
  if (e != hipSuccess) return hip_err(e, "mixed_step_attn launch");
  return rr;
}

int kvp_check_tables(const int32_t* block_tables_host, int maxp, const int32_t* lens, int num_seqs, int num_pages,
                     const kvp_group_prefix* gp) {
  return from_status(kvp::check_tables(block_tables_host, maxp, lens, num_seqs, num_pages, gp));
}

int kvp_plan_decode(const int32_t* seq_lens, int num_seqs, const kvp_group_prefix* gp, int num_q_heads,
                    int num_kv_heads, int32_t* items_out, int cap, int* n_items, int* n_partials,
                    int* pages_per_split) {
  kvp::DecodePlan P;
  kvp::Status st = kvp::plan_decode(seq_lens, num_seqs, 1 << 28, gp, num_q_heads, num_kv_heads, &P);
  if (!st.ok()) return from_status(st);
  std::vector<kvp::DecodeItem> all(P.wave_items);
  all.insert(all.end(), P.group_items.begin(), P.group_items.end());
  for (int i = 0; i < (int)all.size() && i < cap && items_out; ++i) {
    kvp::DecodeItem it = all[i];
    if (it.kind == 0) it.mem_off = it.row;               // private: the member is the row itself
    else it.mem_off = P.members[it.mem_off];             // prefix: first member of the (sub)group
    std::memcpy(items_out + 8 * i, &it, sizeof(it));
  }
  if (n_items) *n_items = (int)all.size();
  if (n_partials) *n_partials = P.total_parts;
  if (pages_per_split) *pages_per_split = P.pages_per_split;
  return KVP_OK;
}

}  // extern "C"
