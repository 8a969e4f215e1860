// Block-granular prefix identification (Sec. 4.4 of the paper: the engine's prefix cache keys every
// full prompt block by a hash, and a request's reusable prefix H is the longest run of its leading full
// blocks whose hashes are cached).  The paper leaves the hash unspecified; the one defined here is
//
//   mix(z)    = SplitMix64 output function of z (Steele, Lea and Flood 2014; constants as published):
//               z += 0x9E3779B97F4A7C15; z = (z ^ z>>30) * 0xBF58476D1CE4E5B9;
//               z = (z ^ z>>27) * 0x94D049BB133111EB; z ^= z>>31
//   local(k)  = x folded over the page's 8 token pairs from x = 0:  x = mix(x ^ (t[2j] | t[2j+1] << 32))
//   h(-1)     = seed;  h(k) = h(k-1) * P + local(k)  (mod 2^64),  P = 0x9E3779B97F4A7C15
//   hash(k)   = mix(h(k))
//
// so hash(k) names tokens [0, 16(k+1)) of a sequence.  The chain is affine in h, so it splits into
// independent 64-page chunks: pass 1 folds every page's tokens (one lane per page) and chains a chunk's
// pages from 0 with an inclusive scan of the affine maps (a, b): h -> a*h + b; pass 2 composes the
// chunk maps before each chunk to get its entering value and finishes every page.  A page's composed
// slope is gamma^(j+1), known without data.
//
// A device hash table (open addressing, linear probing) maps a block hash to the physical page holding
// that block, for the prefix lookup of new requests (probed 64 pages per wave, in two passes: per-chunk
// probes, then the earliest miss of a sequence ends its reusable prefix).  Key 0 marks an empty slot, so a block hash of 0 is
// stored as 1; a slot's page is the largest page id inserted for its key, -1 once erased.
#include "kvp_kernels.h"

namespace kvp {
namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z += kGamma;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t shfl_up64(uint64_t v, int d) {
  const unsigned lo = __shfl_up((unsigned)v, d), hi = __shfl_up((unsigned)(v >> 32), d);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  const unsigned lo = __shfl((unsigned)v, src), hi = __shfl((unsigned)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t table_key(uint64_t h) { return h ? h : 1ull; }

// Inclusive scan over the 64 lanes of the affine maps h -> A*h + B (lane j ends with the composition of
// lanes 0..j, lane 0's map applied first).
__device__ __forceinline__ void affine_scan(uint64_t& A, uint64_t& B, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t pa = shfl_up64(A, d), pb = shfl_up64(B, d);
    if (lane >= d) {
      B = pb * A + B;
      A = pa * A;
    }
  }
}

// Pass 1: one wave per 64-page chunk.  Lane j folds its page's tokens; the scan gives the chunk-local
// chain value B_j (the chain started from 0 at the chunk's first page), kept in the output slot, and the
// chunk's whole map (gamma^n, B_{n-1}) for pass 2.
__global__ __launch_bounds__(64) void hash_chunk_kernel(HashArgs a) {
  const HashChunk ch = a.chunks[blockIdx.x];
  const int lane = threadIdx.x;
  uint64_t A = 1, B = 0;
  if (lane < ch.n) {
    const int32_t* t = a.tokens + ch.t0 + 16 * (int64_t)lane;
    uint64_t x = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint64_t w = (uint64_t)(uint32_t)t[2 * j] | ((uint64_t)(uint32_t)t[2 * j + 1] << 32);
      x = mix64(x ^ w);
    }
    A = kGamma;
    B = x;
  }
  affine_scan(A, B, lane);
  if (lane < ch.n) a.out[ch.o0 + lane] = B;
  if (lane == ch.n - 1) {
    a.totals[2 * (ch.g0 + ch.c)] = A;
    a.totals[2 * (ch.g0 + ch.c) + 1] = B;
  }
}

// Pass 2: one wave per chunk.  The chain value entering chunk c is the composition of chunks 0..c-1
// applied to the seed (scanned 64 chunks at a time); lane j then finishes
// hash = mix(gamma^(j+1) * carry + B_j).
__global__ __launch_bounds__(64) void hash_finish_kernel(HashArgs a) {
  const HashChunk ch = a.chunks[blockIdx.x];
  const int lane = threadIdx.x;
  uint64_t carry = a.seed;
  for (int c0 = 0; c0 < ch.c; c0 += 64) {
    uint64_t A = 1, B = 0;
    if (c0 + lane < ch.c) {
      A = a.totals[2 * (ch.g0 + c0 + lane)];
      B = a.totals[2 * (ch.g0 + c0 + lane) + 1];
    }
    affine_scan(A, B, lane);
    const int last = min(63, ch.c - c0 - 1);
    carry = shfl64(A, last) * carry + shfl64(B, last);
  }
  if (lane < ch.n) {
    uint64_t g = 1, b = kGamma;  // gamma^(lane + 1) by squaring
    for (unsigned e = (unsigned)lane + 1; e; e >>= 1) {
      if (e & 1) g *= b;
      b *= b;
    }
    a.out[ch.o0 + lane] = mix64(g * carry + a.out[ch.o0 + lane]);
  }
}

// One 64-lane workgroup per group: the number of leading pages on which every member's block hash
// equals the first member's (capped by the shortest member).
__global__ __launch_bounds__(64) void group_lcp_kernel(GroupLcpArgs a) {
  const int g = blockIdx.x, lane = threadIdx.x;
  const int m0 = a.grp_off[g], m1 = a.grp_off[g + 1];
  if (m1 <= m0) {
    if (lane == 0) a.shared_pages[g] = 0;
    return;
  }
  int np = 1 << 30;
  for (int m = m0; m < m1; ++m) np = min(np, a.seq_info[a.members[m]].y);
  const int64_t base0 = a.seq_info[a.members[m0]].z;
  int shared = np;
  for (int c = 0; c < np; c += 64) {
    const int k = c + lane;
    bool ok = k < np;
    if (ok) {
      const uint64_t h0 = a.hashes[base0 + k];
      for (int m = m0 + 1; m < m1 && ok; ++m) ok = a.hashes[a.seq_info[a.members[m]].z + k] == h0;
    }
    const uint64_t bad = __ballot(k < np && !ok);
    if (bad) {
      shared = c + __builtin_ctzll(bad);
      break;
    }
  }
  if (lane == 0) a.shared_pages[g] = shared;
}

__global__ void table_insert_kernel(TableArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const uint64_t key = table_key(a.hashes[i]);
  const int page = a.pages[i];
  uint64_t s = key & a.mask;
  for (uint64_t probe = 0; probe <= a.mask; ++probe) {
    unsigned long long* kp = reinterpret_cast<unsigned long long*>(a.keys) + s;
    const unsigned long long prev = atomicCAS(kp, 0ull, (unsigned long long)key);
    if (prev == 0ull || prev == key) {
      atomicMax(a.vals + s, page);
      return;
    }
    s = (s + 1) & a.mask;
  }
  atomicCAS(a.err, 0, KVP_ENOMEM);  // table full: the item is dropped and the table reports it
}

__global__ void table_erase_kernel(TableArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const uint64_t key = table_key(a.hashes[i]);
  uint64_t s = key & a.mask;
  for (uint64_t probe = 0; probe <= a.mask; ++probe) {
    const uint64_t k = a.keys[s];
    if (k == 0) return;
    if (k == key) {
      atomicCAS(a.vals + s, a.pages[i], -1);
      return;
    }
    s = (s + 1) & a.mask;
  }
}

__device__ __forceinline__ int table_find(const TableArgs& a, uint64_t h) {
  const uint64_t key = table_key(h);
  uint64_t s = key & a.mask;
  for (uint64_t probe = 0; probe <= a.mask; ++probe) {
    const uint64_t k = a.keys[s];
    if (k == 0) return -1;
    if (k == key) return a.vals[s];
    s = (s + 1) & a.mask;
  }
  return -1;
}

// Lookup pass 1: one wave per 64-page chunk of a sequence.  Every page is probed; the chunk's first
// miss (a page index within the sequence, or the sequence's page count when it has none) goes to
// scratch.
__global__ __launch_bounds__(64) void lookup_chunk_kernel(TableArgs a) {
  const HashChunk ch = a.chunks[blockIdx.x];
  const int lane = threadIdx.x;
  int page = -1;
  if (lane < ch.n) page = table_find(a, a.hashes[ch.o0 + lane]);
  if (lane < ch.n) a.out_pages[ch.o0 + lane] = page;
  const uint64_t miss = __ballot(lane < ch.n && page < 0);
  if (lane == 0) a.first_miss[ch.g0 + ch.c] = miss ? 64 * ch.c + (int)__builtin_ctzll(miss) : ch.pad[2];
}

// Lookup pass 2: one wave per chunk.  The sequence's reusable prefix ends at the earliest first miss of
// its chunks; pages from there on are reported as -1.
__global__ __launch_bounds__(64) void lookup_finish_kernel(TableArgs a) {
  const HashChunk ch = a.chunks[blockIdx.x];
  const int lane = threadIdx.x;
  const int nch = ch.pad[0];
  int m = 1 << 30;
  for (int c0 = 0; c0 < nch; c0 += 64)
    if (c0 + lane < nch) m = min(m, a.first_miss[ch.g0 + c0 + lane]);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) m = min(m, __shfl_xor(m, d));
  if (lane < ch.n && 64 * ch.c + lane >= m) a.out_pages[ch.o0 + lane] = -1;
  if (ch.c == 0 && lane == 0) a.matched[ch.pad[1]] = m;
}

__global__ void fill_table_kernel(uint64_t* keys, int32_t* vals, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    keys[i] = 0;
    vals[i] = -1;
  }
}

}  // namespace

hipError_t launch_block_hash(const HashArgs& a, int n_chunks, hipStream_t s) {
  if (n_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(hash_chunk_kernel, dim3(n_chunks), dim3(64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(hash_finish_kernel, dim3(n_chunks), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_group_lcp(const GroupLcpArgs& a, int n_groups, hipStream_t s) {
  if (n_groups == 0) return hipSuccess;
  hipLaunchKernelGGL(group_lcp_kernel, dim3(n_groups), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_table(const TableArgs& a, int op, int n_seqs, hipStream_t s) {
  if (op == 0 || op == 1) {
    if (a.n == 0) return hipSuccess;
    const dim3 grid((unsigned)((a.n + 255) / 256));
    if (op == 0) hipLaunchKernelGGL(table_insert_kernel, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(table_erase_kernel, grid, dim3(256), 0, s, a);
  } else if (op == 2) {
    if (n_seqs == 0) return hipSuccess;  // n_seqs: chunk count here
    hipLaunchKernelGGL(lookup_chunk_kernel, dim3(n_seqs), dim3(64), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(lookup_finish_kernel, dim3(n_seqs), dim3(64), 0, s, a);
  } else {
    hipLaunchKernelGGL(fill_table_kernel, dim3(1024), dim3(256), 0, s, a.keys, a.vals, (int64_t)a.mask + 1);
  }
  return hipGetLastError();
}

}  // namespace kvp
