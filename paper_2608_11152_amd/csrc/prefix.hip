// Block-granular prefix identification (Sec. 4.4 of the paper: the engine's prefix cache names every
// full prompt block by a hash, and the longest matching prompt-block hash is a request's reusable prefix
// H).  The paper leaves the hash unspecified; the one defined here is
//
//   mix(z)    = SplitMix64 output function of z (Steele, Lea and Flood 2014; constants as published):
//               z += 0x9E3779B97F4A7C15; z = (z ^ z>>30) * 0xBF58476D1CE4E5B9;
//               z = (z ^ z>>27) * 0x94D049BB133111EB; z ^= z>>31
//   local(k)  = x folded over the page's 8 token pairs from x = 0:  x = mix(x ^ (t[2j] | t[2j+1] << 32))
//   h(-1)     = seed;  h(k) = h(k-1) * P + local(k)  (mod 2^64),  P = 0x9E3779B97F4A7C15
//   hash(k)   = mix(h(k))
//
// so hash(k) names tokens [0, 16(k+1)) of a sequence.  The chain is affine in h, which lets a wave hash
// 64 pages at once: each lane folds its page's tokens, and an inclusive scan of the affine maps
// (a, b): h -> a*h + b over the 64 lanes chains them.
//
// A device hash table (open addressing, linear probing) maps a block hash to the physical page holding
// that block, for the prefix lookup of new requests.  Key 0 marks an empty slot, so a block hash of 0 is
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

// One 64-lane workgroup per sequence; lane j hashes page c + j of each 64-page chunk.
__global__ __launch_bounds__(64) void block_hash_kernel(HashArgs a) {
  const int i = blockIdx.x, lane = threadIdx.x;
  const int64_t t0 = a.seq_info[i].x;
  const int np = a.seq_info[i].y;
  const int64_t o0 = a.seq_info[i].z;
  uint64_t carry = a.seed;
  for (int c = 0; c < np; c += 64) {
    const int k = c + lane;
    uint64_t A = 1, B = 0;
    if (k < np) {
      const int32_t* t = a.tokens + t0 + 16 * (int64_t)k;
      uint64_t x = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint64_t w = (uint64_t)(uint32_t)t[2 * j] | ((uint64_t)(uint32_t)t[2 * j + 1] << 32);
        x = mix64(x ^ w);
      }
      A = kGamma;
      B = x;
    }
    // Inclusive scan of h -> A*h + B: lane j ends with the composition of lanes 0..j.
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t pa = shfl_up64(A, d), pb = shfl_up64(B, d);
      if (lane >= d) {
        B = pb * A + B;
        A = pa * A;
      }
    }
    const uint64_t h = A * carry + B;
    if (k < np) a.out[o0 + k] = mix64(h);
    carry = shfl64(h, min(63, np - c - 1));
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

// One 64-lane workgroup per sequence: the leading pages whose block hash maps to a cached page.
__global__ __launch_bounds__(64) void table_lookup_kernel(TableArgs a) {
  const int i = blockIdx.x, lane = threadIdx.x;
  const int np = a.seq_info[i].y;
  const int64_t o0 = a.seq_info[i].z;
  int matched = np;
  bool done = false;
  for (int c = 0; c < np; c += 64) {
    const int k = c + lane;
    int page = -1;
    if (k < np && !done) page = table_find(a, a.hashes[o0 + k]);
    const uint64_t miss = __ballot(k < np && page < 0);
    const int first = miss ? c + __builtin_ctzll(miss) : np;
    if (k < np) a.out_pages[o0 + k] = (k < first && !done) ? page : -1;
    if (miss && !done) {
      matched = first;
      done = true;
    }
  }
  if (lane == 0) a.matched[i] = matched;
}

__global__ void fill_table_kernel(uint64_t* keys, int32_t* vals, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    keys[i] = 0;
    vals[i] = -1;
  }
}

}  // namespace

hipError_t launch_block_hash(const HashArgs& a, int n_seqs, hipStream_t s) {
  if (n_seqs == 0) return hipSuccess;
  hipLaunchKernelGGL(block_hash_kernel, dim3(n_seqs), dim3(64), 0, s, a);
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
    if (n_seqs == 0) return hipSuccess;
    hipLaunchKernelGGL(table_lookup_kernel, dim3(n_seqs), dim3(64), 0, s, a);
  } else {
    hipLaunchKernelGGL(fill_table_kernel, dim3(1024), dim3(256), 0, s, a.keys, a.vals, (int64_t)a.mask + 1);
  }
  return hipGetLastError();
}

}  // namespace kvp
