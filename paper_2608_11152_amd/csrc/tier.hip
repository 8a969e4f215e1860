// CPU KV tier: whole pool pages copied between HBM and pinned host memory (the host-memory backup tier of
// Sec. 5.5 of the paper, which keeps a copy of GPU-resident KV so evicted pages return without
// recomputation).  One workgroup per page: the GPU reads (restore) or writes (offload) the host copy
// directly over the host link, with eight 16-byte accesses per thread in flight, so a batch of scattered
// pages costs one launch rather than one copy call per page.
#include "kvp_kernels.h"

namespace kvp {
namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <bool kRestore>
__global__ __launch_bounds__(256) void tier_kernel(TierArgs a) {
  const int i = blockIdx.x;
  const TierItem it = a.items[i];
  unsigned char* page = a.layer + (int64_t)it.page * a.page_bytes;
  unsigned char* host = a.host + (int64_t)i * a.page_bytes;
  constexpr int U = 8;
  const int step = 256 * 16;
  for (int64_t off = threadIdx.x * 16; off < a.page_bytes; off += (int64_t)U * step) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t o = off + (int64_t)u * step;
      if (o < a.page_bytes)
        v[u] = kRestore ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(host + o))
                        : __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(page + o));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t o = off + (int64_t)u * step;
      if (o < a.page_bytes) {
        if (kRestore) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(page + o));
        else __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(host + o));
      }
    }
  }
  if (kRestore && a.bt && threadIdx.x == 0) a.bt[(int64_t)it.row * a.maxp + it.lpage] = it.page;
}

}  // namespace

hipError_t launch_tier(const TierArgs& a, bool restore, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  if (restore) hipLaunchKernelGGL(tier_kernel<true>, dim3(a.n), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(tier_kernel<false>, dim3(a.n), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace kvp
