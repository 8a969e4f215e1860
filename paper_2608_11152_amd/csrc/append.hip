// kv_append / kv_gather / pool fill kernels.
//
// kv_append writes new tokens' K/V into their paged slots (a session's retained KV blocks grow, Sec. 3.2
// of the paper); kv_gather reads tokens back in logical order.  Both work on (page run, kv head) units:
// one wave moves every token of one sequence that lands in one page, for one KV head, so each unit's
// writes are whole 16-byte chunks of a single 8 KB page block.
#include "kvp_kernels.h"
#include "kvp_layout.h"

namespace kvp {

namespace {

// Pool writes are streaming stores: left as ordinary dirty lines in the caches, the scattered page
// blocks of a large append slow the next decode's streaming reads when they are evicted.
__device__ __forceinline__ void store_stream(uint16_t* p, uint4 v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4*>(p));
}

template <int D>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  __shared__ uint16_t vstage[4][16 * D];  // one page of V tokens per wave, [slot][dim]
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int unit = blockIdx.x * 4 + w;
  const int run = unit / a.Hkv, head = unit - run * a.Hkv;
  if (run >= a.n_runs) return;
  const PageRun r = a.runs[run];
  const int id = a.bt[(int64_t)r.row * a.maxp + r.lpage];
  if ((unsigned)id >= (unsigned)a.num_pages) {
    if (lane == 0) atomicCAS(a.err, 0, KVP_ERANGE);
    return;
  }
  uint16_t* kblk = a.layer + ((int64_t)id * a.Hkv + head) * (2 * 16 * D);
  uint16_t* vblk = kblk + 16 * D;
  constexpr int CH = D / 8;  // 16-byte chunks per token row
  const int ntok = r.s_hi - r.s_lo;
  uint16_t* vs = vstage[w];
  for (int e = lane; e < ntok * CH; e += 64) {
    const int tt = e / CH, c8 = e - tt * CH;
    const int64_t src = ((r.src0 + tt) * a.Hkv + head) * D + c8 * 8;
    const uint4 kk = *reinterpret_cast<const uint4*>(a.k + src);
    const uint4 vv = *reinterpret_cast<const uint4*>(a.v + src);
    const int s = r.s_lo + tt;
    store_stream(kblk + k_index<D>(s, c8 * 8), kk);
    *reinterpret_cast<uint4*>(vs + s * D + c8 * 8) = vv;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  // V block: 2*D chunks, chunk (dt, h, c) holds slots 8h..8h+7 of dim 16*dt + c.
  for (int e = lane; e < 2 * D; e += 64) {
    const int c = e & 15, h = (e >> 4) & 1, dt = e >> 5;
    const int dim = dt * 16 + c;
    uint16_t* dst = vblk + v_index<D>(/*token of slot 8h*/ slot_token(8 * h), dim);
    bool any = false, all = true;
    for (int j = 0; j < 8; ++j) {
      const int t = slot_token(8 * h + j);
      const bool in = t >= r.s_lo && t < r.s_hi;
      any |= in;
      all &= in;
    }
    if (!any) continue;
    union { uint4 u; uint16_t s[8]; } val;
    if (!all) val.u = *reinterpret_cast<const uint4*>(dst);
    for (int j = 0; j < 8; ++j) {
      const int t = slot_token(8 * h + j);
      if (t >= r.s_lo && t < r.s_hi) val.s[j] = vs[t * D + dim];
    }
    store_stream(dst, val.u);
  }
}

template <int D>
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  __shared__ uint16_t vblock[4][16 * D];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int unit = blockIdx.x * 4 + w;
  const int run = unit / a.Hkv, head = unit - run * a.Hkv;
  if (run >= a.n_runs) return;
  const PageRun r = a.runs[run];
  const int id = a.bt[(int64_t)r.row * a.maxp + r.lpage];
  const bool ok = (unsigned)id < (unsigned)a.num_pages;
  if (!ok && lane == 0) atomicCAS(a.err, 0, KVP_ERANGE);
  const uint16_t* kblk = a.layer + ((int64_t)(ok ? id : 0) * a.Hkv + head) * (2 * 16 * D);
  const uint16_t* vblk = kblk + 16 * D;
  uint16_t* vb = vblock[w];
  for (int e = lane; e < 2 * D; e += 64)
    *reinterpret_cast<uint4*>(vb + e * 8) = *reinterpret_cast<const uint4*>(vblk + e * 8);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  constexpr int CH = D / 8;
  const int ntok = r.s_hi - r.s_lo;
  for (int e = lane; e < ntok * CH; e += 64) {
    const int tt = e / CH, c8 = e - tt * CH;
    const int s = r.s_lo + tt;
    const int64_t dst = ((r.src0 + tt) * a.Hkv + head) * D + c8 * 8;
    uint4 kk = ok ? *reinterpret_cast<const uint4*>(kblk + k_index<D>(s, c8 * 8)) : make_uint4(0, 0, 0, 0);
    union { uint4 u; uint16_t s[8]; } vv;
    for (int j = 0; j < 8; ++j) vv.s[j] = ok ? vb[v_index<D>(s, c8 * 8 + j)] : 0;
    *reinterpret_cast<uint4*>(a.k + dst) = kk;
    *reinterpret_cast<uint4*>(a.v + dst) = vv.u;
  }
}

__global__ void fill_zero_kernel(uint4* p, size_t n16) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) p[i] = make_uint4(0, 0, 0, 0);
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, int D, hipStream_t s) {
  const int64_t units = (int64_t)a.n_runs * a.Hkv;
  if (units == 0) return hipSuccess;
  const dim3 grid((unsigned)((units + 3) / 4));
  if (D == 128) hipLaunchKernelGGL(append_kernel<128>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(append_kernel<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& a, int D, hipStream_t s) {
  const int64_t units = (int64_t)a.n_runs * a.Hkv;
  if (units == 0) return hipSuccess;
  const dim3 grid((unsigned)((units + 3) / 4));
  if (D == 128) hipLaunchKernelGGL(gather_kernel<128>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(gather_kernel<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<size_t>(8192, (n16 + 255) / 256);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<uint4*>(p), n16);
  return hipGetLastError();
}

}  // namespace kvp
