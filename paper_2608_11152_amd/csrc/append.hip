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

// ---------------------------------------------------------------------------------------------------
// FP8 (OCP E4M3) pools: y = fp32(x) * inv_scale is rounded to the nearest E4M3 value, ties to the even
// mantissa, saturating at +-448; NaN stays NaN.  Integer arithmetic on the binary32 bits.
// ---------------------------------------------------------------------------------------------------
__device__ __forceinline__ unsigned e4m3_code(float y) {
  const unsigned u = __float_as_uint(y);
  const unsigned sign = (u >> 24) & 0x80u;
  const unsigned a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return sign | 0x7Fu;             // NaN
  if (a >= 0x43E00000u) return sign | 0x7Eu;            // |y| >= 448 (and infinity): saturate
  if (a >= 0x3C800000u) {                               // |y| >= 2^-6: normal, keep 3 mantissa bits
    const unsigned r = a + 0x7FFFFu + ((a >> 20) & 1u);  // round to nearest even at bit 20
    return sign | ((r >> 20) - ((127u - 7u) << 3));
  }
  return sign | (unsigned)__builtin_rintf(__uint_as_float(a) * 512.0f);  // subnormal: m * 2^-9, m <= 8
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((unsigned)b << 16); }

// Quantised codes of 8 bf16 elements, packed little-endian into two words.
__device__ __forceinline__ uint2 quant8(uint4 x, float inv) {
  const uint16_t* h = reinterpret_cast<const uint16_t*>(&x);
  unsigned w[2] = {0u, 0u};
#pragma unroll
  for (int j = 0; j < 8; ++j) w[j >> 2] |= e4m3_code(bf16_to_f32(h[j]) * inv) << (8 * (j & 3));
  return make_uint2(w[0], w[1]);
}

template <int D>
__global__ __launch_bounds__(256) void append_fp8_kernel(AppendArgs a) {
  __shared__ uint16_t vstage[4][16 * D];  // one page of V tokens per wave, [token][dim] bf16
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
  uint8_t* kblk = reinterpret_cast<uint8_t*>(a.layer) + ((int64_t)id * a.Hkv + head) * (2 * 16 * D);
  uint8_t* vblk = kblk + 16 * D;
  const int ntok = r.s_hi - r.s_lo;
  // K: one 16-byte piece per (token, X): dims 64(X/4) + 8(X%4) + j, then the same + 32.
  constexpr int NX = D / 16;
  for (int e = lane; e < ntok * NX; e += 64) {
    const int tt = e / NX, X = e - tt * NX;
    const int c0 = 64 * (X >> 2) + 8 * (X & 3);
    const int64_t src = ((r.src0 + tt) * a.Hkv + head) * D;
    const uint2 lo = quant8(*reinterpret_cast<const uint4*>(a.k + src + c0), a.inv_scale_k);
    const uint2 hi = quant8(*reinterpret_cast<const uint4*>(a.k + src + c0 + 32), a.inv_scale_k);
    store_stream(reinterpret_cast<uint16_t*>(kblk + (X * 16 + r.s_lo + tt) * 16), make_uint4(lo.x, lo.y, hi.x, hi.y));
  }
  uint16_t* vs = vstage[w];
  constexpr int CH = D / 8;
  for (int e = lane; e < ntok * CH; e += 64) {
    const int tt = e / CH, c8 = e - tt * CH;
    const int64_t src = ((r.src0 + tt) * a.Hkv + head) * D + c8 * 8;
    *reinterpret_cast<uint4*>(vs + (r.s_lo + tt) * D + c8 * 8) = *reinterpret_cast<const uint4*>(a.v + src);
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  // V: D pieces of 16 bytes; piece (Y, h, cc) holds slots 8h..8h+7 of dims 32Y + cc and 32Y + 16 + cc.
  for (int e = lane; e < D; e += 64) {
    const int cc = e & 15, h = (e >> 4) & 1, Y = e >> 5;
    uint8_t* dst = vblk + ((Y * 2 + h) * 16 + cc) * 16;
    bool any = false, all = true;
    for (int j = 0; j < 8; ++j) {
      const int t = slot_token(8 * h + j);
      const bool in = t >= r.s_lo && t < r.s_hi;
      any |= in;
      all &= in;
    }
    if (!any) continue;
    union { uint4 u; uint8_t b[16]; } val;
    if (!all) val.u = *reinterpret_cast<const uint4*>(dst);
    for (int dh = 0; dh < 2; ++dh)
      for (int j = 0; j < 8; ++j) {
        const int t = slot_token(8 * h + j);
        if (t >= r.s_lo && t < r.s_hi)
          val.b[dh * 8 + j] = (uint8_t)e4m3_code(bf16_to_f32(vs[t * D + 32 * Y + 16 * dh + cc]) * a.inv_scale_v);
      }
    store_stream(reinterpret_cast<uint16_t*>(dst), val.u);
  }
}

// bf16(fp32(code value) * scale) of the two codes in half `hi` of w.
__device__ __forceinline__ unsigned dequant2(unsigned w, bool hi, float scale) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  const f2 v = hi ? __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true) : __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  bf2 b;
  b[0] = (__bf16)(v[0] * scale);
  b[1] = (__bf16)(v[1] * scale);
  return __builtin_bit_cast(unsigned, b);
}

template <int D>
__global__ __launch_bounds__(256) void gather_fp8_kernel(GatherArgs a) {
  __shared__ uint8_t vblock[4][16 * D];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int unit = blockIdx.x * 4 + w;
  const int run = unit / a.Hkv, head = unit - run * a.Hkv;
  if (run >= a.n_runs) return;
  const PageRun r = a.runs[run];
  const int id = a.bt[(int64_t)r.row * a.maxp + r.lpage];
  const bool ok = (unsigned)id < (unsigned)a.num_pages;
  if (!ok && lane == 0) atomicCAS(a.err, 0, KVP_ERANGE);
  const uint8_t* kblk = reinterpret_cast<const uint8_t*>(a.layer) + ((int64_t)(ok ? id : 0) * a.Hkv + head) * (2 * 16 * D);
  const uint8_t* vblk = kblk + 16 * D;
  uint8_t* vb = vblock[w];
  for (int e = lane; e < D; e += 64)
    *reinterpret_cast<uint4*>(vb + e * 16) = *reinterpret_cast<const uint4*>(vblk + e * 16);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  constexpr int CH = D / 8;
  const int ntok = r.s_hi - r.s_lo;
  for (int e = lane; e < ntok * CH; e += 64) {
    const int tt = e / CH, c8 = e - tt * CH;
    const int s = r.s_lo + tt;
    const int64_t dst = ((r.src0 + tt) * a.Hkv + head) * D + c8 * 8;
    uint4 kk = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (ok) {
      const uint2 kc = *reinterpret_cast<const uint2*>(kblk + k8_index<D>(s, c8 * 8));  // 8 consecutive dims
      kk = make_uint4(dequant2(kc.x, false, a.scale_k), dequant2(kc.x, true, a.scale_k),
                      dequant2(kc.y, false, a.scale_k), dequant2(kc.y, true, a.scale_k));
      unsigned vw[2] = {0u, 0u};
      for (int j = 0; j < 8; ++j) vw[j >> 2] |= (unsigned)vb[v8_index<D>(s, c8 * 8 + j)] << (8 * (j & 3));
      vv = make_uint4(dequant2(vw[0], false, a.scale_v), dequant2(vw[0], true, a.scale_v),
                      dequant2(vw[1], false, a.scale_v), dequant2(vw[1], true, a.scale_v));
    }
    *reinterpret_cast<uint4*>(a.k + dst) = kk;
    *reinterpret_cast<uint4*>(a.v + dst) = vv;
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

// Copy n bytes from pinned host memory to device memory: 16-byte pieces read over the host link by the
// threads of the grid, the last n mod 16 bytes by one thread.  It runs on the compute queue in stream
// order, so the kernel after it needs no hand-off from the copy engine.
__global__ __launch_bounds__(256) void copy_from_host_kernel(unsigned char* dst, const unsigned char* src, size_t n) {
  const size_t n16 = n / 16;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    reinterpret_cast<uint4*>(dst)[i] = reinterpret_cast<const uint4*>(src)[i];
  if (blockIdx.x == 0 && threadIdx.x == 0)
    for (size_t i = n16 * 16; i < n; ++i) dst[i] = src[i];
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, int D, hipStream_t s) {
  const int64_t units = (int64_t)a.n_runs * a.Hkv;
  if (units == 0) return hipSuccess;
  const dim3 grid((unsigned)((units + 3) / 4));
  if (a.fp8) {
    if (D == 128) hipLaunchKernelGGL(append_fp8_kernel<128>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(append_fp8_kernel<64>, grid, dim3(256), 0, s, a);
  } else if (D == 128) {
    hipLaunchKernelGGL(append_kernel<128>, grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(append_kernel<64>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& a, int D, hipStream_t s) {
  const int64_t units = (int64_t)a.n_runs * a.Hkv;
  if (units == 0) return hipSuccess;
  const dim3 grid((unsigned)((units + 3) / 4));
  if (a.fp8) {
    if (D == 128) hipLaunchKernelGGL(gather_fp8_kernel<128>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(gather_fp8_kernel<64>, grid, dim3(256), 0, s, a);
  } else if (D == 128) {
    hipLaunchKernelGGL(gather_kernel<128>, grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(gather_kernel<64>, grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_copy_from_host(void* dst, const void* src, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<size_t>(256, (n / 16 + 255) / 256 + 1);
  hipLaunchKernelGGL(copy_from_host_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<unsigned char*>(dst),
                     reinterpret_cast<const unsigned char*>(src), n);
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
