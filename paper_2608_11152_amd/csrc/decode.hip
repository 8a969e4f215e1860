// Paged decode attention for prefix-shared rollout groups (gfx950).
//
// The work list (plan.cpp) splits every sequence's pages into ranges; each range of each KV head yields a
// partial softmax state (running max m in log2 units, weight sum l, unnormalised accumulator acc) that
// the merge kernel combines with a log-sum-exp rescale.  A rollout group's shared prompt pages (Sec. 3.1
// group id g_r, Sec. 4.4 block-granular prefix reuse) form ranges of their own whose query columns are
// every member's heads, so those pages are read from HBM once per group rather than once per sample.
//
// Tile shapes.  Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_16x16x32_bf16: the 16 rows
// are 16 tokens (8 of each of two pages), the 16 columns are query columns (member x head of one KV
// head).  The score tile's register layout is exactly the layout of the P^T operand of the next product
// O^T = V^T P^T (16 d-rows x 16 columns, k = 32 token slots of two pages), so probabilities never leave
// registers.  The pool layout (kvp_layout.h) makes every K and V operand a contiguous 16-byte load.
#include <algorithm>
#include <cstring>

#include "decode_dev.h"

namespace kvp {
namespace {

using namespace dec;

// ---------------------------------------------------------------------------------------------------
// Calls without LDS-staged prefix items launch the wave path alone, 8 waves per workgroup: the
// dispatcher starts workgroups at a bounded rate, so half as many workgroups reach the CUs in about
// half the time (a 5-6 us ramp instead of 12-13 us for 2048 waves).
// ---------------------------------------------------------------------------------------------------
template <int D, bool FP8>
__global__ __launch_bounds__(512) void decode_wave_kernel(DecodeArgs a) {
  decode_wave_block<D, FP8>(a, blockIdx.x);
}

// ---------------------------------------------------------------------------------------------------
// Otherwise one launch covers both paths: blocks [0, n_wave_blocks) run 4 wave-path waves each; the
// remaining blocks run the LDS-staged shared-prefix path, one per (prefix item, KV head), whose four
// waves synchronise.  Blocks are dispatched in index order, so the wave blocks take the first round
// and the shared-prefix blocks run in the slots the planner left free for them.  The two paths need
// the same number of registers to within a few, so sharing a launch costs no occupancy and saves a
// launch boundary.
// ---------------------------------------------------------------------------------------------------
template <int D, bool FP8>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a) {
  constexpr int LB = FP8 ? GroupLds8<D>::bytes : GroupLds<D>::bytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[LB];
  if ((int)blockIdx.x < a.n_wave_blocks) {
    decode_wave_block<D, FP8>(a, blockIdx.x);
  } else {
    if constexpr (FP8) decode_group_block_fp8<D>(a, (int)blockIdx.x - a.n_wave_blocks, lds);
    else decode_group_block<D>(a, (int)blockIdx.x - a.n_wave_blocks, lds);
  }
}

// ---------------------------------------------------------------------------------------------------
// Log-sum-exp merge: out = sum_j acc_j 2^(m_j - m) / sum_j l_j 2^(m_j - m), m = max_j m_j, in a fixed
// order (so results are deterministic).  Empty partials (m = -inf, l = 0) carry zero weight; a
// sequence with no partial gets a zero output.  One workgroup per (sequence, KV head, group of hw query
// heads), started from one 16-byte record {seq, first partial, partial count}; hw is chosen per call so
// that few sequences still spread over enough workgroups and many do not pay for extra ones.
// T = 256 / (hw * D / 4) consecutive lanes share each output float4: lane q loads partials q, q + T, ...
// (accumulator and (m, l) together, all in flight at once), folds them with a running max, and the T
// lanes are then combined by shuffles, so the whole merge costs one round of memory latency.
// ---------------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(MergeArgs a) {
  constexpr int V4 = D / 4;  // float4 per head row
  constexpr int U = 16;      // partials in flight per lane
  const int G = a.Hq / a.Hkv;
  const int hw = a.hw;
  const int nsplit = G / hw;
  const int b = blockIdx.x;
  const int rest = b / nsplit;
  const int sub = b - rest * nsplit;
  const int grp = rest / a.Hkv;
  const int kvh = rest - grp * a.Hkv;
  const int4 info = reinterpret_cast<const int4*>(a.merge_info)[grp];
  const int seq = info.x, P = info.z;
  const int64_t base = info.y;
  const int tid = threadIdx.x;
  const int T = 256 / (hw * V4);  // lanes per output float4: 1 to 16 (a divisor of 64)
  const int e = tid / T, q = tid - e * T;
  const int hh = e / V4, d4 = e - hh * V4;
  const int h = kvh * G + sub * hw + hh;
  const int64_t sa = (int64_t)a.Hq * D;
  const float* pa = a.part_acc + (base * a.Hq + h) * D + 4 * d4;
  const float2* pm = a.part_ml + base * a.Hq + h;
  float m = -INFINITY, l = 0.0f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int j0 = q; j0 < P; j0 += U * T) {
    f32x4 v[U];
    float2 ml[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * T;
      if (j < P) {
        v[u] = *reinterpret_cast<const f32x4*>(pa + j * sa);
        ml[u] = pm[(int64_t)j * a.Hq];
      }
    }
    float mr = m;
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (j0 + u * T < P) mr = fmaxf(mr, ml[u].x);
    if (mr != -INFINITY) {
      const float r = fast_exp2(m - mr);  // 0 while nothing has been seen (m = -inf)
      acc *= r;
      l *= r;
      m = mr;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (j0 + u * T < P) {
          const float w = fast_exp2(ml[u].x - m);
          acc += w * v[u];
          l += w * ml[u].y;
        }
    }
  }
  // combine the T lanes of this output (consecutive lanes of one wave)
  float mt = m;
  for (int o = T >> 1; o >= 1; o >>= 1) mt = fmaxf(mt, __shfl_xor(mt, o));
  const float r = mt == -INFINITY ? 0.0f : fast_exp2(m - mt);
  acc *= r;
  l *= r;
  for (int o = T >> 1; o >= 1; o >>= 1) {
    l += __shfl_xor(l, o);
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] += __shfl_xor(acc[c], o);
  }
  if (q != 0) return;
  acc *= (mt != -INFINITY && l > 0.0f) ? 1.0f / l : 0.0f;
  const int64_t oi = ((int64_t)seq * a.Hq + h) * D + 4 * d4;
  if (a.out_f32) {
    *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + oi) = acc;
  } else {
    uint2 u;
    u.x = pack_bf16(acc[0], acc[1]);
    u.y = pack_bf16(acc[2], acc[3]);
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + oi) = u;
  }
}

// ---------------------------------------------------------------------------------------------------
// Host bytes written to device memory through kernel arguments (the allocation-free decode entry point
// stages its work list this way: no pinned host buffer, and the bytes travel by value with the launch).
// ---------------------------------------------------------------------------------------------------
constexpr int kArgChunkBytes = 3840;  // payload per launch; the whole argument block stays under 4 KB

struct ArgChunk {
  unsigned char* dst;
  uint32_t n;  // payload bytes, a multiple of 16
  uint32_t pad;
  uint4 bytes[kArgChunkBytes / 16];
};

__global__ __launch_bounds__(256) void put_bytes_kernel(ArgChunk c) {
  for (uint32_t i = threadIdx.x; i < c.n / 16; i += blockDim.x) reinterpret_cast<uint4*>(c.dst)[i] = c.bytes[i];
}

}  // namespace

hipError_t launch_put_bytes(void* dst, const void* src, size_t n, hipStream_t s) {
  const unsigned char* h = reinterpret_cast<const unsigned char*>(src);
  for (size_t off = 0; off < n; off += kArgChunkBytes) {
    ArgChunk c{};
    const size_t k = std::min<size_t>(kArgChunkBytes, n - off);
    c.dst = reinterpret_cast<unsigned char*>(dst) + off;
    c.n = (uint32_t)((k + 15) & ~size_t(15));
    std::memcpy(c.bytes, h + off, k);
    hipLaunchKernelGGL(put_bytes_kernel, dim3(1), dim3(256), 0, s, c);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_decode(const DecodeArgs& a, int D, hipStream_t s) {
  const int64_t blocks = (int64_t)a.n_wave_blocks + a.n_group_blocks;
  if (blocks == 0) return hipSuccess;
  if (a.n_group_blocks == 0) {
    const dim3 g((unsigned)(((int64_t)a.n_items * a.Hkv + 7) / 8));
    if (a.fp8) {
      if (D == 128) hipLaunchKernelGGL((decode_wave_kernel<128, true>), g, dim3(512), 0, s, a);
      else hipLaunchKernelGGL((decode_wave_kernel<64, true>), g, dim3(512), 0, s, a);
    } else if (D == 128) {
      hipLaunchKernelGGL((decode_wave_kernel<128, false>), g, dim3(512), 0, s, a);
    } else {
      hipLaunchKernelGGL((decode_wave_kernel<64, false>), g, dim3(512), 0, s, a);
    }
    return hipGetLastError();
  }
  const dim3 grid((unsigned)blocks);
  if (a.fp8) {
    if (D == 128) hipLaunchKernelGGL((decode_kernel<128, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((decode_kernel<64, true>), grid, dim3(256), 0, s, a);
  } else if (D == 128) {
    hipLaunchKernelGGL((decode_kernel<128, false>), grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((decode_kernel<64, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_decode_merge(const MergeArgs& a, int D, hipStream_t s) {
  if (a.n_merge == 0) return hipSuccess;
  // Split the query heads of a (sequence, KV head) over up to G workgroups while the grid stays at or
  // under 1024 workgroups; at most 256 threads' worth of float4 outputs per workgroup.
  const int G = a.Hq / a.Hkv;
  const int64_t units = (int64_t)a.n_merge * a.Hkv;
  int nsplit = 1;
  while (2 * nsplit <= G && (units * 2 * nsplit <= 1024 || G / nsplit > 1024 / D)) nsplit *= 2;
  MergeArgs m = a;
  m.hw = G / nsplit;
  const dim3 grid((unsigned)(units * nsplit));
  if (D == 128) hipLaunchKernelGGL(decode_merge_kernel<128>, grid, dim3(256), 0, s, m);
  else hipLaunchKernelGGL(decode_merge_kernel<64>, grid, dim3(256), 0, s, m);
  return hipGetLastError();
}

}  // namespace kvp
