// Chunked prefill of a new turn over a cached history (Eq. 1 of the paper: a later agentic turn only
// prefills its L - H uncached tokens; they attend to the cached H tokens and causally to each other).
//
// One workgroup of kPrefillWaves waves per (session, KV head, 32 x kPrefillWaves flattened query rows, key range).  Query rows are flattened as
// position * G + head-in-group, so every K/V tile loaded serves all G query heads of its KV head.  Keys
// stream through LDS in stages of 4 pages (64 keys), double-buffered: the next stage is loaded into
// registers while this stage's MFMA work runs, then stored to the other buffer.  Wave w owns 32 query
// rows:
//   S^T (64 keys x 32 rows) = K Q^T      v_mfma_f32_32x32x16_bf16, 2 key tiles x D/16 k-steps
//   O^T (D x 32 rows)      += V^T P^T    the score tile's registers are the P^T operand (per page)
// Masking is applied only to stages that reach past the wave's first query position (the diagonal).
// A tile whose history the planner split into key ranges (few tiles over long histories) writes, per
// range, the unnormalised partial state (running max, weight sum, accumulator) instead of its output;
// the decode path's log-sum-exp merge kernel then combines the ranges of each query row.
#include "prefill_dev.h"

namespace kvp {
namespace {

using namespace pf;

template <int D, bool FP8>
__global__ __launch_bounds__(64 * kPrefillWaves, 8 / kPrefillWaves) void prefill_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[PrefillLds<D>::bytes];
  const unsigned item = blockIdx.x;
#include "prefill_body.inc"
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs& a, int D, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  const dim3 grid(a.n_items), block(64 * kPrefillWaves);
  if (a.fp8) {
    if (D == 128) hipLaunchKernelGGL((prefill_kernel<128, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((prefill_kernel<64, true>), grid, block, 0, s, a);
  } else if (D == 128) {
    hipLaunchKernelGGL((prefill_kernel<128, false>), grid, block, 0, s, a);
  } else {
    hipLaunchKernelGGL((prefill_kernel<64, false>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace kvp
