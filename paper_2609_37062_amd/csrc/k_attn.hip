// Paged-attention decode over the block-table KV cache, split-K over context:
// one workgroup per (split, KV head, row); the work item itself is
// attn_unit (attn_core.hpp).
#include "attn_core.hpp"

namespace vsk {

template <int D, int NB>
__global__ __launch_bounds__(64 * kAttnWaves) void k_attn_decode(AttnArgs a) {
  __shared__ AttnLds<D> sm;
  attn_unit<D, NB, false>(a, blockIdx.z, blockIdx.y, blockIdx.x, sm);
}

hipError_t launch_attn_decode(const AttnArgs& a, int n_rows, hipStream_t s) {
  dim3 grid(a.max_splits, a.Hkv, n_rows);
  if (a.hd == 128) {
    hipLaunchKernelGGL((k_attn_decode<128, 4>), grid, dim3(64 * kAttnWaves), 0, s, a);
  } else if (a.hd == 64) {
    hipLaunchKernelGGL((k_attn_decode<64, 4>), grid, dim3(64 * kAttnWaves), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace vsk
