// Backward attention, dQ kernel (gfx950); the per-workgroup body is in
// bwd_dq.hpp.
#include "bwd_dq.hpp"

namespace fck {

template <int D, int HPW>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_kernel(DqParams p) {
  __shared__ __attribute__((aligned(16))) char smem[DqLds<D>::bytes];
  dq_tile<D, HPW>(p, blockIdx.x, smem);
}

template <int D>
static hipError_t launch_dq_d(const DqParams& p, int hpw, hipStream_t s) {
  const dim3 grid(unsigned(p.n_items) * p.hkv * p.head_chunks), block(256);
  switch (hpw) {
    case 1: hipLaunchKernelGGL((attn_bwd_dq_kernel<D, 1>), grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL((attn_bwd_dq_kernel<D, 2>), grid, block, 0, s, p); break;
    case 4: hipLaunchKernelGGL((attn_bwd_dq_kernel<D, 4>), grid, block, 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const DqParams& p, int d, int heads_per_tile, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  if (d == 64) return launch_dq_d<64>(p, heads_per_tile, s);
  if (d == 128) return launch_dq_d<128>(p, heads_per_tile, s);
  return hipErrorInvalidValue;
}

}  // namespace fck
