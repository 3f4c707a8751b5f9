// Backward attention kernels (gfx950): the key-major dK/dV kernel, the
// whole deterministic backward pass (dK/dV and dQ workgroups) in one
// launch, and the non-deterministic pass (key tiles that also add dQ with
// atomics). The per-workgroup bodies are in bwd_dkdv.hpp and bwd_dq.hpp.
#include "bwd_dkdv.hpp"
#include "bwd_dq.hpp"

namespace fck {

template <int D>
__global__ __launch_bounds__(256, 2) void attn_bwd_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) char smem[DkdvLds<D>::bytes];
  dkdv_tile<D>(p, blockIdx.x, smem);
}

// The non-deterministic backward pass: key tiles only, each also adding its
// share of dQ into p.dq (zeroed beforehand) with atomics.
template <int D>
__global__ __launch_bounds__(256, 2) void attn_bwd_atomic_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) char smem[DkdvLds<D, true>::bytes];
  dkdv_tile<D, true>(p, blockIdx.x, smem);
}

// The whole backward pass in one launch: the first n_dkdv workgroups take
// key tiles (dK/dV), the others query tiles (dQ); the dQ workgroups start
// as dK/dV ones finish, so neither pass leaves a tail of its own.
template <int D, int HPW>
__global__ __launch_bounds__(256, 2) void attn_bwd_grid_kernel(BwdParams bp, DqParams dp, int n_dkdv) {
  constexpr uint32_t kBytes = DkdvLds<D>::bytes > DqLds<D>::bytes ? DkdvLds<D>::bytes : DqLds<D>::bytes;
  __shared__ __attribute__((aligned(16))) char smem[kBytes];
  const int b = blockIdx.x;
  if (b < n_dkdv)
    dkdv_tile<D>(bp, b, smem);
  else
    dq_tile<D, HPW>(dp, b - n_dkdv, smem);
}

template <int D>
static hipError_t launch_grid_d(const BwdParams& bp, const DqParams& dp, int hpw, hipStream_t s) {
  const int n_dkdv = bp.n_items * bp.hkv;
  const dim3 grid(unsigned(n_dkdv + dp.n_items * dp.hkv * dp.head_chunks)), block(256);
  switch (hpw) {
    case 1: hipLaunchKernelGGL((attn_bwd_grid_kernel<D, 1>), grid, block, 0, s, bp, dp, n_dkdv); break;
    case 2: hipLaunchKernelGGL((attn_bwd_grid_kernel<D, 2>), grid, block, 0, s, bp, dp, n_dkdv); break;
    case 4: hipLaunchKernelGGL((attn_bwd_grid_kernel<D, 4>), grid, block, 0, s, bp, dp, n_dkdv); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_grid(const BwdParams& bp, const DqParams& dp, int d, int heads_per_tile,
                           hipStream_t s) {
  if (bp.n_items == 0 && dp.n_items == 0) return hipSuccess;
  if (d == 64) return launch_grid_d<64>(bp, dp, heads_per_tile, s);
  if (d == 128) return launch_grid_d<128>(bp, dp, heads_per_tile, s);
  return hipErrorInvalidValue;
}

hipError_t launch_bwd_atomic(const BwdParams& p, int d, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  const dim3 grid(unsigned(p.n_items) * p.hkv), block(256);
  if (d == 64)
    hipLaunchKernelGGL(attn_bwd_atomic_kernel<64>, grid, block, 0, s, p);
  else if (d == 128)
    hipLaunchKernelGGL(attn_bwd_atomic_kernel<128>, grid, block, 0, s, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdParams& p, int d, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  const dim3 grid(unsigned(p.n_items) * p.hkv), block(256);
  if (d == 64)
    hipLaunchKernelGGL(attn_bwd_kernel<64>, grid, block, 0, s, p);
  else if (d == 128)
    hipLaunchKernelGGL(attn_bwd_kernel<128>, grid, block, 0, s, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace fck
