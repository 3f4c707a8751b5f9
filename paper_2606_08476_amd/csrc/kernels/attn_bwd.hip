// Backward attention kernels (gfx950): the key-major dK/dV kernel, the
// whole deterministic backward pass (dK/dV and dQ workgroups) in one
// launch, and the non-deterministic pass (key tiles that also add dQ with
// atomics). The per-workgroup bodies are in bwd_dkdv.hpp and bwd_dq.hpp.
#include "bwd_dkdv.hpp"
#include "bwd_dq.hpp"

namespace fck {

// Query heads per dK/dV iteration: the most of 4, 2, 1 that divides the
// group.
static int heads_per_iteration(int group) { return group % 4 == 0 ? 4 : group % 2 == 0 ? 2 : 1; }

template <int D, int HPI>
__global__ __launch_bounds__(256, 2) void attn_bwd_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) char smem[DkdvLds<D>::bytes];
  dkdv_tile<D, false, HPI>(p, blockIdx.x, smem);
}

// The non-deterministic backward pass: key tiles only, each also adding its
// share of dQ into p.dq (zeroed beforehand) with atomics.
template <int D, int HPI>
__global__ __launch_bounds__(256, 2) void attn_bwd_atomic_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) char smem[DkdvLds<D, true>::bytes];
  dkdv_tile<D, true, HPI>(p, blockIdx.x, smem);
}

// The whole backward pass in one launch: the first n_dkdv workgroups take
// key tiles (dK/dV), the others query tiles (dQ); the dQ workgroups start
// as dK/dV ones finish, so neither pass leaves a tail of its own.
template <int D, int HPW, int HPI>
__global__ __launch_bounds__(256, 2) void attn_bwd_grid_kernel(BwdParams bp, DqParams dp, int n_dkdv) {
  constexpr uint32_t kBytes = DkdvLds<D>::bytes > DqLds<D>::bytes ? DkdvLds<D>::bytes : DqLds<D>::bytes;
  __shared__ __attribute__((aligned(16))) char smem[kBytes];
  const int b = blockIdx.x;
  if (b < n_dkdv)
    dkdv_tile<D, false, HPI>(bp, b, smem);
  else
    dq_tile<D, HPW>(dp, b - n_dkdv, smem);
}

// (HPW, the dQ workgroups' heads per tile, divides the group as HPI does,
// so HPW <= HPI)
template <int D>
static hipError_t launch_grid_d(const BwdParams& bp, const DqParams& dp, int hpw, hipStream_t s) {
  const int n_dkdv = bp.n_items * bp.hkv;
  const dim3 grid(unsigned(n_dkdv + dp.n_items * dp.hkv * dp.head_chunks)), block(256);
  const int hpi = heads_per_iteration(bp.group);
#define FC_GRID(W, I) hipLaunchKernelGGL((attn_bwd_grid_kernel<D, W, I>), grid, block, 0, s, bp, dp, n_dkdv)
  if (hpi == 4 && hpw == 4) FC_GRID(4, 4);
  else if (hpi == 4 && hpw == 2) FC_GRID(2, 4);
  else if (hpi == 4 && hpw == 1) FC_GRID(1, 4);
  else if (hpi == 2 && hpw == 2) FC_GRID(2, 2);
  else if (hpi == 2 && hpw == 1) FC_GRID(1, 2);
  else if (hpi == 1 && hpw == 1) FC_GRID(1, 1);
  else return hipErrorInvalidValue;
#undef FC_GRID
  return hipGetLastError();
}

hipError_t launch_bwd_grid(const BwdParams& bp, const DqParams& dp, int d, int heads_per_tile,
                           hipStream_t s) {
  if (bp.n_items == 0 && dp.n_items == 0) return hipSuccess;
  if (d == 64) return launch_grid_d<64>(bp, dp, heads_per_tile, s);
  if (d == 128) return launch_grid_d<128>(bp, dp, heads_per_tile, s);
  return hipErrorInvalidValue;
}

// the key-tile kernels (dK/dV alone, or with atomic dQ) for head dim D and
// the group's heads per iteration
template <template <int, int> class K, int D>
static hipError_t launch_keys_d(const BwdParams& p, hipStream_t s) {
  const dim3 grid(unsigned(p.n_items) * p.hkv), block(256);
  switch (heads_per_iteration(p.group)) {
    case 4: hipLaunchKernelGGL((K<D, 4>::fn), grid, block, 0, s, p); break;
    case 2: hipLaunchKernelGGL((K<D, 2>::fn), grid, block, 0, s, p); break;
    default: hipLaunchKernelGGL((K<D, 1>::fn), grid, block, 0, s, p); break;
  }
  return hipGetLastError();
}
template <int D, int HPI>
struct DkdvKernel {
  static constexpr auto fn = attn_bwd_kernel<D, HPI>;
};
template <int D, int HPI>
struct AtomicKernel {
  static constexpr auto fn = attn_bwd_atomic_kernel<D, HPI>;
};

hipError_t launch_bwd_atomic(const BwdParams& p, int d, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  if (d == 64) return launch_keys_d<AtomicKernel, 64>(p, s);
  if (d == 128) return launch_keys_d<AtomicKernel, 128>(p, s);
  return hipErrorInvalidValue;
}

hipError_t launch_bwd(const BwdParams& p, int d, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  if (d == 64) return launch_keys_d<DkdvKernel, 64>(p, s);
  if (d == 128) return launch_keys_d<DkdvKernel, 128>(p, s);
  return hipErrorInvalidValue;
}

}  // namespace fck
