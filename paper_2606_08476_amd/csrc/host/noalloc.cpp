// fc_attn_bwd_noalloc: the backward of fc_attn_bwd with its workspace taken
// from a library-owned device array instead of a caller buffer, for callers
// that cannot allocate device memory. The kernels are fc_attn_bwd's; only
// where the workspace lives differs.
//
// The array is a file-scope __device__ variable: every GPU the library runs
// on holds its own copy, at its own address, from module load until the
// process ends. In host code its name is only a stand-in for the symbol, so
// its device address is looked up once per device (hipGetSymbolAddress, with
// that device current) and that address alone is handed to the kernels.
//
// What the workspace holds needs no clearing: the preprocess writes every
// delta the pass reads, and every split key tile's part writes the rows of
// its slot that the reduce reads. Calls on one GPU share the array, so
// calls whose work overlaps on that GPU (other streams, other threads) race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.hpp"
#include "view.hpp"

using fc::fail;

namespace {

constexpr size_t kScratchBytes = size_t(FC_NOALLOC_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

__device__ __attribute__((aligned(256))) char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (looked up on the first
// call made with the device current).
int scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess)
      return fail(FC_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    if (!p) return fail(FC_ERR_HIP, "hipGetSymbolAddress(scratch) returned a null address");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return FC_OK;
}

}  // namespace

extern "C" {

int fc_attn_bwd_noalloc(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                        const void* k_recv, const void* v_recv, const void* o,
                        const float* o_f32, const float* lse, const void* dout, float scale,
                        int32_t deterministic, float* dq,
                        float* dk_loc, float* dv_loc, float* dk_recv, float* dv_recv,
                        void* stream) {
  fc::clear_error();
  if (!view) return fail(FC_ERR_INVALID_ARG, "view is null");
  if (!reinterpret_cast<const fc::View*>(view)->dev_meta)
    return fail(FC_ERR_WORKSPACE, "view is not bound to device metadata");
  size_t need = 0;
  if (int rc = fc_workspace_size(view, FC_TWO_PASS, nullptr, &need, nullptr)) return rc;
  if (need > kScratchBytes)
    return fail(FC_ERR_WORKSPACE, "backward workspace of " + std::to_string(need) +
                                      " bytes exceeds the " + std::to_string(kScratchBytes) +
                                      "-byte static scratch of fc_attn_bwd_noalloc; use "
                                      "fc_attn_bwd with a caller workspace");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(FC_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(FC_ERR_UNSUPPORTED, "device index out of range");
  if (stream) {
    int sdev = 0;
    e = hipStreamGetDevice(reinterpret_cast<hipStream_t>(stream), &sdev);
    if (e != hipSuccess)
      return fail(FC_ERR_HIP, std::string("hipStreamGetDevice: ") + hipGetErrorString(e));
    if (sdev != dev)
      return fail(FC_ERR_INVALID_ARG, "stream belongs to device " + std::to_string(sdev) +
                                          ", the current device is " + std::to_string(dev));
  }
  void* ws = nullptr;
  if (int rc = scratch_address(dev, &ws)) return rc;
  return fc_attn_bwd(view, q, k_loc, v_loc, k_recv, v_recv, o, o_f32, lse, dout, scale,
                     deterministic,
                     dq, dk_loc, dv_loc, dk_recv, dv_recv, ws, kScratchBytes, stream);
}

}  // extern "C"
