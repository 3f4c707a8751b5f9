// Bandwidth-bound kernels: the KV gather (simulated receive), the
// log-sum-exp merge of two partial passes, the backward preprocess (which
// can zero the atomic backward's dQ in the same pass), and a zero fill.
// Each moves whole rows with 16-byte accesses, consecutive lanes on
// consecutive addresses.
#include "common.hpp"
#include "launch.hpp"

namespace fck {

// Row copies: output row i of K/V local (i < t_q) or received (i >= t_q)
// comes from packed row q_gpos[i] or recv_gpos[i - t_q]; rows r0 .. r1-1
// of that concatenation are copied.
__global__ __launch_bounds__(256) void kv_gather_kernel(const uint4* __restrict__ k,
                                                        const uint4* __restrict__ v,
                                                        const int32_t* __restrict__ q_gpos,
                                                        const int32_t* __restrict__ recv_gpos,
                                                        int32_t t_q, int64_t r0, int64_t r1,
                                                        int32_t chunks, uint4* k_loc, uint4* v_loc,
                                                        uint4* k_recv, uint4* v_recv) {
  const int64_t total = (r1 - r0) * chunks;
  for (int64_t c = int64_t(blockIdx.x) * 256 + threadIdx.x; c < total;
       c += int64_t(gridDim.x) * 256) {
    const int32_t row = int32_t(r0 + c / chunks), cc = int32_t(c % chunks);
    const bool loc = row < t_q;
    const int64_t src = int64_t(loc ? q_gpos[row] : recv_gpos[row - t_q]) * chunks + cc;
    const int64_t dst = int64_t(loc ? row : row - t_q) * chunks + cc;
    const uint4 kk = k[src], vv = v[src];
    (loc ? k_loc : k_recv)[dst] = kk;
    (loc ? v_loc : v_recv)[dst] = vv;
  }
}

// One (token, head) row per LPR lanes; each lane handles 4 values.
template <int D>
__global__ __launch_bounds__(256) void lse_merge_kernel(const float* __restrict__ oa,
                                                        const float* __restrict__ la,
                                                        const float* __restrict__ ob,
                                                        const float* __restrict__ lb, int32_t t,
                                                        int32_t h, u16* o, float* of,
                                                        float* lse_out) {
  constexpr int LPR = D / 4;
  const int64_t row = (int64_t(blockIdx.x) * 256 + threadIdx.x) / LPR;
  const int c = threadIdx.x % LPR;
  if (row >= int64_t(t) * h) return;
  const int32_t tok = int32_t(row / h), head = int32_t(row % h);
  const int64_t li = int64_t(head) * t + tok;
  const Merge2 w = merge2(la[li], lb[li]);
  const f32x4 x = reinterpret_cast<const f32x4*>(oa + row * D)[c];
  const f32x4 y = reinterpret_cast<const f32x4*>(ob + row * D)[c];
  f32x4 r;
#pragma unroll
  for (int j = 0; j < 4; ++j) r[j] = merge2_value(w, x[j], y[j]);
  uint2 pk;
  pk.x = uint32_t(f2bf(r[0])) | (uint32_t(f2bf(r[1])) << 16);
  pk.y = uint32_t(f2bf(r[2])) | (uint32_t(f2bf(r[3])) << 16);
  reinterpret_cast<uint2*>(o + row * D)[c] = pk;
  if (of) reinterpret_cast<f32x4*>(of + row * D)[c] = r;
  if (c == 0) lse_out[li] = w.lse;
}

// delta[head, tok] = sum_d dO * O over one (token, head) row, from the bf16
// O or (OF32) the fp32 O; with dq_zero, the same row of that fp32 tensor is
// zeroed too.
template <int D, bool OF32>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const void* __restrict__ o_,
                                                      const u16* __restrict__ dout,
                                                      float* delta, int32_t t, int32_t h,
                                                      float* dq_zero) {
  constexpr int LPR = D / 8;  // lanes per row, 8 values each
  const int64_t row = (int64_t(blockIdx.x) * 256 + threadIdx.x) / LPR;
  const int c = threadIdx.x % LPR;
  const bool ok = row < int64_t(t) * h;
  float acc = 0.f;
  if (ok && dq_zero) {
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    reinterpret_cast<f32x4*>(dq_zero + row * D)[2 * c] = z;
    reinterpret_cast<f32x4*>(dq_zero + row * D)[2 * c + 1] = z;
  }
  if (ok) {
    const uint4 g = reinterpret_cast<const uint4*>(dout + row * D)[c];
    const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
    if constexpr (OF32) {
      const f32x4* op = reinterpret_cast<const f32x4*>(static_cast<const float*>(o_) + row * D);
      const f32x4 a0 = op[2 * c], a1 = op[2 * c + 1];
      const float av[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc += av[2 * j] * bf2f(u16(gw[j] & 0xffff));
        acc += av[2 * j + 1] * bf2f(u16(gw[j] >> 16));
      }
    } else {
      const uint4 a = reinterpret_cast<const uint4*>(static_cast<const u16*>(o_) + row * D)[c];
      const uint32_t aw[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc += bf2f(u16(aw[j] & 0xffff)) * bf2f(u16(gw[j] & 0xffff));
        acc += bf2f(u16(aw[j] >> 16)) * bf2f(u16(gw[j] >> 16));
      }
    }
  }
#pragma unroll
  for (int w = LPR / 2; w >= 1; w >>= 1) acc += __shfl_xor(acc, w);
  if (ok && c == 0) {
    const int32_t tok = int32_t(row / h), head = int32_t(row % h);
    delta[int64_t(head) * t + tok] = acc;
  }
}

// Sum of the partial dK/dV of a split key tile, in slot order. One
// workgroup per (split tile, KV head, 16 of the tile's 128 keys), so that a
// few split tiles still fill the chip; entries are (src, k0, k1, first slot,
// slot count, 0, 0, 0); partial slots hold 128 rows of d values per KV head.
template <int D>
__global__ __launch_bounds__(256) void bwd_reduce_kernel(const int32_t* __restrict__ entries,
                                                         const float* __restrict__ pk,
                                                         const float* __restrict__ pv, int32_t hkv,
                                                         float* dk_loc, float* dv_loc,
                                                         float* dk_recv, float* dv_recv) {
  constexpr int BN = 128, C4 = D / 4, ROWS = 16;  // rows of the key tile per workgroup
  constexpr int PER = ROWS * C4 / 256;            // 16-byte chunks per thread
  const int rb = blockIdx.x % (BN / ROWS);
  const int kvh = (blockIdx.x / (BN / ROWS)) % hkv;
  const int32_t* e = entries + 8 * (blockIdx.x / (BN / ROWS) / hkv);
  const int src = e[0], k0 = e[1], k1 = e[2], s0 = e[3], ns = e[4];
  float* dk = src ? dk_recv : dk_loc;
  float* dv = src ? dv_recv : dv_loc;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int idx = u * 256 + int(threadIdx.x);
    const int r = rb * ROWS + idx / C4, c = idx % C4;
    if (k0 + r >= k1) continue;
    // the slots in their fixed order, two loads of each in flight at once
    f32x4 ak = {0.f, 0.f, 0.f, 0.f}, av = {0.f, 0.f, 0.f, 0.f};
    auto at = [&](int s) { return ((size_t(s0 + s) * hkv + kvh) * BN + r) * D; };
    int s = 0;
    for (; s + 1 < ns; s += 2) {
      const f32x4 x0 = reinterpret_cast<const f32x4*>(pk + at(s))[c];
      const f32x4 y0 = reinterpret_cast<const f32x4*>(pv + at(s))[c];
      const f32x4 x1 = reinterpret_cast<const f32x4*>(pk + at(s + 1))[c];
      const f32x4 y1 = reinterpret_cast<const f32x4*>(pv + at(s + 1))[c];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ak[j] += x0[j];
        ak[j] += x1[j];
        av[j] += y0[j];
        av[j] += y1[j];
      }
    }
    if (s < ns) {
      const f32x4 x = reinterpret_cast<const f32x4*>(pk + at(s))[c];
      const f32x4 y = reinterpret_cast<const f32x4*>(pv + at(s))[c];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ak[j] += x[j];
        av[j] += y[j];
      }
    }
    const size_t g = (size_t(k0 + r) * hkv + kvh) * D;
    reinterpret_cast<f32x4*>(dk + g)[c] = ak;
    reinterpret_cast<f32x4*>(dv + g)[c] = av;
  }
}

// x[0 .. n) = 0 (n a multiple of 4; x 16-byte aligned)
__global__ __launch_bounds__(256) void fill_zero_kernel(f32x4* x, int64_t n4) {
  const f32x4 z = {0.f, 0.f, 0.f, 0.f};
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n4; i += int64_t(gridDim.x) * 256)
    x[i] = z;
}

static unsigned grid_for(int64_t threads) {
  const int64_t b = (threads + 255) / 256;
  return unsigned(b < 1 ? 1 : b);
}

hipError_t launch_kv_gather(const uint16_t* k, const uint16_t* v, const int32_t* q_gpos,
                            const int32_t* recv_gpos, int32_t t_q, int32_t t_r, int64_t r0,
                            int64_t r1, int32_t row_elems, uint16_t* k_loc, uint16_t* v_loc,
                            uint16_t* k_recv, uint16_t* v_recv, hipStream_t s) {
  const int32_t chunks = row_elems / 8;
  if (r0 < 0 || r1 > int64_t(t_q) + t_r || r0 > r1) return hipErrorInvalidValue;
  const int64_t total = (r1 - r0) * chunks;
  if (total == 0) return hipSuccess;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 256 * 64) blocks = 256 * 64;
  hipLaunchKernelGGL(kv_gather_kernel, dim3(unsigned(blocks)), dim3(256), 0, s,
                     reinterpret_cast<const uint4*>(k), reinterpret_cast<const uint4*>(v), q_gpos,
                     recv_gpos, t_q, r0, r1, chunks, reinterpret_cast<uint4*>(k_loc),
                     reinterpret_cast<uint4*>(v_loc), reinterpret_cast<uint4*>(k_recv),
                     reinterpret_cast<uint4*>(v_recv));
  return hipGetLastError();
}

hipError_t launch_lse_merge(const float* o_a, const float* lse_a, const float* o_b,
                            const float* lse_b, int32_t t, int32_t h, int32_t d, uint16_t* o_bf16,
                            float* o_f32, float* lse_out, hipStream_t s) {
  const int64_t rows = int64_t(t) * h;
  if (rows == 0) return hipSuccess;
  if (d == 64)
    hipLaunchKernelGGL(lse_merge_kernel<64>, dim3(grid_for(rows * 16)), dim3(256), 0, s, o_a, lse_a,
                       o_b, lse_b, t, h, o_bf16, o_f32, lse_out);
  else if (d == 128)
    hipLaunchKernelGGL(lse_merge_kernel<128>, dim3(grid_for(rows * 32)), dim3(256), 0, s, o_a,
                       lse_a, o_b, lse_b, t, h, o_bf16, o_f32, lse_out);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_bwd_reduce(const int32_t* entries, int32_t n, const float* part_k,
                             const float* part_v, int32_t hkv, int32_t d, float* dk_loc,
                             float* dv_loc, float* dk_recv, float* dv_recv, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const dim3 grid(unsigned(n) * hkv * 8), block(256);  // 8 row blocks of 16 keys per tile
  if (d == 64)
    hipLaunchKernelGGL(bwd_reduce_kernel<64>, grid, block, 0, s, entries, part_k, part_v, hkv,
                       dk_loc, dv_loc, dk_recv, dv_recv);
  else if (d == 128)
    hipLaunchKernelGGL(bwd_reduce_kernel<128>, grid, block, 0, s, entries, part_k, part_v, hkv,
                       dk_loc, dv_loc, dk_recv, dv_recv);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int D>
static void launch_pre_d(const uint16_t* o, const float* o_f32, const uint16_t* dout,
                         float* delta, int32_t t, int32_t h, float* dq_zero, hipStream_t s) {
  const int64_t rows = int64_t(t) * h;
  const dim3 grid(grid_for(rows * (D / 8))), block(256);
  if (o_f32)
    hipLaunchKernelGGL((bwd_pre_kernel<D, true>), grid, block, 0, s, o_f32, dout, delta, t, h,
                       dq_zero);
  else
    hipLaunchKernelGGL((bwd_pre_kernel<D, false>), grid, block, 0, s, o, dout, delta, t, h,
                       dq_zero);
}

hipError_t launch_bwd_preprocess(const uint16_t* o, const float* o_f32, const uint16_t* dout,
                                 float* delta, int32_t t, int32_t h, int32_t d, float* dq_zero,
                                 hipStream_t s) {
  if (int64_t(t) * h == 0) return hipSuccess;
  if (d == 64)
    launch_pre_d<64>(o, o_f32, dout, delta, t, h, dq_zero, s);
  else if (d == 128)
    launch_pre_d<128>(o, o_f32, dout, delta, t, h, dq_zero, s);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* x, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (n % 4 || reinterpret_cast<uintptr_t>(x) % 16) return hipErrorInvalidValue;
  int64_t blocks = (n / 4 + 255) / 256;
  if (blocks > 256 * 32) blocks = 256 * 32;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(unsigned(blocks)), dim3(256), 0, s,
                     reinterpret_cast<f32x4*>(x), n / 4);
  return hipGetLastError();
}

}  // namespace fck
