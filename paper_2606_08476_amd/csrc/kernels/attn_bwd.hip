// Backward attention, dK/dV part (gfx950), key-major.
//
// One workgroup (4 waves) owns a tile of 128 keys of one source (local or
// received) and one KV head; wave w owns keys 32w..32w+31, so dK and dV for
// the tile accumulate in registers, summed over every query head of the
// group (grouped-query attention) and every query tile that sees the keys.
// K sits in LDS, V in registers. The (query head, 32-query tile) iterations
// are software-pipelined: the next tile's Q and dO are copied from HBM
// straight into a second LDS buffer (asynchronous loads) while the current
// one is computed. Per iteration:
//   S  = Q K^T, dP = dO V^T     MFMA (Q, dO, K from LDS, V from registers);
//   P  = exp(S - LSE), dS = P (dP - D)   D = rowsum(dO * O) from the
//                               preprocess kernel, LSE the merged forward LSE;
//   dV += P^T dO, dK += dS^T Q  P and dS from registers, dO/Q read from LDS
//                               with transpose reads.
// Masking (edge tiles only): local keys are causal in local order; a
// received key is seen by a query iff its index is below the query's
// receive limit.
#include "common.hpp"
#include "launch.hpp"

namespace fck {

template <int D>
__global__ __launch_bounds__(256, 2) void attn_bwd_kernel(BwdParams p) {
  constexpr int BN = 128;       // keys per workgroup
  constexpr int BM = 32;        // queries per iteration
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  __shared__ __attribute__((aligned(16))) u16 sK[BN * D];
  __shared__ __attribute__((aligned(16))) u16 sQ[2][BM * D];
  __shared__ __attribute__((aligned(16))) u16 sO[2][BM * D];  // dO tiles
  __shared__ __attribute__((aligned(16))) float sLD[2][2 * BM];  // LSE, then delta
  __shared__ __attribute__((aligned(16))) int sLim[2][2 * BM];   // receive limits (first BM)

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5;
  const int b = blockIdx.x;
  const int kvh = b % p.hkv;
  const int32_t* it = p.items + 8 * p.perm[b / p.hkv];  // launch list
  const int k0 = it[0], k1 = it[1], q0 = it[2], q1 = it[3], qfull = it[4], src = it[5];
  const u16* Kg = src ? p.k_recv : p.k_loc;
  const u16* Vg = src ? p.v_recv : p.v_loc;
  float* dKg = src ? p.dk_recv : p.dk_loc;
  float* dVg = src ? p.dv_recv : p.dv_loc;
  const size_t kvs = size_t(p.hkv) * D, kvo = size_t(kvh) * D;

  // key tile (rows past k1 repeat the last key; they are masked)
  TileLoader<D, BN>(p.hkv * D).load(sK, Kg + size_t(k0) * kvs + kvo, k1 - k0);
  const int krow = 32 * wave + (lane & 31);  // this lane's key within the tile
  const int kidx = k0 + krow;
  const bool kvalid = kidx < k1;
  // V rows of this lane's key as the B operand of dP = dO V^T
  bf16x8 vreg[KS];
  {
    const u16* vp = Vg + size_t(kidx) * kvs + kvo + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      vreg[ks] = kvalid ? *reinterpret_cast<const bf16x8*>(vp + 16 * ks) : zero8();
  }

  const int ntile = (q1 - q0 + BM - 1) / BM;
  const int n_it = ntile * p.group;

  // next iteration: Q/dO tiles, LSE, D and receive limits, all copied from
  // HBM straight into LDS (rows past q1 repeat the last query; masked)
  const TileLoader<D, BM> ldq(p.hq * D);
  auto fetch = [&](int i_, int buf) {
    const int h = kvh * p.group + i_ / ntile;
    const int t0 = q0 + (i_ % ntile) * BM;
    const size_t base = (size_t(t0) * p.hq + h) * D;
    ldq.load(sQ[buf], p.q + base, q1 - t0);
    ldq.load(sO[buf], p.dout + base, q1 - t0);
    const int qi = min(t0 + (lane & 31), q1 - 1);
    if (wave == 0)
      lds_copy4((half ? p.delta : p.lse) + (size_t)h * p.t_q + qi, sLD[buf]);
    else if (wave == 1 && src)
      lds_copy4(p.lim + qi, sLim[buf]);
  };

  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dk[db] = zero16();
    dv[db] = zero16();
  }
  const bool kfull = k1 - k0 == BN;
  const float sl2 = p.scale * kLog2e;
  const int qb = row_base<D>(0, lane), kb = row_base<D>(32 * wave, lane), trb = tr_base<D>(lane);

  if (n_it > 0) fetch(0, 0);
  wait_async();
  __syncthreads();

  for (int i_ = 0; i_ < n_it; ++i_) {
    const int buf = i_ & 1;
    const int t0 = q0 + (i_ % ntile) * BM;
    if (i_ + 1 < n_it) fetch(i_ + 1, buf ^ 1);
    const u16* Q = sQ[buf];
    const u16* O = sO[buf];

    f32x16 sacc = zero16(), dpacc = zero16();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sacc = mfma32(tread8_ks<D>(Q, qb, ks), tread8_ks<D>(sK, kb, ks), sacc);
      dpacc = mfma32(tread8_ks<D>(O, qb, ks), vreg[ks], dpacc);
    }
    // this lane's 16 query rows are 8g + 4*half + 0..3, g = 0..3
    const bool diag = t0 < qfull;
    const bool edge = diag || !kfull || t0 + BM > q1;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sLD[buf][8 * g + 4 * half]);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sLD[buf][BM + 8 * g + 4 * half]);
      int4 m4 = {0, 0, 0, 0};
      if (diag && src) m4 = *reinterpret_cast<const int4*>(&sLim[buf][8 * g + 4 * half]);
      const int lim[4] = {m4.x, m4.y, m4.z, m4.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = 4 * g + j;
        float pij = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[i], sl2, -l4[j] * kLog2e));
        if (edge) {
          const int qi = t0 + 8 * g + 4 * half + j;
          bool vis = kvalid && qi < q1;
          if (diag) vis = vis && (src ? kidx < lim[j] : kidx <= qi);
          pij = vis ? pij : 0.f;
        }
        sacc[i] = pij;
        dpacc[i] = pij * (dpacc[i] - d4[j]);
      }
    }
    // dV += P^T dO and dK += dS^T Q (scale applied at the end)
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
      const bf16x8 pa = pack8(sacc, 8 * kh);
      const bf16x8 sa = pack8(dpacc, 8 * kh);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        dv[db] = mfma32(pa, tread_tr2<D>(O, trb, 16 * kh, db), dv[db]);
        dk[db] = mfma32(sa, tread_tr2<D>(Q, trb, 16 * kh, db), dk[db]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // keep this tile's MFMAs ahead of the wait
    wait_async();
    __syncthreads();
  }

  // dK/dV of this tile, or of this part of a split tile (partial slot)
  const int slot = it[7];
  float* outK = dKg;
  float* outV = dVg;
  size_t rs = size_t(p.hkv) * D, base = size_t(kvh) * D;
  int r0 = k0;
  if (slot >= 0) {
    outK = p.part_k;
    outV = p.part_v;
    rs = D;
    base = (size_t(slot) * p.hkv + kvh) * BN * D;
    r0 = 0;
  }
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = 32 * wave + 8 * (i >> 2) + 4 * half + (i & 3);
      if (k0 + r < k1) {
        const size_t g = base + size_t(r0 + r) * rs + 32 * db + (lane & 31);
        outK[g] = p.scale * dk[db][i];
        outV[g] = dv[db][i];
      }
    }
  }
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
