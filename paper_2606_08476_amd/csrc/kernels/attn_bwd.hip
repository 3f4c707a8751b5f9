// Backward attention over one rank's share (gfx950), key-major.
//
// One workgroup (4 waves) owns a tile of 128 keys of one source (local or
// received) and one KV head; wave w owns keys 32w..32w+31, so dK and dV for
// the tile accumulate in registers, summed over every query head of the
// group (grouped-query attention) and every query tile that sees the keys.
// Per (query head, 32-query tile):
//   S  = Q K^T, dP = dO V^T     MFMA, both operands straight from LDS;
//   P  = exp(S - LSE), dS = P (dP - D)   D = rowsum(dO * O) from the
//                               preprocess kernel, LSE the merged forward LSE;
//   dV += P^T dO, dK += dS^T Q  P and dS from registers, dO/Q read from LDS
//                               with transpose reads;
//   dQ += dS K                  dS^T staged in LDS, dQ accumulated in fp32
//                               with atomics (several key tiles feed a row).
// Masking: local keys are causal in local order; a received key is seen by
// a query iff its index is below the query's receive limit.
#include "common.hpp"
#include "launch.hpp"

namespace fck {

template <int D>
__global__ __launch_bounds__(256) void attn_bwd_kernel(BwdParams p) {
  constexpr int BN = 128;       // keys per workgroup
  constexpr int BM = 32;        // queries per inner tile
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int LD = D + 8;
  constexpr int LDT = BM + 8;   // row stride of dS^T in LDS
  constexpr int CH = D / 8;
  constexpr int KSPLIT = 4 / DB;            // waves sharing one dQ column block
  constexpr int DQ_STEPS = (BN / 16) / KSPLIT;
  __shared__ __attribute__((aligned(16))) u16 sK[BN * LD];
  __shared__ __attribute__((aligned(16))) u16 sV[BN * LD];
  __shared__ __attribute__((aligned(16))) u16 sQ[BM * LD];
  __shared__ __attribute__((aligned(16))) u16 sO[BM * LD];   // dO tile
  __shared__ __attribute__((aligned(16))) u16 sS[BN * LDT];  // dS^T tile
  __shared__ float sLse[BM], sDel[BM];
  __shared__ int sLim[BM];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5;
  const int b = blockIdx.x;
  const int kvh = b % p.hkv;
  const int32_t* it = p.items + 8 * p.perm[b / p.hkv];
  const int k0 = it[0], k1 = it[1], q0 = it[2], q1 = it[3], qfull = it[4], src = it[5];
  const u16* Kg = src ? p.k_recv : p.k_loc;
  const u16* Vg = src ? p.v_recv : p.v_loc;
  float* dKg = src ? p.dk_recv : p.dk_loc;
  float* dVg = src ? p.dv_recv : p.dv_loc;

  for (int c = threadIdx.x; c < BN * CH; c += 256) {
    const int r = c / CH, cc = c % CH;
    bf16x8 kv = zero8(), vv = zero8();
    if (k0 + r < k1) {
      const size_t g = ((size_t)(k0 + r) * p.hkv + kvh) * D + cc * 8;
      kv = *reinterpret_cast<const bf16x8*>(Kg + g);
      vv = *reinterpret_cast<const bf16x8*>(Vg + g);
    }
    *reinterpret_cast<bf16x8*>(sK + r * LD + cc * 8) = kv;
    *reinterpret_cast<bf16x8*>(sV + r * LD + cc * 8) = vv;
  }

  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dk[db] = zero16();
    dv[db] = zero16();
  }
  const int krow = 32 * wave + (lane & 31);  // this lane's key within the tile
  const int kidx = k0 + krow;
  const bool kvalid = kidx < k1;
  const float sl2 = p.scale * kLog2e;
  const int nb = wave % DB, part = wave / DB;

  for (int hh = 0; hh < p.group; ++hh) {
    const int h = kvh * p.group + hh;
    for (int t0 = q0; t0 < q1; t0 += BM) {
      __syncthreads();  // LDS of the previous tile is consumed
      for (int c = threadIdx.x; c < BM * CH; c += 256) {
        const int r = c / CH, cc = c % CH;
        bf16x8 qv = zero8(), ov = zero8();
        if (t0 + r < q1) {
          const size_t g = ((size_t)(t0 + r) * p.hq + h) * D + cc * 8;
          qv = *reinterpret_cast<const bf16x8*>(p.q + g);
          ov = *reinterpret_cast<const bf16x8*>(p.dout + g);
        }
        *reinterpret_cast<bf16x8*>(sQ + r * LD + cc * 8) = qv;
        *reinterpret_cast<bf16x8*>(sO + r * LD + cc * 8) = ov;
      }
      if (threadIdx.x < BM) {
        const int qi = t0 + threadIdx.x;
        const bool ok = qi < q1;
        sLse[threadIdx.x] = ok ? p.lse[(size_t)h * p.t_q + qi] * kLog2e : 0.f;
        sDel[threadIdx.x] = ok ? p.delta[(size_t)h * p.t_q + qi] : 0.f;
        sLim[threadIdx.x] = ok ? p.lim[qi] : 0;
      }
      __syncthreads();

      f32x16 sacc = zero16(), dpacc = zero16();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int eq = (lane & 31) * LD + 16 * ks + 8 * half;
        const int ek = krow * LD + 16 * ks + 8 * half;
        sacc = mfma32(lds_read8(sQ, eq), lds_read8(sK, ek), sacc);
        dpacc = mfma32(lds_read8(sO, eq), lds_read8(sV, ek), dpacc);
      }
      const bool diag = t0 < qfull;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int qr = 8 * (i >> 2) + 4 * half + (i & 3);
        const int qi = t0 + qr;
        bool vis = kvalid && qi < q1;
        if (diag) vis = vis && (src ? kidx < sLim[qr] : kidx <= qi);
        const float pij = vis ? exp2f(sacc[i] * sl2 - sLse[qr]) : 0.f;
        sacc[i] = pij;
        dpacc[i] = pij * (dpacc[i] - sDel[qr]);
      }
      // dV += P^T dO and dK += dS^T Q (scale applied at the end)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {
        const bf16x8 pa = pack8(sacc, 8 * kh);
        const bf16x8 sa = pack8(dpacc, 8 * kh);
        const int rb = 16 * kh + 4 * half;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dv[db] = mfma32(pa, lds_operand_tr(sO, LD, rb, rb + 8, 32 * db, lane), dv[db]);
          dk[db] = mfma32(sa, lds_operand_tr(sQ, LD, rb, rb + 8, 32 * db, lane), dk[db]);
        }
      }
      // dS^T -> LDS: this lane's key row, queries 8g + 4*half + 0..3
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 w;
        w.x = uint32_t(f2bf(dpacc[4 * g])) | (uint32_t(f2bf(dpacc[4 * g + 1])) << 16);
        w.y = uint32_t(f2bf(dpacc[4 * g + 2])) | (uint32_t(f2bf(dpacc[4 * g + 3])) << 16);
        *reinterpret_cast<uint2*>(sS + krow * LDT + 8 * g + 4 * half) = w;
      }
      __syncthreads();
      // dQ[:, 32nb .. 32nb+31] += dS K over this wave's share of the keys
      f32x16 dq = zero16();
#pragma unroll
      for (int s = 0; s < DQ_STEPS; ++s) {
        const int ks = part * DQ_STEPS + s;
        const int rb = 16 * ks + 8 * half;
        dq = mfma32(lds_operand_tr(sS, LDT, rb, rb + 4, 0, lane),
                    lds_operand_tr(sK, LD, rb, rb + 4, 32 * nb, lane), dq);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int qi = t0 + 8 * (i >> 2) + 4 * half + (i & 3);
        if (qi < q1)
          atomicAdd(p.dq + ((size_t)qi * p.hq + h) * D + 32 * nb + (lane & 31), p.scale * dq[i]);
      }
    }
  }

#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int kr = k0 + 32 * wave + 8 * (i >> 2) + 4 * half + (i & 3);
      if (kr < k1) {
        const size_t g = ((size_t)kr * p.hkv + kvh) * D + 32 * db + (lane & 31);
        dKg[g] = p.scale * dk[db][i];
        dVg[g] = dv[db][i];
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
