#pragma once
// Backward attention, dQ part (gfx950), query-major.
//
// Same work items and schedule as the fused forward: one workgroup takes a
// tile of query tokens of one piece for `heads_per_tile` query heads of one
// KV head, and walks the received key range (no mask) and then the local key
// range (intra-document causal). Key/value tiles of 64 keys are
// double-buffered in LDS (asynchronous HBM-to-LDS copies) and shared by the
// waves, i.e. by the heads of the group. Per tile, with a query per lane:
//   S^T = K Q^T, dP^T = V dO^T      Q and dO held in registers;
//   P = exp(S - LSE), dS = P (dP - D)  LSE and D are per-lane scalars;
//   dQ^T += K^T dS^T                 K^T read from LDS with transpose reads.
// dQ is produced whole by the workgroup that owns the query rows, so it is
// written once, without atomics, and is deterministic. Recomputing S and dP
// here costs two extra products per key tile compared with accumulating dQ
// inside the key-major kernel, but removes that kernel's dQ traffic and
// frees the registers and LDS that limit its occupancy.
#include "common.hpp"
#include "launch.hpp"

#include <type_traits>

namespace fck {

template <int D>
struct DqLds {
  static constexpr uint32_t bytes = 4 * 64 * D * 2;
};

// One workgroup's query tile (workgroup index b); smem: DqLds<D>::bytes of
// shared memory.
template <int D, int HPW>
__device__ __forceinline__ void dq_tile(const DqParams& p, int b, char* smem) {
  constexpr int BN = 64;
  constexpr int RPW = 32 / HPW;  // query rows per wave and head
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr uint32_t TILE = BN * D * 2;  // bytes of one K or V tile
  // LDS: K0 | V0 | K1 | V1 (double buffer); the loop is unrolled by two so
  // every read names its buffer with a compile-time offset
  static_assert(4 * TILE == DqLds<D>::bytes, "LDS layout");

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5;
  const int kvh = b % p.hkv;
  const int rest = b / p.hkv;
  const int hc = rest % p.head_chunks;
  const int32_t* it = p.items + 8 * (rest / p.head_chunks);
  const int q0 = it[0], q1 = it[1], r0 = it[2], r1 = it[3], l0 = it[4], l1 = it[5];
  const int ldiag = it[6];

  // lane -> (query row, head) as in the forward: RPW rows of each of the
  // HPW heads per wave; a wave with no row skips the products
  const int l31 = lane & 31;
  const int h = kvh * p.group + hc * HPW + l31 / RPW;
  const int qrow = q0 + wave * RPW + l31 % RPW;
  const bool qvalid = qrow < q1;
  const bool active = q0 + wave * RPW < q1;  // wave-uniform
  const float sl2 = p.scale * kLog2e;

  const int n_r = (r1 - r0 + BN - 1) / BN;
  const int n_t = n_r + (l1 - l0 + BN - 1) / BN;

  const TileLoader<D, BN> ld(p.hkv * D);
  auto fetch = [&](int j, uint32_t kofs) {
    const bool rs = j < n_r;
    const int k0 = rs ? r0 + j * BN : l0 + (j - n_r) * BN;
    const int hi = rs ? r1 : l1;
    const size_t base = (size_t(k0) * p.hkv + kvh) * D;
    ld.load_at(lds_addr(smem) + kofs, (rs ? p.k_recv : p.k_loc) + base, hi - k0);
    ld.load_at(lds_addr(smem) + kofs + TILE, (rs ? p.v_recv : p.v_loc) + base, hi - k0);
  };

  // the workgroup's Q and dO rows through LDS first (Q over the second K/V
  // buffer, dO over the first), then key tile 0
  const int h0 = kvh * p.group + hc * HPW;
  load_pairs<D, RPW>(lds_addr(smem) + 2 * TILE, p.q, q0, q1, p.hq, h0);
  load_pairs<D, RPW>(lds_addr(smem), p.dout, q0, q1, p.hq, h0);

  bf16x8 qreg[KS], oreg[KS];
  float lse2 = 0.f, del = 0.f;
  if (qvalid) {
    lse2 = p.lse[(size_t)h * p.t_q + qrow] * kLog2e;
    del = p.delta[(size_t)h * p.t_q + qrow];
  }

  // per-lane LDS byte offsets: K/V rows for k-step ks, and the two transpose
  // reads of K^T block db
  uint32_t pr[KS], pt[DB][2];
  {
    const int rb = row_base<D>(0, lane), tb = tr_base<D>(lane);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) pr[ks] = 2u * uint32_t(rb ^ (ks << 4));
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      pt[db][0] = 2u * uint32_t(tb ^ (db << 5));
      pt[db][1] = 2u * uint32_t((tb ^ ((db << 5) | 16)) + 8 * D);
    }
  }

  f32x16 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dq[db] = zero16();
  wait_async();
  __syncthreads();
  if (active) {
    const int qb = row_base<D>(32 * wave, lane);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qreg[ks] = lds_b128(smem, 2u * uint32_t(qb ^ (ks << 4)), 2 * TILE);
      oreg[ks] = lds_b128(smem, 2u * uint32_t(qb ^ (ks << 4)), 0);
    }
  }
  __syncthreads();  // every wave holds its rows before tile 0 overwrites them
  if (n_t > 0) fetch(0, 0);
  wait_async();
  __syncthreads();

  // One key tile. Its MFMAs run as one software pipeline of slots:
  //   S^T, keys 0-31; S^T, keys 32-63 (with P of keys 0-31); dP^T, keys 0-31
  //   (with P of keys 32-63); dP^T, keys 32-63 (with dS of keys 0-31);
  //   dQ^T += K^T dS^T over keys 0-31 (with dS of keys 32-63), then 32-63.
  // Each slot issues the LDS reads of the slot two ahead, its MFMA and its
  // share of the vector work, which runs while the MFMA does; a scheduling
  // barrier after each slot keeps this order.
  constexpr int NS = 4 * KS + 4 * DB;        // slots per tile
  constexpr int EP = 16 / KS, EQ = 8 / DB;   // elements per slot (P, dS)
  auto step = [&](int j, auto buf) {
    constexpr uint32_t KO = decltype(buf)::value * 2 * TILE, VO = KO + TILE;
    if (j + 1 < n_t) fetch(j + 1, 2 * TILE - KO);
    const bool rs = j < n_r;
    const int k0 = rs ? r0 + j * BN : l0 + (j - n_r) * BN;
    const int hi = rs ? r1 : l1;
    if (active) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) pr[ks] = opaque(pr[ks]);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        pt[db][0] = opaque(pt[db][0]);
        pt[db][1] = opaque(pt[db][1]);
      }
      // key k0 + 4*half + c (c = 32*mb + 8*(i/4) + i%4 for register i) is seen
      // iff c < rel: keys past the range, and later keys on diagonal tiles,
      // give P = 0. Only edge tiles (diagonal, or running past the range)
      // mask, in one branch before each half's dS.
      const bool diag = !rs && k0 >= ldiag;
      const int rel = (diag ? min(hi, qrow + 1) : hi) - k0 - 4 * half;
      const bool edge = diag || k0 + BN > hi;

      f32x16 s[2] = {zero16(), zero16()}, dp[2] = {zero16(), zero16()};
      bf16x8 ring[3], sb[4];
      auto rd = [&](int n) {
        bf16x8& a = ring[n % 3];
        if (n < 4 * KS) {  // K rows (S) or V rows (dP)
          const int ks = n % KS, mb = (n / KS) & 1;
          a = lds_b128(smem, pr[ks], (n < 2 * KS ? KO : VO) + mb * 64 * D);
        } else {  // K^T for dQ
          const int u = n - 4 * KS, kk = u / DB, db = u % DB;
          const uint32_t ro = KO + kk * 32 * D;
          a = cat8(lds_tr(smem, pt[db][0], ro), lds_tr(smem, pt[db][1], ro));
        }
      };
      auto pexp = [&](int mb, int i) {
        s[mb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mb][i], sl2, -lse2));
      };
      auto mask = [&](int mb) {
        if (edge) {
#pragma unroll
          for (int i = 0; i < 16; ++i)
            s[mb][i] = 32 * mb + 8 * (i >> 2) + (i & 3) < rel ? s[mb][i] : 0.f;
        }
      };
      auto dsv = [&](int mb, int i) { dp[mb][i] = s[mb][i] * (dp[mb][i] - del); };
      rd(0);
      rd(1);
      static_for<0, NS>([&](auto nc) {
        constexpr int n = decltype(nc)::value;
        if (n + 2 < NS) rd(n + 2);
        const bf16x8& a = ring[n % 3];
        if (n < 2 * KS) {
          const int ks = n % KS, mb = n / KS;
          s[mb] = mfma32(a, qreg[ks], s[mb]);
          if (mb == 1)
#pragma unroll
            for (int e = ks * EP; e < (ks + 1) * EP; ++e) pexp(0, e);
        } else if (n < 4 * KS) {
          const int ks = n % KS, mb = (n - 2 * KS) / KS;
          dp[mb] = mfma32(a, oreg[ks], dp[mb]);
          if (mb == 1 && ks == 0) mask(0);
          if (mb == 0) {
#pragma unroll
            for (int e = ks * EP; e < (ks + 1) * EP; ++e) pexp(1, e);
          } else {
#pragma unroll
            for (int e = ks * EP; e < (ks + 1) * EP; ++e) dsv(0, e);
            if ((ks + 1) * EP == 8) sb[0] = pack8(dp[0], 0);
            if ((ks + 1) * EP == 16) sb[1] = pack8(dp[0], 8);
          }
        } else {
          const int u = n - 4 * KS, kk = u / DB, db = u % DB;
          dq[db] = mfma32(a, sb[kk], dq[db]);
          if (u == 0) mask(1);
          if (u < 2 * DB) {
#pragma unroll
            for (int e = u * EQ; e < (u + 1) * EQ; ++e) dsv(1, e);
            if ((u + 1) * EQ == 8) sb[2] = pack8(dp[1], 0);
            if ((u + 1) * EQ == 16) sb[3] = pack8(dp[1], 8);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    wait_async();
    __syncthreads();
  };
  for (int j = 0; j < n_t; j += 2) {
    step(j, std::integral_constant<int, 0>());
    if (j + 1 < n_t) step(j + 1, std::integral_constant<int, 1>());
  }

  // dQ rows out through this wave's share of the (now free) K/V buffers,
  // 1 KiB per store instruction
  store_rows<D, RPW>(
      smem + size_t(wave) * (32 * D * 4), active,
      [&](int db, int g) {
        f32x4 v;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) v[jj] = p.scale * dq[db][4 * g + jj];
        return v;
      },
      q0 + wave * RPW, q1, p.hq, kvh * p.group + hc * HPW, p.dq, nullptr);
}

}  // namespace fck
