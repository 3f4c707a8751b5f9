#pragma once
// Backward attention, dK/dV part (gfx950), key-major.
//
// One workgroup (4 waves) owns a tile of 128 keys of one source (local or
// received) and one KV head; wave w owns keys 32w..32w+31, so dK and dV for
// the tile accumulate in registers, summed over every query head of the
// group (grouped-query attention) and every query tile that sees the keys.
// K sits in LDS, V in registers. An iteration takes 32 (query row, query
// head) pairs: 32/HPI consecutive query rows of each of HPI heads of the
// group (HPI = 4 when the group allows it), so the last, short block of a
// query range pads to 32/HPI rows rather than 32. The iterations are
// software-pipelined: the next block's Q and dO are copied from HBM
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
//
// With DQ (the non-deterministic backward), the same workgroup also adds
// this key tile's share of dQ = scale dS K into dQ: each wave writes its dS
// block, transposed, into an LDS tile of all 128 keys (dS holds a key per
// lane here; the dQ product needs the keys along the contraction), and after
// a barrier wave w computes dQ for the query tile's 32 rows and head-dim
// columns 32w..32w+31 (MFMA, dS and K both read from LDS with transpose
// reads) and adds it into dQ with fp32 atomics. No second pass recomputes S
// and dP; the order of the additions into dQ, and so its last bits, varies
// from run to run.
#include "common.hpp"
#include "launch.hpp"

#include <type_traits>

namespace fck {

template <int D, bool DQ = false>
struct DkdvLds {
  // LSE/delta/limit slots, the key tile, two Q and two dO tiles; with DQ the
  // transposed dS tile (128 keys x 32 queries, bf16) after them
  static constexpr uint32_t bytes = 6 * 256 + (128 + 4 * 32) * D * 2 + (DQ ? 128 * 32 * 2 : 0);
};

// One workgroup's key tile (workgroup index b); smem: DkdvLds<D, DQ>::bytes
// of shared memory. HPI (1, 2 or 4) must divide the group size.
template <int D, bool DQ = false, int HPI = 1>
__device__ __forceinline__ void dkdv_tile(const BwdParams& p, int b, char* smem) {
  constexpr int BN = 128;       // keys per workgroup
  constexpr int BM = 32;        // (query row, head) pairs per iteration
  constexpr int RPI = BM / HPI; // query rows per iteration and head
  static_assert(HPI == 1 || HPI == 2 || HPI == 4, "heads per iteration");
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr uint32_t KT = BN * D * 2;  // bytes of the key tile
  constexpr uint32_t QT = BM * D * 2;  // bytes of a Q or dO tile
  // LDS layout (bytes): per buffer b, LSE at 256*3b, delta at +256, receive
  // limits at +512 (a wave-wide copy each, the first BM entries used); then
  // the key tile; then Q and dO of buffer 0 and of buffer 1. The loop is
  // unrolled by two, so every read names its buffer with a compile-time
  // offset (all below 64 KiB, the reach of the offset field).
  constexpr uint32_t OK = 6 * 256;
  constexpr uint32_t OQ0 = OK + KT, OO0 = OQ0 + QT, OQ1 = OO0 + QT, OO1 = OQ1 + QT;
  // dS^T tile (DQ only): row k (key) holds the tile's 32 queries, 64 bytes;
  // the 8-byte chunk c (queries 4c..4c+3) of row k sits at chunk position
  // c ^ ((k >> 2) & 7), so that the row writes of a wave (32 keys, one
  // chunk) and the transpose reads (4 keys x 16 queries per 16 lanes) both
  // spread over the 64 banks
  constexpr uint32_t ODS = OO1 + QT;
  static_assert(ODS + (DQ ? 128 * 32 * 2 : 0) == DkdvLds<D, DQ>::bytes, "LDS layout");

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5;
  const int kvh = b % p.hkv;
  const int item = b / p.hkv;  // the launch list is in launch order
  const int32_t* it = p.items + 8 * item;  // launch list
  const int k0 = it[0], k1 = it[1], q0 = it[2], q1 = it[3], qfull = it[4], src = it[5];
  const u16* Kg = src ? p.k_recv : p.k_loc;
  const u16* Vg = src ? p.v_recv : p.v_loc;
  float* dKg = src ? p.dk_recv : p.dk_loc;
  float* dVg = src ? p.dv_recv : p.dv_loc;
  const size_t kvs = size_t(p.hkv) * D, kvo = size_t(kvh) * D;

  // first query row that sees this wave's first key (host table: local rows
  // from the key's own index on, received rows once their receive limit
  // exceeds it)
  const int kw = k0 + 32 * wave;
  const int qfirst = p.qfirst[4 * item + wave];

  // key tile, and the same rows of V over the Q/dO buffers (read into
  // registers before the first Q/dO copy); rows past k1 repeat the last
  // key, whose P is masked to 0
  {
    const TileLoader<D, BN> ldk(p.hkv * D);
    ldk.load_at(lds_addr(smem) + OK, Kg + size_t(k0) * kvs + kvo, k1 - k0);
    ldk.load_at(lds_addr(smem) + OQ0, Vg + size_t(k0) * kvs + kvo, k1 - k0);
  }
  // V rows of this lane's key as the B operand of dP = dO V^T
  bf16x8 vreg[KS];

  const int ntile = (q1 - q0 + RPI - 1) / RPI;
  const int n_it = ntile * (p.group / HPI);

  // iteration i covers query heads kvh * group + HPI * (i / ntile) + 0 ..
  // HPI-1 and query rows q0 + RPI * (i % ntile) + 0 .. RPI-1; block and head
  // set are carried from one iteration to the next (no integer division
  // per iteration). Pair m (0..31) of an iteration is row m % RPI of head
  // m / RPI: the row order of the Q/dO tiles, of the LSE, delta and limit
  // slots and of the MFMA rows.
  int cur_t = 0, cur_h = 0;   // row block and head set of the current iteration
  int nxt_t = 0, nxt_h = 0;   // row block and head set of the next copy
  auto advance = [&]() {
    if (++nxt_t == ntile) {
      nxt_t = 0;
      ++nxt_h;
    }
  };

  // next iteration: Q/dO tiles, LSE, D and receive limits, all copied from
  // HBM straight into LDS (rows past q1 repeat the last query; masked)
  const TileLoader<D, BM, 256, RPI> ldq(p.hq * D, D);
  auto fetch = [&](int hh, int tt, int buf) {
    const int h = kvh * p.group + hh * HPI;
    const int t0 = q0 + tt * RPI;
    const size_t base = (size_t(t0) * p.hq + h) * D;
    const uint32_t sb = lds_addr(smem);
    ldq.load_at(sb + (buf ? OQ1 : OQ0), p.q + base, q1 - t0);
    ldq.load_at(sb + (buf ? OO1 : OO0), p.dout + base, q1 - t0);
    const int m = lane & 31;
    const uint32_t roff = 4u * uint32_t(min(t0 + m % RPI, q1 - 1));
    const uint32_t qoff = roff + 4u * uint32_t(m / RPI) * uint32_t(p.t_q);
    const uint32_t sm = sb + 768u * buf;
    if (wave == 0)
      lds_copy4(p.lse + (size_t)h * p.t_q, qoff, sm);
    else if (wave == 1)
      lds_copy4(p.delta + (size_t)h * p.t_q, qoff, sm + 256);
    else if (wave == 2 && src)
      lds_copy4(p.lim, roff, sm + 512);
  };

  // per-lane LDS byte offsets (swizzled tiles): row reads of a 32-row block
  // (Q and dO tiles; the key rows are the same plus this wave's block) and
  // transpose reads; a k-step or column block is an XOR of a constant
  uint32_t pr = 2u * uint32_t(row_base<D>(0, lane));
  uint32_t pt = 2u * uint32_t(tr_base<D>(lane));
  const uint32_t kofs = OK + uint32_t(wave) * 64u * D;  // this wave's key rows

  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dk[db] = zero16();
    dv[db] = zero16();
  }
  const bool kfull = k1 - k0 == BN;
  const float sl2 = p.scale * kLog2e;

  wait_async();
  __syncthreads();
  {
    const int vb = row_base<D>(32 * wave, lane);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) vreg[ks] = lds_b128(smem, 2u * uint32_t(vb ^ (ks << 4)), OQ0);
  }
  __syncthreads();  // every wave holds its V rows before the Q/dO copies
  if (n_it > 0) fetch(0, 0, 0);
  advance();
  wait_async();
  __syncthreads();

  // One query tile. The 4*KS... MFMAs of the step run as one software
  // pipeline of slots, in this order:
  //   S = Q K^T (KS slots); dP = dO V^T (KS slots, each also computing part of
  //   P = exp(S - LSE)); dV += P^T dO (2*DB slots, each also computing part
  //   of dS = P (dP - D)); dK += dS^T Q (2*DB slots).
  // Each slot issues the LDS reads of the slot two ahead, its MFMA, and its
  // share of the vector work, which then runs while the MFMA does; a
  // scheduling barrier after each slot keeps this order.
  constexpr int NS = 2 * KS + 4 * DB;       // slots per step
  constexpr int EP = 16 / KS, ES = 8 / DB;  // P / dS elements per slot
  // The compute of one query tile; P is masked (a branch after its last
  // slot) only on edge tiles.
  // DQ: store this wave's dS block (bf16; w0 holds queries 4h..4h+3 and
  // 8+4h..8+4h+3 of this lane's key, w1 the same plus 16) as rows of the
  // dS^T tile: four 8-byte chunk writes per lane
  // (the lane-derived addresses of the dQ stage are recomputed from an
  // opaque copy of the lane index, not hoisted and held across the loop)
  auto put_ds = [&](const uint4& w0, const uint4& w1) {
    const uint32_t krow = 32 * wave + (opaque(uint32_t(lane)) & 31);
    const uint32_t row = ODS + krow * 64, sw = (krow >> 2) & 7;
    *reinterpret_cast<uint2*>(smem + row + 8 * (uint32_t(half) ^ sw)) = make_uint2(w0.x, w0.y);
    *reinterpret_cast<uint2*>(smem + row + 8 * ((2u + half) ^ sw)) = make_uint2(w0.z, w0.w);
    *reinterpret_cast<uint2*>(smem + row + 8 * ((4u + half) ^ sw)) = make_uint2(w1.x, w1.y);
    *reinterpret_cast<uint2*>(smem + row + 8 * ((6u + half) ^ sw)) = make_uint2(w1.z, w1.w);
  };
  auto tile = [&](int t0, auto bufc, bool edge) {
    constexpr int B = decltype(bufc)::value;
    constexpr uint32_t QO = B ? OQ1 : OQ0, OO = B ? OO1 : OO0, SO = 768u * B;
    // masks: this lane's key against query rows t0 + 4*half + cq, cq =
    // (8g) % RPI + j (register 4g + j, pair 8g + 4*half + j): rows cq < hiq
    // exist; on a local diagonal the key is
    // seen by rows cq >= lo; on a received diagonal by rows whose receive
    // limit exceeds the key index
    // (this lane's key is recomputed here from an opaque lane index rather
    // than held across the loop)
    const bool diag = t0 < qfull;
    const uint32_t ln = opaque(uint32_t(lane));
    const int hf = int(ln >> 5);
    const int kid = k0 + 32 * wave + int(ln & 31);
    const bool kval = kid < k1;
    const int hiq = q1 - t0 - 4 * hf;
    const int lo = !kval ? 0x40000000 : (diag && !src) ? kid - t0 - 4 * hf : -0x40000000;
    const int kl = (diag && src) ? (kval ? kid : 0x7fffffff) : -0x7fffffff;

    f32x16 sacc = zero16(), dpacc = zero16();
    bf16x8 ra[3], rb[3], pa[2], sa[2];
    // Where P is large (short documents, keys near the diagonal) the bf16
    // rounding of P and dS dominates the dV/dK error. On a wave's tile with
    // any P above 1/16 (rare on long documents) the bf16 residuals of P and
    // dS also go through the dV and dK products: after the last dV slot,
    // where P and the whole dS are still in fp32 registers, one branch forms
    // both residuals and multiplies them by their operands (read again) into
    // the same accumulators. Elsewhere each rounding error is at most 2^-13
    // of a term.
    constexpr float kSplitP = 1.0f / 16.0f;
    bool split = false;
    auto residual = [&](const bf16x8 (&lo)[2], uint32_t base, f32x16 (&acc)[DB]) {
      static_for<0, 2 * DB>([&](auto uc) {
        constexpr int u = decltype(uc)::value, kh = u / DB, db = u % DB;
        const uint32_t t0_ = pt ^ (db << 6), t1_ = (pt ^ ((db << 6) | 32)) + 16 * D;
        const bf16x8 b = cat8(lds_tr(smem, t0_, base + kh * 32 * D),
                              lds_tr(smem, t1_, base + kh * 32 * D));
        acc[db] = mfma32(lo[kh], b, acc[db]);
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    f32x4 l4[4], d4[4];
    // P = 0 where the key is not seen: keys past the range, later keys on a
    // local diagonal, keys at or past a row's receive limit on a received
    // diagonal (edge tiles only)
    auto mask_p = [&](f32x16& pv) {
      int4 m4[4];
#pragma unroll
      for (int g = 0; g < 4; ++g)
        m4[g] = *reinterpret_cast<const int4*>(smem + SO + 512 + 4 * (8 * g + 4 * half));
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int g = e >> 2, j = e & 3, cq = (8 * g) % RPI + j;
        // (local tiles never copy limits into LDS: what is there is stale
        // and must not be compared)
        const int lim = !src ? 0x7fffffff
                        : j == 0 ? m4[g].x : j == 1 ? m4[g].y : j == 2 ? m4[g].z : m4[g].w;
        pv[e] = ((cq >= lo) & (cq < hiq) & (kl < lim)) ? pv[e] : 0.f;
      }
    };
    // LDS operand reads of slot n into ring entry n % 3
    auto rd = [&](int n) {
      bf16x8& a = ra[n % 3];
      if (n < KS) {
        const uint32_t r = pr ^ (n << 5);
        a = lds_b128(smem, r, QO);
        rb[n % 3] = lds_b128(smem, r + kofs, 0);
      } else if (n < 2 * KS) {
        a = lds_b128(smem, pr ^ ((n - KS) << 5), OO);
      } else {
        const int u = n < 2 * KS + 2 * DB ? n - 2 * KS : n - 2 * KS - 2 * DB;
        const int kh = u / DB, db = u % DB;
        const uint32_t base = (n < 2 * KS + 2 * DB ? OO : QO) + kh * 32 * D;
        const uint32_t t0_ = pt ^ (db << 6), t1_ = (pt ^ ((db << 6) | 32)) + 16 * D;
        a = cat8(lds_tr(smem, t0_, base), lds_tr(smem, t1_, base));
      }
    };
    rd(0);
    rd(1);
    static_for<0, NS>([&](auto nc) {
      constexpr int n = decltype(nc)::value;
      if (n + 2 < NS) rd(n + 2);
      // LSE and delta of rows 8g + 4*half + 0..3, read two slots before the
      // first slot that uses them
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if (KS + 4 * g / EP == n + 2)
          l4[g] = *reinterpret_cast<const f32x4*>(smem + SO + 4 * (8 * g + 4 * half));
        if (2 * KS + 4 * g / ES == n + 2)
          d4[g] = *reinterpret_cast<const f32x4*>(smem + SO + 256 + 4 * (8 * g + 4 * half));
      }
      const bf16x8& a = ra[n % 3];
      if (n < KS) {
        sacc = mfma32(a, rb[n % 3], sacc);
      } else if (n < 2 * KS) {
        dpacc = mfma32(a, vreg[n - KS], dpacc);
#pragma unroll
        for (int e = (n - KS) * EP; e < (n - KS + 1) * EP; ++e) {
          const int g = e >> 2, j = e & 3;
          sacc[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[e], sl2, -l4[g][j] * kLog2e));
        }
        if ((n - KS + 1) * EP == 8) pa[0] = pack8(sacc, 0);
        if (n == 2 * KS - 1) {
          if (edge) {
            mask_p(sacc);
            pa[0] = pack8(sacc, 0);
          }
          pa[1] = pack8(sacc, 8);
          float pmax = sacc[0];
#pragma unroll
          for (int e = 1; e < 16; ++e) pmax = fmaxf(pmax, sacc[e]);
          split = __any(pmax > kSplitP);
        }
      } else if (n < 2 * KS + 2 * DB) {
        const int u = n - 2 * KS, kh = u / DB, db = u % DB;
        dv[db] = mfma32(pa[kh], a, dv[db]);
#pragma unroll
        for (int e = u * ES; e < (u + 1) * ES; ++e)
          dpacc[e] = sacc[e] * (dpacc[e] - d4[e >> 2][e & 3]);
        if ((u + 1) * ES == 8) sa[0] = pack8(dpacc, 0);
        if ((u + 1) * ES == 16) sa[1] = pack8(dpacc, 8);
        if (u == 2 * DB - 1 && split) {
          // (P and dS through opaque copies: the compiler would otherwise
          // share their bf16 conversions with the packs above, converting
          // element by element on the common path for this rare one)
          f32x16 pf = sacc, sf = dpacc;
          asm volatile("" : "+v"(pf), "+v"(sf));
          residual({pack8_lo(pf, 0), pack8_lo(pf, 8)}, OO, dv);
          residual({pack8_lo(sf, 0), pack8_lo(sf, 8)}, QO, dk);
        }
      } else {
        const int u = n - 2 * KS - 2 * DB, kh = u / DB, db = u % DB;
        dk[db] = mfma32(sa[kh], a, dk[db]);
        if constexpr (DQ) {
          if (u == 0) put_ds(__builtin_bit_cast(uint4, sa[0]), __builtin_bit_cast(uint4, sa[1]));
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // DQ: after a barrier (every wave's dS rows are in the dS^T tile), wave w
  // computes dQ for the iteration's 32 query rows and head-dim columns
  // 32w..32w+31 over the tile's 128 keys, and adds it into dQ. Operands by
  // transpose reads: A (dS, 32 queries x 16 keys per k-step s) from the
  // dS^T tile -- lane 32h + 16g + t reads rows 16s + 4h + t/4 (then + 8),
  // chunk 4g + t%4, whose swizzle is (4s + h) & 7 (then (4s + 2 + h) & 7):
  // the base below XOR 32*(s & 1) (and XOR 16) -- and B (K, 16 keys x 32
  // columns) from the key tile, as the Q/dO tiles are read for dV and dK.
  // With D = 64 there are two column blocks; waves 2 and 3 take the second
  // half of the keys for them (two partial sums per column block).
  constexpr int KPARTS = 4 / DB;         // key parts of the dQ product
  constexpr int QSTEPS = 8 / KPARTS;     // 16-key steps per wave
  auto dq_part = [&](f32x16& qacc) {
    __syncthreads();
    const int cb = wave % DB, kpart = wave / DB;
    const uint32_t ln = opaque(uint32_t(lane));
    const int t = ln & 15, g = (ln >> 4) & 1, hf = ln >> 5;
    // (a key part starts at a multiple of 64 rows: its offset leaves the
    // low bits the XORs act on untouched)
    const uint32_t a0 = uint32_t((4 * hf + (t >> 2)) * 64 + 8 * ((4 * g + (t & 3)) ^ hf)) +
                        uint32_t(kpart) * QSTEPS * 1024u;
    const uint32_t kofs_q = uint32_t(kpart) * QSTEPS * 32u * D;
    const uint32_t b0 = (pt ^ uint32_t(cb << 6)) + kofs_q;
    const uint32_t b1 = (pt ^ uint32_t((cb << 6) | 32)) + 16 * D + kofs_q;
    qacc = zero16();
    // operands of k-step j into ring entry j % 3, two steps ahead of the
    // MFMA that uses them (QSTEPS is even, so the parity of j is that of the
    // k-step)
    bf16x8 ra[3], rb[3];
    auto rdq = [&](int j) {
      const uint32_t x = 32u * uint32_t(j & 1);
      ra[j % 3] = cat8(lds_tr(smem, a0 ^ x, ODS + 1024u * j),
                       lds_tr(smem, a0 ^ x ^ 16u, ODS + 1024u * j + 512u));
      rb[j % 3] = cat8(lds_tr(smem, b0, OK + uint32_t(j) * 32u * D),
                       lds_tr(smem, b1, OK + uint32_t(j) * 32u * D));
    };
    rdq(0);
    rdq(1);
    static_for<0, QSTEPS>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      if (j + 2 < QSTEPS) rdq(j + 2);
      qacc = mfma32(ra[j % 3], rb[j % 3], qacc);
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  // DQ: add the iteration's dQ block into dQ. Issued after the iteration's
  // closing wait and barrier, so the atomics complete while the next
  // iteration computes (its closing vmcnt(0) wait, which also covers them,
  // comes an iteration later) instead of stalling this one.
  auto dq_add = [&](int t0, int hh, const f32x16& qacc) {
    const int cb = wave % DB;
    const uint32_t ln = opaque(uint32_t(lane));
    const int hf = ln >> 5;
    // C layout: register i is pair 8*(i/4) + 4h + i%4 (query row
    // (8*(i/4)) % RPI + 4h + i%4 of head set member (8*(i/4)) / RPI), column
    // 32cb + lane%32; each register's 64 lanes cover two 128-byte row
    // segments.
    // Addresses: a wave-uniform row base per register (scalar registers)
    // plus one 32-bit lane offset shared by all sixteen.
    // (the stride goes through an empty asm per iteration, so the row bases
    // are recomputed here by scalar arithmetic rather than kept, sixteen
    // 64-bit values, across the loop)
    uint32_t rs = uint32_t(p.hq) * D;
    asm volatile("" : "+s"(rs));
    const uint32_t loff = uint32_t(4 * hf) * rs + 32u * cb + (ln & 31);
    float* const base = p.dq + (size_t(t0) * p.hq + kvh * p.group + hh * HPI) * D;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r0 = (8 * (i >> 2)) % RPI + (i & 3), hm = (8 * (i >> 2)) / RPI;
      float* const bi = base + size_t(r0) * rs + hm * D;
      if (t0 + r0 + 4 * hf < q1) atomicAdd(bi + loff, p.scale * qacc[i]);
    }
  };
  // One pipelined iteration: start the next tile's copies, compute this one,
  // wait for the copies. Each wave picks its own variant of the compute:
  // unmasked where every row of the tile sees all of the wave's 32 keys
  // (past the diagonal, a whole tile of rows, all keys in range); skipped
  // where no row sees any of them (the tile ends before qfirst, or the keys
  // are past the range); masked otherwise.
  auto step = [&](int i_, auto bufc) {
    const int t0 = q0 + cur_t * RPI, hh = cur_h;
    if (i_ + 1 < n_it) fetch(nxt_h, nxt_t, decltype(bufc)::value ^ 1);
    cur_t = nxt_t;
    cur_h = nxt_h;
    advance();
    pr = opaque(pr);
    pt = opaque(pt);
    const int tlast = min(t0 + RPI, q1) - 1;
    const bool computed = !(kw >= k1 || tlast < qfirst);
    if (computed) tile(t0, bufc, !(t0 >= qfull && t0 + RPI <= q1 && kw + 32 <= k1));
    f32x16 qacc;
    if constexpr (DQ) {
      if (!computed) put_ds(uint4{0u, 0u, 0u, 0u}, uint4{0u, 0u, 0u, 0u});
      dq_part(qacc);
    }
    wait_async();
    __syncthreads();
    if constexpr (DQ) dq_add(t0, hh, qacc);
  };
  for (int i_ = 0; i_ < n_it; i_ += 2) {
    step(i_, std::integral_constant<int, 0>());
    if (i_ + 1 < n_it) step(i_ + 1, std::integral_constant<int, 1>());
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

}  // namespace fck
