// Forward attention over one rank's share (gfx950).
//
// One workgroup (4 waves) takes one work item -- a tile of query tokens
// with a received key range (no mask inside it, FlashCP Sec. 3.2: every
// query of a piece sees the same received prefix) and a local key range
// (intra-document causal, Sec. 2.1) -- for `heads_per_tile` query heads of
// one KV head. Each wave owns 32/heads_per_tile query rows of every one of
// those heads (a query per lane). Key tiles of 64 keys are double-buffered
// in LDS and shared by the waves (and so by the heads of the group); later
// tiles are copied from HBM straight into LDS (asynchronous loads, no
// staging registers) while the current one is computed, and the loop is
// software-pipelined across tiles (the scores of the next tile are computed
// beside the softmax of the current one):
//   S^T = K Q^T        MFMA 32x32x16, Q held in registers (B operand), so a
//                      query is a lane and its row statistics are per lane;
//   online softmax     base 2, scale folded into one FMA per score; a row's
//                      output is rescaled only when its maximum grows by
//                      more than 2^8 (the result is the same: numerator and
//                      denominator share the stale maximum). The decision is
//                      per row, so a row's arithmetic does not depend on the
//                      other rows of its tile (any query tiling gives the
//                      same bits);
//   O^T += V^T P^T     V^T read from LDS with transpose reads, P^T straight
//                      from the S^T accumulator registers.
// Output (template OUT): the final O (bf16, optionally fp32) and LSE; or an
// fp32 partial O/LSE for the log-sum-exp merge; or, for items that carry a
// received and a local range, both partials: the received range is run
// first and its partial written when the local range starts, so the query
// tile is loaded once and the tile pipeline runs on across the switch; or
// (merged) the same two passes followed by their log-sum-exp merge in the
// epilogue: the received partial's O is written to a workspace at the
// switch and read back at the end, its LSE kept in a register, and the
// final O and LSE are written as the merge kernel would write them.
#include "common.hpp"
#include "launch.hpp"

#include <type_traits>

namespace fck {

enum { kOutPartial = 0, kOutFinal = 1, kOutPaired = 2, kOutMerged = 3 };

template <int D, int HPW, int OUT>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(FwdParams p) {
  constexpr bool FINAL = OUT == kOutFinal, MERGED = OUT == kOutMerged;
  constexpr bool PAIRED = OUT == kOutPaired || MERGED;
  constexpr int BN = 64;        // keys per tile
  constexpr int RPW = 32 / HPW;  // query rows per wave and head
  constexpr int KS = D / 16;    // MFMA k-steps over the head dim
  constexpr int DB = D / 32;    // 32-wide output blocks of the head dim
  constexpr float kLazy = 8.0f; // log2 headroom before rescaling
  constexpr uint32_t TILE = BN * D * 2;  // bytes of one K or V tile
  // LDS: K0 | K1 | V0 | V1; key tile j uses K buffer j % 2 and V buffer
  // j % 2. K runs one tile ahead of V: iteration j reads K of tile j+1 and V
  // of tile j while the copies of K of tile j+2 and V of tile j+1 fill the
  // other two buffers. The loop is unrolled by two, so every read names its
  // buffer with a compile-time offset.
  // Ordering rule: a buffer is refilled only after a barrier that follows
  // every wave's last read of it. Iteration j refills K buffer j % 2, last
  // read in iteration j-1 (before its closing barrier) -- or, for j = 0, in
  // the prologue, which therefore ends with a barrier of its own.
  __shared__ __attribute__((aligned(16))) char smem[4 * TILE];

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int half = lane >> 5;
  const int b = blockIdx.x;
  const int kvh = b % p.hkv;
  const int rest = b / p.hkv;
  const int hc = rest % p.head_chunks;
  const int32_t* it = p.items + 8 * (rest / p.head_chunks);
  const int q0 = it[0], q1 = it[1], r0 = it[2], r1 = it[3], l0 = it[4], l1 = it[5];
  const int ldiag = it[6];

  // lane -> (query row, head): a wave takes RPW consecutive rows of each of
  // the HPW heads, so a short query range leaves whole waves without rows
  // (they skip the products and only help with the copies and barriers)
  // instead of padding every head's rows to 32
  const int l31 = lane & 31;
  const int h = kvh * p.group + hc * HPW + l31 / RPW;
  const int qrow = q0 + wave * RPW + l31 % RPW;
  const bool qvalid = qrow < q1;
  const bool active = q0 + wave * RPW < q1;  // wave-uniform
  const float c = p.scale_log2;

  // key tiles: first the received range, then the local range
  const int n_r = (r1 - r0 + BN - 1) / BN;
  const int n_t = n_r + (l1 - l0 + BN - 1) / BN;

  // async copy of the K (or V) rows of key tile j into the buffer at byte
  // offset `ofs`; rows past the range repeat the last row (finite data;
  // those keys are masked)
  const TileLoader<D, BN> ld(p.hkv * D);
  auto fetch = [&](int j, uint32_t ofs, bool v) {
    const bool rs = j < n_r;
    const int k0 = rs ? r0 + j * BN : l0 + (j - n_r) * BN;
    const int hi = rs ? r1 : l1;
    const size_t base = (size_t(k0) * p.hkv + kvh) * D;
    const u16* src = v ? (rs ? p.v_recv : p.v_loc) : (rs ? p.k_recv : p.k_loc);
    ld.load_at(lds_addr(smem) + ofs, src + base, hi - k0);
  };

  if (n_t > 0) {
    fetch(0, 0, false);
    fetch(0, 2 * TILE, true);
  }
  if (n_t > 1) fetch(1, TILE, false);

  bf16x8 qreg[KS];
  {
    const u16* qp = p.q + ((size_t)qrow * p.hq + h) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = qvalid ? *reinterpret_cast<const bf16x8*>(qp + 16 * ks) : zero8();
  }

  // per-lane LDS byte offsets of the MFMA operand reads (swizzled tiles):
  // K rows for k-step ks, and the two transpose reads of V^T block db
  uint32_t pk[KS], pv[DB][2];
  {
    const int kb = row_base<D>(0, lane), vb = tr_base<D>(lane);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) pk[ks] = 2u * uint32_t(kb ^ (ks << 4));
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      pv[db][0] = 2u * uint32_t(vb ^ (db << 5));
      pv[db][1] = 2u * uint32_t((vb ^ ((db << 5) | 16)) + 8 * D);
    }
  }

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = zero16();
  float m = -INFINITY;  // reference row maximum (scaled, log2 units)
  float lsum = 0.f;     // this lane's share of the row sum

  // this wave's slot of the merged mode's workspace: 32 x D floats, held in
  // register order (instruction k of lane l at 256k + 4l), so that the
  // received partial goes out and comes back with 1 KiB stores and loads
  // (the lane's address is formed where it is used, from an opaque copy of
  // the lane index, not held across the loop)
  auto slot = [&]() {
    return p.o_f32_recv + (size_t(blockIdx.x) * 4 + wave) * (32 * D) + 4 * opaque(uint32_t(lane));
  };
  // paired items: the received partial is complete when the local range
  // starts; write it (merged: to the slot, with its LSE kept in a register)
  // and start the local one from empty
  float lse_recv = -INFINITY;  // merged: the received partial's LSE
  auto switch_source = [&]() {
    const float tot = sum_halves(lsum);
    const float inv = tot > 0.f ? 1.f / tot : 0.f;
    const float lse = tot > 0.f ? (m + __log2f(tot)) * kLn2 : -INFINITY;
    if (MERGED) {
      lse_recv = lse;
      if (active) {
        float* const sl = slot();
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            f32x4 v;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) v[jj] = oacc[db][4 * g + jj] * inv;
            *reinterpret_cast<f32x4*>(sl + 256 * (4 * db + g)) = v;
          }
      }
    } else if (qvalid) {
      // (paired partial passes: the caller's [T_q, Hq, D] tensor, stored
      // from the registers; this is not the benchmarked path)
      const size_t ob = ((size_t)qrow * p.hq + h) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 v;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) v[jj] = oacc[db][4 * g + jj] * inv;
          *reinterpret_cast<f32x4*>(p.o_f32_recv + ob + 32 * db + 8 * g + 4 * half) = v;
        }
      if (half == 0) p.lse_recv[(size_t)h * p.t_q + qrow] = lse;
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = zero16();
    m = -INFINITY;
    lsum = 0.f;
  };

  // S^T = K Q^T for the K tile at byte offset ko (prologue only; the loop
  // interleaves the same products with the softmax), two independent
  // accumulator chains (32 keys each)
  auto scores = [&](f32x16 (&s)[2], uint32_t ko) {
    s[0] = zero16();
    s[1] = zero16();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
        s[mb] = mfma32(lds_b128(smem, pk[ks], ko + mb * 64 * D), qreg[ks], s[mb]);
  };
  // scores of tile j: keys past the range and, on diagonal tiles, keys after
  // the query are masked (element i of block mb is key k0 + 4*half +
  // cst(mb, i), visible iff cst < rel: one compare per score, edge tiles only)
  auto mask = [&](f32x16 (&s)[2], int j) {
    const bool rs = j < n_r;
    const int k0 = rs ? r0 + j * BN : l0 + (j - n_r) * BN;
    const int hi = rs ? r1 : l1;
    const bool diag = !rs && k0 >= ldiag;
    if (diag || k0 + BN > hi) {
      const int rel = (diag ? min(hi, qrow + 1) : hi) - k0 - 4 * half;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          s[mb][i] = mb * 32 + 8 * (i >> 2) + (i & 3) < rel ? s[mb][i] : -INFINITY;
    }
  };
  // row maximum of masked scores (scaled, log2 units)
  auto row_max = [&](const f32x16 (&s)[2]) {
    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[mb][i]);
    return max_halves(mx) * c;
  };

  wait_async();
  __syncthreads();
  f32x16 sa[2], sb[2];  // scores of the current and of the next tile
  float mxa = -INFINITY, mxb = -INFINITY;
  if (n_t > 0 && active) {
    scores(sa, 0);
    mask(sa, 0);
    mxa = row_max(sa);
  }
  // every wave has read K of tile 0 before iteration 0 copies tile 2 into
  // the same buffer
  if (n_t > 2) __syncthreads();

  // Iteration j runs the online softmax of tile j (scores sc and row maximum
  // mxc, both from the previous iteration) beside the MFMAs of tile j+1's
  // scores into sn, then O^T += V^T P^T for tile j beside tile j+1's mask
  // and row maximum (to mxn). The MFMAs form a fixed sequence of slots: a
  // slot issues the LDS reads of the slot two ahead, its MFMA and its share
  // of the vector work, then a scheduling barrier, so the softmax runs in
  // the MFMAs' shadow. The last iteration computes the scores of a tile that
  // does not exist (from whatever its K buffer holds: finite data or stale
  // bits, never read past the buffer) and drops them; one iteration body,
  // with no branch per slot and no second copy for the last tile.
  constexpr int NS = 2 * KS + 4 * DB;  // score slots, then PV slots
  constexpr int EX = 32 / (2 * KS);    // exponentials per score slot
  constexpr int MX = 3;                // first PV slot that takes maxima
  constexpr int MPS = (32 + (4 * DB - MX) - 1) / (4 * DB - MX);  // maxima per slot
  auto step = [&](int j, auto par, f32x16 (&sc)[2], float mxc, f32x16 (&sn)[2], float& mxn) {
    constexpr int PAR = decltype(par)::value;
    constexpr uint32_t KN = (1 - PAR) * TILE, VC = (2 + PAR) * TILE;
    if (j + 1 < n_t) fetch(j + 1, (3 - PAR) * TILE, true);   // V of tile j+1
    if (j + 2 < n_t) fetch(j + 2, PAR * TILE, false);        // K of tile j+2
    if (PAIRED && j == n_r) switch_source();
    if (active) {
      // a row's output is rescaled only when its maximum grows by more than
      // the headroom; rows that do not grow keep their maximum and scale by 1
      const bool grow = mxc > m + kLazy;  // implies mxc > m
      if (__any(grow)) {
        const float alpha =
            !grow ? 1.f : m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mxc);
        m = grow ? mxc : m;
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
      }
      const float mref = m == -INFINITY ? 0.f : m;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) pk[ks] = opaque(pk[ks]);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        pv[db][0] = opaque(pv[db][0]);
        pv[db][1] = opaque(pv[db][1]);
      }

      bf16x8 ring[3], pb[4];
      // operand of slot n: K rows of tile j+1 (score slots), V^T of tile j
      // (PV slots)
      auto rd = [&](int n) {
        if (n < 2 * KS) {
          ring[n % 3] = lds_b128(smem, pk[n / 2], KN + (n % 2) * 64 * D);
        } else {
          const int u = n - 2 * KS, kk = u / DB, db = u % DB;
          const uint32_t ro = VC + kk * 32 * D;  // rows 16*kk..
          ring[n % 3] = cat8(lds_tr(smem, pv[db][0], ro), lds_tr(smem, pv[db][1], ro));
        }
      };
      float ps = 0.f, mx = -INFINITY;
      sn[0] = zero16();
      sn[1] = zero16();
      rd(0);
      rd(1);
      static_for<0, NS>([&](auto nc) {
        constexpr int n = decltype(nc)::value;
        if (n + 2 < NS) rd(n + 2);
        if constexpr (n < 2 * KS) {
          sn[n % 2] = mfma32(ring[n % 3], qreg[n / 2], sn[n % 2]);
#pragma unroll
          for (int e = n * EX; e < (n + 1) * EX; ++e) {
            const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[e / 16][e % 16], c, -mref));
            sc[e / 16][e % 16] = x;
            ps += x;
            if (e % 8 == 7) {
              pb[e / 8] = pack8(sc[e / 16], 8 * ((e / 8) & 1));
              // complete here: keeps the exponentials in the score slots
              // rather than sunk past the masking branch into the PV slots
              asm volatile("" ::"v"(pb[e / 8]));
            }
          }
          if (n == 2 * KS - 1) {
            lsum += ps;
            asm volatile("" : "+v"(lsum));  // the row sum too, not sunk into the next step
          }
        } else {
          constexpr int u = n - 2 * KS;
          oacc[u % DB] = mfma32(ring[n % 3], pb[u / DB], oacc[u % DB]);
          if constexpr (u == MX - 1) mask(sn, j + 1);
          if constexpr (u >= MX) {
#pragma unroll
            for (int e = (u - MX) * MPS; e < (u - MX + 1) * MPS && e < 32; ++e)
              mx = fmaxf(mx, sn[e / 16][e % 16]);
          }
          if constexpr (u == 4 * DB - 1) mxn = max_halves(mx) * c;
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    wait_async();
    __syncthreads();
  };
  for (int j = 0; j < n_t; j += 2) {
    step(j, std::integral_constant<int, 0>(), sa, mxa, sb, mxb);
    if (j + 1 < n_t) step(j + 1, std::integral_constant<int, 1>(), sb, mxb, sa, mxa);
  }

  if (PAIRED && n_r == n_t) switch_source();  // no local tile (never empty in practice)
  // the local (or only) partial, normalised, and its LSE
  const float tot = sum_halves(lsum);
  const float inv = tot > 0.f ? 1.f / tot : 0.f;
  const float lse_own = tot > 0.f ? (m + __log2f(tot)) * kLn2 : -INFINITY;
  // rows go out through the LDS tile buffers, free once the loop's last
  // barrier has passed: wave w's region is bytes 32*D*4*w ..
  char* const region = smem + size_t(wave) * (32 * D * 4);
  const int h0 = kvh * p.group + hc * HPW;
  if constexpr (MERGED) {
    // local partial (registers) merged with the received one (this wave's
    // slot, written at the switch; the waits since have completed it)
    wait_async();
    const Merge2 w = merge2(lse_own, lse_recv);
    // every read of the received partial is issued before the first use
    f32x4 y[DB][4];
    if (active) {  // (a wave without rows wrote no slot)
      const float* const sl = slot();
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          y[db][g] = *reinterpret_cast<const f32x4*>(sl + 256 * (4 * db + g));
    }
    store_rows<D, RPW>(
        region, active,
        [&](int db, int g) {
          f32x4 v;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) v[jj] = merge2_value(w, oacc[db][4 * g + jj] * inv, y[db][g][jj]);
          return v;
        },
        q0 + wave * RPW, q1, p.hq, h0, p.o_f32, p.o_bf16);
    if (qvalid && half == 0) p.lse[(size_t)h * p.t_q + qrow] = w.lse;
  } else {
    store_rows<D, RPW>(
        region, active,
        [&](int db, int g) {
          f32x4 v;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) v[jj] = oacc[db][4 * g + jj] * inv;
          return v;
        },
        q0 + wave * RPW, q1, p.hq, h0, p.o_f32, FINAL ? p.o_bf16 : nullptr);
    if (qvalid && half == 0) p.lse[(size_t)h * p.t_q + qrow] = lse_own;
  }
}

template <int D, int HPW>
static hipError_t launch_fwd_t(const FwdParams& p, int out, hipStream_t s) {
  const dim3 grid(unsigned(p.n_items) * p.hkv * p.head_chunks), block(256);
  if (out == kOutFinal)
    hipLaunchKernelGGL((attn_fwd_kernel<D, HPW, kOutFinal>), grid, block, 0, s, p);
  else if (out == kOutPaired)
    hipLaunchKernelGGL((attn_fwd_kernel<D, HPW, kOutPaired>), grid, block, 0, s, p);
  else if (out == kOutMerged)
    hipLaunchKernelGGL((attn_fwd_kernel<D, HPW, kOutMerged>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((attn_fwd_kernel<D, HPW, kOutPartial>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_fwd_d(const FwdParams& p, int hpw, int out, hipStream_t s) {
  switch (hpw) {
    case 1: return launch_fwd_t<D, 1>(p, out, s);
    case 2: return launch_fwd_t<D, 2>(p, out, s);
    case 4: return launch_fwd_t<D, 4>(p, out, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fwd(const FwdParams& p, int d, int heads_per_tile, bool final_out,
                      hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  const int out = p.o_f32_recv ? (final_out ? kOutMerged : kOutPaired)
                  : final_out ? kOutFinal : kOutPartial;
  if (d == 64) return launch_fwd_d<64>(p, heads_per_tile, out, s);
  if (d == 128) return launch_fwd_d<128>(p, heads_per_tile, out, s);
  return hipErrorInvalidValue;
}

}  // namespace fck
