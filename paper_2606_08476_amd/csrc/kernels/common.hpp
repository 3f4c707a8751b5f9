// Device helpers shared by the gfx950 kernels: bf16 conversion, MFMA and
// LDS operand fetches.
//
// MFMA v_mfma_f32_32x32x16_bf16 operand layout (wave of 64 lanes, l = lane):
//   A (32 x 16): lane l holds A[l % 32][8*(l/32) + j], j = 0..7
//   B (16 x 32): lane l holds B[8*(l/32) + j][l % 32]
//   C (32 x 32): lane l, register i holds C[8*(i/4) + 4*(l/32) + i%4][l % 32]
// ds_read_b64_tr_b16: within each group of 16 lanes, lane t addresses row
// R0 + t/4, columns C0 + 4*(t%4) .. +3 of a row-major bf16 matrix, and
// receives column C0 + t of rows R0 .. R0+3.
// global_load_lds_dwordx4: lane i's 16 bytes land at the wave's LDS base
// + 16*i.
//
// LDS tiles are unpadded row-major bf16 (D columns); the 16-byte chunk c of
// row r is stored at chunk position c ^ swz<D>(r). The LDS serves 256 bytes
// (64 banks) per cycle; with the swizzle both access patterns fill them
// without conflicts: 16-byte row reads (16 lanes = 16 consecutive rows, one
// chunk) and transpose reads (32 lanes = 4 consecutive rows x 4 chunks).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace fck {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) u16 lds_u16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ u16 f2bf(float x) {
  __bf16 b = (__bf16)x;  // round to nearest even
  return __builtin_bit_cast(u16, b);
}

__device__ __forceinline__ float bf2f(u16 x) {
  return __uint_as_float(uint32_t(x) << 16);
}

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int j = 0; j < 8; ++j) z[j] = (__bf16)0.0f;
  return z;
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int j = 0; j < 16; ++j) z[j] = 0.0f;
  return z;
}

// 16-byte LDS read of 8 consecutive bf16 at element offset `e` of `base`.
__device__ __forceinline__ bf16x8 lds_read8(const u16* base, int e) {
  return *reinterpret_cast<const bf16x8*>(base + e);
}

// Transposed 4-row read (see header comment); `e` is this lane's element
// offset (row R0 + t/4, column C0 + 4*(t%4)).
__device__ __forceinline__ bf16x4 lds_read_tr4(const u16* base, int e) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4*)((lds_u16*)(base) + e));
}

__device__ __forceinline__ bf16x8 cat8(const bf16x4& a, const bf16x4& b) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    r[j] = a[j];
    r[4 + j] = b[j];
  }
  return r;
}

// MFMA operand holding X[k][nbase + l%32] of a row-major LDS matrix X (row
// stride ld elements) for 8 values of k taken as two runs of four rows:
// rows r0(l)..r0(l)+3 then r1(l)..r1(l)+3, where the caller picks r0/r1.
__device__ __forceinline__ bf16x8 lds_operand_tr(const u16* X, int ld, int r0, int r1,
                                                 int nbase, int lane) {
  const int t = lane & 15;
  const int col = nbase + 16 * ((lane >> 4) & 1) + 4 * (t & 3);
  const bf16x4 a = lds_read_tr4(X, (r0 + (t >> 2)) * ld + col);
  const bf16x4 b = lds_read_tr4(X, (r1 + (t >> 2)) * ld + col);
  return cat8(a, b);
}

// Pack 8 fp32 of a C-layout accumulator (registers i0 .. i0+7) as a bf16
// operand; with the C layout this covers rows {4*(l/32)+0..3} and
// {8+4*(l/32)+0..3} of a 16-row band.
__device__ __forceinline__ bf16x8 pack8(const f32x16& c, int i0) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)c[i0 + j];
  return r;
}

// The bf16 residuals of the same 8 values: c - bf16(c), rounded to bf16.
// With pack8 it splits each value into a high and a low bf16 part whose sum
// carries about 16 significant bits (a product taken over both parts is as
// exact as its fp32 accumulation).
__device__ __forceinline__ bf16x8 pack8_lo(const f32x16& c, int i0) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)(c[i0 + j] - (float)(__bf16)c[i0 + j]);
  return r;
}

template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128)
    return ((r & 3) << 2) | ((r >> 2) & 3);           // one row per 256 bytes
  else
    return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);    // two rows per 256 bytes
}

// Element offset of (row r, column col) in a swizzled tile; col % 4 == 0.
template <int D>
__device__ __forceinline__ int toff(int r, int col) {
  return r * D + ((((col >> 3) ^ swz<D>(r)) << 3) | (col & 7));
}

// 8 consecutive bf16 of row r starting at column col (col % 8 == 0).
template <int D>
__device__ __forceinline__ bf16x8 tread8(const u16* T, int r, int col) {
  return *reinterpret_cast<const bf16x8*>(T + toff<D>(r, col));
}

// MFMA operand holding X[k][nbase + l%32] of a swizzled tile for 8 values of
// k taken as two runs of four rows, r0(l)..r0(l)+3 then r1(l)..r1(l)+3.
template <int D>
__device__ __forceinline__ bf16x8 tread_tr(const u16* T, int r0, int r1, int nbase, int lane) {
  const int t = lane & 15;
  const int col = nbase + 16 * ((lane >> 4) & 1) + 4 * (t & 3);
  const bf16x4 a = lds_read_tr4(T, toff<D>(r0 + (t >> 2), col));
  const bf16x4 b = lds_read_tr4(T, toff<D>(r1 + (t >> 2), col));
  return cat8(a, b);
}

// Cheap addressing of the swizzled tiles: every MFMA operand read below is a
// per-lane base XOR a compile-time constant, plus a constant row offset.
//
// Row reads: rows base_row + (lane & 31) (base_row a multiple of 32), 8
// columns from 16*ks + 8*(lane/32); offset = row_base ^ (ks << 4).
template <int D>
__device__ __forceinline__ int row_base(int base_row, int lane) {
  const int r = base_row + (lane & 31), half = lane >> 5, f = swz<D>(r);
  return (r * D) | ((half ^ (f & 1)) << 3) | ((f >> 1) << 4);
}
template <int D>
__device__ __forceinline__ bf16x8 tread8_ks(const u16* T, int base, int ks) {
  return *reinterpret_cast<const bf16x8*>(T + (base ^ (ks << 4)));
}

// Transpose reads forming an operand with k = rows R + 4*(lane/32) + 0..3 and
// R + 8 + 4*(lane/32) + 0..3 (R a multiple of 16) and n = columns
// 32*db + (lane % 32); tr_base is per lane, R and db compile-time.
template <int D>
__device__ __forceinline__ int tr_base(int lane) {
  const int half = lane >> 5, t = lane & 15, g = (lane >> 4) & 1;
  const int t4 = D == 128 ? ((t >> 2) << 2) : (((t >> 3) & 1) << 2);
  const int x = (2 * g + ((t & 3) >> 1)) ^ half;
  return ((4 * half + (t >> 2)) * D + (t & 1) * 4) | (x << 3) | (t4 << 3);
}
template <int D>
__device__ __forceinline__ bf16x8 tread_tr2(const u16* T, int base, int R, int db) {
  const bf16x4 a = lds_read_tr4(T, (base ^ (db << 5)) + R * D);
  const bf16x4 b = lds_read_tr4(T, (base ^ ((db << 5) | 16)) + (R + 8) * D);
  return cat8(a, b);
}

// LDS reads at byte addresses: `smem` is a kernel's shared array, `v` a
// per-lane byte offset in a register and `imm` a compile-time byte offset
// (buffer, row block), which the compiler folds into the instruction's
// offset field.
__device__ __forceinline__ bf16x8 lds_b128(const void* smem, uint32_t v, uint32_t imm) {
  return *reinterpret_cast<const bf16x8*>(static_cast<const char*>(smem) + v + imm);
}
__device__ __forceinline__ bf16x4 lds_tr(const void* smem, uint32_t v, uint32_t imm) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4*)((__attribute__((address_space(3))) char*)smem + v + imm));
}

// A copy of `x` the compiler cannot see through. Taken once per loop
// iteration of a per-lane address, it keeps `x + constant` inside the loop,
// so the constant lands in the LDS instruction's offset field instead of a
// register of its own per distinct constant.
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Asynchronous HBM-to-LDS copies. Lane i's 16 (or 4) bytes at `gbase` +
// `voff` land at LDS byte address `lds` + 16*i (4*i); `gbase` and `lds` are
// wave-uniform. The instruction is issued from inline assembly so that the
// compiler does not track it: with the builtin form the compiler waits for
// every outstanding copy before any later LDS read it cannot prove disjoint,
// which serialises the double buffering (reads of the current tile would
// wait for the copy of the next). Completion is the caller's business:
// wait_async() then a barrier before the destination is read. M0 holds the
// LDS address; nothing else in these kernels uses M0.
__device__ __forceinline__ void lds_copy16(const void* gbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(lds), "v"(voff), "s"(gbase) : "memory");
}
__device__ __forceinline__ void lds_copy4(const void* gbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2"
               :: "s"(lds), "v"(voff), "s"(gbase) : "memory");
}

// LDS byte address of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// Calls f(std::integral_constant<int, I>()) for I = B .. E-1: a fully
// unrolled loop whose index is a compile-time constant, whatever the size of
// the body (a plain unroll pragma gives up past the unroller's size limit).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>());
    static_for<B + 1, E>(f);
  }
}

// Lane l combined with lane l ^ 32 (the other half of the wave) through
// v_permlane32_swap, a VALU exchange with no LDS round trip: after the swap
// one register holds x of lanes 0-31 in both halves and the other x of lanes
// 32-63, so one max or add of the two gives each lane the pair's result
// (addition commutes exactly, so the bits equal x + x[l ^ 32]).
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Index of this thread's wave in the workgroup, as a wave-uniform value.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// Asynchronous copies of ROWS x D bf16 tiles into a swizzled LDS tile by a
// workgroup of NT threads. Tile row r is HBM row (r % RPB) * row_stride +
// (r / RPB) * block_stride elements from the base: RPB consecutive rows of
// one block (one query head, say), then the next block (RPB = ROWS: one
// block of rows row_stride apart). Each thread's chunk byte offsets are
// computed once; a copy is then one uniform base address plus those
// offsets. Rows whose index within their block is at or past `nvalid`
// repeat row nvalid-1 of the same block (finite data for masked rows, no
// read past the range).
template <int D, int ROWS, int NT = 256, int RPB = ROWS>
struct TileLoader {
  static constexpr int CH = D / 8;
  static constexpr int N = ROWS * CH / NT;
  static_assert((ROWS * CH) % NT == 0, "tile must be a multiple of NT chunks");
  static_assert(ROWS % RPB == 0, "whole blocks of rows");
  uint32_t off[N];
  int row_stride, block_stride;

  __device__ __forceinline__ explicit TileLoader(int stride, int bstride = 0)
      : row_stride(stride), block_stride(bstride) {
#pragma unroll
    for (int u = 0; u < N; ++u) {
      const int L = u * NT + threadIdx.x;
      const int r = L / CH;
      off[u] = 2u * uint32_t((r % RPB) * stride + (r / RPB) * bstride + 8 * ((L % CH) ^ swz<D>(r)));
    }
  }

  __device__ __forceinline__ void load(u16* T, const u16* g, int nvalid) const {
    load_at(lds_addr(T), g, nvalid);
  }
  // the same with the tile's LDS byte address
  __device__ __forceinline__ void load_at(uint32_t tile, const u16* g, int nvalid) const {
    const uint32_t lds = tile + 1024u * wave_id();
    if (nvalid >= RPB) {  // uniform: whole blocks, the offsets as computed
#pragma unroll
      for (int u = 0; u < N; ++u) lds_copy16(g, off[u], lds + 16u * NT * u);
    } else {  // the last, ragged rows of a range: a per-lane select, no branch
#pragma unroll
      for (int u = 0; u < N; ++u) {
        const int L = u * NT + threadIdx.x;
        const int r = L / CH;
        const uint32_t alt = 2u * uint32_t((nvalid - 1) * row_stride + (r / RPB) * block_stride +
                                           8 * ((L % CH) ^ swz<D>(r)));
        lds_copy16(g, r % RPB >= nvalid ? alt : off[u], lds + 16u * NT * u);
      }
    }
  }
};

// Asynchronous copy of a workgroup's 128 (query row, head) rows of D bf16
// from a [rows, hq, D] tensor into a swizzled 128 x D LDS tile, whose row
// 32w + p is pair p of wave w: row row0 + RPW*w + p % RPW, head h0 + p / RPW
// (the lane-to-pair map of the forward and dQ workgroups). Each wave then
// reads its 32 rows as an MFMA operand with row reads (row_base(32w, lane)).
// Loaded lane by lane into registers, these rows cost one scattered 16-byte
// piece per row and instruction; copied this way every instruction moves
// 1 KiB in whole 16-byte chunks. Rows at or past row_end repeat row
// row_end - 1 (finite data for lanes without a row).
template <int D, int RPW>
__device__ __forceinline__ void load_pairs(uint32_t tile, const u16* g, int row0, int row_end,
                                           int hq, int h0) {
  constexpr int CH = D / 8;
  constexpr int N = 128 * CH / 256;
  const u16* base = g + (size_t(row0) * hq + h0) * D;
  const uint32_t lds = tile + 1024u * wave_id();
  const int last = row_end - 1 - row0;
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int L = u * 256 + int(threadIdx.x);
    const int R = L / CH, w = R / 32, pr = R % 32;
    const int rr = min(RPW * w + pr % RPW, last);
    const uint32_t off = 2u * uint32_t((rr * hq + pr / RPW) * D + 8 * ((L % CH) ^ swz<D>(R)));
    lds_copy16(base, off, lds + 16u * 256 * u);
  }
}

// Coalesced store of one wave's 32 output rows (query row, head) of D
// values. Lane l holds, for pair p = l % 32, columns 32db + 8g + 4(l/32) +
// 0..3 in val(db, g) (the MFMA accumulator layout of O^T or dQ^T); pair p
// is row row0 + p % RPW of head h0 + p / RPW of a [rows, hq, D] tensor, so
// the heads of a row lie side by side in memory. Stored straight from the
// registers, every store instruction would scatter over 32 rows; here the
// wave first writes its rows to its own LDS region (32 x D floats, 16-byte
// chunks XOR-swizzled by row) and then stores them so that each
// instruction covers 1 KiB of consecutive addresses (fp32), or 1 KiB of
// bf16. Rows at or past row_end are not stored; out_f32 or out_bf16 may be
// null. Every wave of the workgroup must call it (it contains a barrier);
// `active` false skips the wave's stores, and the LDS regions must be free
// of other use.
template <int D, int RPW, class Val>
__device__ __forceinline__ void store_rows(char* region, bool active, Val val, int row0,
                                           int row_end, int hq, int h0, float* out_f32,
                                           u16* out_bf16) {
  constexpr int CH = D / 4;           // 16-byte chunks per row
  constexpr int U = (32 / RPW) * D;   // values per row0 + r: its heads side by side
  const int lane = threadIdx.x & 63, p = lane & 31, half = lane >> 5;
  float* st = reinterpret_cast<float*>(region);
  if (active) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = 8 * db + 2 * g + half;
        *reinterpret_cast<f32x4*>(st + p * D + 4 * (c ^ (p % CH))) = val(db, g);
      }
  }
  __syncthreads();
  if (!active) return;
  // value e of the wave's output, in memory order: row row0 + e / U, head
  // h0 + (e % U) / D, column e % D
  auto at = [&](int e, int& pr, int& row, size_t& gofs) {
    const int r = e / U, u = e % U, hoff = u / D, dd = u % D;
    pr = hoff * RPW + r;
    row = row0 + r;
    gofs = (size_t(row) * hq + h0 + hoff) * D + dd;
    return dd;
  };
  if (out_f32) {
#pragma unroll
    for (int s = 0; s < D / 8; ++s) {
      int pr, row;
      size_t go;
      const int dd = at(256 * s + 4 * lane, pr, row, go);
      const f32x4 v = *reinterpret_cast<const f32x4*>(st + pr * D + 4 * ((dd / 4) ^ (pr % CH)));
      if (row < row_end) *reinterpret_cast<f32x4*>(out_f32 + go) = v;
    }
  }
  if (out_bf16) {
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      int pr, row;
      size_t go;
      const int dd = at(512 * s + 8 * lane, pr, row, go);
      const f32x4 a = *reinterpret_cast<const f32x4*>(st + pr * D + 4 * ((dd / 4) ^ (pr % CH)));
      const f32x4 b = *reinterpret_cast<const f32x4*>(st + pr * D + 4 * ((dd / 4 + 1) ^ (pr % CH)));
      uint4 pk;
      pk.x = uint32_t(f2bf(a[0])) | (uint32_t(f2bf(a[1])) << 16);
      pk.y = uint32_t(f2bf(a[2])) | (uint32_t(f2bf(a[3])) << 16);
      pk.z = uint32_t(f2bf(b[0])) | (uint32_t(f2bf(b[1])) << 16);
      pk.w = uint32_t(f2bf(b[2])) | (uint32_t(f2bf(b[3])) << 16);
      if (row < row_end) *reinterpret_cast<uint4*>(out_bf16 + go) = pk;
    }
  }
}

// Log-sum-exp merge of two partial results over disjoint key sets (weights
// of the partials and the merged LSE, natural log; a -inf partial has
// weight 0, so two empty partials merge to O = 0, LSE = -inf). One
// definition for the merge kernel and the forward's merging epilogue, so
// that both give the same bits.
struct Merge2 {
  float ca, cb, lse;
};
__device__ __forceinline__ Merge2 merge2(float la, float lb) {
  const float mx = fmaxf(la, lb);
  const float m = mx == -INFINITY ? 0.f : mx;
  const float wa = __expf(la - m), wb = __expf(lb - m);
  const float tot = wa + wb;
  const bool any = tot > 0.f;
  return {any ? wa / tot : 0.f, any ? wb / tot : 0.f, m + __logf(tot)};
}
__device__ __forceinline__ float merge2_value(const Merge2& w, float a, float b) {
  return __builtin_fmaf(w.ca, a, w.cb * b);
}

// Wait until every outstanding vector memory load of this wave, the LDS
// copies included, has completed (s_waitcnt vmcnt(0); the expcnt and
// lgkmcnt fields are left at their no-wait maxima). Issued through the
// builtin so that the compiler knows its own earlier loads are complete too
// and does not add waits of its own inside the loops.
__device__ __forceinline__ void wait_async() { __builtin_amdgcn_s_waitcnt(0x0F70); }

}  // namespace fck
