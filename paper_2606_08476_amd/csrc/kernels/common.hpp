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
// row r is stored at chunk position c ^ swz(r). With that swizzle the 16-byte
// row reads (eight rows per phase) and the 4-row transpose reads (two chunks
// of four consecutive rows) both touch distinct banks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

__device__ __forceinline__ int swz(int r) { return ((r & 3) << 1) | ((r >> 2) & 1); }

// Element offset of (row r, column col) in a swizzled tile; col % 4 == 0.
template <int D>
__device__ __forceinline__ int toff(int r, int col) {
  return r * D + ((((col >> 3) ^ swz(r)) << 3) | (col & 7));
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

// Asynchronous copy of ROWS rows of D bf16 into a swizzled LDS tile, 256
// threads; rowptr(r) is the global address of the row that goes to tile row
// r. Completion: wait_async() then a barrier.
template <int D, int ROWS, class RowPtr>
__device__ __forceinline__ void tile_load_async(u16* T, RowPtr rowptr) {
  constexpr int CH = D / 8;
  static_assert((ROWS * CH) % 256 == 0, "tile must be a multiple of 256 chunks");
#pragma unroll
  for (int u = 0; u < ROWS * CH / 256; ++u) {
    const int L = u * 256 + threadIdx.x;
    const int r = L / CH;
    const int c = (L % CH) ^ swz(r);
    const u16* src = rowptr(r) + 8 * c;
    u16* dst = T + (u * 256 + (threadIdx.x & ~63)) * 8;  // wave-uniform base
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
  }
}

__device__ __forceinline__ void wait_async() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

}  // namespace fck
