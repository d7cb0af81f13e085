// Matrix-core building blocks for gfx950 (CDNA4), shared by the boundary kernels.
//
// Every contraction is expressed with 16x16 output tiles.  A lane l of a
// 64-wide wave is addressed as (row16 = l % 16, grp = l / 16).  For one
// 32-deep step of K the A operand fragment of lane l holds A[row16][8*grp + e]
// and the B fragment holds B[8*grp + e][row16], e = 0..7; the accumulator
// holds D[4*grp + v][row16], v = 0..3.  Because A and B use the same
// lane/slot -> k assignment, the exact order in which the hardware visits k
// inside the step does not matter.
//
// Two element types are supported:
//   bf16 I/O  (default)   : one v_mfma_f32_16x16x32_bf16 per bf16 x bf16 product.
//                           float32 operands (weights, on-chip gradients) are
//                           split into hi + lo bf16 parts, hi = rne(w),
//                           lo = rne(w - hi), which keeps ~16 significant bits.
//   f32 I/O (validation)  : eight v_mfma_f32_16x16x4_f32 per step, slot e of
//                           every lane feeding the e-th instruction.
#pragma once

#ifndef RESBM_IO_F32_BUILD
#define RESBM_IO_F32_BUILD 0
#endif

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resbm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// ---------------------------------------------------------------- bf16 helpers
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// float32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

// hi + lo split of a float32 value.  Infinite hi parts get a zero lo part so
// that an infinite weight multiplies as infinity rather than inf + (-inf).
__device__ __forceinline__ void split_hi_lo(float w, __bf16& hi, __bf16& lo) {
  hi = to_bf16(w);
  float h = (float)hi;
  lo = __builtin_isinf(h) ? to_bf16(0.0f) : to_bf16(w - h);
}

// ---------------------------------------------------------------- fragments
// An "exact" fragment carries 8 values that are representable in the I/O type
// (activations, payloads).  A "split" fragment carries 8 float32 values
// (weights, float32 intermediates) in the form the matrix cores consume.
#if RESBM_IO_F32_BUILD
struct XFrag { float v[8]; };
struct SFrag { float v[8]; };
#else
struct XFrag { bf16x8 v; };
struct SFrag { bf16x8 hi, lo; };
#endif

__device__ __forceinline__ XFrag xfrag_zero() {
  XFrag f;
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) f.v[e] = 0.0f;
#else
  f.v = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
#endif
  return f;
}

__device__ __forceinline__ SFrag sfrag_from(const float (&w)[8]) {
  SFrag f;
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) f.v[e] = w[e];
#else
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    __bf16 h, l;
    split_hi_lo(w[e], h, l);
    f.hi[e] = h;
    f.lo[e] = l;
  }
#endif
  return f;
}

__device__ __forceinline__ SFrag sfrag_zero() {
  float w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  return sfrag_from(w);
}

// An exact fragment reinterpreted as a split one (lo = 0); used where a bf16
// operand meets a split operand in the 3-product form.
__device__ __forceinline__ float xfrag_get(const XFrag& f, int e) {
#if RESBM_IO_F32_BUILD
  return f.v[e];
#else
  return (float)f.v[e];
#endif
}

// ---------------------------------------------------------------- products
#if RESBM_IO_F32_BUILD
__device__ __forceinline__ f32x4 mma8(const float (&a)[8], const float (&b)[8], f32x4 c) {
#pragma unroll
  for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
  return c;
}
// split (A) x exact (B)
__device__ __forceinline__ f32x4 mma_sx(const SFrag& a, const XFrag& b, f32x4 c) { return mma8(a.v, b.v, c); }
// exact (A) x split (B)
__device__ __forceinline__ f32x4 mma_xs(const XFrag& a, const SFrag& b, f32x4 c) { return mma8(a.v, b.v, c); }
// exact x exact
__device__ __forceinline__ f32x4 mma_xx(const XFrag& a, const XFrag& b, f32x4 c) { return mma8(a.v, b.v, c); }
// split x split
__device__ __forceinline__ f32x4 mma_ss(const SFrag& a, const SFrag& b, f32x4 c) { return mma8(a.v, b.v, c); }
#else
__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma_sx(const SFrag& a, const XFrag& b, f32x4 c) {
  c = mfma(a.lo, b.v, c);
  return mfma(a.hi, b.v, c);
}
__device__ __forceinline__ f32x4 mma_xs(const XFrag& a, const SFrag& b, f32x4 c) {
  c = mfma(a.v, b.lo, c);
  return mfma(a.v, b.hi, c);
}
__device__ __forceinline__ f32x4 mma_xx(const XFrag& a, const XFrag& b, f32x4 c) {
  return mfma(a.v, b.v, c);
}
// (ah + al)(bh + bl) without the al*bl term (below 2^-16 relative).
__device__ __forceinline__ f32x4 mma_ss(const SFrag& a, const SFrag& b, f32x4 c) {
  c = mfma(a.lo, b.hi, c);
  c = mfma(a.hi, b.lo, c);
  return mfma(a.hi, b.hi, c);
}
#endif

// ---------------------------------------------------------------- I/O element
#if RESBM_IO_F32_BUILD
typedef float io_t;
#else
typedef __bf16 io_t;
#endif

__device__ __forceinline__ float io_to_f32(io_t x) { return (float)x; }
__device__ __forceinline__ io_t f32_to_io(float x) {
#if RESBM_IO_F32_BUILD
  return x;
#else
  return to_bf16(x);
#endif
}

// 8 consecutive I/O elements starting at p (16-byte aligned for bf16,
// 32-byte aligned for f32).
__device__ __forceinline__ XFrag load_x8(const io_t* p) {
  XFrag f;
#if RESBM_IO_F32_BUILD
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
#else
  f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
#endif
  return f;
}

// 4 consecutive I/O elements (8-byte aligned for bf16, 16 for f32).
__device__ __forceinline__ void load_x4(const io_t* p, float (&out)[4]) {
#if RESBM_IO_F32_BUILD
  float4 a = *reinterpret_cast<const float4*>(p);
  out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
#else
  uint2 u = *reinterpret_cast<const uint2*>(p);
  out[0] = bf16_bits_to_f32(u.x & 0xffffu);
  out[1] = bf16_bits_to_f32(u.x >> 16);
  out[2] = bf16_bits_to_f32(u.y & 0xffffu);
  out[3] = bf16_bits_to_f32(u.y >> 16);
#endif
}

__device__ __forceinline__ void store_x4(io_t* p, const float (&v)[4]) {
#if RESBM_IO_F32_BUILD
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
#else
  bf16x4 h;
  h[0] = to_bf16(v[0]); h[1] = to_bf16(v[1]); h[2] = to_bf16(v[2]); h[3] = to_bf16(v[3]);
  *reinterpret_cast<uint2*>(p) = __builtin_bit_cast(uint2, h);
#endif
}

// ---------------------------------------------------------------- LDS tile layouts
// Bank model of the gfx950 LDS, measured with timing probes of single access
// patterns (cycles per instruction for 8 waves issuing the same pattern):
//   ds_read_b128        64 banks of 4 bytes; 16 lanes per cycle, in the groups
//                       {0-3, 12-15, 20-23, 24-27} and {4-11, 16-19, 28-31}
//                       of each half-wave;
//   ds_read_b64 and     64 banks; 32 lanes per cycle (lanes 0-31, 32-63);
//   ds_read_b64_tr_b16
//   ds_write_b128       32 banks (128 bytes); 8 consecutive lanes per cycle;
//   ds_write_b64        32 banks; 16 consecutive lanes per cycle.
// A group of lanes takes as many cycles as the largest number of distinct
// 4-byte words that it addresses in one bank.  The layouts below permute the
// 16-byte (8-element) chunks of a row-major tile by an XOR with a function of
// the row, chosen so that the accesses of the kernels take one cycle per
// group: whole-row copies (consecutive lanes on consecutive chunks), matrix-core
// fragments (one chunk from each of 16 rows, lane group g on chunk c0 + g),
// per-lane row pieces (lane (i, g) of a 16 x 8g tile writing row i, chunk g),
// and transposed reads (ds_read_b64_tr_b16: 32 lanes on two adjacent chunks of
// the 8 rows r0 .. r0 + 3 and r0 + 8 .. r0 + 11, r0 % 4 == 0).  Chunks stay
// contiguous and never leave their row.

// XOR applied to the low four chunk bits of row `row` of a tile whose rows are
// a multiple of 256 bytes: chunk bit 1 <- row bit 0, bit 2 <- row bit 1,
// bit 3 <- row bits 2 ^ 3, bit 0 <- row bit 3.  A bijection of the row's low
// four bits (16 rows, one chunk each: 16 distinct slots, for either lane
// grouping of ds_read_b128), and bits 1-3 take 8 distinct values over the rows
// of a transposed read (the two chunks of a row share bits 1-3).  XORing with
// the row's low four bits instead leaves rows r and r + 1 of a transposed read
// on the same banks (twice the cycles).
__device__ __forceinline__ int wide_xor(int row) {
  const int rr = row & 15;
  return (((rr << 1) | (rr >> 3)) & 15) ^ (rr & 8);
}

// Column permutation of a row-major tile with WC elements per row (32 or 64:
// 4 or 8 chunks, i.e. 4 or 2 rows per 256-byte bank window); other widths are
// left as is.  The XOR keeps the rows written by one 8-lane write group (8
// consecutive rows of a 16-row tile, one chunk each) on distinct banks of the
// 128-byte write window, and serves fragments and transposed reads as above.
template <int WC>
__device__ __forceinline__ int tile_col(int row, int col) {
  constexpr int CPR = WC / 8;
  int x;
  if constexpr (CPR == 8) {
    x = (row & 7) ^ (((row >> 3) & 1) * 5);
  } else if constexpr (CPR == 4) {
    x = ((row >> 1) & 3) ^ (((row >> 3) & 1) * 3);
  } else if constexpr (CPR == 2) {
    x = (row >> 3) & 1;
  } else {
    return col;
  }
  return ((((col >> 3) ^ x) & (CPR - 1)) << 3) | (col & 7);
}

// Column permutation of a block-wide row-major tile (WIDE elements per row, a
// multiple of 128): the low four chunk bits are XORed with wide_xor(row).
__device__ __forceinline__ int wide_col(int row, int col) {
  return ((((col >> 3) ^ wide_xor(row)) & 15) | ((col >> 3) & ~15)) << 3 | (col & 7);
}

// Either layout, by row width (elements).
template <int W>
__device__ __forceinline__ int lds_col(int row, int col) {
  if constexpr (W % 128 == 0) {
    return wide_col(row, col);
  } else {
    return tile_col<W>(row, col);
  }
}

// Activation function and its derivative (float32).
__device__ __forceinline__ float act_phi(float a, int act) {
  return act == 1 ? a / (1.0f + expf(-a)) : a;
}
__device__ __forceinline__ float act_dphi(float a, int act) {
  if (act != 1) return 1.0f;
  float s = 1.0f / (1.0f + expf(-a));
  return s * (1.0f + a * (1.0f - s));
}

// SiLU'(a) = s (1 + a (1 - s)), s = 1 / (1 + e^-a) = 1 / (1 + 2^(-a log2 e)),
// with the hardware exp2 and reciprocal (about 1 ulp each) in place of expf and
// a division; exp2 overflowing to inf gives s = 0, underflowing gives s = 1.
__device__ __forceinline__ float silu_grad(float a) {
  const float s = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-a * 1.44269504088896341f));
  return s * (1.0f + a * (1.0f - s));
}

}  // namespace resbm
