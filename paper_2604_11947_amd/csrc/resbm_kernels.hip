// HIP kernels of the ResBM boundary module for gfx950 and the C ABI around them.
//
// Paper: ResBM, Sec. 3.2 (encoder after the FFN, decoder before the next
// attention, only b crosses the boundary), Sec. 3.3 Eq. 5 (the identity path
// keeps columns [0, r) on the way down and zero-pads on the way up), App. A.3
// (bf16 payload).  The backward kernels are the adjoints of these maps.
//
// Work split (T tokens, hidden n, rank r; every streaming tensor is T x n):
//   encode_fwd  a = z W_e: a block owns a token tile; its waves split the
//               n-contraction and add their partial sums in LDS in wave order
//               before phi, the skip and the bf16 rounding.
//   decode_fwd  z~ = b W_d: waves own column strips (W_d held in registers) and
//               walk tokens, writing 64 contiguous bytes per row per store.
//   decode_bwd  one pass over g_z~ gives g_b (contraction over n; the 8 waves'
//               column partials meet in LDS, one barrier per 32-token step) and
//               dW_d (contraction over tokens, accumulated in registers); the
//               token-major tiles are read back transposed from LDS.
//   encode_bwd  one pass reads z and writes g_z; g_h = g_b phi'(a) comes from a
//               small prologue kernel in the two fragment orders the matrix cores
//               want; dW_e accumulates in registers and meets once per block.
// Every partial sum is added in a fixed order, so results are reproducible bit
// for bit.
//
// Streaming tensors are accessed through buffer descriptors: the hardware range
// check returns zeros for loads and drops stores outside a descriptor, so token
// tails and padding need no branches inside the loops, and every loop keeps two
// register sets in flight (the next step's loads are issued before the current
// step's math), which lets the compiler place each memory wait at its use.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "resbm.h"
#include "resbm_buffer.hpp"
#include "resbm_host.hpp"
#include "resbm_mfma.hpp"
#include "resbm_plan.hpp"

namespace resbm {

// ---------------------------------------------------------------- buffer access
constexpr int kEs = (int)sizeof(io_t);

// Cache policy of the T x n streams, read or written once per op: non-temporal
// loads, and non-temporal device-scope stores (streamed out instead of left
// dirty in the caches for the next kernel to write back).  Everything reused
// (weights, payload rows, partial sums) keeps the default policy.
// (gfx950 cache-policy operand bits: 1 = sc0, 2 = nt, 16 = sc1; measured on the
// four-op step: loads nt and stores nt|sc1 took it from ~196 to ~178 us, the
// gain being mostly the next kernel's reads no longer competing with
// write-backs of the previous kernel's output.)
#ifndef RESBM_LD_STREAM
#define RESBM_LD_STREAM 2   // nt
#endif
#ifndef RESBM_ST_STREAM
#define RESBM_ST_STREAM 18  // nt | sc1
#endif
constexpr int kLdStream = RESBM_LD_STREAM;
constexpr int kStStream = RESBM_ST_STREAM;

// Byte extent of rows [0, rows) of a row-major matrix with n used columns.
__device__ __forceinline__ int64_t rows_bytes(int64_t rows, int n, int64_t ld, int es) {
  return rows > 0 ? ((rows - 1) * ld + n) * es : 0;
}

// 8 consecutive I/O elements of a streamed T x n matrix at byte offset off.
__device__ __forceinline__ XFrag bld_x8(rsrc_t r, uint32_t off) {
  XFrag f;
#if RESBM_IO_F32_BUILD
  const uint4 a = bld16<kLdStream>(r, off), b = bld16<kLdStream>(r, off == kOOB ? kOOB : off + 16);
  f.v[0] = __builtin_bit_cast(float, a.x); f.v[1] = __builtin_bit_cast(float, a.y);
  f.v[2] = __builtin_bit_cast(float, a.z); f.v[3] = __builtin_bit_cast(float, a.w);
  f.v[4] = __builtin_bit_cast(float, b.x); f.v[5] = __builtin_bit_cast(float, b.y);
  f.v[6] = __builtin_bit_cast(float, b.z); f.v[7] = __builtin_bit_cast(float, b.w);
#else
  f.v = __builtin_bit_cast(bf16x8, bld16<kLdStream>(r, off));
#endif
  return f;
}

// 4 consecutive I/O elements at byte offset off, widened to float.
__device__ __forceinline__ void bld_x4(rsrc_t r, uint32_t off, float (&out)[4]) {
#if RESBM_IO_F32_BUILD
  const uint4 a = bld16(r, off);
  out[0] = __builtin_bit_cast(float, a.x); out[1] = __builtin_bit_cast(float, a.y);
  out[2] = __builtin_bit_cast(float, a.z); out[3] = __builtin_bit_cast(float, a.w);
#else
  const uint2 u = bld8(r, off);
  out[0] = bf16_bits_to_f32(u.x & 0xffffu);
  out[1] = bf16_bits_to_f32(u.x >> 16);
  out[2] = bf16_bits_to_f32(u.y & 0xffffu);
  out[3] = bf16_bits_to_f32(u.y >> 16);
#endif
}

// Rounds and stores CNT (4 or 8) consecutive values of a streamed T x n matrix
// at byte offset off.
template <int CNT>
__device__ __forceinline__ void bst_n(rsrc_t r, uint32_t off, const float* v) {
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int q = 0; q < CNT / 4; ++q)
    bst16<kStStream>(r, off == kOOB ? kOOB : off + 16 * q,
          make_uint4(__builtin_bit_cast(uint32_t, v[4 * q]), __builtin_bit_cast(uint32_t, v[4 * q + 1]),
                     __builtin_bit_cast(uint32_t, v[4 * q + 2]), __builtin_bit_cast(uint32_t, v[4 * q + 3])));
#else
  if constexpr (CNT == 8) {
    bf16x8 h;
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = to_bf16(v[e]);
    bst16<kStStream>(r, off, __builtin_bit_cast(uint4, h));
  } else {
    bf16x4 h;
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = to_bf16(v[e]);
    bst8<kStStream>(r, off, __builtin_bit_cast(uint2, h));
  }
#endif
}

// Stores 8 consecutive I/O elements read from LDS at src (16-byte aligned) into
// a streamed T x n matrix.
__device__ __forceinline__ void bst_x8(rsrc_t r, uint32_t off, const io_t* src) {
#if RESBM_IO_F32_BUILD
  bst16<kStStream>(r, off, *reinterpret_cast<const uint4*>(src));
  bst16<kStStream>(r, off == kOOB ? kOOB : off + 16, *reinterpret_cast<const uint4*>(src + 4));
#else
  bst16<kStStream>(r, off, *reinterpret_cast<const uint4*>(src));
#endif
}

// Stores the 8 elements of an exact fragment into a streamed T x n matrix.
__device__ __forceinline__ void bst_frag(rsrc_t r, uint32_t off, const XFrag& f) {
#if RESBM_IO_F32_BUILD
  bst16<kStStream>(r, off, make_uint4(__builtin_bit_cast(uint32_t, f.v[0]), __builtin_bit_cast(uint32_t, f.v[1]),
                           __builtin_bit_cast(uint32_t, f.v[2]), __builtin_bit_cast(uint32_t, f.v[3])));
  bst16<kStStream>(r, off == kOOB ? kOOB : off + 16,
        make_uint4(__builtin_bit_cast(uint32_t, f.v[4]), __builtin_bit_cast(uint32_t, f.v[5]),
                   __builtin_bit_cast(uint32_t, f.v[6]), __builtin_bit_cast(uint32_t, f.v[7])));
#else
  bst16<kStStream>(r, off, __builtin_bit_cast(uint4, f.v));
#endif
}

// 8 consecutive elements m[row][kb .. kb + 8) of a packed matrix with r columns
// (payload, wire gradient), zeros at columns >= r; r % 4 == 0, so a lane gets 8,
// 4 or 0 of them.  `row_off` is the row's byte offset in the descriptor (or kOOB).
// R8: the caller knows r % 8 == 0 (at compile time), so the 8 elements are in
// range together and one aligned 16-byte load fetches them.  A run-time test
// here would put a branch around the loads of the callers' loops.
template <bool R8 = false>
__device__ __forceinline__ XFrag bld_r8(rsrc_t m, uint32_t row_off, int r, int kb) {
  const bool lo = kb < r, hi = kb + 4 < r;
  const uint32_t olo = (row_off == kOOB || !lo) ? kOOB : row_off + kb * kEs;
  XFrag f;
#if RESBM_IO_F32_BUILD
  const uint32_t ohi = (row_off == kOOB || !hi) ? kOOB : row_off + (kb + 4) * kEs;
  const uint4 a = bld16(m, olo), b = bld16(m, ohi);
  f.v[0] = __builtin_bit_cast(float, a.x); f.v[1] = __builtin_bit_cast(float, a.y);
  f.v[2] = __builtin_bit_cast(float, a.z); f.v[3] = __builtin_bit_cast(float, a.w);
  f.v[4] = __builtin_bit_cast(float, b.x); f.v[5] = __builtin_bit_cast(float, b.y);
  f.v[6] = __builtin_bit_cast(float, b.z); f.v[7] = __builtin_bit_cast(float, b.w);
#else
  if constexpr (R8) {
    f.v = __builtin_bit_cast(bf16x8, bld16(m, olo));
  } else {
    const uint32_t ohi = (row_off == kOOB || !hi) ? kOOB : row_off + (kb + 4) * kEs;
    const uint2 a = bld8(m, olo), b = bld8(m, ohi);
    f.v = __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
  }
#endif
  return f;
}

// Split (weight-like) fragment f of a fragment-ordered buffer: per fragment and
// lane 2 x 16 bytes (hi, lo bf16 in the bf16 build; 8 floats in the f32 build).
__device__ __forceinline__ SFrag bld_sfrag(rsrc_t r, int64_t f, int l, bool ok = true) {
  SFrag s;
#if RESBM_IO_F32_BUILD
  const uint32_t o = ok ? (uint32_t)((f * 64 + l) * 32) : kOOB;
  const uint4 a = bld16(r, o), b = bld16(r, ok ? o + 16 : kOOB);
  s.v[0] = __builtin_bit_cast(float, a.x); s.v[1] = __builtin_bit_cast(float, a.y);
  s.v[2] = __builtin_bit_cast(float, a.z); s.v[3] = __builtin_bit_cast(float, a.w);
  s.v[4] = __builtin_bit_cast(float, b.x); s.v[5] = __builtin_bit_cast(float, b.y);
  s.v[6] = __builtin_bit_cast(float, b.z); s.v[7] = __builtin_bit_cast(float, b.w);
#else
  s.hi = __builtin_bit_cast(bf16x8, bld16(r, ok ? (uint32_t)(((f * 2 + 0) * 64 + l) * 16) : kOOB));
  s.lo = __builtin_bit_cast(bf16x8, bld16(r, ok ? (uint32_t)(((f * 2 + 1) * 64 + l) * 16) : kOOB));
#endif
  return s;
}
constexpr int kSFragBytes = 2048;  // one split fragment for the 64 lanes

__device__ __forceinline__ void store_sfrag(void* __restrict__ base, int64_t f, int l, const float (&w)[8]) {
#if RESBM_IO_F32_BUILD
  float4* out = reinterpret_cast<float4*>(base) + (f * 64 + l) * 2;
  out[0] = make_float4(w[0], w[1], w[2], w[3]);
  out[1] = make_float4(w[4], w[5], w[6], w[7]);
#else
  SFrag s = sfrag_from(w);
  uint4* out = reinterpret_cast<uint4*>(base);
  out[(f * 2 + 0) * 64 + l] = __builtin_bit_cast(uint4, s.hi);
  out[(f * 2 + 1) * 64 + l] = __builtin_bit_cast(uint4, s.lo);
#endif
}

// ---------------------------------------------------------------- LDS helpers
// Orders this wave's LDS accesses: waits for its outstanding LDS operations and
// keeps the compiler from moving memory accesses across.  Sufficient for LDS
// regions that only this wave touches.
__device__ __forceinline__ void wave_lds_fence() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Index of this wave in its block, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// The value v, opaque to the optimizer.  Used for the first index of the
// streaming loops, which start before their range on zeroed registers: the
// compiler then cannot peel the first iterations off the loop, which would
// leave it fewer memory operations in flight at the loop entry than the loop
// itself keeps, and so make it wait too early inside the loop.  32-bit on
// purpose: this toolchain encodes a negative 64-bit constant moved into a scalar
// register pair as a 32-bit literal, which the hardware zero-extends.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+s"(v));
  return v;
}

// Loads 8 consecutive elements at (row, col) of a WC-wide tile (col % 8 == 0).
template <int WC>
__device__ __forceinline__ XFrag tile_get8(const io_t* tile, int row, int col) {
  const io_t* p = tile + row * WC + tile_col<WC>(row, col);
  XFrag f;
#if RESBM_IO_F32_BUILD
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w; f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
#else
  f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
#endif
  return f;
}

// Stores 8 consecutive elements at (row, col) of a WC-wide tile (col % 8 == 0).
template <int WC>
__device__ __forceinline__ void tile_put8(io_t* tile, int row, int col, const XFrag& v) {
  io_t* d = tile + row * WC + tile_col<WC>(row, col);
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) d[e] = v.v[e];
#else
  *reinterpret_cast<uint4*>(d) = __builtin_bit_cast(uint4, v.v);
#endif
}

// Transposed fragment from a row-major 32 x WC tile in LDS: lane (row16, grp)
// receives tile[8 grp + e][c0 + row16], e = 0..7, i.e. the operand of a
// contraction over the 32 rows (tokens) of the tile.
// bf16: two ds_read_b64_tr_b16.  Within a 16-lane group that instruction hands
// lane i element i % 4 of the 8-byte chunks addressed by group lanes 4 e + i / 4,
// e = 0..3; so group lane j addresses row 8 grp + 4 h + j / 4, columns
// c0 + 4 (j % 4) .. + 3, and lane i collects 4 consecutive rows of column c0 + i.
template <int WC>
__device__ __forceinline__ XFrag tr_frag(const io_t* tile, int c0, int row16, int grp) {
  XFrag f;
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int row = 8 * grp + e;
    f.v[e] = tile[row * WC + tile_col<WC>(row, c0 + row16)];
  }
#else
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  s16x4 h[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int row = 8 * grp + 4 * q + (row16 >> 2);
    const io_t* p = tile + row * WC + tile_col<WC>(row, c0 + 4 * (row16 & 3));
    h[q] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  }
  f.v = __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){h[0][0], h[0][1], h[0][2], h[0][3],
                                                                               h[1][0], h[1][1], h[1][2], h[1][3]});
#endif
  return f;
}

// Transposed fragment from a block-wide tile (see wide_col): lane (row16, grp)
// receives tile[row0 + 8 grp + e][c0 + row16], e = 0..7 (addressed as tr_frag).
template <int WIDE>
__device__ __forceinline__ XFrag tr_frag_wide(const io_t* tile, int row0, int c0, int row16, int grp) {
  XFrag f;
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int row = row0 + 8 * grp + e;
    f.v[e] = tile[row * WIDE + wide_col(row, c0 + row16)];
  }
#else
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  s16x4 h[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int row = row0 + 8 * grp + 4 * q + (row16 >> 2);
    const io_t* p = tile + row * WIDE + wide_col(row, c0 + 4 * (row16 & 3));
    h[q] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  }
  f.v = __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){h[0][0], h[0][1], h[0][2], h[0][3],
                                                                               h[1][0], h[1][1], h[1][2], h[1][3]});
#endif
  return f;
}

// Output-column permutation of the "expand" contractions (decode_fwd, the g_z
// part of encode_bwd).  A wave's A operand covers 16*CT columns starting at c0;
// row i of column tile ct stands for column
//     c0 + 32 (ct / 2) + W grp + 4 (ct % 2) + i % 4,   grp = i / 4, W = 8 (CT >= 2) or 4,
// so that lane group grp ends up holding runs of W consecutive columns and the
// four lane groups of one token cover 4W contiguous columns per store.
template <int CT>
__device__ __forceinline__ int expand_col(int c0, int ct, int i) {
  constexpr int W = CT >= 2 ? 8 : 4;
  return c0 + 32 * (ct >> 1) + W * (i >> 2) + 4 * (ct & 1) + (i & 3);
}

// ============================================================ encode forward
// Fragment-ordered hi/lo copy of W_e for the A operand of a = z W_e:
// fragment f = ks * NT + nt, lane (row16, grp) holds W_e[32 ks + 8 grp + e][16 nt + row16].
// One wave per block, so that the few fragments spread over many compute units.
__global__ __launch_bounds__(64) void k_enc_fwd_prep(const float* __restrict__ W_e, int n, int r, int NT,
                                                     void* __restrict__ wf) {
  const int64_t gid = (int64_t)blockIdx.x * 64 + threadIdx.x;
  const int64_t total = (int64_t)(n / 32) * NT * 64;
  if (gid >= total) return;
  const int l = (int)(gid & 63);
  const int64_t f = gid >> 6;
  const int nt = (int)(f % NT);
  const int ks = (int)(f / NT);
  const int col = nt * 16 + (l & 15);
  const int grp = l >> 4;
  float w[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int k = ks * 32 + grp * 8 + e;
    w[e] = col < r ? W_e[(int64_t)k * r + col] : 0.0f;
  }
  store_sfrag(wf, f, l, w);
}

// a = z W_e for 16*MT tokens per block.  A stage covers KW * SC columns of the
// n-contraction: the block loads its TOK x (KW SC) tile cooperatively, whole
// row segments per load instruction (1 KiB at r <= 32), into a block-wide LDS
// tile; after the stage's barrier wave w contracts columns [w SC, (w + 1) SC)
// of it, with the W_e fragments of those rows from the prologue kernel.
template <int NT, int MT, int KW>
__global__ __launch_bounds__(KW * 64) void k_enc_fwd(int64_t T, int n, int r, int act,
                                                     const io_t* __restrict__ x_attn, int64_t ld_x,
                                                     const io_t* __restrict__ z, int64_t ld_z,
                                                     const void* __restrict__ wf, const float* __restrict__ W_e,
                                                     io_t* __restrict__ b, float* __restrict__ a_save) {
  constexpr int U = ef_u(NT);           // k-steps per wave and stage
  constexpr bool PW = NT <= 4;          // W_e fragments travel with the stage
  constexpr int NW = PW ? NT : 1;
  constexpr bool WL = ef_we_lds(NT);    // W_e split in the kernel, through LDS (no fragments in wf)
  constexpr int TOK = 16 * MT;
  constexpr int RPT = 16 * NT;
  constexpr int SC = 32 * U;            // z columns per wave and stage
  constexpr int BC = KW * SC;           // z columns per stage (tile row)
  constexpr int LPR = BC / 8;           // lanes per tile row in the cooperative loads
  constexpr int NQ = TOK * LPR / (64 * KW);  // cooperative loads per lane per stage
  constexpr int ZB = RESBM_IO_F32_BUILD ? 1 : 2;  // tile buffers
  constexpr int TILE = TOK * BC * (int)sizeof(io_t);
  constexpr int RED = KW * TOK * (RPT + 4) * 4;
  static_assert(TOK * LPR % (64 * KW) == 0, "tile rows must split evenly over the waves");
  __shared__ __attribute__((aligned(16))) char smem[ZB * TILE > RED ? ZB * TILE : RED];

  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
  const int64_t tok0 = (int64_t)blockIdx.x * TOK;
  const int nks = n / 32;
  const int nst = (n + BC - 1) / BC;  // stages

  // rows at or beyond T fall outside the descriptor (ld >= n)
  const rsrc_t zr = make_rsrc(z + tok0 * ld_z, rows_bytes(min((int64_t)TOK, T - tok0), n, ld_z, kEs));
  const rsrc_t wr = make_rsrc(WL ? nullptr : wf, WL ? 0 : (int64_t)nks * NT * kSFragBytes);
  // WL: wave w's rows [w SC, (w + 1) SC) of the stage's W_e slice, float32, 16
  // bytes per lane and load (WLL lanes per row), split into hi / lo planes of
  // its own LDS region [SC][RPT] (tile_col layout) and read back transposed.
  // Stage i + 1's rows are split while stage i is multiplied (two plane
  // buffers per wave), and loaded two stages before they are split.
  constexpr int WLL = RPT / 4, WRPI = 64 / WLL, WQ = WL ? SC * RPT / 256 : 1;
  constexpr int WPL = SC * RPT;  // elements of one plane
  static_assert(!WL || (RPT % 4 == 0 && 64 % WLL == 0 && SC % WRPI == 0), "W_e rows must split over the lanes");
  __shared__ __attribute__((aligned(16))) __bf16 s_w[WL ? KW * 4 * WPL : 8];
  const rsrc_t we = make_rsrc(W_e, WL ? (int64_t)n * r * 4 : 0);
  // cooperative load q of this lane: tile row zrow[q], columns zc .. zc + 8 of the stage
  const int zc = 8 * (l % LPR);
  int zrow[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) zrow[q] = (wave * NQ * 64 + q * 64 + l) / LPR;

  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Blocks start at different stages (rotating through all of them), so that
  // concurrently running blocks read different column ranges.  Consecutive
  // blocks go to the 8 XCDs in turn, so the rotation steps every 8 blocks: the
  // blocks sharing an XCD start at different stages (stepping with every block
  // put all of an XCD's blocks on one column range; 2-3 us slower).  Stages
  // before 0 or past the last load zeros and add nothing.
  const int srot = (int)((blockIdx.x / 8u) % (unsigned)nst);
  auto stage_col = [&](int i) {  // first column of stage i, or n outside [0, nst)
    if (i < 0 || i >= nst) return n;
    const int ir = i + srot < nst ? i + srot : i + srot - nst;
    return ir * BC;
  };
  auto load_z = [&](XFrag (&zz)[NQ], int i) {
    const int c = stage_col(i) + zc;
#pragma unroll
    for (int q = 0; q < NQ; ++q) zz[q] = bld_x8(zr, c < n ? (uint32_t)((zrow[q] * ld_z + c) * kEs) : kOOB);
  };
  auto load_w = [&](SFrag (&ww)[U][NW], int i) {
    if constexpr (PW) {
      const int ks = (stage_col(i) + wave * SC) / 32;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) ww[u][nt] = bld_sfrag(wr, (int64_t)(ks + u) * NT + nt, l, ks + u < nks);
    }
  };

  auto load_wq = [&](uint4 (&qq)[WQ], int i) {
    if constexpr (WL) {
      const int c0 = stage_col(i) + wave * SC;  // n (all zeros) outside the stages
      const int col = 4 * (l % WLL);
#pragma unroll
      for (int q = 0; q < WQ; ++q) {
        const int row = q * WRPI + l / WLL;
        const bool ok = c0 + row < n && col < r;
        qq[q] = bld16(we, ok ? (uint32_t)(((c0 + row) * r + col) * 4) : kOOB);
      }
    }
  };
  // fragment (u, nt) of this wave's planes: lane (row16, grp) gets rows
  // 32 u + 8 grp + e of column 16 nt + row16 (two transposed 8-byte reads)
  auto wl_frag = [&](const __bf16* plane, int u, int nt) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    s16x4 h[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int row = 32 * u + 8 * grp + 4 * q + (row16 >> 2);
      const __bf16* pp = plane + row * RPT + tile_col<RPT>(row, 16 * nt + 4 * (row16 & 3));
      h[q] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pp));
    }
    return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){h[0][0], h[0][1], h[0][2], h[0][3],
                                                                                 h[1][0], h[1][1], h[1][2], h[1][3]});
  };

  // this wave's hi plane of stage i's buffer (the lo plane follows it)
  auto wl_plane = [&](int i) { return s_w + (WL ? (wave * 4 + 2 * (i & 1)) * WPL : 0); };
  // split the W_e rows in qq (stage i) into this wave's planes of stage i
  auto wl_split = [&](const uint4 (&qq)[WQ], int i) {
    __bf16* const ph = wl_plane(i);
    __bf16* const pl = ph + WPL;
    const int col = 4 * (l % WLL);
#pragma unroll
    for (int q = 0; q < WQ; ++q) {
      const int row = q * WRPI + l / WLL;
      const uint4 v = qq[q];
      const float f4[4] = {__builtin_bit_cast(float, v.x), __builtin_bit_cast(float, v.y),
                           __builtin_bit_cast(float, v.z), __builtin_bit_cast(float, v.w)};
      bf16x4 h, lo;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        __bf16 a, c;
        split_hi_lo(f4[e], a, c);
        h[e] = a;
        lo[e] = c;
      }
      const int pos = row * RPT + tile_col<RPT>(row, col);
      *reinterpret_cast<uint2*>(ph + pos) = __builtin_bit_cast(uint2, h);
      *reinterpret_cast<uint2*>(pl + pos) = __builtin_bit_cast(uint2, lo);
    }
  };

  // One stage; zz / ww are reloaded with the z rows / W_e fragments of stage
  // i + 2; WL: qn holds stage i + 1's W_e rows, split here and reloaded with
  // stage i + 3's.
  auto body = [&](XFrag (&zz)[NQ], SFrag (&ww)[U][NW], uint4 (&qn)[WQ], int i) {
    io_t* tile = reinterpret_cast<io_t*>(smem + (ZB == 2 ? (i & 1) : 0) * TILE);
    if constexpr (ZB == 1) __syncthreads();  // the previous stage's readers of the single tile are done
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      io_t* d = tile + zrow[q] * BC + wide_col(zrow[q], zc);
#if RESBM_IO_F32_BUILD
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = zz[q].v[e];
#else
      *reinterpret_cast<uint4*>(d) = __builtin_bit_cast(uint4, zz[q].v);
#endif
    }
    load_z(zz, i + 2);
    __syncthreads();  // the stage's tile is complete; the other buffer's readers are done
    const int ks = (stage_col(i) + wave * SC) / 32;
    const __bf16* const ph = wl_plane(i);  // written by this wave during stage i - 1
    const __bf16* const pl = ph + WPL;
    // fp32 build: the stage's products go to a zeroed partial added to the
    // total afterwards (n / 4 products of K = 4 would otherwise round as one
    // chain); the bf16 build accumulates directly
    constexpr bool PART = RESBM_IO_F32_BUILD;
    f32x4 part[PART ? MT : 1][PART ? NT : 1];
    if constexpr (PART) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) part[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      XFrag f[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int row = 16 * mt + row16;
        const io_t* p = tile + row * BC + wide_col(row, wave * SC + 32 * u + 8 * grp);
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) f[mt].v[e] = p[e];
#else
        f[mt].v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
#endif
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        SFrag w;
        if constexpr (WL) {
#if !RESBM_IO_F32_BUILD
          w.hi = wl_frag(ph, u, nt);
          w.lo = wl_frag(pl, u, nt);
#endif
        } else if constexpr (PW) {
          w = ww[u][nt];
        } else {
          w = bld_sfrag(wr, (int64_t)(ks + u) * NT + nt, l, ks + u < nks);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          if constexpr (PART) part[mt][nt] = mma_sx(w, f[mt], part[mt][nt]);
          else acc[mt][nt] = mma_sx(w, f[mt], acc[mt][nt]);
        }
      }
    }
    if constexpr (PART) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] += part[mt][nt];
    }
    if constexpr (WL) {
      wl_split(qn, i + 1);
      load_wq(qn, i + 3);
      wave_lds_fence();  // stage i + 1's planes are written before this wave reads them
    } else {
      load_w(ww, i + 2);
    }
  };

  // Every memory operation sits in one unconditional loop body (the loop starts
  // two stages early on zeroed registers instead of after a prologue of loads),
  // which lets the compiler place each wait at its exact distance.
  XFrag za[NQ], zb[NQ];
  SFrag wa[U][NW], wb[U][NW];
  uint4 qa[WQ], qb[WQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) za[q] = zb[q] = xfrag_zero();
#pragma unroll
  for (int q = 0; q < WQ; ++q) qa[q] = qb[q] = make_uint4(0, 0, 0, 0);
  if constexpr (PW && !WL) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) wa[u][nt] = wb[u][nt] = sfrag_zero();
  }
  if constexpr (WL) {
    wl_split(qa, -2);  // zeros: stage -2 multiplies its planes with a zero tile (no stale LDS bits)
    load_wq(qa, 0);    // stage 0's rows, split during stage -1
  }
  for (int i = opaque(-2); i < nst; i += 2) {
    body(za, wa, qb, i);
    body(zb, wb, qa, i + 1);
  }
  __syncthreads();  // the reduction area overlaps the tiles
  float (*s_red)[TOK][RPT + 4] = reinterpret_cast<float (*)[TOK][RPT + 4]>(smem);

  // acc[mt][nt][v] = partial a[tok0 + 16 mt + row16][16 nt + 4 grp + v]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      *reinterpret_cast<float4*>(&s_red[wave][16 * mt + row16][16 * nt + 4 * grp]) =
          make_float4(acc[mt][nt][0], acc[mt][nt][1], acc[mt][nt][2], acc[mt][nt][3]);
  __syncthreads();

  // Sum the KW partials in wave order, then a_save = a, b = x_attn[:, :r] + phi(a).
  constexpr int Q = RPT / 4;
  for (int idx = threadIdx.x; idx < TOK * Q; idx += KW * 64) {
    const int tt = idx / Q;
    const int j0 = (idx % Q) * 4;
    const int64_t t = tok0 + tt;
    if (t >= T || j0 >= r) continue;
    float a[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < KW; ++w) {
      const float4 p = *reinterpret_cast<const float4*>(&s_red[w][tt][j0]);
      a[0] += p.x; a[1] += p.y; a[2] += p.z; a[3] += p.w;
    }
    if (a_save) *reinterpret_cast<float4*>(a_save + t * r + j0) = make_float4(a[0], a[1], a[2], a[3]);
    float x[4];
    load_x4(x_attn + t * ld_x + j0, x);
    float o[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) o[v] = x[v] + act_phi(a[v], act);
    store_x4(b + t * r + j0, o);
  }
}

// sum_{c < cnt} p[c stride .. + 4), added in order of c; the loads of eight
// terms are issued together.
__device__ __forceinline__ float4 sum_ordered4(const float* __restrict__ p, int64_t stride, int cnt) {
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int c0 = 0; c0 < cnt; c0 += 8) {
    float4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      v[k] = c0 + k < cnt ? *reinterpret_cast<const float4*>(p + (int64_t)(c0 + k) * stride)
                          : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      s.x += v[k].x; s.y += v[k].y; s.z += v[k].z; s.w += v[k].w;
    }
  }
  return s;
}

// ============================================================ decode backward
// One pass over g_z~ for the token range [tg TB, ...), columns [cg 512, cg 512 + 512)
// and j-tiles [16 jt0, 16 (jt0 + JT)) of r:
//   gbp[cg][t][j] = sum over the block's columns of g_z~[t][c] W_d[j][c]
//   dwp[tg][j][c] = sum over the block's tokens of b[t][j] g_z~[t][c]
// Per 32-token step the block loads its 32 x 512 tile of g_z~ cooperatively,
// one 1 KiB row segment per load instruction (wave w: rows 4 w .. 4 w + 3, two
// steps ahead), into a block-wide LDS tile; after the step's barrier each wave
// reads its 64 columns back in fragment order for its g_b partial (W_d held in
// registers) and transposed for dW_d.  The payload rows of a step are staged
// once per block.  The 8 waves' g_b partials of a step are added in wave order
// behind the next step's barrier.
// Position of float [row][j] (j % 4 == 0) in a 32-row tile of JW-float rows of
// partial sums, written as 16-byte pieces by lane (row16, grp) at row 16 th +
// row16, chunk 4 jt + grp (8-lane write groups: 8 rows, one chunk) and read
// back row by row (consecutive lanes on consecutive chunks).  With 4, 8 or 16
// chunks per row the chunk index is XORed with (row / 2) % 4, row % 8 or row % 8,
// which puts both patterns on distinct banks; other widths pad rows by 4 floats.
template <int JW>
__device__ __forceinline__ int gb_pos(int row, int j) {
  constexpr int C = JW / 4;
  if constexpr (C == 4) {
    return row * JW + (((j >> 2) ^ ((row >> 1) & 3)) << 2);
  } else if constexpr (C == 8 || C == 16) {
    return row * JW + (((j >> 2) ^ (row & 7)) << 2);
  } else {
    return row * (JW + 4) + j;
  }
}
template <int JW>
constexpr int gb_rowsz() { return (JW == 16 || JW == 32 || JW == 64) ? JW : JW + 4; }

template <int JT>
__global__ __launch_bounds__(kDbWaves * 64) void k_dec_bwd(int64_t T, int n, int r, int RP,
                                                           const io_t* __restrict__ b,
                                                           const float* __restrict__ W_d,
                                                           const io_t* __restrict__ g_zt, int64_t ld_g,
                                                           float* __restrict__ gbp, float* __restrict__ dwp,
                                                           int TB) {
  constexpr int KSW = kDbWC / 32;  // 32-column steps per wave
  constexpr int CTW = kDbWC / 16;  // 16-column tiles per wave
  constexpr int BW = kDbWaves * kDbWC;  // block columns (one 1 KiB bf16 row segment)
  constexpr int JW = JT * 16;      // j values per pass
  constexpr int NBUF = JT <= 2 ? 2 : 1;                 // g_b partial buffers
  constexpr int GZB = RESBM_IO_F32_BUILD ? 1 : 2;       // g_z~ tile buffers
  constexpr int BQ = JW / 8;       // 16-byte payload chunks per token row
  constexpr int RPW = 32 / kDbWaves;  // tile rows loaded per wave
  __shared__ __attribute__((aligned(16))) io_t s_gz[GZB][32 * BW];
  __shared__ __attribute__((aligned(16))) io_t s_b[2][32 * JW];
  __shared__ __attribute__((aligned(16))) float s_gb[NBUF][kDbWaves][32 * gb_rowsz<JW>()];

  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
#if RESBM_XCD_SPREAD
  const int tg = blockIdx.x, cg = blockIdx.y;  // token groups vary fastest: every XCD sees every column group
#else
  const int cg = blockIdx.x, tg = blockIdx.y;
#endif
  const int jt0 = blockIdx.z * JT;
  const int bc0 = cg * BW;
  const int wc0 = bc0 + wave * kDbWC;
  const bool won = wc0 < n;  // n % 64 == 0: a wave's columns lie in [0, n) in whole runs of 64

  // W_d as the A operand of g_b: lane (row16, grp) holds W_d[16 (jt0 + jt) + row16][wc0 + 32 ks + 8 grp + e].
  SFrag wdf[JT][KSW];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt)
#pragma unroll
    for (int ks = 0; ks < KSW; ++ks) {
      const int j = 16 * (jt0 + jt) + row16;
      float w[8];
      if (wc0 + 32 * ks + 8 * grp < n && j < r) {
        const float4* p = reinterpret_cast<const float4*>(W_d + (int64_t)j * n + wc0 + 32 * ks + 8 * grp);
        const float4 a = p[0], c = p[1];
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w; w[4] = c.x; w[5] = c.y; w[6] = c.z; w[7] = c.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) w[e] = 0.0f;
      }
      wdf[jt][ks] = sfrag_from(w);
    }

  f32x4 dw[CTW][JT];
#pragma unroll
  for (int ct = 0; ct < CTW; ++ct)
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) dw[ct][jt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t t_begin = (int64_t)tg * TB;
  const int64_t t_end = min(T, t_begin + TB);

  // payload rows of one step: threads [0, 32 BQ) each carry one 16-byte chunk
  const bool bthr = threadIdx.x < 32 * BQ;
  const int btt = bthr ? threadIdx.x / BQ : 0, bch = threadIdx.x % BQ;
  // g_z~ loads: lane l takes columns bc0 + 8 l .. + 8 of rows RPW wave + q (outside [0, n): zeros)
  const bool lon = bc0 + 8 * l < n;
  const uint32_t gz_lane = (uint32_t)((RPW * wave * ld_g + bc0 + 8 * l) * kEs);

  // Registers of step s: its tile rows and the payload rows of step s + 1.
  // Steps before 0 or past the range read zeros and store nothing.
  struct Step {
    XFrag gz[RPW];
    XFrag bp;
  };
  auto load_gz = [&](Step& st, int64_t s) {
    const int64_t t0 = t_begin + 32 * s;
    const int64_t rows = s < 0 ? 0 : min((int64_t)32, t_end - t0);
    const rsrc_t gr = make_rsrc(g_zt + t0 * ld_g, rows_bytes(rows, n, ld_g, kEs));
#pragma unroll
    for (int q = 0; q < RPW; ++q)
      st.gz[q] = bld_x8(gr, lon ? gz_lane + (uint32_t)(q * ld_g * kEs) : kOOB);
  };
  auto load_bp = [&](Step& st, int64_t s) {
    const int64_t t0 = t_begin + 32 * s;
    const int64_t rows1 = s + 1 < 0 ? 0 : min((int64_t)32, t_end - t0 - 32);
    const rsrc_t br = make_rsrc(b + (t0 + 32) * r, rows1 > 0 ? rows1 * r * kEs : 0);
    st.bp = bld_r8(br, bthr ? (uint32_t)(btt * r * kEs) : kOOB, r, 16 * jt0 + 8 * bch);
  };

  // One 32-token step; `st` is reloaded with the registers of step s + 2.
  auto body = [&](Step& st, int64_t s) {
    const int tb = GZB == 2 ? (int)(s & 1) : 0;
    const int gcur = NBUF == 2 ? (int)(s & 1) : 0, gprev = NBUF == 2 ? (int)((s + 1) & 1) : 0;
    io_t* tile = s_gz[tb];
    if constexpr (GZB == 1) __syncthreads();  // the previous step's readers of the single tile are done
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      const int row = RPW * wave + q;
      io_t* d = tile + row * BW + wide_col(row, 8 * l);
#if RESBM_IO_F32_BUILD
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = st.gz[q].v[e];
#else
      *reinterpret_cast<uint4*>(d) = __builtin_bit_cast(uint4, st.gz[q].v);
#endif
    }
    load_gz(st, s + 2);  // in flight across the barrier
    __syncthreads();  // the step's tile, its payload rows and the previous step's partials are complete
    // the next step's payload rows go to the other buffer (its readers passed this barrier)
    if (bthr) tile_put8<JW>(s_b[(s + 1) & 1], btt, 8 * bch, st.bp);
    load_bp(st, s + 2);
    // add the previous step's 8 partials of g_b in wave order; rows outside the range are dropped
    {
      const int64_t t0 = t_begin + 32 * (s - 1);
      const rsrc_t pr = make_rsrc(gbp + ((int64_t)cg * T + t0) * RP, s - 1 < 0 ? 0 : (t_end - t0) * RP * 4);
      // four consecutive j per thread (r % 4 == 0: all four in range or none)
#pragma unroll
      for (int idx0 = 0; idx0 < 32 * JW / 4; idx0 += kDbWaves * 64) {
        const int idx = idx0 + threadIdx.x;
        const int tt = idx / (JW / 4), jj = 4 * (idx % (JW / 4));
        const int j = 16 * jt0 + jj;
        if (32 * JW / 4 % (kDbWaves * 64) == 0 || idx < 32 * JW / 4) {
          float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int w = 0; w < kDbWaves; ++w) {
            const float4 p = *reinterpret_cast<const float4*>(&s_gb[gprev][w][gb_pos<JW>(tt, jj)]);
            v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
          }
          bst16(pr, j < r ? (uint32_t)((tt * RP + j) * 4) : kOOB,
                make_uint4(__builtin_bit_cast(uint32_t, v.x), __builtin_bit_cast(uint32_t, v.y),
                           __builtin_bit_cast(uint32_t, v.z), __builtin_bit_cast(uint32_t, v.w)));
        }
      }
    }
    if constexpr (NBUF == 1) __syncthreads();  // the single partial buffer is refilled below
    // g_b partial over this wave's 64 columns: D[j][t], B = g_z~ rows in fragment order
#pragma unroll
    for (int th = 0; th < 2; ++th) {
      XFrag f[KSW];
#pragma unroll
      for (int ks = 0; ks < KSW; ++ks) {
        const int row = 16 * th + row16;
        const io_t* p = tile + row * BW + wide_col(row, wave * kDbWC + 32 * ks + 8 * grp);
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) f[ks].v[e] = p[e];
#else
        f[ks].v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
#endif
      }
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks) acc = mma_sx(wdf[jt][ks], f[ks], acc);
        *reinterpret_cast<float4*>(&s_gb[gcur][wave][gb_pos<JW>(16 * th + row16, 16 * jt + 4 * grp)]) =
            make_float4(acc[0], acc[1], acc[2], acc[3]);
      }
    }
    // dW_d: D[c][j] = sum_t g_z~[t][c] b[t][j], A = g_z~^T, B = b^T (both transposed from LDS)
    XFrag bt[JT];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) bt[jt] = tr_frag<JW>(s_b[s & 1], 16 * jt, row16, grp);
#pragma unroll
    for (int ct = 0; ct < CTW; ++ct) {
      const XFrag a = tr_frag_wide<BW>(tile, 0, wave * kDbWC + 16 * ct, row16, grp);
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) dw[ct][jt] = mma_xx(a, bt[jt], dw[ct][jt]);
    }
  };

  // Every memory operation sits in one unconditional loop body: the loop starts
  // three (empty) steps early on zeroed registers instead of after a prologue of
  // loads, so the compiler can place each wait at its exact distance, and runs
  // one step past the range to add the last step's partials.  Step -1 stages
  // the payload rows of step 0.
  const int64_t nsteps = (t_end - t_begin + 31) / 32;
  // The first (empty) step reads payload buffer 1 before any step has filled
  // it; LDS starts with whatever the previous kernel left, and a NaN or Inf
  // there would survive the product with the zero tile.  Both buffers start at
  // zero (ordered before those reads by the first step's barrier).
  for (int i = threadIdx.x; i < (int)(sizeof(s_b) / 16); i += kDbWaves * 64)
    reinterpret_cast<uint4*>(&s_b[0][0])[i] = make_uint4(0, 0, 0, 0);
  Step sa, sb;
#pragma unroll
  for (int q = 0; q < RPW; ++q) sa.gz[q] = sb.gz[q] = xfrag_zero();
  sa.bp = sb.bp = xfrag_zero();
  for (int64_t s = opaque(-3); s <= nsteps; s += 2) {
    body(sb, s);      // odd steps
    body(sa, s + 1);  // even steps
  }

  // dw[ct][jt][v] = dW_d partial [16 (jt0 + jt) + row16][wc0 + 16 ct + 4 grp + v]
  if (won) {
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const int j = 16 * (jt0 + jt) + row16;
      if (j >= r) continue;
#pragma unroll
      for (int ct = 0; ct < CTW; ++ct)
        if (wc0 + 16 * ct < n)
          *reinterpret_cast<float4*>(dwp + ((int64_t)tg * RP + j) * n + wc0 + 16 * ct + 4 * grp) =
              make_float4(dw[ct][jt][0], dw[ct][jt][1], dw[ct][jt][2], dw[ct][jt][3]);
    }
  }
}

// Blocks [0, nb_gb): g_b = sum_cg gbp[cg] + g_id[:, :r], rounded once.
// Blocks [nb_gb, ...): dW_d (+)= sum_tg dwp[tg]; a block covers 64 four-column
// groups, its 4 thread quarters sum consecutive quarters of the token groups and
// the quarters are added in order.
__global__ __launch_bounds__(256) void k_dec_bwd_fin(int64_t T, int n, int r, int RP,
                                                     const float* __restrict__ gbp, int ncg,
                                                     const io_t* __restrict__ g_id, int64_t ld_gid,
                                                     io_t* __restrict__ g_b,
                                                     const float* __restrict__ dwp, int ntg,
                                                     float* __restrict__ dW_d, int accumulate,
                                                     int64_t nb_gb) {
  __shared__ float4 s_q[4][64];
  if ((int64_t)blockIdx.x < nb_gb) {
    const int nq = r / 4;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (gid >= T * nq) return;
    const int64_t t = gid / nq;
    const int j0 = (int)(gid % nq) * 4;
    const float4 p = sum_ordered4(gbp + t * RP + j0, T * RP, ncg);
    float s[4] = {p.x, p.y, p.z, p.w};
    if (g_id) {
      float x[4];
      load_x4(g_id + t * ld_gid + j0, x);
#pragma unroll
      for (int v = 0; v < 4; ++v) s[v] += x[v];
    }
    store_x4(g_b + t * r + j0, s);
    return;
  }
  const int nq = n / 4;
  const int q = threadIdx.x >> 6;
  const int64_t cidx = ((int64_t)blockIdx.x - nb_gb) * 64 + (threadIdx.x & 63);
  const bool ok = cidx < (int64_t)r * nq;
  const int j = ok ? (int)(cidx / nq) : 0;
  const int c0 = ok ? (int)(cidx % nq) * 4 : 0;
  const int g0 = q * ntg / 4, g1 = (q + 1) * ntg / 4;
  const float4 acc = ok ? sum_ordered4(dwp + ((int64_t)g0 * RP + j) * n + c0, (int64_t)RP * n, g1 - g0)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
  s_q[q][threadIdx.x & 63] = acc;
  __syncthreads();
  if (q == 0 && ok) {
    float4 s = accumulate ? *reinterpret_cast<const float4*>(dW_d + (int64_t)j * n + c0)
                          : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 tot = s_q[0][threadIdx.x];
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      const float4 p = s_q[k][threadIdx.x];
      tot.x += p.x; tot.y += p.y; tot.z += p.z; tot.w += p.w;
    }
    s.x += tot.x; s.y += tot.y; s.z += tot.z; s.w += tot.w;
    *reinterpret_cast<float4*>(dW_d + (int64_t)j * n + c0) = s;
  }
}

// ============================================================ encode backward
// Two streams, one kernel each: k_enc_bwd reads z for dW_e, k_expand (GZ)
// writes g_z; a read-only and a write-only pass each run closer to their own
// bandwidth ceilings than one pass that does both.
//
// k_enc_bwd: a block has CW x TW waves.  Wave (cw, tw) owns the 16 CT columns
// starting at bc0 + cw 16 CT and, in every block step of 32 TW tokens, the 32
// tokens starting at t0 + 32 tw.  Per block step:
//   1. the block forms g_h = g_b phi'(a) for the step's tokens in LDS, in split
//      form, with zeros in the columns r .. 32 KS (each column block also writes
//      its share of the rows out, split, for k_expand),
//   2. the block loads the step's 32 TW x 16 CT CW tile of z cooperatively,
//      whole row segments per load instruction, into a double-buffered LDS tile,
//   3. dW_e[c][j] += sum_t z[t][c] g_h[t][j]: A = g_h^T and B = z^T, both read
//      transposed from LDS, accumulated in registers over the token group.
// One barrier per step covers the tile and g_h.  The TW partial dW_e of a
// column slice are added in LDS in wave order; the finishing blocks add the
// token groups in order.

// Row pitch (elements) of a staged [rows][KP] plane of 16-bit values that is
// read transposed: KP itself where lds_col has a layout for it, else KP + 8
// (the padding moves consecutive rows to different banks).
constexpr int plane_pitch(int KP) { return (KP % 128 == 0 || KP == 32 || KP == 64) ? KP : KP + 8; }

// LDS of one block (gfx950: 160 KiB per compute unit).
constexpr int kLdsBytes = 160 * 1024;
// k_tokc_wide: pitch of its staged r-wide planes, and the tokens per step
// (32 TSM) it takes: 64 where two buffers of the 64-token tiles fit in LDS.
constexpr int tw_ypitch(int NT) {
  return RESBM_IO_F32_BUILD ? 32 * ((NT + 1) / 2) + 8 : plane_pitch(32 * ((NT + 1) / 2));
}
constexpr int tw_lds(int NT, bool DWD, int tsm) {
  const int planes = (!DWD && !RESBM_IO_F32_BUILD) ? 2 : 1;
  return 2 * (32 * tsm * 128 + planes * 32 * tsm * tw_ypitch(NT)) * (int)sizeof(io_t);
}
constexpr int tw_tsm(int NT, bool DWD) {
  return (RESBM_TW_TSM >= 4 && tw_lds(NT, DWD, 4) <= kLdsBytes)   ? 4
         : (RESBM_TW_TSM >= 2 && tw_lds(NT, DWD, 2) <= kLdsBytes) ? 2
                                                                   : 1;
}

// Split g_h tile of TS tokens x RPS columns: bf16 build: hi and lo planes in
// the lds_col<RPS> layout; f32 build: one float plane, row-major.
template <int TS, int RPS>
struct GhTile {
#if RESBM_IO_F32_BUILD
  float v[TS][RPS];
#else
  __bf16 hi[TS][RPS];
  __bf16 lo[TS][RPS];
#endif
};

template <int TS, int RPS>
__device__ __forceinline__ void gh_put4(GhTile<TS, RPS>& t, int row, int col, const float (&g)[4]) {
#if RESBM_IO_F32_BUILD
  *reinterpret_cast<float4*>(&t.v[row][col]) = make_float4(g[0], g[1], g[2], g[3]);
#else
  bf16x4 h, l;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    __bf16 a, b;
    split_hi_lo(g[e], a, b);
    h[e] = a;
    l[e] = b;
  }
  const int c = lds_col<RPS>(row, col);  // col % 4 == 0: the four stay in one chunk
  *reinterpret_cast<uint2*>(&t.hi[row][c]) = __builtin_bit_cast(uint2, h);
  *reinterpret_cast<uint2*>(&t.lo[row][c]) = __builtin_bit_cast(uint2, l);
#endif
}

// Transposed 16-bit fragment from a plane with PITCH elements per row in the
// lds_col<PITCH> layout: lane (row16, grp) receives plane[row0 + 8 grp + e][c0 + row16],
// e = 0..7 (two ds_read_b64_tr_b16, addressed as in tr_frag).
template <int PITCH>
__device__ __forceinline__ bf16x8 tr_plane(const __bf16* plane, int row0, int c0, int row16, int grp) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  s16x4 h[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int row = row0 + 8 * grp + 4 * q + (row16 >> 2);
    const __bf16* p = plane + row * PITCH + lds_col<PITCH>(row, c0 + 4 * (row16 & 3));
    h[q] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  }
  return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){h[0][0], h[0][1], h[0][2], h[0][3],
                                                                               h[1][0], h[1][1], h[1][2], h[1][3]});
}

// g_h[row0 + 8 grp + e][c0 + row16] as the A operand of dW_e (k = t).
template <int TS, int RPS>
__device__ __forceinline__ SFrag gh_tr(const GhTile<TS, RPS>& t, int row0, int c0, int row16, int grp) {
  SFrag f;
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) f.v[e] = t.v[row0 + 8 * grp + e][c0 + row16];
#else
  f.hi = tr_plane<RPS>(&t.hi[0][0], row0, c0, row16, grp);
  f.lo = tr_plane<RPS>(&t.lo[0][0], row0, c0, row16, grp);
#endif
  return f;
}

template <int KS, int NT, int CT, int CW, int TW>
__global__ __launch_bounds__(CW * TW * 64) void k_enc_bwd(int64_t T, int n, int r, int RP, int silu,
                                                          const io_t* __restrict__ z, int64_t ld_z,
                                                          const float* __restrict__ a_save,
                                                          const io_t* __restrict__ g_b, io_t* __restrict__ gh_hi,
                                                          io_t* __restrict__ gh_lo, float* __restrict__ dwp,
                                                          int TB) {
  constexpr int EW = CW * TW, NTH = EW * 64;
  constexpr int WC = 16 * CT, BC = CW * WC;
  constexpr int TS = 32 * TW;
  constexpr int KP = 32 * KS, RPT = 16 * NT, RPS = RESBM_IO_F32_BUILD ? KP + 8 : plane_pitch(KP);
  constexpr int GQ = TS * KP / 4;          // 4-column chunks of the g_h tile
  constexpr int NCH = (GQ + NTH - 1) / NTH;
  constexpr int GH_BYTES = (int)sizeof(GhTile<TS, RPS>);
  constexpr int Z_BYTES = TS * BC * (int)sizeof(io_t);  // block tile of one step
  constexpr int MAIN_LDS = 2 * GH_BYTES + 2 * Z_BYTES;
  constexpr int LPR = BC / 8;                 // lanes per tile row
  constexpr int NQ = TS * LPR / NTH;          // cooperative loads per lane and step
  static_assert(TS * LPR % NTH == 0 && 64 % LPR == 0, "tile rows must split evenly over the block");
  // wide_col needs rows of a multiple of 128 elements; narrower tiles (one
  // token wave) use tile_col, whose rows hold 8 chunks
  constexpr bool kWideZ = BC % 128 == 0;
  static_assert(kWideZ || (TW == 1 && BC / 8 == 8), "narrow z tiles hold 32 rows of 8 chunks");
  constexpr int RED_LDS = (TW - 1) * BC * (RPT + 4) * 4;
  constexpr int LDS = MAIN_LDS > RED_LDS ? MAIN_LDS : RED_LDS;
  __shared__ __attribute__((aligned(16))) char smem[LDS];

  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
  const int cw = wave % CW, tw = wave / CW;
#if RESBM_XCD_SPREAD
  const int cbi = blockIdx.y, tg = blockIdx.x;  // token groups vary fastest: every XCD sees every column block
  const int ncb = gridDim.y;
#else
  const int cbi = blockIdx.x, tg = blockIdx.y;
  const int ncb = gridDim.x;
#endif
  const int wc0 = cbi * BC + cw * WC;
  const bool on = wc0 < n;  // whole waves fall inside or outside [0, n): n % 64 == 0, WC | 64
  const int64_t t_begin = (int64_t)tg * TB;
  const int64_t t_end = min(T, t_begin + TB);
  GhTile<TS, RPS>* s_gh = reinterpret_cast<GhTile<TS, RPS>*>(smem);
  io_t* s_zb = reinterpret_cast<io_t*>(smem + 2 * GH_BYTES);
  const int bc0 = cbi * BC;
  const int bcv = min(BC, n - bc0);  // valid columns of the block (a multiple of 64, or <= 0)
  const int zc = 8 * (l % LPR);
  int zrow[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) zrow[q] = (wave * NQ * 64 + q * 64 + l) / LPR;

  f32x4 dw[CT][NT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int jt = 0; jt < NT; ++jt) dw[ct][jt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // g_h inputs of one block step: chunk q = threadIdx + i NTH covers token q / (KP / 4),
  // columns 4 (q % (KP / 4)) .. + 3 (zeros at or beyond r and past the token range).
  // Raw loaded bits: converting at load time would make the compiler wait for
  // the load right where it is issued.
  struct Gin {
#if RESBM_IO_F32_BUILD
    uint4 gb[NCH];
#else
    uint2 gb[NCH];
#endif
    uint4 a[NCH];
  };
  auto load_gin = [&](Gin& g, int64_t t0) {
    const int64_t rows = min((int64_t)TS, t_end - t0);
    const rsrc_t gbr = make_rsrc(g_b + t0 * r, rows * r * kEs);
    const rsrc_t ar = make_rsrc(silu ? a_save + t0 * r : a_save, silu ? rows * r * 4 : 0);
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int q = threadIdx.x + i * NTH;
      const int tt = q / (KP / 4), j0 = 4 * (q % (KP / 4));
      const bool ok = q < GQ && j0 < r;
#if RESBM_IO_F32_BUILD
      g.gb[i] = bld16(gbr, ok ? (uint32_t)((tt * r + j0) * kEs) : kOOB);
#else
      g.gb[i] = bld8(gbr, ok ? (uint32_t)((tt * r + j0) * kEs) : kOOB);
#endif
      g.a[i] = bld16(ar, ok ? (uint32_t)((tt * r + j0) * 4) : kOOB);  // zeros without SiLU
    }
  };
  // g_h of one block step into LDS (split).  Every column block forms the same
  // g_h; row tt of the step also goes to gh_hi / gh_lo for the g_z kernel from
  // column block tt mod ncb (one writer per row), which spreads those writes
  // over the grid.
  auto put_gh = [&](const Gin& g, int buf, int64_t s, int64_t t0) {
    const int64_t grows = s >= 0 ? min((int64_t)TS, t_end - t0) : 0;
    const rsrc_t ghr = make_rsrc(gh_hi + t0 * r, grows * r * kEs);
#if !RESBM_IO_F32_BUILD
    const rsrc_t glr = make_rsrc(gh_lo + t0 * r, grows * r * kEs);
#endif
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int q = threadIdx.x + i * NTH;
      if (GQ % NTH == 0 || q < GQ) {
        const int tt = q / (KP / 4), j0 = 4 * (q % (KP / 4));
        float gbv[4], av[4], v[4];
#if RESBM_IO_F32_BUILD
        gbv[0] = __builtin_bit_cast(float, g.gb[i].x); gbv[1] = __builtin_bit_cast(float, g.gb[i].y);
        gbv[2] = __builtin_bit_cast(float, g.gb[i].z); gbv[3] = __builtin_bit_cast(float, g.gb[i].w);
#else
        gbv[0] = bf16_bits_to_f32(g.gb[i].x & 0xffffu); gbv[1] = bf16_bits_to_f32(g.gb[i].x >> 16);
        gbv[2] = bf16_bits_to_f32(g.gb[i].y & 0xffffu); gbv[3] = bf16_bits_to_f32(g.gb[i].y >> 16);
#endif
        av[0] = __builtin_bit_cast(float, g.a[i].x); av[1] = __builtin_bit_cast(float, g.a[i].y);
        av[2] = __builtin_bit_cast(float, g.a[i].z); av[3] = __builtin_bit_cast(float, g.a[i].w);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = silu ? gbv[e] * silu_grad(av[e]) : gbv[e];
        gh_put4(s_gh[buf], tt, j0, v);
        const uint32_t go = j0 < r && tt % ncb == cbi ? (uint32_t)((tt * r + j0) * kEs) : kOOB;
#if RESBM_IO_F32_BUILD
        bst16(ghr, go, make_uint4(__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                                  __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])));
#else
        bf16x4 h, lo;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          __bf16 a, b;
          split_hi_lo(v[e], a, b);
          h[e] = a;
          lo[e] = b;
        }
        bst8(ghr, go, __builtin_bit_cast(uint2, h));
        bst8(glr, go, __builtin_bit_cast(uint2, lo));
#endif
      }
    }
  };
  auto load_z = [&](XFrag (&zz)[NQ], int64_t t0) {
    const int64_t rows = min((int64_t)TS, t_end - t0);  // <= 0 past the range: zeros
    const rsrc_t zr = make_rsrc(z + t0 * ld_z + bc0, bcv > 0 ? rows_bytes(rows, bcv, ld_z, kEs) : 0);
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      zz[q] = bld_x8(zr, zc < bcv ? (uint32_t)((zrow[q] * ld_z + zc) * kEs) : kOOB);
  };

  // One block step.  zz and gin hold this step's z tile and g_h inputs and are
  // reloaded with those of the step after next.  Steps outside [0, nsb) see
  // zero inputs and store nothing.
  auto body = [&](int64_t s, XFrag (&zz)[NQ], Gin& gin) {
    const int buf = (int)(s & 1);
    const int64_t t0 = t_begin + s * TS;
    io_t* tile = s_zb + buf * (TS * BC);
    put_gh(gin, buf, s, t0);
    load_gin(gin, t0 + 2 * TS);
    // this buffer's readers (two steps back) passed the previous step's barrier
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      io_t* d = tile + zrow[q] * BC + (kWideZ ? wide_col(zrow[q], zc) : tile_col<BC>(zrow[q], zc));
#if RESBM_IO_F32_BUILD
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = zz[q].v[e];
#else
      *reinterpret_cast<uint4*>(d) = __builtin_bit_cast(uint4, zz[q].v);
#endif
    }
    load_z(zz, t0 + 2 * TS);
    __syncthreads();  // g_h and the z tile of this step are complete

    // dW_e: D[j][c] = sum_t g_h[t][j] z[t][c], A = g_h^T, B = z^T
    {
      XFrag zb[CT];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
        zb[ct] = kWideZ ? tr_frag_wide<BC>(tile, 32 * tw, cw * WC + 16 * ct, row16, grp)
                        : tr_frag<BC>(tile, cw * WC + 16 * ct, row16, grp);
#pragma unroll
      for (int jt = 0; jt < NT; ++jt) {
        const SFrag g = gh_tr(s_gh[buf], 32 * tw, 16 * jt, row16, grp);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) dw[ct][jt] = mma_sx(g, zb[ct], dw[ct][jt]);
      }
    }

  };

  // The z tiles and g_h inputs of two steps are in flight at all times.  The
  // loop starts two (empty) steps early with zeroed registers instead of a
  // prologue of loads, and runs an even number of steps, so that every memory
  // operation sits inside one unconditional loop body and the compiler can
  // place each wait at its exact distance.
  const int64_t nsb = (t_end - t_begin + TS - 1) / TS;
  Gin ga, gb;
  XFrag z0[NQ], z1[NQ];
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    ga.gb[i] = gb.gb[i] = {};
    ga.a[i] = gb.a[i] = make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) z0[q] = z1[q] = xfrag_zero();
  for (int64_t s = opaque(-2); s < nsb; s += 2) {
    body(s, z0, ga);
    body(s + 1, z1, gb);
  }

  // dw[ct][jt][v] = partial dW_e[wc0 + 16 ct + row16][16 jt + 4 grp + v]
  if constexpr (TW > 1) {
    __syncthreads();  // the reduction area overlaps the step buffers
    float (*s_red)[BC][RPT + 4] = reinterpret_cast<float (*)[BC][RPT + 4]>(smem);
    if (tw > 0) {
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int jt = 0; jt < NT; ++jt)
          *reinterpret_cast<float4*>(&s_red[tw - 1][cw * WC + 16 * ct + row16][16 * jt + 4 * grp]) =
              make_float4(dw[ct][jt][0], dw[ct][jt][1], dw[ct][jt][2], dw[ct][jt][3]);
    }
    __syncthreads();
    if (tw > 0) return;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int jt = 0; jt < NT; ++jt)
#pragma unroll
        for (int u = 0; u < TW - 1; ++u) {
          const float4 p = *reinterpret_cast<const float4*>(&s_red[u][cw * WC + 16 * ct + row16][16 * jt + 4 * grp]);
          dw[ct][jt][0] += p.x; dw[ct][jt][1] += p.y; dw[ct][jt][2] += p.z; dw[ct][jt][3] += p.w;
        }
  }
  if (!on) return;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int jt = 0; jt < NT; ++jt)
      *reinterpret_cast<float4*>(dwp + ((int64_t)tg * n + wc0 + 16 * ct + row16) * RP + 16 * jt + 4 * grp) =
          make_float4(dw[ct][jt][0], dw[ct][jt][1], dw[ct][jt][2], dw[ct][jt][3]);
}

// Finishing work of encode_bwd, one 256-thread block per call (bid = its index):
// blocks [0, nb_dw): dW_e (+)= sum_tg dwp[tg]; a block covers 64 four-column
// groups, its 4 thread quarters sum consecutive quarters of the token groups and
// the quarters are added in order.  Remaining blocks (when g_x is given apart
// from g_z): g_x[t][0:r] += g_b[t][0:r], rounded once.  These blocks ride along
// with the g_z pass (extra blocks of its launch), whose stream they do not touch.
__device__ __forceinline__ void enc_bwd_fin_block(int64_t bid, int64_t T, int n, int r, int RP,
                                                  const float* __restrict__ dwp, int ntg,
                                                  float* __restrict__ dW_e, int accumulate, int64_t nb_dw,
                                                  const io_t* __restrict__ g_b, io_t* __restrict__ g_x,
                                                  int64_t ld_gx) {
  __shared__ float4 s_q[4][64];
  const int nq = r / 4;
  if (bid >= nb_dw) {
    const int64_t gid = (bid - nb_dw) * 256 + threadIdx.x;
    if (gid >= T * nq) return;
    const int64_t t = gid / nq;
    const int j0 = (int)(gid % nq) * 4;
    float gb[4], x[4];
    load_x4(g_b + t * r + j0, gb);
    load_x4(g_x + t * ld_gx + j0, x);
#pragma unroll
    for (int v = 0; v < 4; ++v) x[v] += gb[v];
    store_x4(g_x + t * ld_gx + j0, x);
    return;
  }
  const int q = threadIdx.x >> 6;
  const int64_t cidx = bid * 64 + (threadIdx.x & 63);
  const bool ok = cidx < (int64_t)n * nq;
  const int c = ok ? (int)(cidx / nq) : 0;
  const int j0 = ok ? (int)(cidx % nq) * 4 : 0;
  const int g0 = q * ntg / 4, g1 = (q + 1) * ntg / 4;
  const float4 acc = ok ? sum_ordered4(dwp + ((int64_t)g0 * n + c) * RP + j0, (int64_t)n * RP, g1 - g0)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
  s_q[q][threadIdx.x & 63] = acc;
  __syncthreads();
  if (q == 0 && ok) {
    float4 s = accumulate ? *reinterpret_cast<const float4*>(dW_e + (int64_t)c * r + j0)
                          : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 tot = s_q[0][threadIdx.x];
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      const float4 p = s_q[k][threadIdx.x];
      tot.x += p.x; tot.y += p.y; tot.z += p.z; tot.w += p.w;
    }
    s.x += tot.x; s.y += tot.y; s.z += tot.z; s.w += tot.w;
    *reinterpret_cast<float4*>(dW_e + (int64_t)c * r + j0) = s;
  }
}

// The finishing work of encode_bwd as a kernel of its own (wide r: the g_z
// kernel's register allocation would leave its finishing blocks one wave per
// SIMD, behind the g_z blocks).
__global__ __launch_bounds__(256) void k_enc_bwd_fin(int64_t T, int n, int r, int RP, const float* __restrict__ dwp,
                                                     int ntg, float* __restrict__ dW_e, int accumulate,
                                                     int64_t nb_dw, const io_t* __restrict__ g_b,
                                                     io_t* __restrict__ g_x, int64_t ld_gx) {
  enc_bwd_fin_block(blockIdx.x, T, n, r, RP, dwp, ntg, dW_e, accumulate, nb_dw, g_b, g_x, ld_gx);
}

// ============================================================ expand contractions
// out = in W (+ idsrc I_{r x n} when ADD), an r-wide input times an r x n map:
//   decode_fwd (GZ = false): z~ = b W_d (+ b I_{r x n}, reading A); in = b, W = W_d [r][n];
//   encode_bwd (GZ = true):  g_z = g_h W_e^T (+ g_b I_{r x n} when g_x is g_z);
//     in = g_h as hi and lo bf16 planes [T][r] (one fp32 plane in the fp32 build),
//     W = W_e [n][r].
// A wave owns columns [c0, c0 + 16 CT) (see expand_col) and walks the token range
// [blockIdx.y tpg, ...) 16 tokens at a time.
// Finishing work that rides along with the g_z pass (GZ): the dW_e partial sums
// and a separate g_x update, in extra rows of the grid (see enc_bwd_fin_block).
struct FinArgs {
  int RP;
  const float* dwp;
  int ntg;
  float* dW_e;
  int accumulate;
  int64_t nb_dw, nb_all;
  const io_t* g_b;
  io_t* g_x;
  int64_t ld_gx;
};

template <int KS, int CT, bool ADD, bool GZ, bool R8>
__global__ __launch_bounds__(256) void k_expand(int64_t T, int n, int r,
                                                const io_t* __restrict__ in, const io_t* __restrict__ in_lo,
                                                const io_t* __restrict__ idsrc, const float* __restrict__ W,
                                                io_t* __restrict__ out, int64_t ld_out, int tpg, int main_y,
                                                FinArgs fin) {
  if constexpr (GZ) {
    if ((int)blockIdx.y >= main_y) {  // a finishing block
      const int64_t bid = (int64_t)(blockIdx.y - main_y) * gridDim.x + blockIdx.x;
      if (bid < fin.nb_all)
        enc_bwd_fin_block(bid, T, n, r, fin.RP, fin.dwp, fin.ntg, fin.dW_e, fin.accumulate, fin.nb_dw, fin.g_b,
                          fin.g_x, fin.ld_gx);
      return;
    }
  }
  constexpr int W8 = CT >= 2 ? 8 : 4;       // consecutive columns per lane run
  constexpr int NH = CT >= 2 ? CT / 2 : 1;  // runs per lane
  constexpr int NI = ADD ? NH * W8 / 4 : 1;  // 4-column identity chunks per lane
  constexpr int WC = 16 * CT;               // columns of the wave
  constexpr int CPR = WC / 8;               // 8-element chunks per output row
  constexpr int NS = (16 * CPR + 63) / 64;  // coalesced stores per lane per tile
  constexpr bool LO = GZ && !RESBM_IO_F32_BUILD;  // a second (lo) input plane
  __shared__ __attribute__((aligned(16))) io_t s_out[4][16 * WC];
  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
  io_t* tile = s_out[wave];
#if RESBM_DF_TOKEN_FASTEST
  // token groups vary fastest: the blocks of one token group share an XCD and
  // its L2 holds their input rows once
  const int strip = blockIdx.y * 4 + wave;
  const int tgi = blockIdx.x;
#else
  const int strip = blockIdx.x * 4 + wave;
  const int tgi = blockIdx.y;
#endif
  const int c0 = strip * 16 * CT;
  if (c0 >= n) return;  // whole strips only: n % 64 == 0 and 16 CT divides 64

  // the map as the A operand: lane (row16, grp) holds W(k = 32 ks + 8 grp + e, column)
  SFrag wfr[KS][CT];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int col = expand_col<CT>(c0, ct, row16);
      float w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = ks * 32 + grp * 8 + e;
        w[e] = k < r ? (GZ ? W[(int64_t)col * r + k] : W[(int64_t)k * n + col]) : 0.0f;
      }
      wfr[ks][ct] = sfrag_from(w);
    }

  const int64_t t_begin = (int64_t)tgi * tpg;
  const int64_t rows = min((int64_t)tpg, T - t_begin);
  const rsrc_t br = make_rsrc(in + t_begin * r, rows * r * kEs);
  const rsrc_t lr = make_rsrc(LO ? in_lo + t_begin * r : in, LO ? rows * r * kEs : 0);
  const rsrc_t ir = make_rsrc(idsrc + t_begin * r, ADD ? rows * r * kEs : 0);
  const rsrc_t zr = make_rsrc(out + t_begin * ld_out, rows_bytes(rows, n, ld_out, kEs));
  const int cl = c0 + W8 * grp;  // first column of this lane's run 0

  struct Tile {
    XFrag p[KS];
    XFrag q[LO ? KS : 1];  // lo plane
#if RESBM_IO_F32_BUILD
    uint4 id[NI];  // idsrc[t][column chunk] below r, zeros elsewhere (raw bits)
#else
    uint2 id[NI];
#endif
  };
  auto load = [&](Tile& x, int64_t tt) {  // tt: tile start relative to t_begin
    const int64_t t = tt + row16;
    const uint32_t ro = (uint32_t)(t * r * kEs);  // rows >= `rows` are out of range
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      x.p[ks] = bld_r8<R8>(br, ro, r, ks * 32 + grp * 8);
      if constexpr (LO) x.q[ks] = bld_r8<R8>(lr, ro, r, ks * 32 + grp * 8);
    }
    if constexpr (ADD) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int cb = cl + 32 * (i / (W8 / 4)) + 4 * (i % (W8 / 4));
        const uint32_t o = cb < r ? (uint32_t)((t * r + cb) * kEs) : kOOB;
#if RESBM_IO_F32_BUILD
        x.id[i] = bld16(ir, o);
#else
        x.id[i] = bld8(ir, o);
#endif
      }
    }
  };
  auto compute = [&](const Tile& x, int64_t tt) {
    f32x4 acc[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if constexpr (GZ) {
        SFrag g;  // the split input
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) g.v[e] = x.p[ks].v[e];
#else
        g.hi = x.p[ks].v;
        g.lo = x.q[ks].v;
#endif
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct] = mma_ss(wfr[ks][ct], g, acc[ct]);
      } else {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct] = mma_sx(wfr[ks][ct], x.p[ks], acc[ct]);
      }
    }
    const int64_t t = tt + row16;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      float v[W8];
#pragma unroll
      for (int q = 0; q < W8 / 4; ++q) {
        float id[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (ADD) {
          const auto u = x.id[h * (W8 / 4) + q];
#if RESBM_IO_F32_BUILD
          id[0] = __builtin_bit_cast(float, u.x); id[1] = __builtin_bit_cast(float, u.y);
          id[2] = __builtin_bit_cast(float, u.z); id[3] = __builtin_bit_cast(float, u.w);
#else
          id[0] = bf16_bits_to_f32(u.x & 0xffffu); id[1] = bf16_bits_to_f32(u.x >> 16);
          id[2] = bf16_bits_to_f32(u.y & 0xffffu); id[3] = bf16_bits_to_f32(u.y >> 16);
#endif
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) v[4 * q + e] = ADD ? acc[2 * h + q][e] + id[e] : acc[2 * h + q][e];
      }
      // round into the wave's tile (row = token)
      io_t* d = tile + row16 * WC + tile_col<WC>(row16, cl - c0 + 32 * h);
#pragma unroll
      for (int e = 0; e < W8; ++e) d[e] = f32_to_io(v[e]);
    }
    (void)t;
    // write the tile out row by row, 8 lanes per 128 bytes
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const int idx = l + 64 * q;
      const int row = idx / CPR, c8 = 8 * (idx % CPR);
      const XFrag o = tile_get8<WC>(tile, row < 16 ? row : 0, c8);
      bst_frag(zr, (tt < 0 || row >= 16) ? kOOB : (uint32_t)(((tt + row) * ld_out + c0 + c8) * kEs), o);
    }
  };

  // Every memory operation sits in one unconditional loop body: the loop starts
  // two (empty) tiles early on zeroed registers instead of after a prologue of
  // loads, so the compiler can place each wait at its exact distance.
  Tile xa, xb;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) xa.p[ks] = xb.p[ks] = xfrag_zero();
  if constexpr (LO) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) xa.q[ks] = xb.q[ks] = xfrag_zero();
  }
  if constexpr (ADD) {
#pragma unroll
    for (int i = 0; i < NI; ++i) xa.id[i] = xb.id[i] = {};
  }
  // (the scheduling barriers keep the compiler from hoisting a tile's math
  // above the loads issued before it, which would wait for those loads)
  for (int64_t tt = opaque(-32); tt < rows; tt += 32) {
    compute(xa, tt);
    load(xa, tt + 32);
    __builtin_amdgcn_sched_barrier(0);
    compute(xb, tt + 16);  // past the range: loads were zeros, stores are dropped
    load(xb, tt + 48);
    __builtin_amdgcn_sched_barrier(0);
  }
}


// ============================================================ wide rank (r > 64)
// Above r = 64 the matrix-core work per streamed byte grows with r, and the
// kernels above, shaped for r <= 64, re-read their r-wide operands too often:
// encode_fwd reads all of W_e's fragments per 16 tokens, the expand kernel
// fetches the input rows once per wave, encode_bwd forms g_h again in every
// column block.  The kernels below keep the streaming structure and share the
// r-wide operands instead: blocks of 64 tokens whose waves split the r outputs
// (one read of the weight fragments per 64 tokens), input rows staged once per
// block in LDS, g_h formed once by a kernel of its own.  decode_bwd becomes a
// row contraction (g_b) and a token contraction (dW_d) over g_z~, which reads
// g_z~ twice but needs no g_b partial sums (at r = 256 those were 134 MB).

// Fragment-ordered hi/lo copy of W_d (r x n, contiguous along the contraction
// over n) for the A operand of g_b = g_z~ W_d^T: fragment f = ks * NT + nt,
// lane (row16, grp) holds W_d[16 nt + row16][32 ks + 8 grp + e], zeros at rows >= r.
__global__ __launch_bounds__(64) void k_wd_prep(const float* __restrict__ W_d, int n, int r, int NT,
                                                void* __restrict__ wf) {
  const int64_t gid = (int64_t)blockIdx.x * 64 + threadIdx.x;
  const int64_t total = (int64_t)(n / 32) * NT * 64;
  if (gid >= total) return;
  const int l = (int)(gid & 63);
  const int64_t f = gid >> 6;
  const int nt = (int)(f % NT), ks = (int)(f / NT);
  const int j = nt * 16 + (l & 15), k0 = ks * 32 + (l >> 4) * 8;
  float w[8];
  if (j < r) {
    const float4* p = reinterpret_cast<const float4*>(W_d + (int64_t)j * n + k0);
    const float4 a = p[0], c = p[1];
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w; w[4] = c.x; w[5] = c.y; w[6] = c.z; w[7] = c.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) w[e] = 0.0f;
  }
  store_sfrag(wf, f, l, w);
}

// Row contraction for wide r: C[t][j] = sum_c X[t][c] M(c, j) over the n
// columns of a streamed T x n matrix X, M given as split fragments (W_e for
// encode_fwd, W_d^T for the g_b of decode_bwd).  A block of NWV waves owns
// TOK = 64 RH tokens and one of RH groups of j-tiles; it stages TOK x 256 tiles
// of X cooperatively in LDS (512-byte row segments) and wave w contracts them
// against the fragments of j-tiles [w NTW, w NTW + NTW) of its group, so every
// wave ends with whole sums of its columns and the block reads each weight
// fragment of its group once per TOK tokens.  With RH = 2 the two blocks of a
// token group are 8 apart in a run of 16 (same XCD, dispatched together), so
// their shared X rows come from HBM once.  The weight fragments run kRwRing - 1
// k-steps ahead of their use in a ring of kRwRing registers.
//   GB = false: a_save = a, b = x_attn[:, :r] + phi(a)        (encode_fwd)
//   GB = true:  g_b = C + g_id[:, :r] (g_id may be NULL)        (decode_bwd)
template <int NT, int NTW, bool GB, int NWV, int RH>
__global__ __launch_bounds__(64 * NWV) void k_rowc_wide(int64_t T, int n, int r, int act, const io_t* __restrict__ X,
                                                        int64_t ld_x, const void* __restrict__ wf,
                                                        const io_t* __restrict__ skip, int64_t ld_s,
                                                        io_t* __restrict__ out, float* __restrict__ a_save) {
  constexpr int TOK = 64 * RH, MT = TOK / 16, BC = 256, KSS = BC / 32;
  constexpr int NTG = (NT + RH - 1) / RH;     // j-tiles of a group
  constexpr int LPR = BC / 8;                 // lanes per tile row
  constexpr int NQ = TOK * LPR / (64 * NWV);  // cooperative loads per lane and stage
  static_assert(NWV * NTW >= NTG, "the waves must cover the j-tiles of a group");
  constexpr int ZB = RESBM_IO_F32_BUILD ? 1 : 2;
  constexpr int TILE = TOK * BC * (int)sizeof(io_t);
  __shared__ __attribute__((aligned(16))) char smem[ZB * TILE];

  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
  const int bid = (int)blockIdx.x;
  const int tg = RH == 1 ? bid : (bid >> 4) * 8 + (bid & 7);  // token group
  const int jg0 = RH == 1 ? 0 : ((bid >> 3) & 1) * NTG;       // first j-tile of the group
  const int jg1 = min(NT, jg0 + NTG);
  const int64_t tok0 = (int64_t)tg * TOK;
  if (tok0 >= T) return;  // the last run of 16 can hold token groups past T (whole block)
  const int nks = n / 32;
  const int nst = (n + BC - 1) / BC;
  const rsrc_t zr = make_rsrc(X + tok0 * ld_x, rows_bytes(min((int64_t)TOK, T - tok0), n, ld_x, kEs));
  const rsrc_t wr = make_rsrc(wf, (int64_t)nks * NT * kSFragBytes);
  const int zc = 8 * (l % LPR);
  int zrow[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) zrow[q] = (wave * NQ * 64 + q * 64 + l) / LPR;

  // stages start rotated per group of 8 token groups (one per XCD), as in k_enc_fwd
  const int srot = (int)((unsigned)(tg / 8) % (unsigned)nst);
  auto stage_col = [&](int i) {
    if (i < 0 || i >= nst) return n;
    const int ir = i + srot < nst ? i + srot : i + srot - nst;
    return ir * BC;
  };
  auto load_z = [&](XFrag (&zz)[NQ], int i) {
    const int c = stage_col(i) + zc;
#pragma unroll
    for (int q = 0; q < NQ; ++q) zz[q] = bld_x8(zr, c < n ? (uint32_t)((zrow[q] * ld_x + c) * kEs) : kOOB);
  };
  constexpr int RG = kRwRing, AH = RG - 1;  // ring of weight fragments, loaded AH k-steps ahead
  static_assert(KSS % RG == 0, "a stage's k-steps must fill whole rings");
  SFrag wring[RG][NTW];
  // the weight fragments of k-step ks of stage i (zeros outside [0, nks) or past NT)
  auto load_wf = [&](SFrag (&dst)[NTW], int i, int ks) {
    const int kg = (stage_col(i) >> 5) + ks;
#pragma unroll
    for (int jt = 0; jt < NTW; ++jt) {
      const int jtg = jg0 + wave * NTW + jt;
      dst[jt] = bld_sfrag(wr, (int64_t)kg * NT + jtg, l, kg < nks && jtg < jg1);
    }
  };

  f32x4 acc[MT][NTW];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int jt = 0; jt < NTW; ++jt) acc[mt][jt] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto body = [&](XFrag (&zz)[NQ], int i) {
    io_t* tile = reinterpret_cast<io_t*>(smem + (ZB == 2 ? (i & 1) : 0) * TILE);
    if constexpr (ZB == 1) __syncthreads();  // the previous stage's readers of the single tile are done
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      io_t* d = tile + zrow[q] * BC + wide_col(zrow[q], zc);
#if RESBM_IO_F32_BUILD
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = zz[q].v[e];
#else
      *reinterpret_cast<uint4*>(d) = __builtin_bit_cast(uint4, zz[q].v);
#endif
    }
    load_z(zz, i + 2);
    __syncthreads();  // the stage's tile is complete; the other buffer's readers are done
    const bool live = i >= 0 && i < nst;  // stages outside hold zeros: only their weight loads matter
    // fp32 build: each stage sums into a zeroed partial that is then added to
    // the total, so a long contraction (n / 4 products of K = 4) rounds as two
    // short ones; the bf16 build accumulates directly
    constexpr bool PART = RESBM_IO_F32_BUILD;
    f32x4 part[PART ? MT : 1][PART ? NTW : 1];
    if constexpr (PART) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int jt = 0; jt < NTW; ++jt) part[mt][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int ks = 0; ks < KSS; ++ks) {
      if (ks + AH < KSS) load_wf(wring[(ks + AH) % RG], i, ks + AH);
      else load_wf(wring[(ks + AH) % RG], i + 1, ks + AH - KSS);
      if (!live) continue;
      XFrag f[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int row = 16 * mt + row16;
        const io_t* p = tile + row * BC + wide_col(row, 32 * ks + 8 * grp);
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) f[mt].v[e] = p[e];
#else
        f[mt].v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
#endif
      }
      // waves whose last j-tiles lie past the group multiply zero fragments (never stored)
#pragma unroll
      for (int jt = 0; jt < NTW; ++jt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          if constexpr (PART) part[mt][jt] = mma_sx(wring[ks % RG][jt], f[mt], part[mt][jt]);
          else acc[mt][jt] = mma_sx(wring[ks % RG][jt], f[mt], acc[mt][jt]);
        }
    }
    if constexpr (PART) {
      if (live) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int jt = 0; jt < NTW; ++jt) acc[mt][jt] += part[mt][jt];
      }
    }
  };
  XFrag za[NQ], zb[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) za[q] = zb[q] = xfrag_zero();
  {
    const int i0 = opaque(-2);
#pragma unroll
    for (int u = 0; u < AH; ++u) load_wf(wring[u], i0, u);
  }
  for (int i = opaque(-2); i < nst; i += 2) {
    body(za, i);
    body(zb, i + 1);
  }

  // acc[mt][jt][v] = C[tok0 + 16 mt + row16][16 (jg0 + w NTW + jt) + 4 grp + v]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int jt = 0; jt < NTW; ++jt) {
      const int jtg = jg0 + wave * NTW + jt;
      const int64_t t = tok0 + 16 * mt + row16;
      const int j0 = 16 * jtg + 4 * grp;
      if (jtg >= jg1 || t >= T || j0 >= r) continue;
      float a[4] = {acc[mt][jt][0], acc[mt][jt][1], acc[mt][jt][2], acc[mt][jt][3]};
      if constexpr (GB) {
        if (skip) {
          float x[4];
          load_x4(skip + t * ld_s + j0, x);
#pragma unroll
          for (int v = 0; v < 4; ++v) a[v] += x[v];
        }
        store_x4(out + t * r + j0, a);
      } else {
        if (a_save) *reinterpret_cast<float4*>(a_save + t * r + j0) = make_float4(a[0], a[1], a[2], a[3]);
        float x[4], o[4];
        load_x4(skip + t * ld_s + j0, x);
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = x[v] + act_phi(a[v], act);
        store_x4(out + t * r + j0, o);
      }
    }
}

// g_h = g_b phi'(a), formed once for encode_bwd's wide-rank kernels: hi and lo
// bf16 planes [T][r] (one float plane in the fp32 build); 4 columns per thread.
__global__ __launch_bounds__(256) void k_gh(int64_t T, int r, int silu, const io_t* __restrict__ g_b,
                                            const float* __restrict__ a_save, io_t* __restrict__ gh_hi,
                                            io_t* __restrict__ gh_lo) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int nq = r / 4;
  if (q >= T * nq) return;
  const int64_t t = q / nq;
  const int j0 = (int)(q % nq) * 4;
  float g[4];
  load_x4(g_b + t * r + j0, g);
  if (silu) {
    const float4 a = *reinterpret_cast<const float4*>(a_save + t * r + j0);
    g[0] *= silu_grad(a.x);
    g[1] *= silu_grad(a.y);
    g[2] *= silu_grad(a.z);
    g[3] *= silu_grad(a.w);
  }
#if RESBM_IO_F32_BUILD
  (void)gh_lo;
  *reinterpret_cast<float4*>(gh_hi + t * r + j0) = make_float4(g[0], g[1], g[2], g[3]);
#else
  bf16x4 h, lo;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    __bf16 a, b;
    split_hi_lo(g[e], a, b);
    h[e] = a;
    lo[e] = b;
  }
  *reinterpret_cast<uint2*>(gh_hi + t * r + j0) = __builtin_bit_cast(uint2, h);
  *reinterpret_cast<uint2*>(gh_lo + t * r + j0) = __builtin_bit_cast(uint2, lo);
#endif
}

// Transposed fragment of a [rows][PITCH] plane of the I/O type (bf16 build:
// lds_col<PITCH> layout; f32 build: row-major): lane (row16, grp) receives
// plane[row0 + 8 grp + e][c0 + row16], e = 0..7 (row0 % 16 == 0).
template <int PITCH>
__device__ __forceinline__ XFrag tr_rows(const io_t* plane, int row0, int c0, int row16, int grp) {
  XFrag f;
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int e = 0; e < 8; ++e) f.v[e] = plane[(row0 + 8 * grp + e) * PITCH + c0 + row16];
#else
  f.v = tr_plane<PITCH>(plane, row0, c0, row16, grp);
#endif
  return f;
}

// Token contraction for wide r over a token group, for 128 columns c of the
// streamed matrix X and all r columns j of the r-wide operand Y:
//   DWD = false (encode_bwd): dwp[tg][c][j] = sum_t X[t][c] Y[t][j], Y = g_h
//                             (split: hi and lo planes; one float plane in the fp32 build)
//   DWD = true  (decode_bwd): dwp[tg][j][c] = sum_t Y[t][j] X[t][c], Y = b (exact)
// 8 waves: wave (cw, jq) owns columns [64 cw, 64 cw + 64) of the block and
// j-tiles [jq NTW, jq NTW + NTW).  Per step of TS = 32 TSM tokens the block
// stages the TS x 128 tile of X and the TS x r tile(s) of Y in LDS (double
// buffered, the next steps' loads in registers: X 128 tokens or two steps
// ahead, Y two steps); both operands are read back transposed (the contraction runs over
// the tile's rows, 32 at a time).  TSM = 2 halves the barriers per token where
// the buffers fit in LDS.
template <int NT, int NTW, bool DWD, bool R8, int TSM>
__global__ __launch_bounds__(512) void k_tokc_wide(int64_t T, int n, int r, int RP, const io_t* __restrict__ X,
                                                   int64_t ld_x, const io_t* __restrict__ Y,
                                                   const io_t* __restrict__ Y_lo, float* __restrict__ dwp, int TB) {
  constexpr int BCc = 128, TS = 32 * TSM, KS = (NT + 1) / 2, KP = 32 * KS;
  constexpr int YP = tw_ypitch(NT);  // Y plane pitch (lds_col<YP> layout)
  constexpr bool SPLIT = !DWD && !RESBM_IO_F32_BUILD;
  constexpr int PL = SPLIT ? 2 : 1;
  constexpr int XE = TS * BCc, YE = TS * YP;  // elements of the X tile and of one Y plane
  constexpr int YC = TS * (KP / 8);           // 8-element chunks of one Y plane
  constexpr int NYQ = (PL * YC + 511) / 512;  // Y chunk loads per thread and step
  constexpr int XA = RESBM_TW_XTOK / TS >= 2 ? RESBM_TW_XTOK / TS : 2;  // steps of X loads in flight (even)
  static_assert(2 * (XE + PL * YE) * (int)sizeof(io_t) <= kLdsBytes, "tiles exceed LDS");
  __shared__ __attribute__((aligned(16))) io_t s_x[2][XE];
  __shared__ __attribute__((aligned(16))) io_t s_y[2][PL][YE];

  const int tid = threadIdx.x, l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
  const int cw = wave & 1, jq = wave >> 1;
  const int tg = blockIdx.x, cbi = blockIdx.y;  // token groups vary fastest
  const int bc0 = cbi * BCc;
  const int bcv = min(BCc, n - bc0);          // valid columns of the block (a multiple of 64)
  const int64_t t_begin = (int64_t)tg * TB;
  const int64_t t_end = min(T, t_begin + TB);
  // X loads: thread tid takes rows tid / 16 + 32 q, columns 8 (tid % 16) .. + 8
  const int xrow = tid >> 4, xc = 8 * (tid & 15);

  f32x4 acc[4][NTW];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int jt = 0; jt < NTW; ++jt) acc[ct][jt] = f32x4{0.f, 0.f, 0.f, 0.f};

  struct XRegs {
    XFrag x[TSM];
  };
  struct YRegs {
    XFrag y[NYQ];
  };
  auto rows_of = [&](int64_t s, int64_t& t0) {
    t0 = t_begin + s * TS;
    return s < 0 ? (int64_t)0 : min((int64_t)TS, t_end - t0);
  };
  auto load_x = [&](XRegs& x, int64_t s) {
    int64_t t0;
    const int64_t rows = rows_of(s, t0);
    const rsrc_t xr_ = make_rsrc(X + t0 * ld_x + bc0, bcv > 0 ? rows_bytes(rows, bcv, ld_x, kEs) : 0);
#pragma unroll
    for (int q = 0; q < TSM; ++q)
      x.x[q] = bld_x8(xr_, xc < bcv ? (uint32_t)(((xrow + 32 * q) * ld_x + xc) * kEs) : kOOB);
  };
  auto load_y = [&](YRegs& g, int64_t s) {
    int64_t t0;
    const int64_t rows = rows_of(s, t0);
    const rsrc_t yr_ = make_rsrc(Y + t0 * r, rows > 0 ? rows * r * kEs : 0);
    const rsrc_t yl_ = make_rsrc(SPLIT ? Y_lo + t0 * r : Y, SPLIT && rows > 0 ? rows * r * kEs : 0);
#pragma unroll
    for (int i = 0; i < NYQ; ++i) {
      const int qq = tid + 512 * i;
      const int pl = qq / YC, rem = qq % YC;
      const int yrow = rem / (KP / 8), c8 = 8 * (rem % (KP / 8));
      const bool ok = qq < PL * YC;
      g.y[i] = bld_r8<R8>(pl ? yl_ : yr_, ok ? (uint32_t)(yrow * r * kEs) : kOOB, r, c8);
    }
  };
  auto put = [&](const XRegs& x, const YRegs& g, int buf) {
#pragma unroll
    for (int q = 0; q < TSM; ++q) {
      io_t* dx = &s_x[buf][(xrow + 32 * q) * BCc + wide_col(xrow + 32 * q, xc)];
#if RESBM_IO_F32_BUILD
#pragma unroll
      for (int e = 0; e < 8; ++e) dx[e] = x.x[q].v[e];
#else
      *reinterpret_cast<uint4*>(dx) = __builtin_bit_cast(uint4, x.x[q].v);
#endif
    }
#pragma unroll
    for (int i = 0; i < NYQ; ++i) {
      const int qq = tid + 512 * i;
      if (NYQ * 512 == PL * YC || qq < PL * YC) {
        const int pl = qq / YC, rem = qq % YC;
        const int yrow = rem / (KP / 8), c8 = 8 * (rem % (KP / 8));
        io_t* dy = &s_y[buf][pl][yrow * YP + (RESBM_IO_F32_BUILD ? c8 : lds_col<YP>(yrow, c8))];
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) dy[e] = g.y[i].v[e];
#else
        *reinterpret_cast<uint4*>(dy) = __builtin_bit_cast(uint4, g.y[i].v);
#endif
      }
    }
  };
  // fp32 build: each step sums into a zeroed partial that is then added to the
  // total, so a token group's long sum rounds as a short one per step plus one
  // addition per step; the bf16 build accumulates directly
  constexpr bool PART = RESBM_IO_F32_BUILD;
  auto compute = [&](int buf) {
    f32x4 part[PART ? 4 : 1][PART ? NTW : 1];
    if constexpr (PART) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int jt = 0; jt < NTW; ++jt) part[ct][jt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int ks = 0; ks < TSM; ++ks) {  // 32 tokens of the step at a time
      XFrag xf[4];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) xf[ct] = tr_frag_wide<BCc>(s_x[buf], 32 * ks, 64 * cw + 16 * ct, row16, grp);
#pragma unroll
      for (int jt = 0; jt < NTW; ++jt) {
        const int jtg = jq * NTW + jt;
        if constexpr (NT % 4 != 0) {
          if (jtg >= NT) continue;  // wave-uniform; the tile's columns end at 32 KS
        }
        if constexpr (DWD) {
          const XFrag yb = tr_rows<YP>(s_y[buf][0], 32 * ks, 16 * jtg, row16, grp);
#pragma unroll
          for (int ct = 0; ct < 4; ++ct) {
            if constexpr (PART) part[ct][jt] = mma_xx(xf[ct], yb, part[ct][jt]);
            else acc[ct][jt] = mma_xx(xf[ct], yb, acc[ct][jt]);
          }
        } else {
          SFrag g;
#if RESBM_IO_F32_BUILD
          const XFrag y = tr_rows<YP>(s_y[buf][0], 32 * ks, 16 * jtg, row16, grp);
#pragma unroll
          for (int e = 0; e < 8; ++e) g.v[e] = y.v[e];
#else
          g.hi = tr_rows<YP>(s_y[buf][0], 32 * ks, 16 * jtg, row16, grp).v;
          g.lo = tr_rows<YP>(s_y[buf][PL - 1], 32 * ks, 16 * jtg, row16, grp).v;
#endif
#pragma unroll
          for (int ct = 0; ct < 4; ++ct) {
            if constexpr (PART) part[ct][jt] = mma_sx(g, xf[ct], part[ct][jt]);
            else acc[ct][jt] = mma_sx(g, xf[ct], acc[ct][jt]);
          }
        }
      }
    }
    if constexpr (PART) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int jt = 0; jt < NTW; ++jt) acc[ct][jt] += part[ct][jt];
    }
  };

  // The X tiles (HBM) run XA steps ahead of their use, the Y tiles (L2) two.
  // Steps before 0 or past the range load zeros (the LDS buffers are fully
  // written with them before they are read) and skip the products.
  const int64_t nsb = (t_end - t_begin + TS - 1) / TS;
  XRegs xr[XA];
  YRegs yr[2];
#pragma unroll
  for (int i = 0; i < XA; ++i)
#pragma unroll
    for (int q = 0; q < TSM; ++q) xr[i].x[q] = xfrag_zero();
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < NYQ; ++i) yr[h].y[i] = xfrag_zero();
  auto body = [&](int64_t s, XRegs& xs, YRegs& ys) {
    put(xs, ys, (int)(s & 1));
    load_x(xs, s + XA);
    load_y(ys, s + 2);
    __syncthreads();  // this step's tiles are complete; the other buffers' readers are done
    if (s >= 0 && s < nsb) compute((int)(s & 1));
  };
  for (int64_t s = opaque(-XA); s < nsb; s += XA) {
#pragma unroll
    for (int u = 0; u < XA; ++u) body(s + u, xr[u], yr[u & 1]);
  }

#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int jt = 0; jt < NTW; ++jt) {
      const int jtg = jq * NTW + jt;
      if (jtg >= NT) continue;
      if constexpr (DWD) {
        // acc[ct][jt][v] = partial dW_d[16 jtg + row16][bc0 + 64 cw + 16 ct + 4 grp + v]
        const int j = 16 * jtg + row16, c = bc0 + 64 * cw + 16 * ct + 4 * grp;
        if (j < r && c < n)
          *reinterpret_cast<float4*>(dwp + ((int64_t)tg * RP + j) * n + c) =
              make_float4(acc[ct][jt][0], acc[ct][jt][1], acc[ct][jt][2], acc[ct][jt][3]);
      } else {
        // acc[ct][jt][v] = partial dW_e[bc0 + 64 cw + 16 ct + row16][16 jtg + 4 grp + v]
        const int c = bc0 + 64 * cw + 16 * ct + row16, j = 16 * jtg + 4 * grp;
        if (c < n && j < r)
          *reinterpret_cast<float4*>(dwp + ((int64_t)tg * n + c) * RP + j) =
              make_float4(acc[ct][jt][0], acc[ct][jt][1], acc[ct][jt][2], acc[ct][jt][3]);
      }
    }
}

// Expand contraction for wide r (decode_fwd, the g_z pass of encode_bwd):
// k_expand's work split and epilogue, with the input rows of each 32-token
// step staged once per block in LDS, in fragment order (fragment q = (16-token
// tile, k-step, plane), 64 lanes x one exact fragment each), every wave
// fetching a quarter of them, instead of every wave fetching all of them.
// A wave whose strip lies past n still fetches its share and meets the
// barriers.  Double-buffered, with the next step's fetches two steps ahead in
// registers.
template <int KS, int CT, bool ADD, bool GZ, bool R8>
__global__ __launch_bounds__(256) void k_expand_wide(int64_t T, int n, int r, const io_t* __restrict__ in,
                                                     const io_t* __restrict__ in_lo, const io_t* __restrict__ idsrc,
                                                     const float* __restrict__ W, io_t* __restrict__ out,
                                                     int64_t ld_out, int tpg, int main_y, FinArgs fin) {
  if constexpr (GZ) {
    if ((int)blockIdx.y >= main_y) {  // a finishing block
      const int64_t bid = (int64_t)(blockIdx.y - main_y) * gridDim.x + blockIdx.x;
      if (bid < fin.nb_all)
        enc_bwd_fin_block(bid, T, n, r, fin.RP, fin.dwp, fin.ntg, fin.dW_e, fin.accumulate, fin.nb_dw, fin.g_b,
                          fin.g_x, fin.ld_gx);
      return;
    }
  }
  constexpr int W8 = CT >= 2 ? 8 : 4;
  constexpr int NH = CT >= 2 ? CT / 2 : 1;
  constexpr int NI = ADD ? NH * W8 / 4 : 1;
  constexpr int WC = 16 * CT;
  constexpr int CPR = WC / 8;
  constexpr int NS = (16 * CPR + 63) / 64;
  constexpr bool LO = GZ && !RESBM_IO_F32_BUILD;
  constexpr int PL = LO ? 2 : 1;
  constexpr int NF = 2 * KS * PL;   // input fragments of a 32-token step
  constexpr int NFW = (NF + 3) / 4;  // fetched per wave (the last round partly, when NF % 4 != 0)
  __shared__ __attribute__((aligned(16))) XFrag s_in[2][NF][64];
  __shared__ __attribute__((aligned(16))) io_t s_out[4][16 * WC];
  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = wave_id();
  io_t* tile = s_out[wave];
#if RESBM_DF_TOKEN_FASTEST
  const int strip = blockIdx.y * 4 + wave;
  const int tgi = blockIdx.x;
#else
  const int strip = blockIdx.x * 4 + wave;
  const int tgi = blockIdx.y;
#endif
  const int c0 = strip * 16 * CT;
  const bool won = c0 < n;  // whole strips: n % 64 == 0 and 16 CT divides 64

  SFrag wfr[KS][CT];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int col = expand_col<CT>(c0, ct, row16);
      float w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = ks * 32 + grp * 8 + e;
        w[e] = (won && k < r) ? (GZ ? W[(int64_t)col * r + k] : W[(int64_t)k * n + col]) : 0.0f;
      }
      wfr[ks][ct] = sfrag_from(w);
    }

  const int64_t t_begin = (int64_t)tgi * tpg;
  const int64_t rows = min((int64_t)tpg, T - t_begin);
  const rsrc_t br = make_rsrc(in + t_begin * r, rows * r * kEs);
  const rsrc_t lr = make_rsrc(LO ? in_lo + t_begin * r : in, LO ? rows * r * kEs : 0);
  const rsrc_t ir = make_rsrc(idsrc + t_begin * r, ADD ? rows * r * kEs : 0);
  const rsrc_t zr = make_rsrc(out + t_begin * ld_out, rows_bytes(rows, n, ld_out, kEs));
  const int cl = c0 + W8 * grp;  // first column of this lane's run 0

#if RESBM_IO_F32_BUILD
  typedef uint4 IdT;
#else
  typedef uint2 IdT;
#endif
  struct Step {
    XFrag f[NFW];    // this wave's share of the step's input fragments
    IdT id[2][NI];   // idsrc of the step's two tiles, this lane's columns below r (raw bits)
  };
  // fragment q = wave + 4 i of a step: with two planes NF is a multiple of 4
  // and q % PL = wave % PL, so every load of a wave uses one descriptor; only a
  // last round with NF % 4 != 0 tests q < NF
  const rsrc_t mine = (PL == 2 && (wave & 1)) ? lr : br;
  auto load = [&](Step& x, int64_t tt) {  // tt: first token of the step, relative to t_begin
#pragma unroll
    for (int i = 0; i < NFW; ++i) {
      const int q = wave + 4 * i;
      const int tile16 = q / (KS * PL), ks = (q % (KS * PL)) / PL;
      const int64_t t = tt + 16 * tile16 + row16;
      // rows >= `rows` fall outside the descriptor
      const uint32_t ro = (4 * i + 4 <= NF || q < NF) ? (uint32_t)(t * r * kEs) : kOOB;
      x.f[i] = bld_r8<R8>(mine, ro, r, ks * 32 + grp * 8);
    }
    if constexpr (ADD) {
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int64_t t = tt + 16 * h2 + row16;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          const int cb = cl + 32 * (i / (W8 / 4)) + 4 * (i % (W8 / 4));
          const uint32_t o = (won && cb < r) ? (uint32_t)((t * r + cb) * kEs) : kOOB;
#if RESBM_IO_F32_BUILD
          x.id[h2][i] = bld16(ir, o);
#else
          x.id[h2][i] = bld8(ir, o);
#endif
        }
      }
    }
  };
  auto put = [&](const Step& x, int buf) {
#pragma unroll
    for (int i = 0; i < NFW; ++i)
      if (4 * i + 4 <= NF || wave + 4 * i < NF) s_in[buf][wave + 4 * i][l] = x.f[i];
  };
  // The products of one step (two 16-token tiles) from buffer buf.  Both tiles
  // and, at CT <= 2, two k-step parities accumulate separately, so that at
  // least eight independent accumulation chains keep the matrix cores busy;
  // the parities are added at the end.
  constexpr int PAR = CT <= 2 ? 2 : 1;
  auto products = [&](int buf, f32x4 (&acc)[2][CT]) {
    f32x4 part[2][PAR][CT];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int pa = 0; pa < PAR; ++pa)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) part[h2][pa][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the fragments of k-step ks + 1 are read while those of ks are multiplied
    XFrag cur[2][PL], nxt[2][PL];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int pl = 0; pl < PL; ++pl) cur[h2][pl] = s_in[buf][h2 * KS * PL + pl][l];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
          for (int pl = 0; pl < PL; ++pl) nxt[h2][pl] = s_in[buf][(h2 * KS + ks + 1) * PL + pl][l];
      }
      // keep the next k-step's reads ahead of this k-step's products (left to
      // itself the compiler issues each read right before its first use and
      // waits for it there)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        if constexpr (GZ) {
          SFrag g;
#if RESBM_IO_F32_BUILD
#pragma unroll
          for (int e = 0; e < 8; ++e) g.v[e] = cur[h2][0].v[e];
#else
          g.hi = cur[h2][0].v;
          g.lo = cur[h2][PL - 1].v;
#endif
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) part[h2][ks % PAR][ct] = mma_ss(wfr[ks][ct], g, part[h2][ks % PAR][ct]);
        } else {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
            part[h2][ks % PAR][ct] = mma_sx(wfr[ks][ct], cur[h2][0], part[h2][ks % PAR][ct]);
        }
      }
      if (ks + 1 < KS) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
          for (int pl = 0; pl < PL; ++pl) cur[h2][pl] = nxt[h2][pl];
      }
    }
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        acc[h2][ct] = part[h2][0][ct];
#pragma unroll
        for (int pa = 1; pa < PAR; ++pa) acc[h2][ct] += part[h2][pa][ct];
      }
  };
  // rounds and stores one 16-token tile (tokens tt .. tt + 15 relative to t_begin)
  auto epilogue = [&](const f32x4 (&acc)[CT], int64_t tt, const IdT* idr) {
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      float v[W8];
#pragma unroll
      for (int q = 0; q < W8 / 4; ++q) {
        float id[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (ADD) {
          const auto u = idr[h * (W8 / 4) + q];
#if RESBM_IO_F32_BUILD
          id[0] = __builtin_bit_cast(float, u.x); id[1] = __builtin_bit_cast(float, u.y);
          id[2] = __builtin_bit_cast(float, u.z); id[3] = __builtin_bit_cast(float, u.w);
#else
          id[0] = bf16_bits_to_f32(u.x & 0xffffu); id[1] = bf16_bits_to_f32(u.x >> 16);
          id[2] = bf16_bits_to_f32(u.y & 0xffffu); id[3] = bf16_bits_to_f32(u.y >> 16);
#endif
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) v[4 * q + e] = ADD ? acc[2 * h + q][e] + id[e] : acc[2 * h + q][e];
      }
      io_t* d = tile + row16 * WC + tile_col<WC>(row16, cl - c0 + 32 * h);
#pragma unroll
      for (int e = 0; e < W8; ++e) d[e] = f32_to_io(v[e]);
    }
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const int idx = l + 64 * q;
      const int row = idx / CPR, c8 = 8 * (idx % CPR);
      const XFrag o = tile_get8<WC>(tile, row < 16 ? row : 0, c8);
      bst_frag(zr, (tt < 0 || row >= 16) ? kOOB : (uint32_t)(((tt + row) * ld_out + c0 + c8) * kEs), o);
    }
  };

  Step sa, sb;
#pragma unroll
  for (int i = 0; i < NFW; ++i) sa.f[i] = sb.f[i] = xfrag_zero();
  if constexpr (ADD) {
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int i = 0; i < NI; ++i) sa.id[h2][i] = sb.id[h2][i] = {};
  }
  const int64_t nsteps = (rows + 31) / 32;
  // step s covers tokens [32 s, 32 s + 32) of the group; its fetches were
  // issued two steps earlier
  auto body = [&](Step& x, int64_t s) {
    put(x, (int)(s & 1));
    IdT idr[2][NI];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int i = 0; i < NI; ++i) idr[h2][i] = x.id[h2][i];
    load(x, 32 * (s + 2));
    __syncthreads();  // the step's fragments are complete; the other buffer's readers are done
    if (won && s >= 0 && s < nsteps) {
      f32x4 acc[2][CT];
      products((int)(s & 1), acc);
      epilogue(acc[0], 32 * s, idr[0]);
      epilogue(acc[1], 32 * s + 16, idr[1]);
    }
  };
  for (int64_t s = opaque(-2); s < nsteps; s += 2) {
    body(sa, s);
    body(sb, s + 1);
  }
}

}  // namespace resbm

// ============================================================ host side
using namespace resbm;

namespace {

constexpr size_t kIoBytes = sizeof(io_t);

using resbm_host::aligned;
using resbm_host::extent;
using resbm_host::launch_status;
using resbm_host::ld_ok;
using resbm_host::overlap;

// Whether `rows` rows of a streamed T x n matrix with row stride ld fit one
// buffer descriptor (the kernels address a block's rows through one
// descriptor with 32-bit byte offsets).
bool window_ok(int64_t rows, int64_t ld) { return rows * ld * (int64_t)kIoBytes <= kMaxRange; }
// rows of the streamed T x n matrix one block of the row contraction addresses
// through one descriptor: k_rowc_wide's token group, or k_enc_fwd's 16 MT
// tokens (decode_bwd's narrow kernel rebases per 32-token step)
int64_t rowc_rows(const Plan& p, int64_t narrow) { return p.wide ? rw_tok(p.NT) : narrow; }

int32_t check_common(int64_t T, int n, int r, int64_t ws_need, const void* ws, size_t ws_bytes) {
  if (T < 0 || !shape_ok(n, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  if (ws_need > 0) {
    if (!ws) return RESBM_E_NULL;
    if (!aligned(ws, kWsAlign)) return RESBM_E_ALIGN;
    if (ws_bytes < (size_t)ws_need) return RESBM_E_WORKSPACE;
  }
  return RESBM_OK;
}

template <int NT>
void launch_enc_fwd(const Plan& p, int act, const io_t* x, int64_t ld_x, const io_t* z, int64_t ld_z,
                    const void* wf, const float* W_e, io_t* b, float* a_save, hipStream_t st) {
  if constexpr (NT >= kWideNT) {
    hipLaunchKernelGGL((k_rowc_wide<NT, rw_ntw(NT), false, rw_waves(NT), rw_rh(NT)>), dim3(p.rw_nblk),
                       dim3(64 * rw_waves(NT)), 0, st, p.T, p.n, p.r, act,
                       z, ld_z, wf, x, ld_x, b, a_save);
  } else {
    constexpr int MT = ef_mt(NT);
    constexpr int KW = ef_kw(NT);
    hipLaunchKernelGGL((k_enc_fwd<NT, MT, KW>), dim3(p.ef_nblk), dim3(KW * 64), 0, st, p.T, p.n, p.r, act, x, ld_x,
                       z, ld_z, wf, W_e, b, a_save);
  }
}

// The expand kernel's input rows are fetched 8 elements per 16-byte load when
// r % 8 == 0 (else as two 8-byte halves, one of them past r at r % 8 == 4);
// at r = 64 that took decode_fwd from 40 to 28 us and encode_bwd from 112 to 86.
bool expand_r8(int r) { return r % 8 == 0; }

template <int KS>
void launch_dec_fwd(const Plan& p, int add_id, const io_t* b, const float* W_d, io_t* zt, int64_t ld,
                    hipStream_t st) {
  constexpr int CT = df_ct(KS);
#if RESBM_DF_TOKEN_FASTEST
  dim3 grid(p.df_ngrp, p.df_nwg);
#else
  dim3 grid(p.df_nwg, p.df_ngrp);
#endif
  const FinArgs none{};
  const bool r8 = expand_r8(p.r);
#define CALL_DF(ADD, R8)                                                                                           \
  do {                                                                                                             \
    if constexpr (KS >= kExpandWideKS)                                                                            \
      hipLaunchKernelGGL((k_expand_wide<KS, CT, ADD, false, R8>), grid, dim3(256), 0, st, p.T, p.n, p.r, b, b, b, \
                         W_d, zt, ld, p.df_tpg, (int)grid.y, none);                                                \
    else                                                                                                           \
      hipLaunchKernelGGL((k_expand<KS, CT, ADD, false, R8>), grid, dim3(256), 0, st, p.T, p.n, p.r, b, b, b, W_d,  \
                         zt, ld, p.df_tpg, (int)grid.y, none);                                                     \
  } while (0)
  if (add_id) {
    if (r8) CALL_DF(true, true); else CALL_DF(true, false);
  } else {
    if (r8) CALL_DF(false, true); else CALL_DF(false, false);
  }
#undef CALL_DF
}

template <int JT>
void launch_dec_bwd(const Plan& p, const io_t* b, const float* W_d, const io_t* g, int64_t ld, float* gbp,
                    float* dwp, hipStream_t st) {
#if RESBM_XCD_SPREAD
  dim3 grid(p.db_ntg, p.db_ncg, p.db_njg);
#else
  dim3 grid(p.db_ncg, p.db_ntg, p.db_njg);
#endif
  hipLaunchKernelGGL((k_dec_bwd<JT>), grid, dim3(kDbWaves * 64), 0, st, p.T, p.n, p.r, p.RP, b, W_d, g, ld, gbp,
                     dwp, p.db_TB);
}

template <int NT>
void launch_enc_bwd(const Plan& p, int act, const io_t* z, int64_t ld_z, const float* W_e, const float* a_save,
                    const io_t* g_b, io_t* g_z, int64_t ld_gz, int fused, float* dwp, io_t* gh_hi, io_t* gh_lo,
                    FinArgs fin, hipStream_t st) {
  constexpr int KS = (NT + 1) / 2;
  const int silu = act == RESBM_ACT_SILU;
  const bool r8 = expand_r8(p.r);
  if constexpr (NT >= kWideNT) {
    // g_h once, then the dW_e partials of the token groups
    hipLaunchKernelGGL(k_gh, dim3((unsigned)ceil_div(p.T * (p.r / 4), 256)), dim3(256), 0, st, p.T, p.r, silu, g_b,
                       a_save, gh_hi, gh_lo);
    if (r8)
      hipLaunchKernelGGL((k_tokc_wide<NT, tw_ntw(NT), false, true, tw_tsm(NT, false)>), dim3(p.tw_ntg, p.tw_ncb), dim3(512), 0, st,
                         p.T, p.n, p.r, p.RP, z, ld_z, gh_hi, gh_lo, dwp, p.tw_TB);
    else
      hipLaunchKernelGGL((k_tokc_wide<NT, tw_ntw(NT), false, false, tw_tsm(NT, false)>), dim3(p.tw_ntg, p.tw_ncb), dim3(512), 0, st,
                         p.T, p.n, p.r, p.RP, z, ld_z, gh_hi, gh_lo, dwp, p.tw_TB);
  } else {
    constexpr int CT = eb_ct(KS), CW = eb_cw(KS), TW = eb_tw(KS);
#if RESBM_XCD_SPREAD
    dim3 grid(p.eb_ntg, p.eb_ncb);
#else
    dim3 grid(p.eb_ncb, p.eb_ntg);
#endif
    hipLaunchKernelGGL((k_enc_bwd<KS, NT, CT, CW, TW>), grid, dim3(CW * TW * 64), 0, st, p.T, p.n, p.r, p.RP, silu,
                       z, ld_z, a_save, g_b, gh_hi, gh_lo, dwp, p.eb_TB);
  }
  // g_z = g_h W_e^T (+ g_b I_{r x n} when g_x is g_z): the expand kernel of decode_fwd on the split g_h
  constexpr int GCT = df_ct(KS);
#if RESBM_DF_TOKEN_FASTEST
  dim3 ggrid(p.df_ngrp, p.df_nwg);
#else
  dim3 ggrid(p.df_nwg, p.df_ngrp);
#endif
  // the finishing blocks follow in extra grid rows (dispatched after the g_z
  // blocks, run beside them); wide r: a kernel of their own after g_z
  const int main_y = (int)ggrid.y;
  if constexpr (NT < kWideNT) ggrid.y += (unsigned)ceil_div(fin.nb_all, (int64_t)ggrid.x);
#define CALL_GZ(ADD, R8)                                                                                         \
  do {                                                                                                           \
    if constexpr (NT >= kWideNT || KS >= kExpandWideKSGZ)                                                        \
      hipLaunchKernelGGL((k_expand_wide<KS, GCT, ADD, true, R8>), ggrid, dim3(256), 0, st, p.T, p.n, p.r, gh_hi, \
                         gh_lo, g_b, W_e, g_z, ld_gz, p.df_tpg, main_y, fin);                                   \
    else                                                                                                         \
      hipLaunchKernelGGL((k_expand<KS, GCT, ADD, true, R8>), ggrid, dim3(256), 0, st, p.T, p.n, p.r, gh_hi,      \
                         gh_lo, g_b, W_e, g_z, ld_gz, p.df_tpg, main_y, fin);                                   \
  } while (0)
  if (fused) {
    if (r8) CALL_GZ(true, true); else CALL_GZ(true, false);
  } else {
    if (r8) CALL_GZ(false, true); else CALL_GZ(false, false);
  }
#undef CALL_GZ
  if constexpr (NT >= kWideNT)
    hipLaunchKernelGGL(k_enc_bwd_fin, dim3((unsigned)fin.nb_all), dim3(256), 0, st, p.T, p.n, p.r, fin.RP, fin.dwp,
                       fin.ntg, fin.dW_e, fin.accumulate, fin.nb_dw, fin.g_b, fin.g_x, fin.ld_gx);
}

#define RESBM_DISPATCH_NT(NTV, CALL) \
  switch (NTV) {                     \
    case 1: CALL(1); break;          \
    case 2: CALL(2); break;          \
    case 3: CALL(3); break;          \
    case 4: CALL(4); break;          \
    case 5: CALL(5); break;          \
    case 6: CALL(6); break;          \
    case 7: CALL(7); break;          \
    case 8: CALL(8); break;          \
    case 9: CALL(9); break;          \
    case 10: CALL(10); break;        \
    case 11: CALL(11); break;        \
    case 12: CALL(12); break;        \
    case 13: CALL(13); break;        \
    case 14: CALL(14); break;        \
    case 15: CALL(15); break;        \
    case 16: CALL(16); break;        \
    default: return RESBM_E_SHAPE;   \
  }

}  // namespace

// The fixed device-resident scratch of resbm_encode_bwd_noalloc: one array per
// device, held until the process ends and shared by every such call on that
// device.  Host code never uses its name as an address: the device address is
// looked up once per device (scratch_address) and passed to the kernels.
static __device__ __align__(256) unsigned char scratch[RESBM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];

// Device address of `scratch` on the device that runs `stream` (the current
// device for the null stream), taken with hipGetSymbolAddress once per device
// with that device current.
int32_t scratch_address(hipStream_t stream, void** out) {
  int dev = -1;
  if (stream ? hipStreamGetDevice(stream, &dev) != hipSuccess : hipGetDevice(&dev) != hipSuccess) return RESBM_E_HIP;
  if (dev < 0 || dev >= kMaxDevices) return RESBM_E_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return RESBM_E_HIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return RESBM_E_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) return RESBM_E_HIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return RESBM_OK;
}

// encode_bwd with the caller's workspace, or (noalloc) with the device's fixed
// scratch; every argument is validated before the first HIP call.
int32_t encode_bwd_impl(int64_t T, int32_t n, int32_t r, int32_t act, const void* z, int64_t ld_z,
                        const float* W_e, const float* a_save, const void* g_b, void* g_z, int64_t ld_gz,
                        void* g_x, int64_t ld_gx, float* dW_e, int32_t accumulate, void* ws, size_t ws_bytes,
                        bool noalloc, void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (T < 0 || !shape_ok(n, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan p = make_plan(T, n, r);
  if (noalloc) {
    if (p.eb_ws > (size_t)RESBM_NOALLOC_SCRATCH_BYTES) return RESBM_E_WORKSPACE;
  } else {
    int32_t st = check_common(T, n, r, (int64_t)p.eb_ws, ws, ws_bytes);
    if (st) return st;
  }
  if (!z || !W_e || !g_b || !g_z || !dW_e) return RESBM_E_NULL;
  if (act == RESBM_ACT_SILU && !a_save) return RESBM_E_ACT;
  if (!ld_ok(ld_z, n) || !ld_ok(ld_gz, n) || (g_x && !ld_ok(ld_gx, n)) || !window_ok(64, ld_z) ||
      !window_ok(p.df_tpg, ld_gz))
    return RESBM_E_SHAPE;
  if (!aligned(z, 16) || !aligned(W_e, 16) || !aligned(g_b, 16) || !aligned(g_z, 16) || !aligned(dW_e, 16) ||
      (a_save && !aligned(a_save, 16)) || (g_x && !aligned(g_x, 16)))
    return RESBM_E_ALIGN;
  const int fused = g_x != nullptr && g_x == g_z;
  if (fused && ld_gx != ld_gz) return RESBM_E_ALIAS;
  const size_t bz = extent(T, n, ld_z, kIoBytes), bgz = extent(T, n, ld_gz, kIoBytes);
  const size_t bx = (g_x && !fused) ? extent(T, n, ld_gx, kIoBytes) : 0;
  const size_t bb = (size_t)T * r * kIoBytes, ba = a_save ? (size_t)T * r * 4 : 0, bw = (size_t)n * r * 4;
  if (overlap(g_z, bgz, z, bz) || overlap(g_z, bgz, g_b, bb) || overlap(g_z, bgz, a_save, ba) ||
      overlap(g_z, bgz, W_e, bw) || overlap(g_z, bgz, dW_e, bw) || overlap(g_x, bx, z, bz) ||
      overlap(g_x, bx, g_z, bgz) || overlap(g_x, bx, g_b, bb) || overlap(g_x, bx, a_save, ba) ||
      overlap(g_x, bx, W_e, bw) || overlap(g_x, bx, dW_e, bw) || overlap(dW_e, bw, z, bz) ||
      overlap(dW_e, bw, g_b, bb) || overlap(dW_e, bw, a_save, ba) || overlap(dW_e, bw, W_e, bw) ||
      overlap(ws, p.eb_ws, z, bz) || overlap(ws, p.eb_ws, g_z, bgz) || overlap(ws, p.eb_ws, g_x, bx) ||
      overlap(ws, p.eb_ws, g_b, bb) || overlap(ws, p.eb_ws, a_save, ba) || overlap(ws, p.eb_ws, dW_e, bw) ||
      overlap(ws, p.eb_ws, W_e, bw))
    return RESBM_E_ALIAS;
  hipStream_t s = (hipStream_t)stream;
  if (noalloc) {
    const int32_t e = scratch_address(s, &ws);
    if (e) return e;
  }
  float* dwp = (float*)((char*)ws + p.eb_dwp_off);
  io_t* gh_hi = (io_t*)((char*)ws + p.eb_gh_off);
  io_t* gh_lo = gh_hi + (RESBM_IO_F32_BUILD ? 0 : T * r);  // bf16 build: hi and lo planes
  const io_t* Z = (const io_t*)z;
  const io_t* GB = (const io_t*)g_b;
  io_t* GZ = (io_t*)g_z;
  const float* AS = act == RESBM_ACT_SILU ? a_save : nullptr;
  const int64_t nb_dw = ceil_div((int64_t)n * (r / 4), 64);
  const int64_t nb_gx = (g_x && !fused) ? ceil_div(T * (r / 4), 256) : 0;
  const FinArgs fin{p.RP, dwp, p.eb_ntg, dW_e, accumulate, nb_dw, nb_dw + nb_gx, GB, (io_t*)g_x, ld_gx};
#define CALL(NTV) launch_enc_bwd<NTV>(p, act, Z, ld_z, W_e, AS, GB, GZ, ld_gz, fused, dwp, gh_hi, gh_lo, fin, s)
  RESBM_DISPATCH_NT(p.NT, CALL)
#undef CALL
  return launch_status();
}

}  // namespace

extern "C" {

int32_t resbm_encode_fwd(int64_t T, int32_t n, int32_t r, int32_t act, const void* x_attn, int64_t ld_x,
                         const void* z, int64_t ld_z, const float* W_e, void* b, float* a_save, void* ws,
                         size_t ws_bytes, void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (T < 0 || !shape_ok(n, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan p = make_plan(T, n, r);
  int32_t st = check_common(T, n, r, (int64_t)p.ef_ws, ws, ws_bytes);
  if (st) return st;
  if (!x_attn || !z || !W_e || !b) return RESBM_E_NULL;
  if (!ld_ok(ld_x, n) || !ld_ok(ld_z, n) || !window_ok(rowc_rows(p, 16 * p.ef_mt), ld_z)) return RESBM_E_SHAPE;
  if (!aligned(x_attn, 16) || !aligned(z, 16) || !aligned(W_e, 16) || !aligned(b, 16) ||
      (a_save && !aligned(a_save, 16)))
    return RESBM_E_ALIGN;
  const size_t bx = extent(T, n, ld_x, kIoBytes), bz = extent(T, n, ld_z, kIoBytes);
  const size_t bb = (size_t)T * r * kIoBytes, ba = (size_t)T * r * 4, bw = (size_t)n * r * 4;
  if (overlap(b, bb, x_attn, bx) || overlap(b, bb, z, bz) || overlap(b, bb, W_e, bw) ||
      overlap(a_save, ba, x_attn, bx) || overlap(a_save, ba, z, bz) || overlap(a_save, ba, W_e, bw) ||
      overlap(a_save, ba, b, bb) || overlap(ws, p.ef_ws, x_attn, bx) || overlap(ws, p.ef_ws, z, bz) ||
      overlap(ws, p.ef_ws, b, bb) || overlap(ws, p.ef_ws, a_save, ba) || overlap(ws, p.ef_ws, W_e, bw))
    return RESBM_E_ALIAS;

  hipStream_t s = (hipStream_t)stream;
  char* w = (char*)ws;
  void* wf = w + p.ef_wf_off;
  if (!ef_we_lds(p.NT)) {  // fragments for the kernels that read them prepared
    const int64_t nprep = (int64_t)(n / 32) * p.NT * 64;
    hipLaunchKernelGGL(k_enc_fwd_prep, dim3((unsigned)ceil_div(nprep, 64)), dim3(64), 0, s, W_e, n, r, p.NT, wf);
  }
  const io_t* X = (const io_t*)x_attn;
  const io_t* Z = (const io_t*)z;
  io_t* B = (io_t*)b;
#define CALL(NTV) launch_enc_fwd<NTV>(p, act, X, ld_x, Z, ld_z, wf, W_e, B, a_save, s)
  RESBM_DISPATCH_NT(p.NT, CALL)
#undef CALL
  return launch_status();
}

int32_t resbm_decode_fwd(int64_t T, int32_t n, int32_t r, int32_t add_identity, const void* b, const float* W_d,
                         void* z_tilde, int64_t ld_zt, void* ws, size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (T < 0 || !shape_ok(n, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan p = make_plan(T, n, r);
  if (!b || !W_d || !z_tilde) return RESBM_E_NULL;
  if (!ld_ok(ld_zt, n) || !window_ok(p.df_tpg, ld_zt)) return RESBM_E_SHAPE;
  if (!aligned(b, 16) || !aligned(W_d, 16) || !aligned(z_tilde, 16)) return RESBM_E_ALIGN;
  const size_t bz = extent(T, n, ld_zt, kIoBytes), bb = (size_t)T * r * kIoBytes, bw = (size_t)n * r * 4;
  if (overlap(z_tilde, bz, b, bb) || overlap(z_tilde, bz, W_d, bw)) return RESBM_E_ALIAS;
  hipStream_t s = (hipStream_t)stream;
  const io_t* B = (const io_t*)b;
  io_t* Z = (io_t*)z_tilde;
  switch (p.KS) {
    case 1: launch_dec_fwd<1>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 2: launch_dec_fwd<2>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 3: launch_dec_fwd<3>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 4: launch_dec_fwd<4>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 5: launch_dec_fwd<5>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 6: launch_dec_fwd<6>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 7: launch_dec_fwd<7>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    case 8: launch_dec_fwd<8>(p, add_identity, B, W_d, Z, ld_zt, s); break;
    default: return RESBM_E_SHAPE;
  }
  return launch_status();
}

int32_t resbm_decode_bwd(int64_t T, int32_t n, int32_t r, const void* b, const float* W_d, const void* g_zt,
                         int64_t ld_gzt, const void* g_id, int64_t ld_gid, void* g_b, float* dW_d,
                         int32_t accumulate, void* ws, size_t ws_bytes, void* stream) {
  if (T < 0 || !shape_ok(n, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan p = make_plan(T, n, r);
  int32_t st = check_common(T, n, r, (int64_t)p.db_ws, ws, ws_bytes);
  if (st) return st;
  if (!b || !W_d || !g_zt || !g_b || !dW_d) return RESBM_E_NULL;
  if (!ld_ok(ld_gzt, n) || (g_id && !ld_ok(ld_gid, n)) || !window_ok(rowc_rows(p, 32), ld_gzt))
    return RESBM_E_SHAPE;
  if (!aligned(b, 16) || !aligned(W_d, 16) || !aligned(g_zt, 16) || !aligned(g_b, 16) || !aligned(dW_d, 16) ||
      (g_id && !aligned(g_id, 16)))
    return RESBM_E_ALIGN;
  const size_t bb = (size_t)T * r * kIoBytes, bw = (size_t)n * r * 4, bg = extent(T, n, ld_gzt, kIoBytes);
  const size_t bi = g_id ? extent(T, n, ld_gid, kIoBytes) : 0;
  if (overlap(g_b, bb, b, bb) || overlap(g_b, bb, g_zt, bg) || overlap(g_b, bb, g_id, bi) ||
      overlap(g_b, bb, W_d, bw) || overlap(g_b, bb, dW_d, bw) || overlap(dW_d, bw, b, bb) ||
      overlap(dW_d, bw, g_zt, bg) || overlap(dW_d, bw, g_id, bi) || overlap(dW_d, bw, W_d, bw) ||
      overlap(ws, p.db_ws, b, bb) || overlap(ws, p.db_ws, g_zt, bg) || overlap(ws, p.db_ws, g_id, bi) ||
      overlap(ws, p.db_ws, g_b, bb) || overlap(ws, p.db_ws, dW_d, bw) || overlap(ws, p.db_ws, W_d, bw))
    return RESBM_E_ALIAS;
  hipStream_t s = (hipStream_t)stream;
  char* w = (char*)ws;
  float* gbp = (float*)(w + p.db_gbp_off);
  float* dwp = (float*)(w + p.db_dwp_off);
  const io_t* B = (const io_t*)b;
  const io_t* G = (const io_t*)g_zt;
  if (p.wide) {
    void* wf = w + p.db_wf_off;
    const int64_t nprep = (int64_t)(n / 32) * p.NT * 64;
    hipLaunchKernelGGL(k_wd_prep, dim3((unsigned)ceil_div(nprep, 64)), dim3(64), 0, s, W_d, n, r, p.NT, wf);
    const bool r8 = expand_r8(r);
#define CALL(NTV)                                                                                                   \
  do {                                                                                                              \
    if constexpr (NTV >= kWideNT) {                                                                                 \
      hipLaunchKernelGGL((k_rowc_wide<NTV, rw_ntw(NTV), true, rw_waves(NTV), rw_rh(NTV)>), dim3(p.rw_nblk),    \
                         dim3(64 * rw_waves(NTV)), 0, s, T, n, r, 0, G,                                         \
                         ld_gzt, (const void*)wf, (const io_t*)g_id, ld_gid, (io_t*)g_b, (float*)nullptr);         \
      if (r8)                                                                                                       \
        hipLaunchKernelGGL((k_tokc_wide<NTV, tw_ntw(NTV), true, true, tw_tsm(NTV, true)>), dim3(p.tw_ntg, p.tw_ncb), dim3(512), 0, s,  \
                           T, n, r, p.RP, G, ld_gzt, B, B, dwp, p.tw_TB);                                          \
      else                                                                                                          \
        hipLaunchKernelGGL((k_tokc_wide<NTV, tw_ntw(NTV), true, false, tw_tsm(NTV, true)>), dim3(p.tw_ntg, p.tw_ncb), dim3(512), 0, s, \
                           T, n, r, p.RP, G, ld_gzt, B, B, dwp, p.tw_TB);                                          \
    }                                                                                                               \
  } while (0)
    RESBM_DISPATCH_NT(p.NT, CALL)
#undef CALL
    // the ordered sum of the dW_d partials (g_b is complete)
    const int64_t nb_dw = ceil_div((int64_t)r * (n / 4), 64);
    hipLaunchKernelGGL(k_dec_bwd_fin, dim3((unsigned)nb_dw), dim3(256), 0, s, T, n, r, p.RP, (const float*)nullptr, 0,
                       (const io_t*)nullptr, ld_gid, (io_t*)nullptr, (const float*)dwp, p.tw_ntg, dW_d, accumulate,
                       (int64_t)0);
    return launch_status();
  }
  switch (p.db_jt) {
    case 1: launch_dec_bwd<1>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    case 2: launch_dec_bwd<2>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    case 3: launch_dec_bwd<3>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    case 4: launch_dec_bwd<4>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    default: return RESBM_E_SHAPE;
  }
  const int64_t nb_gb = ceil_div(T * (r / 4), 256);
  const int64_t nb_dw = ceil_div((int64_t)r * (n / 4), 64);
  hipLaunchKernelGGL(k_dec_bwd_fin, dim3((unsigned)(nb_gb + nb_dw)), dim3(256), 0, s, T, n, r, p.RP,
                     (const float*)gbp, p.db_ncg, (const io_t*)g_id, ld_gid, (io_t*)g_b, (const float*)dwp,
                     p.db_ntg, dW_d, accumulate, nb_gb);
  return launch_status();
}

int32_t resbm_encode_bwd(int64_t T, int32_t n, int32_t r, int32_t act, const void* z, int64_t ld_z,
                         const float* W_e, const float* a_save, const void* g_b, void* g_z, int64_t ld_gz,
                         void* g_x, int64_t ld_gx, float* dW_e, int32_t accumulate, void* ws, size_t ws_bytes,
                         void* stream) {
  return encode_bwd_impl(T, n, r, act, z, ld_z, W_e, a_save, g_b, g_z, ld_gz, g_x, ld_gx, dW_e, accumulate, ws,
                         ws_bytes, false, stream);
}

int32_t resbm_encode_bwd_noalloc(int64_t T, int32_t n, int32_t r, int32_t act, const void* z, int64_t ld_z,
                                 const float* W_e, const float* a_save, const void* g_b, void* g_z, int64_t ld_gz,
                                 void* g_x, int64_t ld_gx, float* dW_e, int32_t accumulate, void* stream) {
  return encode_bwd_impl(T, n, r, act, z, ld_z, W_e, a_save, g_b, g_z, ld_gz, g_x, ld_gx, dW_e, accumulate,
                         nullptr, 0, true, stream);
}

size_t resbm_workspace_bytes(int64_t T, int32_t n, int32_t r) {
  if (T < 0 || !shape_ok(n, r)) return 0;
  return make_plan(T, n, r).ws_total;
}

int32_t resbm_io_dtype(void) { return RESBM_IO_F32_BUILD ? RESBM_IO_F32 : RESBM_IO_BF16; }

const char* resbm_strerror(int32_t status) {
  switch (status) {
    case RESBM_OK: return "ok";
    case RESBM_E_NULL: return "a required pointer is NULL";
    case RESBM_E_SHAPE: return "T, n, r or a leading dimension breaks the shape rules";
    case RESBM_E_ALIGN: return "a pointer is not aligned as required";
    case RESBM_E_WORKSPACE: return "workspace smaller than the op requires";
    case RESBM_E_ACT: return "unknown activation, or SiLU backward without a_save";
    case RESBM_E_HIP: return "a HIP kernel launch failed";
    case RESBM_E_ALIAS: return "an output overlaps an input it may not alias";
    default: return "unknown status";
  }
}

}  // extern "C"
