// HIP kernels of the ResBM boundary module for gfx950 and the C ABI around them.
//
// Paper: ResBM, Sec. 3.2 (encoder after the FFN, decoder before the next
// attention, only b crosses the boundary), Sec. 3.3 Eq. 5 (the identity path
// keeps columns [0, r) on the way down and zero-pads on the way up), App. A.3
// (bf16 payload).  The backward kernels are the adjoints of these maps.
//
// Work split (T tokens, hidden n, rank r; every streaming tensor is T x n):
//   encode_fwd  a = z W_e over n: waves own token tiles and walk n; blockIdx.y
//               splits n, and a second kernel adds the splits in a fixed order,
//               then applies phi, the skip and the bf16 rounding.
//   decode_fwd  z~ = b W_d: waves own column strips (W_d held in registers) and
//               walk tokens, writing full 16-byte rows.
//   decode_bwd  one pass over g_z~ gives g_b (contraction over n, per-block
//               partial) and dW_d (contraction over tokens, per-block partial);
//               the token-major tile is transposed through LDS for the latter.
//   encode_bwd  one pass reads z and writes g_z; g_h = g_b phi'(a) is formed
//               once per 32-token step in LDS; dW_e partials as in decode_bwd.
// Partial sums are added by small reduction kernels in index order, so every
// result is reproducible bit for bit.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "resbm.h"
#include "resbm_mfma.hpp"
#include "resbm_plan.hpp"

namespace resbm {

// ============================================================ encode forward
// Fragment-ordered copy of W_e for the A operand of a = z W_e:
// fragment f = ks * NT + nt, lane (row16, grp) holds W_e[32 ks + 8 grp + e][16 nt + row16].
__global__ __launch_bounds__(256) void k_enc_fwd_prep(const float* __restrict__ W_e, int n,
                                                      int r, int NT, void* __restrict__ wf) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
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
#if RESBM_IO_F32_BUILD
  float4* out = reinterpret_cast<float4*>(wf) + (f * 64 + l) * 2;
  out[0] = make_float4(w[0], w[1], w[2], w[3]);
  out[1] = make_float4(w[4], w[5], w[6], w[7]);
#else
  SFrag s = sfrag_from(w);
  uint4* out = reinterpret_cast<uint4*>(wf);
  out[(f * 2 + 0) * 64 + l] = __builtin_bit_cast(uint4, s.hi);
  out[(f * 2 + 1) * 64 + l] = __builtin_bit_cast(uint4, s.lo);
#endif
}

__device__ __forceinline__ SFrag load_wfrag(const void* __restrict__ wf, int64_t f, int l) {
  SFrag s;
#if RESBM_IO_F32_BUILD
  const float4* p = reinterpret_cast<const float4*>(wf) + (f * 64 + l) * 2;
  float4 a = p[0], b = p[1];
  s.v[0] = a.x; s.v[1] = a.y; s.v[2] = a.z; s.v[3] = a.w;
  s.v[4] = b.x; s.v[5] = b.y; s.v[6] = b.z; s.v[7] = b.w;
#else
  const uint4* p = reinterpret_cast<const uint4*>(wf);
  s.hi = __builtin_bit_cast(bf16x8, p[(f * 2 + 0) * 64 + l]);
  s.lo = __builtin_bit_cast(bf16x8, p[(f * 2 + 1) * 64 + l]);
#endif
  return s;
}

// Final encoder epilogue for 4 consecutive columns j0..j0+3 of token t:
// a_save = a; b = x_attn[t, j0:j0+4] + phi(a), rounded once.
__device__ __forceinline__ void enc_fwd_epilogue(int64_t t, int j0, int r, int act, const float (&a)[4],
                                                 const io_t* __restrict__ x_attn, int64_t ld_x,
                                                 io_t* __restrict__ b, float* __restrict__ a_save) {
  if (a_save) *reinterpret_cast<float4*>(a_save + t * r + j0) = make_float4(a[0], a[1], a[2], a[3]);
  float x[4];
  load_x4(x_attn + t * ld_x + j0, x);
  float o[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) o[v] = x[v] + act_phi(a[v], act);
  store_x4(b + t * r + j0, o);
}

// a = z W_e over the k-steps [s*kspl, min(nks, (s+1)*kspl)), 16*MT tokens per wave.
template <int NT, int MT>
__global__ __launch_bounds__(256) void k_enc_fwd(int64_t T, int n, int r, int RP, int act,
                                                 const io_t* __restrict__ x_attn, int64_t ld_x,
                                                 const io_t* __restrict__ z, int64_t ld_z,
                                                 const void* __restrict__ wf, io_t* __restrict__ b,
                                                 float* __restrict__ a_save, float* __restrict__ part,
                                                 int S, int kspl) {
  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = threadIdx.x >> 6;
  const int64_t tok0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * MT);
  const int s = blockIdx.y;
  const int nks = n / 32;
  const int ks0 = s * kspl;
  const int ks1 = min(nks, ks0 + kspl);

  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const io_t* zrow[MT];
  bool ok[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int64_t t = tok0 + 16 * mt + row16;
    ok[mt] = t < T;
    zrow[mt] = z + (ok[mt] ? t : 0) * ld_z + grp * 8;
  }

  XFrag cur[MT], nxt[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    cur[mt] = (ok[mt] && ks0 < ks1) ? load_x8(zrow[mt] + ks0 * 32) : xfrag_zero();

  for (int ks = ks0; ks < ks1; ++ks) {
    const bool more = ks + 1 < ks1;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      nxt[mt] = (ok[mt] && more) ? load_x8(zrow[mt] + (ks + 1) * 32) : xfrag_zero();
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const SFrag w = load_wfrag(wf, (int64_t)ks * NT + nt, l);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt][nt] = mma_sx(w, cur[mt], acc[mt][nt]);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) cur[mt] = nxt[mt];
  }

  // acc[mt][nt][v] = a[tok0 + 16 mt + row16][16 nt + 4 grp + v]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int64_t t = tok0 + 16 * mt + row16;
    if (!ok[mt]) continue;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j0 = nt * 16 + grp * 4;
      if (j0 >= r) continue;
      if (S == 1) {
        float a[4] = {acc[mt][nt][0], acc[mt][nt][1], acc[mt][nt][2], acc[mt][nt][3]};
        enc_fwd_epilogue(t, j0, r, act, a, x_attn, ld_x, b, a_save);
      } else {
        *reinterpret_cast<float4*>(part + ((int64_t)s * T + t) * RP + j0) =
            make_float4(acc[mt][nt][0], acc[mt][nt][1], acc[mt][nt][2], acc[mt][nt][3]);
      }
    }
  }
}

// Adds the S split-n partials of a in split order, then the epilogue.
__global__ __launch_bounds__(256) void k_enc_fwd_fin(int64_t T, int r, int RP, int act,
                                                     const io_t* __restrict__ x_attn, int64_t ld_x,
                                                     const float* __restrict__ part, int S,
                                                     io_t* __restrict__ b, float* __restrict__ a_save) {
  const int nq = r / 4;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= T * nq) return;
  const int64_t t = gid / nq;
  const int j0 = (int)(gid % nq) * 4;
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < S; ++s) {
    const float4 p = *reinterpret_cast<const float4*>(part + ((int64_t)s * T + t) * RP + j0);
    a[0] += p.x; a[1] += p.y; a[2] += p.z; a[3] += p.w;
  }
  enc_fwd_epilogue(t, j0, r, act, a, x_attn, ld_x, b, a_save);
}

// ============================================================ decode forward
// 8 consecutive payload elements b[t][kb .. kb+8) with zeros at k >= r.
__device__ __forceinline__ XFrag load_payload8(const io_t* __restrict__ b, int64_t t, int r, int kb, bool ok) {
  if (!ok || kb >= r) return xfrag_zero();
  const io_t* p = b + t * r + kb;
#if RESBM_IO_F32_BUILD
  XFrag f = xfrag_zero();
  float4 a = *reinterpret_cast<const float4*>(p);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  if (kb + 8 <= r) {
    float4 c = *reinterpret_cast<const float4*>(p + 4);
    f.v[4] = c.x; f.v[5] = c.y; f.v[6] = c.z; f.v[7] = c.w;
  }
  return f;
#else
  if (kb + 8 <= r && (r & 7) == 0) return load_x8(p);
  uint2 lo = *reinterpret_cast<const uint2*>(p);
  uint2 hi = kb + 8 <= r ? *reinterpret_cast<const uint2*>(p + 4) : make_uint2(0, 0);
  XFrag f;
  f.v = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
  return f;
#endif
}

// Stores cnt = 4*CT consecutive values (16-byte aligned when cnt >= 8 for bf16).
template <int CNT>
__device__ __forceinline__ void store_row(io_t* __restrict__ p, const float (&v)[CNT]) {
#if RESBM_IO_F32_BUILD
#pragma unroll
  for (int q = 0; q < CNT / 4; ++q)
    *reinterpret_cast<float4*>(p + 4 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
#else
  if constexpr (CNT >= 8) {
#pragma unroll
    for (int q = 0; q < CNT / 8; ++q) {
      bf16x8 h;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = to_bf16(v[8 * q + e]);
      *reinterpret_cast<uint4*>(p + 8 * q) = __builtin_bit_cast(uint4, h);
    }
  } else {
    float w[4] = {v[0], v[1], v[2], v[3]};
    store_x4(p, w);
  }
#endif
}

// z~ = b W_d (+ b I_{r x n}).  A wave owns columns [c0, c0 + 16 CT) with the
// A-operand row i of column tile ct mapped to column c0 + 4 CT (i / 4) + 4 ct + i % 4,
// so that lane (row16, grp) ends up holding 4 CT consecutive columns of token row16.
template <int KS, int CT>
__global__ __launch_bounds__(256) void k_dec_fwd(int64_t T, int n, int r, int add_id,
                                                 const io_t* __restrict__ b, const float* __restrict__ W_d,
                                                 io_t* __restrict__ zt, int64_t ld_zt, int tpg) {
  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = threadIdx.x >> 6;
  const int strip = blockIdx.x * 4 + wave;
  const int c0 = strip * 16 * CT;
  if (c0 >= n) return;  // whole strips only: n % 64 == 0 and 16 CT divides 64

  SFrag wfr[KS][CT];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int col = c0 + 4 * CT * (row16 >> 2) + 4 * ct + (row16 & 3);
      float w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = ks * 32 + grp * 8 + e;
        w[e] = k < r ? W_d[(int64_t)k * n + col] : 0.0f;
      }
      wfr[ks][ct] = sfrag_from(w);
    }

  const int64_t t_begin = (int64_t)blockIdx.y * tpg;
  const int64_t t_end = min(T, t_begin + tpg);
  const int cl = c0 + 4 * CT * grp;  // first column held by this lane

  XFrag cur[KS], nxt[KS];
  {
    const int64_t t = t_begin + row16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) cur[ks] = load_payload8(b, t, r, ks * 32 + grp * 8, t < t_end);
  }
  for (int64_t tt = t_begin; tt < t_end; tt += 16) {
    const int64_t t = tt + row16;
    const bool ok = t < t_end;
    {
      const int64_t tn = t + 16;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) nxt[ks] = load_payload8(b, tn, r, ks * 32 + grp * 8, tn < t_end);
    }
    f32x4 acc[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) acc[ct] = mma_sx(wfr[ks][ct], cur[ks], acc[ct]);
    if (ok) {
      float v[4 * CT];
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * ct + q] = acc[ct][q];
      if (add_id && cl < r) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const int cb = cl + 4 * ct;
          if (cb < r) {
            float x[4];
            load_x4(b + t * r + cb, x);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[4 * ct + q] += x[q];
          }
        }
      }
      store_row<4 * CT>(zt + t * ld_zt + cl, v);
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) cur[ks] = nxt[ks];
  }
}

// ============================================================ decode backward
// LDS pitches (elements) chosen to spread the transposed 2-byte reads over banks.
constexpr int kDbWaves = 8;
constexpr int kDbWC = 64;                 // columns per wave
constexpr int kDbGzPitch = kDbWC + 8;     // s_gz row pitch
constexpr int kBtPitch = 32 + 8;          // transposed payload / g_h row pitch

// One pass over g_z~ for token range [tg*TB, ...) and columns [cg*512, cg*512 + 512),
// j-tiles [16 jt0, 16 (jt0 + JT)) of r:
//   gbp[cg][t][j]  = sum_{c in block} g_z~[t][c] W_d[j][c]
//   dwp[tg][j][c]  = sum_{t in block} b[t][j] g_z~[t][c]
template <int JT>
__global__ __launch_bounds__(512) void k_dec_bwd(int64_t T, int n, int r, int RP,
                                                 const io_t* __restrict__ b, const float* __restrict__ W_d,
                                                 const io_t* __restrict__ g_zt, int64_t ld_g,
                                                 float* __restrict__ gbp, float* __restrict__ dwp, int TB) {
  constexpr int KSW = kDbWC / 32;  // 32-column steps per wave
  constexpr int CTW = kDbWC / 16;  // 16-column tiles per wave
  constexpr int JW = JT * 16;      // j values per pass
  __shared__ __attribute__((aligned(16))) io_t s_gz[kDbWaves][32][kDbGzPitch];
  __shared__ __attribute__((aligned(16))) io_t s_bT[JW][kBtPitch];
  __shared__ __attribute__((aligned(16))) float s_gb[kDbWaves][32][JW];

  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = threadIdx.x >> 6;
  const int cg = blockIdx.x, tg = blockIdx.y;
  const int jt0 = blockIdx.z * JT;
  const int wc0 = cg * (kDbWaves * kDbWC) + wave * kDbWC;
  const bool won = wc0 < n;  // n % 64 == 0: a wave's 64 columns are all in or all out

  // W_d as the A operand of g_b: lane (row16, grp) holds W_d[16 (jt0 + jt) + row16][wc0 + 32 ks + 8 grp + e].
  SFrag wdf[JT][KSW];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt)
#pragma unroll
    for (int ks = 0; ks < KSW; ++ks) {
      const int j = 16 * (jt0 + jt) + row16;
      float w[8];
      if (won && j < r) {
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

  for (int64_t t0 = t_begin; t0 < t_end; t0 += 32) {
    // 1. g_z~ rows of this step: gz[th][ks] = g_z~[t0 + 16 th + row16][wc0 + 32 ks + 8 grp + e]
    XFrag gz[2][KSW];
#pragma unroll
    for (int th = 0; th < 2; ++th) {
      const int64_t t = t0 + 16 * th + row16;
      const bool ok = won && t < t_end;
#pragma unroll
      for (int ks = 0; ks < KSW; ++ks)
        gz[th][ks] = ok ? load_x8(g_zt + t * ld_g + wc0 + 32 * ks + 8 * grp) : xfrag_zero();
    }
    // 2. payload transposed into LDS: s_bT[jj][tt] = b[t0 + tt][16 jt0 + jj]
    for (int idx = threadIdx.x; idx < 32 * JW; idx += kDbWaves * 64) {
      const int tt = idx / JW, jj = idx % JW;
      const int64_t t = t0 + tt;
      const int j = 16 * jt0 + jj;
      s_bT[jj][tt] = (t < t_end && j < r) ? b[t * r + j] : f32_to_io(0.0f);
    }
    // 3. g_b partial over this wave's 64 columns: D[j][t]
#pragma unroll
    for (int th = 0; th < 2; ++th)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks) acc = mma_sx(wdf[jt][ks], gz[th][ks], acc);
        *reinterpret_cast<float4*>(&s_gb[wave][16 * th + row16][16 * jt + 4 * grp]) =
            make_float4(acc[0], acc[1], acc[2], acc[3]);
      }
    // 4. stage the wave's tile row-major for the transposed reads
#pragma unroll
    for (int th = 0; th < 2; ++th)
#pragma unroll
      for (int ks = 0; ks < KSW; ++ks) {
#if RESBM_IO_F32_BUILD
        float* d = &s_gz[wave][16 * th + row16][32 * ks + 8 * grp];
#pragma unroll
        for (int e = 0; e < 8; ++e) d[e] = gz[th][ks].v[e];
#else
        *reinterpret_cast<uint4*>(&s_gz[wave][16 * th + row16][32 * ks + 8 * grp]) =
            __builtin_bit_cast(uint4, gz[th][ks].v);
#endif
      }
    __syncthreads();

    // 5. dW_d: D[c][j] = sum_t g_z~[t][c] b[t][j], A = g_z~^T (LDS), B = b^T (LDS)
#pragma unroll
    for (int ct = 0; ct < CTW; ++ct) {
      XFrag a;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
#if RESBM_IO_F32_BUILD
        a.v[e] = s_gz[wave][8 * grp + e][16 * ct + row16];
#else
        a.v[e] = s_gz[wave][8 * grp + e][16 * ct + row16];
#endif
      }
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
        XFrag bb;
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) bb.v[e] = s_bT[16 * jt + row16][8 * grp + e];
#else
        bb.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&s_bT[16 * jt + row16][8 * grp]));
#endif
        dw[ct][jt] = mma_xx(a, bb, dw[ct][jt]);
      }
    }
    // 6. sum the 8 waves' g_b partials in wave order and store this block's partial
    for (int idx = threadIdx.x; idx < 32 * JW; idx += kDbWaves * 64) {
      const int tt = idx / JW, jj = idx % JW;
      const int64_t t = t0 + tt;
      const int j = 16 * jt0 + jj;
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < kDbWaves; ++w) s += s_gb[w][tt][jj];
      if (t < t_end && j < r) gbp[((int64_t)cg * T + t) * RP + j] = s;
    }
    __syncthreads();
  }

  // dw[ct][jt][v] = dW_d partial [16 (jt0 + jt) + row16][wc0 + 16 ct + 4 grp + v]
  if (won) {
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const int j = 16 * (jt0 + jt) + row16;
      if (j >= r) continue;
#pragma unroll
      for (int ct = 0; ct < CTW; ++ct)
        *reinterpret_cast<float4*>(dwp + ((int64_t)tg * RP + j) * n + wc0 + 16 * ct + 4 * grp) =
            make_float4(dw[ct][jt][0], dw[ct][jt][1], dw[ct][jt][2], dw[ct][jt][3]);
    }
  }
}

// g_b = sum_cg gbp[cg] + g_id[:, :r]  (rounded once), then
// dW_d (+)= sum_tg dwp[tg]; blocks [0, nb_gb) do the first part.
__global__ __launch_bounds__(256) void k_dec_bwd_fin(int64_t T, int n, int r, int RP,
                                                     const float* __restrict__ gbp, int ncg,
                                                     const io_t* __restrict__ g_id, int64_t ld_gid,
                                                     io_t* __restrict__ g_b,
                                                     const float* __restrict__ dwp, int ntg,
                                                     float* __restrict__ dW_d, int accumulate,
                                                     int64_t nb_gb) {
  if ((int64_t)blockIdx.x < nb_gb) {
    const int nq = r / 4;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (gid >= T * nq) return;
    const int64_t t = gid / nq;
    const int j0 = (int)(gid % nq) * 4;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < ncg; ++c) {
      const float4 p = *reinterpret_cast<const float4*>(gbp + ((int64_t)c * T + t) * RP + j0);
      s[0] += p.x; s[1] += p.y; s[2] += p.z; s[3] += p.w;
    }
    if (g_id) {
      float x[4];
      load_x4(g_id + t * ld_gid + j0, x);
#pragma unroll
      for (int v = 0; v < 4; ++v) s[v] += x[v];
    }
    store_x4(g_b + t * r + j0, s);
  } else {
    const int nq = n / 4;
    const int64_t gid = ((int64_t)blockIdx.x - nb_gb) * 256 + threadIdx.x;
    if (gid >= (int64_t)r * nq) return;
    const int j = (int)(gid / nq);
    const int c0 = (int)(gid % nq) * 4;
    float4 s = accumulate ? *reinterpret_cast<const float4*>(dW_d + (int64_t)j * n + c0)
                          : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int g = 0; g < ntg; ++g) {
      const float4 p = *reinterpret_cast<const float4*>(dwp + ((int64_t)g * RP + j) * n + c0);
      acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
    }
    s.x += acc.x; s.y += acc.y; s.z += acc.z; s.w += acc.w;
    *reinterpret_cast<float4*>(dW_d + (int64_t)j * n + c0) = s;
  }
}

// ============================================================ encode backward
// One pass for token range [tg*TB, ...) and columns [cg*64*CT, ...):
//   g_z[t][c] = sum_j g_h[t][j] W_e[c][j]          (written, + g_b when fused with g_x)
//   dwp[tg][c][j] = sum_t z[t][c] g_h[t][j]
// with g_h = g_b * phi'(a_save) formed per 32-token step in LDS (row-major and
// transposed, as hi/lo split fragments).
template <int KS, int NT, int CT>
__global__ __launch_bounds__(256) void k_enc_bwd(int64_t T, int n, int r, int RP, int act,
                                                 const io_t* __restrict__ z, int64_t ld_z,
                                                 const float* __restrict__ W_e, const float* __restrict__ a_save,
                                                 const io_t* __restrict__ g_b,
                                                 io_t* __restrict__ g_z, int64_t ld_gz,
                                                 io_t* __restrict__ g_x, int64_t ld_gx, int gx_fused,
                                                 float* __restrict__ dwp, int TB) {
  constexpr int W = 4;
  constexpr int WC = 16 * CT;          // columns per wave
  constexpr int KP = 32 * KS;          // r padded for the contraction over r
  constexpr int RPT = 16 * NT;         // r padded to output tiles
  constexpr int GP = KP + 8;           // row-major g_h pitch
  constexpr int ZP = WC + 8;           // z tile pitch
#if RESBM_IO_F32_BUILD
  __shared__ __attribute__((aligned(16))) float s_ghr[32][GP];
  __shared__ __attribute__((aligned(16))) float s_ght[RPT][kBtPitch];
#else
  __shared__ __attribute__((aligned(16))) __bf16 s_ghr[2][32][GP];      // [hi/lo][t][j]
  __shared__ __attribute__((aligned(16))) __bf16 s_ght[2][RPT][kBtPitch];  // [hi/lo][j][t]
#endif
  __shared__ __attribute__((aligned(16))) io_t s_z[W][32][ZP];

  const int l = lane_id(), row16 = l & 15, grp = l >> 4, wave = threadIdx.x >> 6;
  const int cg = blockIdx.x, tg = blockIdx.y;
  const int wc0 = (cg * W + wave) * WC;
  const bool won = wc0 < n;  // n % 64 == 0 and WC divides 64

  // W_e as the A operand of g_z: lane (row16, grp) holds W_e[col][32 ks + 8 grp + e],
  // col = wc0 + 4 CT (row16 / 4) + 4 ct + row16 % 4.
  SFrag wef[KS][CT];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int col = wc0 + 4 * CT * (row16 >> 2) + 4 * ct + (row16 & 3);
      float w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = ks * 32 + grp * 8 + e;
        w[e] = (won && j < r) ? W_e[(int64_t)col * r + j] : 0.0f;
      }
      wef[ks][ct] = sfrag_from(w);
    }

  f32x4 dw[CT][NT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int jt = 0; jt < NT; ++jt) dw[ct][jt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t t_begin = (int64_t)tg * TB;
  const int64_t t_end = min(T, t_begin + TB);
  const int cl = wc0 + 4 * CT * grp;  // first g_z column held by this lane

  for (int64_t t0 = t_begin; t0 < t_end; t0 += 32) {
    // 1. g_h for 32 tokens x KP, both layouts
    for (int idx = threadIdx.x; idx < 32 * KP; idx += W * 64) {
      const int tt = idx / KP, j = idx % KP;
      const int64_t t = t0 + tt;
      float gh = 0.0f;
      if (t < t_end && j < r) {
        const float gb = io_to_f32(g_b[t * r + j]);
        const float d = a_save ? act_dphi(a_save[t * r + j], act) : 1.0f;
        gh = gb * d;
        if (g_x && !gx_fused && cg == 0) {
          io_t* px = g_x + t * ld_gx + j;
          *px = f32_to_io(io_to_f32(*px) + gb);
        }
      }
#if RESBM_IO_F32_BUILD
      s_ghr[tt][j] = gh;
      if (j < RPT) s_ght[j][tt] = gh;
#else
      __bf16 h, lo;
      split_hi_lo(gh, h, lo);
      s_ghr[0][tt][j] = h;
      s_ghr[1][tt][j] = lo;
      if (j < RPT) {
        s_ght[0][j][tt] = h;
        s_ght[1][j][tt] = lo;
      }
#endif
    }
    // 2. this wave's z tile, 32 tokens x WC columns, row-major into LDS
#pragma unroll
    for (int q = 0; q < WC / 16; ++q) {
      const int idx = l + 64 * q;
      const int tt = idx / (WC / 8), ch = idx % (WC / 8);
      const int64_t t = t0 + tt;
      XFrag v = (won && t < t_end) ? load_x8(z + t * ld_z + wc0 + 8 * ch) : xfrag_zero();
#if RESBM_IO_F32_BUILD
#pragma unroll
      for (int e = 0; e < 8; ++e) s_z[wave][tt][8 * ch + e] = v.v[e];
#else
      *reinterpret_cast<uint4*>(&s_z[wave][tt][8 * ch]) = __builtin_bit_cast(uint4, v.v);
#endif
    }
    __syncthreads();

    // 3. g_z for two 16-token halves: D[c][t] = sum_j W_e[c][j] g_h[t][j]
    if (won) {
#pragma unroll
      for (int th = 0; th < 2; ++th) {
        f32x4 acc[CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          SFrag g;
#if RESBM_IO_F32_BUILD
#pragma unroll
          for (int e = 0; e < 8; ++e) g.v[e] = s_ghr[16 * th + row16][32 * ks + 8 * grp + e];
#else
          g.hi = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&s_ghr[0][16 * th + row16][32 * ks + 8 * grp]));
          g.lo = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&s_ghr[1][16 * th + row16][32 * ks + 8 * grp]));
#endif
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) acc[ct] = mma_ss(wef[ks][ct], g, acc[ct]);
        }
        const int64_t t = t0 + 16 * th + row16;
        if (t < t_end) {
          float v[4 * CT];
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int q = 0; q < 4; ++q) v[4 * ct + q] = acc[ct][q];
          if (gx_fused && cl < r) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
              const int cb = cl + 4 * ct;
              if (cb < r) {
                float x[4];
                load_x4(g_b + t * r + cb, x);
#pragma unroll
                for (int q = 0; q < 4; ++q) v[4 * ct + q] += x[q];
              }
            }
          }
          store_row<4 * CT>(g_z + t * ld_gz + cl, v);
        }
      }
    }

    // 4. dW_e: D[j][c] = sum_t g_h[t][j] z[t][c], A = g_h^T (LDS), B = z^T (LDS)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      XFrag zb;
#pragma unroll
      for (int e = 0; e < 8; ++e) zb.v[e] = s_z[wave][8 * grp + e][16 * ct + row16];
#pragma unroll
      for (int jt = 0; jt < NT; ++jt) {
        SFrag g;
#if RESBM_IO_F32_BUILD
#pragma unroll
        for (int e = 0; e < 8; ++e) g.v[e] = s_ght[16 * jt + row16][8 * grp + e];
#else
        g.hi = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&s_ght[0][16 * jt + row16][8 * grp]));
        g.lo = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&s_ght[1][16 * jt + row16][8 * grp]));
#endif
        dw[ct][jt] = mma_sx(g, zb, dw[ct][jt]);
      }
    }
    __syncthreads();
  }

  // dw[ct][jt][v] = dW_e partial [wc0 + 16 ct + row16][16 jt + 4 grp + v]
  if (won) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int c = wc0 + 16 * ct + row16;
#pragma unroll
      for (int jt = 0; jt < NT; ++jt) {
        const int j0 = 16 * jt + 4 * grp;
        if (j0 >= r) continue;
        *reinterpret_cast<float4*>(dwp + ((int64_t)tg * n + c) * RP + j0) =
            make_float4(dw[ct][jt][0], dw[ct][jt][1], dw[ct][jt][2], dw[ct][jt][3]);
      }
    }
  }
}

// dW_e (+)= sum_tg dwp[tg] in token-group order.
__global__ __launch_bounds__(256) void k_enc_bwd_fin(int n, int r, int RP, const float* __restrict__ dwp,
                                                     int ntg, float* __restrict__ dW_e, int accumulate) {
  const int nq = r / 4;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (int64_t)n * nq) return;
  const int c = (int)(gid / nq);
  const int j0 = (int)(gid % nq) * 4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int g = 0; g < ntg; ++g) {
    const float4 p = *reinterpret_cast<const float4*>(dwp + ((int64_t)g * n + c) * RP + j0);
    acc.x += p.x; acc.y += p.y; acc.z += p.z; acc.w += p.w;
  }
  float4 s = accumulate ? *reinterpret_cast<const float4*>(dW_e + (int64_t)c * r + j0)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
  s.x += acc.x; s.y += acc.y; s.z += acc.z; s.w += acc.w;
  *reinterpret_cast<float4*>(dW_e + (int64_t)c * r + j0) = s;
}

}  // namespace resbm

// ============================================================ host side
using namespace resbm;

namespace {

constexpr size_t kIoBytes = sizeof(io_t);

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Byte extent of a T x n matrix with row stride ld.
size_t extent(int64_t T, int64_t n, int64_t ld, size_t es) {
  return T > 0 ? (size_t)(((T - 1) * ld + n) * (int64_t)es) : 0;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return pa < pb + nb && pb < pa + na;
}

int32_t launch_status() {
  return hipGetLastError() == hipSuccess ? RESBM_OK : RESBM_E_HIP;
}

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

bool ld_ok(int64_t ld, int n) { return ld >= n && ld % 8 == 0; }

template <int NT>
void launch_enc_fwd(const Plan& p, int act, const io_t* x, int64_t ld_x, const io_t* z, int64_t ld_z,
                    const void* wf, io_t* b, float* a_save, float* part, hipStream_t st) {
  constexpr int MT = NT <= 2 ? 4 : (NT <= 4 ? 2 : 1);
  dim3 grid(p.ef_nblk, p.ef_S);
  hipLaunchKernelGGL((k_enc_fwd<NT, MT>), grid, dim3(256), 0, st, p.T, p.n, p.r, p.RP, act, x, ld_x, z,
                     ld_z, wf, b, a_save, part, p.ef_S, p.ef_kspl);
}

template <int KS>
void launch_dec_fwd(const Plan& p, int add_id, const io_t* b, const float* W_d, io_t* zt, int64_t ld,
                    hipStream_t st) {
  constexpr int CT = KS <= 2 ? 4 : (KS <= 4 ? 2 : 1);
  dim3 grid(p.df_nwg, p.df_ngrp);
  hipLaunchKernelGGL((k_dec_fwd<KS, CT>), grid, dim3(256), 0, st, p.T, p.n, p.r, add_id, b, W_d, zt, ld,
                     p.df_tpg);
}

template <int JT>
void launch_dec_bwd(const Plan& p, const io_t* b, const float* W_d, const io_t* g, int64_t ld, float* gbp,
                    float* dwp, hipStream_t st) {
  dim3 grid(p.db_ncg, p.db_ntg, p.db_njg);
  hipLaunchKernelGGL((k_dec_bwd<JT>), grid, dim3(512), 0, st, p.T, p.n, p.r, p.RP, b, W_d, g, ld, gbp, dwp,
                     p.db_TB);
}

template <int NT>
void launch_enc_bwd(const Plan& p, int act, const io_t* z, int64_t ld_z, const float* W_e, const float* a_save,
                    const io_t* g_b, io_t* g_z, int64_t ld_gz, io_t* g_x, int64_t ld_gx, int fused, float* dwp,
                    hipStream_t st) {
  constexpr int KS = (NT + 1) / 2;
  constexpr int CT = KS <= 2 ? 4 : (KS <= 4 ? 2 : 1);
  dim3 grid(p.eb_ncg, p.eb_ntg);
  hipLaunchKernelGGL((k_enc_bwd<KS, NT, CT>), grid, dim3(256), 0, st, p.T, p.n, p.r, p.RP, act, z, ld_z, W_e,
                     a_save, g_b, g_z, ld_gz, g_x, ld_gx, fused, dwp, p.eb_TB);
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
  if (!ld_ok(ld_x, n) || !ld_ok(ld_z, n)) return RESBM_E_SHAPE;
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
  float* part = (float*)(w + p.ef_part_off);
  const int64_t nprep = (int64_t)(n / 32) * p.NT * 64;
  hipLaunchKernelGGL(k_enc_fwd_prep, dim3((unsigned)ceil_div(nprep, 256)), dim3(256), 0, s, W_e, n, r, p.NT, wf);
  const io_t* X = (const io_t*)x_attn;
  const io_t* Z = (const io_t*)z;
  io_t* B = (io_t*)b;
#define CALL(NTV) launch_enc_fwd<NTV>(p, act, X, ld_x, Z, ld_z, wf, B, a_save, part, s)
  RESBM_DISPATCH_NT(p.NT, CALL)
#undef CALL
  if (p.ef_S > 1) {
    const int64_t nth = T * (r / 4);
    hipLaunchKernelGGL(k_enc_fwd_fin, dim3((unsigned)ceil_div(nth, 256)), dim3(256), 0, s, T, r, p.RP, act, X,
                       ld_x, (const float*)part, p.ef_S, B, a_save);
  }
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
  if (!ld_ok(ld_zt, n)) return RESBM_E_SHAPE;
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
  if (!ld_ok(ld_gzt, n) || (g_id && !ld_ok(ld_gid, n))) return RESBM_E_SHAPE;
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
  switch (p.db_JT) {
    case 1: launch_dec_bwd<1>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    case 2: launch_dec_bwd<2>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    case 3: launch_dec_bwd<3>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    case 4: launch_dec_bwd<4>(p, B, W_d, G, ld_gzt, gbp, dwp, s); break;
    default: return RESBM_E_SHAPE;
  }
  const int64_t nb_gb = ceil_div(T * (r / 4), 256);
  const int64_t nb_dw = ceil_div((int64_t)r * (n / 4), 256);
  hipLaunchKernelGGL(k_dec_bwd_fin, dim3((unsigned)(nb_gb + nb_dw)), dim3(256), 0, s, T, n, r, p.RP,
                     (const float*)gbp, p.db_ncg, (const io_t*)g_id, ld_gid, (io_t*)g_b, (const float*)dwp,
                     p.db_ntg, dW_d, accumulate, nb_gb);
  return launch_status();
}

int32_t resbm_encode_bwd(int64_t T, int32_t n, int32_t r, int32_t act, const void* z, int64_t ld_z,
                         const float* W_e, const float* a_save, const void* g_b, void* g_z, int64_t ld_gz,
                         void* g_x, int64_t ld_gx, float* dW_e, int32_t accumulate, void* ws, size_t ws_bytes,
                         void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (T < 0 || !shape_ok(n, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan p = make_plan(T, n, r);
  int32_t st = check_common(T, n, r, (int64_t)p.eb_ws, ws, ws_bytes);
  if (st) return st;
  if (!z || !W_e || !g_b || !g_z || !dW_e) return RESBM_E_NULL;
  if (act == RESBM_ACT_SILU && !a_save) return RESBM_E_ACT;
  if (!ld_ok(ld_z, n) || !ld_ok(ld_gz, n) || (g_x && !ld_ok(ld_gx, n))) return RESBM_E_SHAPE;
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
  float* dwp = (float*)((char*)ws + p.eb_dwp_off);
  const io_t* Z = (const io_t*)z;
  const io_t* GB = (const io_t*)g_b;
  io_t* GZ = (io_t*)g_z;
  io_t* GX = (io_t*)g_x;
  const float* AS = act == RESBM_ACT_SILU ? a_save : nullptr;
#define CALL(NTV) launch_enc_bwd<NTV>(p, act, Z, ld_z, W_e, AS, GB, GZ, ld_gz, GX, ld_gx, fused, dwp, s)
  RESBM_DISPATCH_NT(p.NT, CALL)
#undef CALL
  const int64_t nth = (int64_t)n * (r / 4);
  hipLaunchKernelGGL(k_enc_bwd_fin, dim3((unsigned)ceil_div(nth, 256)), dim3(256), 0, s, n, r, p.RP,
                     (const float*)dwp, p.eb_ntg, dW_e, accumulate);
  return launch_status();
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
    case RESBM_E_WORKSPACE: return "workspace smaller than resbm_workspace_bytes(T, n, r)";
    case RESBM_E_ACT: return "unknown activation, or SiLU backward without a_save";
    case RESBM_E_HIP: return "a HIP kernel launch failed";
    case RESBM_E_ALIAS: return "an output overlaps an input it may not alias";
    default: return "unknown status";
  }
}

}  // extern "C"
