// resbm_matrix.hip -- optimizer-side kernels on the bottleneck weights, gfx950.
//
// Sec. 3.4 pairs the bottleneck weights with Muon: a weight matrix moves along
// its gradient momentum orthogonalised by a Newton-Schulz iteration; Sec. 4.1
// trains every bottleneck model that way.  App. B.1 measures a bottleneck
// projection by its effective rank r_eff = sum sigma_i^2 / max sigma_i^2.
// These matrices are n x r or r x n with r <= 256 -- a few MiB at most, tiny
// next to the module's T x n streams -- so every kernel here is latency-bound:
// the design keeps launches few, blocks busy for about a microsecond, and the
// arithmetic in float64 (full vector rate on CDNA4), which costs nothing at
// this size and keeps results within rounding of a float64 reference.
//
// Logical layout.  A p x q matrix is viewed as X (L x s), s = min(p, q),
// L = max(p, q): the matrix itself when p >= q, its transpose otherwise.  X
// lives in the workspace as float64, row-major [L][s4] (s4 = s rounded up to
// a multiple of 4; the padding columns are zero and stay zero).  On the short
// side one Newton-Schulz step is
//     A = X^T X,   B = b A + c A^2,   X <- a X + X B,
// the transpose of the wide-form step X_w <- a X_w + (b A + c A^2) X_w.
//
// Launches per call: k_mx_rows in load mode (float32 input, momentum, X and
// the per-chunk partial Grams), then per step k_mx_reduce (partials -> A in
// chunk order), k_mx_poly (B, and on the first step the Frobenius scale
// kappa = 1 / (||U||_F + eps); for s4 <= 64 the row kernel forms B itself),
// and k_mx_rows (X <- kappa (a X + X B) and the partial Grams of the result;
// on the last step the float32 outputs instead).
// Short side s4 <= 64, few steps: the iteration runs on the s x s Gram alone.
// With X_0 = kappa U and Q_k = a I + b A_k + c A_k^2, X_{k+1} = X_k Q_k, so
// X_k = X_0 P_k with P_0 = I, P_{k+1} = P_k Q_k, and the next Gram is
// A_{k+1} = Q_k A_k Q_k (Q_k is a polynomial in the symmetric A_k).  One block
// (k_mx_small) takes the Gram of U (k_mx_reduce), runs that recurrence in LDS
// and writes R = kappa P_n; one row pass then forms X_n = U R.  Four launches
// instead of 1 + 2n.  Equal to the row-by-row iteration in exact arithmetic;
// in float64 the two agree to ~1e-12 of max |X_n| at the default 5 quintic
// steps.  A direction of A_0 whose computed eigenvalue is a rounding error
// (~1e-16 of the largest, possibly negative) grows by about a^2 per step in
// the recurrence, where the row iteration keeps every Gram positive
// semidefinite: on rank-one inputs the difference reaches ~1e-6 of max |X_n|
// at a^(2n) ~ 1e11.  The recurrence is used only while a^(2n) <= 1e9 (the
// quintic: n <= 8; the cubic: n <= 25), where it stays below ~1e-10.
// No atomics and no waits between blocks: every sum has a fixed order, so
// results are reproducible run to run.
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdint.h>

#include "resbm.h"
#include "resbm_host.hpp"

namespace resbm_mx {

constexpr int kThreads = 256;
constexpr int kMaxShort = 256;        // s <= 256
constexpr int kEigLdsMax = 128;         // the eigen-solver keeps s x s in LDS up to here
constexpr int64_t kMaxLong = 1 << 20;
constexpr int kMaxSteps = 100;
constexpr double kNsEps = 1e-7;       // added to ||U||_F before the division
constexpr int kLdsDoubles = 17408;    // 136 KiB of LDS per block

enum Mode { kLoad = 0, kStep = 1, kOutO = 2, kOutW = 3 };

struct Dims {
  int L, s, s4;  // logical rows, short side, short side rounded up to 4
  int tall;      // 1: X is the matrix; 0: X is its transpose
  int q;         // columns (row stride) of the matrix as stored
  int sub;       // rows per LDS sub-chunk of the row kernel
  int ch;        // rows per block
  int nch;       // blocks of the row kernel = partial Grams per step
  int b_lds;     // B fits LDS beside a sub-chunk
  int fuse_b;    // the row kernel forms B (and kappa) itself from A (s4 <= 64)
};

// Index of logical element (row l, column k) in the stored p x q matrix.
__device__ __forceinline__ int64_t phys(const Dims& d, int64_t l, int k) {
  return d.tall ? l * d.q + k : (int64_t)k * d.q + l;
}

// M <- float32(mu M + G); returns the matrix to orthogonalise, M or G + mu M.
// Separate roundings in that order, so that the float32 momentum matches a
// float64 reference bit for bit.
__device__ __forceinline__ double momentum_step(float* m, double gv, double mu, int nesterov) {
#pragma clang fp contract(off)
  const float mn = (float)(mu * (double)*m + gv);
  *m = mn;
  return nesterov ? gv + mu * (double)mn : (double)mn;
}

// ---------------------------------------------------------------- rows
// Block b owns logical rows [b ch, b ch + ch).
//  kLoad: X = U from the float32 input (momentum applied first when given);
//  kStep: X <- kappa (a X + X B);
//  kOutO: out = float32(kappa (a X + X B)) in the stored layout;
//  kOutW: out = float32(W - lr (scale X' + wd W)), X' = kappa (a X + X B);
//  the output modes write from registers and leave X as it was.
// kLoad and kStep then write the chunk's partial Gram part[b] = X^T X (rows of
// the chunk only, s4 x s4).
struct RowArgs {
  double* X;
  double* part;
  const double* B;
  const double* scal;  // scal[0] = kappa (when B comes from k_mx_poly)
  const double* A;     // the reduced Gram (when the row kernel forms B)
  int first;           // first step: kappa = 1 / (sqrt(trace A) + eps)
  double a, cb, cc;    // Newton-Schulz coefficients
  const float* src;    // kLoad: gradient G
  float* mom;          // kLoad: momentum buffer M or NULL
  double mu;
  int nesterov;
  float* out;          // kOutO: O; kOutW: W (read and written)
  double lr, scale, wd;
};

// Results y of logical elements (l0, k0 .. k0 + 3) and, when two, (l1, k0 ..
// k0 + 3) of the row update: kStep keeps them in X; kOutO stores float32(y)
// and kOutW the updated weights at the elements' places in the stored matrix
// (columns >= s are padding and are dropped).  kOutW loads all of its weights
// before the first store.
template <int MODE>
__device__ __forceinline__ void put_rows(const Dims& d, const RowArgs& g, int64_t l0, int64_t l1, bool two, int k0,
                                         const double (&y)[8]) {
  if constexpr (MODE == kStep) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      g.X[l0 * d.s4 + k0 + v] = y[v];
      if (two) g.X[l1 * d.s4 + k0 + v] = y[4 + v];
    }
  } else {
    int64_t pi[8];
    bool ok[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      ok[q] = k0 + (q & 3) < d.s && (q < 4 || two);
      pi[q] = ok[q] ? phys(d, q < 4 ? l0 : l1, k0 + (q & 3)) : 0;
    }
    if constexpr (MODE == kOutO) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (ok[q]) g.out[pi[q]] = (float)y[q];
    } else {
      double w[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = ok[q] ? (double)g.out[pi[q]] : 0.0;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (ok[q]) g.out[pi[q]] = (float)(w[q] - g.lr * (g.scale * y[q] + g.wd * w[q]));
    }
  }
}

template <int MODE>
__global__ __launch_bounds__(kThreads) void k_mx_rows(Dims d, RowArgs g) {
  __shared__ double s_mem[kLdsDoubles];
  const int t = threadIdx.x;
  const int s = d.s, s4 = d.s4;
  const int ts = s4 + 1;  // LDS row stride: an odd number of doubles puts consecutive rows on other banks
  const int64_t r0 = (int64_t)blockIdx.x * d.ch;
  const int64_t r1 = r0 + d.ch < d.L ? r0 + d.ch : d.L;
  if (r0 >= r1) return;  // uniform per block

  if constexpr (MODE == kLoad) {
    // logical rows of the chunk in order of the stored layout (coalesced reads)
    const int rows = (int)(r1 - r0);
    const int total = rows * s;  // <= 2^28
    // eight elements per thread at a time: all their loads are issued before
    // the first store (the stores to M could alias the next loads otherwise)
    constexpr int kB = 8;
    for (int e0 = t; e0 < total; e0 += kB * kThreads) {
      double gv[kB];
      float mv[kB];
      int64_t pis[kB];
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int e = e0 + q * kThreads;
        const int i = d.tall ? e / s : e % rows;
        const int k = d.tall ? e % s : e / rows;
        pis[q] = e < total ? phys(d, r0 + i, k) : -1;
        gv[q] = e < total ? (double)g.src[pis[q]] : 0.0;
        mv[q] = (e < total && g.mom) ? g.mom[pis[q]] : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int e = e0 + q * kThreads;
        if (e >= total) continue;
        const int i = d.tall ? e / s : e % rows;
        const int k = d.tall ? e % s : e / rows;
        double u = gv[q];
        if (g.mom) {
          float m = mv[q];
          u = momentum_step(&m, gv[q], g.mu, g.nesterov);
          g.mom[pis[q]] = m;
        }
        g.X[(r0 + i) * s4 + k] = u;
        if (rows <= d.sub) s_mem[i * ts + k] = u;  // the Gram pass's tile, staged here
      }
    }
    for (int e = t; e < rows * (s4 - s); e += kThreads) {
      g.X[(r0 + e / (s4 - s)) * s4 + s + e % (s4 - s)] = 0.0;
      if (rows <= d.sub) s_mem[(e / (s4 - s)) * ts + s + e % (s4 - s)] = 0.0;
    }
  } else {
    // X <- kappa (a X + X B), one sub-chunk of rows at a time through LDS
    __shared__ double s_kappa;
    double* s_b = s_mem;
    double* tile = s_mem + (d.b_lds ? s4 * s4 : 0);
    const double* Bm = d.b_lds ? s_b : g.B;
    if (d.fuse_b) {
      // B = b kappa^2 A + c kappa^4 A^2 from the reduced Gram, in LDS (A sits in
      // the tile area until B is formed; A is exactly symmetric, so (A^2)[i][j]
      // is the dot product of rows i and j)
      double* s_a = tile;
      for (int e = t; e < s4 * s4; e += kThreads) s_a[(e / s4) * ts + e % s4] = g.A[e];
      __syncthreads();
      if (t == 0) {
        double k = 1.0;
        if (g.first) {
          double tr = 0.0;
          for (int i = 0; i < s4; ++i) tr += s_a[i * ts + i];
          k = 1.0 / (sqrt(tr) + kNsEps);
        }
        s_kappa = k;
      }
      __syncthreads();
      const double k2 = s_kappa * s_kappa;
      for (int e = t; e < s4 * s4; e += kThreads) {
        const double* ri = s_a + (e / s4) * ts;
        const double* rj = s_a + (e % s4) * ts;
        double sq = 0.0;
        for (int m = 0; m < s4; ++m) sq = fma(ri[m], rj[m], sq);
        s_b[e] = g.cb * k2 * ri[e % s4] + g.cc * (k2 * k2) * sq;
      }
    } else {
      if (d.b_lds) {
        for (int e = t; e < s4 * s4; e += kThreads) s_b[e] = g.B[e];
      }
      if (t == 0) s_kappa = g.scal[0];
    }
    __syncthreads();
    const double kappa = s_kappa;
    const int ncg = s4 / 4;
    const int nrg = kThreads / ncg > 0 ? kThreads / ncg : 1;
    const int cg = t % ncg, rg = t / ncg;
    for (int64_t t0 = r0; t0 < r1; t0 += d.sub) {
      const int rows = (int)(r1 - t0 < d.sub ? r1 - t0 : d.sub);
      for (int e = t; e < rows * s4; e += kThreads) tile[(e / s4) * ts + e % s4] = g.X[t0 * s4 + e];
      __syncthreads();
      if (rg < nrg) {
        // two rows per pass share the B loads
        for (int i = rg; i < rows; i += 2 * nrg) {
          const int i2 = i + nrg < rows ? i + nrg : i;
          double acc0[4] = {0.0, 0.0, 0.0, 0.0}, acc1[4] = {0.0, 0.0, 0.0, 0.0};
          const double* x0 = tile + i * ts;
          const double* x1 = tile + i2 * ts;
#pragma unroll 4
          for (int m = 0; m < s4; ++m) {
            const double* br = Bm + m * s4 + 4 * cg;
            double bv[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) bv[v] = br[v];
            const double a0 = x0[m], a1 = x1[m];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              acc0[v] = fma(a0, bv[v], acc0[v]);
              acc1[v] = fma(a1, bv[v], acc1[v]);
            }
          }
          double y[8];
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            y[v] = kappa * fma(g.a, x0[4 * cg + v], acc0[v]);
            y[4 + v] = kappa * fma(g.a, x1[4 * cg + v], acc1[v]);
          }
          put_rows<MODE>(d, g, t0 + i, t0 + i2, i2 != i, 4 * cg, y);
        }
      }
      __syncthreads();  // the tile is reloaded next
    }
  }

  if constexpr (MODE == kOutO || MODE == kOutW) {
    return;  // the outputs were written by the row update
  } else {
    // partial Gram of the chunk: part[b][i][j] = sum over its rows of X[l][i] X[l][j],
    // 4 x 4 entry blocks per thread; row groups (small s4) are added in order
    __syncthreads();  // this block's rows of X are complete
    double* tile = s_mem;
    double* red = s_mem + d.sub * ts;
    const int nb4 = s4 / 4, nblk = nb4 * nb4;
    const int R = nblk < kThreads ? kThreads / nblk : 1;
    const int groups = nblk <= kThreads ? 1 : (nblk + 4 * kThreads - 1) / (4 * kThreads);
    double* part = g.part + (int64_t)blockIdx.x * s4 * s4;
    for (int grp = 0; grp < groups; ++grp) {
      // this pass: blocks blk = t + kThreads (4 grp + u), u < 4 (large s4), or blk = t % nblk (small s4)
      double acc[4][4][4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) acc[u][x][y] = 0.0;
      const int rgp = R > 1 ? t / nblk : 0;
      for (int64_t t0 = r0; t0 < r1; t0 += d.sub) {
        const int rows = (int)(r1 - t0 < d.sub ? r1 - t0 : d.sub);
        // in load mode a chunk of one sub-chunk is in the tile already
        if (MODE != kLoad || r1 - r0 > d.sub)
          for (int e = t; e < rows * s4; e += kThreads) tile[(e / s4) * ts + e % s4] = g.X[t0 * s4 + e];
        __syncthreads();
        if (rgp < R) {
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int blk = R > 1 ? t % nblk : t + kThreads * (4 * grp + u);
            if ((R > 1 && u > 0) || blk >= nblk) continue;
            const int bi = blk / nb4, bj = blk % nb4;
            for (int i = rgp; i < rows; i += R) {
              const double* xr = tile + i * ts;
              double xa[4], xb[4];
#pragma unroll
              for (int v = 0; v < 4; ++v) { xa[v] = xr[4 * bi + v]; xb[v] = xr[4 * bj + v]; }
#pragma unroll
              for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) acc[u][x][y] = fma(xa[x], xb[y], acc[u][x][y]);
            }
          }
        }
        __syncthreads();
      }
      if (R > 1) {
        // row groups meet in LDS, added in group order
        const int blk = t % nblk;
        if (rgp < R) {
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) red[(rgp * nblk + blk) * 16 + 4 * x + y] = acc[0][x][y];
        }
        __syncthreads();
        if (t < nblk) {
          const int bi = t / nb4, bj = t % nb4;
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) {
              double v = red[t * 16 + 4 * x + y];
              for (int k = 1; k < R; ++k) v += red[(k * nblk + t) * 16 + 4 * x + y];
              part[(4 * bi + x) * s4 + 4 * bj + y] = v;
            }
        }
        __syncthreads();
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int blk = t + kThreads * (4 * grp + u);
          if (blk >= nblk) continue;
          const int bi = blk / nb4, bj = blk % nb4;
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) part[(4 * bi + x) * s4 + 4 * bj + y] = acc[u][x][y];
        }
      }
    }
  }
}

// ---------------------------------------------------------------- reduce
// A[e] = sum over chunks, in chunk order, of part[chunk][e].
__global__ __launch_bounds__(kThreads) void k_mx_reduce(int ne, int nch, const double* part, double* A) {
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= ne) return;
  double v = 0.0;
  int c = 0;
  for (; c + 32 <= nch; c += 32) {
    double p[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) p[k] = part[(int64_t)(c + k) * ne + e];
#pragma unroll
    for (int k = 0; k < 32; ++k) v += p[k];
  }
  for (; c < nch; ++c) v += part[(int64_t)c * ne + e];
  A[e] = v;
}

// ---------------------------------------------------------------- poly
// B = b Ah + c Ah^2 with Ah = kappa^2 A; kappa = 1 / (sqrt(trace A) + eps) on
// the first step (X_0 = U / (||U||_F + eps)), else 1.  A is exactly symmetric
// (its (i, j) and (j, i) partial sums take the same products in the same
// order), so (A^2)[i][j] is the dot product of rows i and j.  Block bx owns
// rows [16 bx, 16 bx + 16) of B and walks the rows j in chunks of 16, both
// operands in LDS; block 0 publishes kappa for the row kernel.
__global__ __launch_bounds__(kThreads) void k_mx_poly(int s4, const double* A, double* B, double* scal, int first,
                                                      double cb, double cc) {
  __shared__ double s_i[16 * (kMaxShort + 1)];
  __shared__ double s_j[16 * (kMaxShort + 1)];
  __shared__ double s_kappa;
  const int t = threadIdx.x;
  const int ts = s4 + 1;  // padded LDS row stride
  const int i0 = blockIdx.x * 16;
  const int ni = s4 - i0 < 16 ? s4 - i0 : 16;
  for (int e = t; e < ni * s4; e += kThreads) s_i[(e / s4) * ts + e % s4] = A[(int64_t)i0 * s4 + e];
  for (int i = t; i < s4; i += kThreads) s_j[i] = A[(int64_t)i * s4 + i];  // the diagonal, for the trace
  __syncthreads();
  if (t == 0) {
    double k = 1.0;
    if (first) {
      double tr = 0.0;
      for (int i = 0; i < s4; ++i) tr += s_j[i];
      k = 1.0 / (sqrt(tr) + kNsEps);
    }
    s_kappa = k;
    if (blockIdx.x == 0) scal[0] = k;
  }
  const int ii = t / 16, jj = t % 16;
  for (int j0 = 0; j0 < s4; j0 += 16) {
    const int nj = s4 - j0 < 16 ? s4 - j0 : 16;
    __syncthreads();  // kappa and s_i are ready; the previous chunk's readers are done
    for (int e = t; e < nj * s4; e += kThreads) s_j[(e / s4) * ts + e % s4] = A[(int64_t)j0 * s4 + e];
    __syncthreads();
    if (ii < ni && jj < nj) {
      const double* ri = s_i + ii * ts;
      const double* rj = s_j + jj * ts;
      double sq = 0.0;
      for (int m = 0; m < s4; ++m) sq = fma(ri[m], rj[m], sq);
      const double k2 = s_kappa * s_kappa;
      B[(int64_t)(i0 + ii) * s4 + j0 + jj] = cb * k2 * ri[j0 + jj] + cc * (k2 * k2) * sq;
    }
  }
}

// ---------------------------------------------------------------- short-side recurrence
constexpr int kSmallThreads = 1024;
constexpr int kSmallMax = 64;               // s4 of the short-side recurrence
constexpr int kSmallLd = kSmallMax + 1;     // padded LDS row stride (doubles)

// Z = X Y for s4 x s4 matrices in LDS (row stride ld, zero beyond s4 up to a
// multiple of 16) on the float64 matrix cores: v_mfma_f64_16x16x4_f64 per
// 16 x 16 tile and 4-deep k-step, one tile per wave.  Lane (row16, grp) holds
// A[row16][grp] and B[grp][row16]; its accumulator element v is
// D[grp + 4 v][row16] (measured on gfx950).
// NT = tiles per side (s4 <= 16 NT); the k-steps run to 16 NT over the zero
// padding, all operand loads issued before the products.
template <int NT>
__device__ __forceinline__ void small_mm(const double* X, const double* Y, double* Z, int ld) {
  typedef double d4 __attribute__((ext_vector_type(4)));
  constexpr int KSTEPS = 4 * NT;
  const int l = threadIdx.x & 63, row16 = l & 15, grp = l >> 4, wave = threadIdx.x >> 6;
  if (wave >= NT * NT) return;  // one tile per wave (16 waves >= NT^2)
  const int i0 = 16 * (wave / NT), j0 = 16 * (wave % NT);
  double xa[KSTEPS], yb[KSTEPS];
#pragma unroll
  for (int q = 0; q < KSTEPS; ++q) {
    xa[q] = X[(i0 + row16) * ld + 4 * q + grp];
    yb[q] = Y[(4 * q + grp) * ld + j0 + row16];
  }
  d4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int q = 0; q < KSTEPS; ++q) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(xa[q], yb[q], acc, 0, 0, 0);
#pragma unroll
  for (int v = 0; v < 4; ++v) Z[(i0 + grp + 4 * v) * ld + j0 + row16] = acc[v];
}

// One block: from the reduced Gram A_0 (s4 x s4, row-major), kappa =
// 1 / (sqrt(trace A_0) + eps), then n steps of the recurrence on
// Ab = kappa^2 A_0; writes R = kappa P_n to Rout (s4 x s4, row-major) and 1 to
// scal[0] (the row pass scales by it).
template <int NT>
__global__ __launch_bounds__(kSmallThreads) void k_mx_small(int s4, const double* A0, int n, double a, double b,
                                                            double c, double* Rout, double* scal) {
  __shared__ double s_a[kSmallMax * kSmallLd], s_p[kSmallMax * kSmallLd];
  __shared__ double s_q[kSmallMax * kSmallLd], s_t[kSmallMax * kSmallLd];
  __shared__ double s_kappa;
  const int t = threadIdx.x, ld = kSmallLd, ne = s4 * s4;
  // the matrix-core tiles read up to a multiple of 16 rows and columns: zeros there
  for (int e = t; e < kSmallMax * kSmallLd; e += kSmallThreads) s_a[e] = s_p[e] = s_q[e] = s_t[e] = 0.0;
  __syncthreads();
  for (int e = t; e < ne; e += kSmallThreads) {
    s_a[(e / s4) * ld + e % s4] = A0[e];
    s_p[(e / s4) * ld + e % s4] = (e / s4 == e % s4) ? 1.0 : 0.0;
  }
  __syncthreads();
  if (t == 0) {
    double tr = 0.0;
    for (int i = 0; i < s4; ++i) tr += s_a[i * ld + i];
    s_kappa = 1.0 / (sqrt(tr) + kNsEps);
  }
  __syncthreads();
  const double kappa = s_kappa, k2 = kappa * kappa;
  for (int e = t; e < ne; e += kSmallThreads) s_a[(e / s4) * ld + e % s4] *= k2;
  __syncthreads();
  double* P = s_p;  // P_k and a scratch matrix swap roles after every P Q
  double* U = s_t;
  for (int k = 0; k < n; ++k) {
    small_mm<NT>(s_a, s_a, s_q, ld);  // A^2
    __syncthreads();
    for (int e = t; e < ne; e += kSmallThreads) {
      const int i = e / s4, j = e % s4;
      s_q[i * ld + j] = (i == j ? a : 0.0) + b * s_a[i * ld + j] + c * s_q[i * ld + j];  // Q
    }
    __syncthreads();
    small_mm<NT>(P, s_q, U, ld);  // P Q
    __syncthreads();
    double* w = P;
    P = U;
    U = w;
    if (k + 1 < n) {
      small_mm<NT>(s_a, s_q, U, ld);  // A Q
      __syncthreads();
      small_mm<NT>(s_q, U, s_a, ld);  // next A = Q (A Q)
      __syncthreads();
    }
  }
  for (int e = t; e < ne; e += kSmallThreads) Rout[e] = kappa * P[(e / s4) * ld + e % s4];
  if (t == 0) scal[0] = 1.0;
}

// Whether the short-side recurrence applies: s4 <= 64 and |a|^(2n) <= 1e9.
bool small_ok(int s4, int n, double a) {
  return s4 <= kSmallMax && 2.0 * n * log10(fabs(a) > 1.0 ? fabs(a) : 1.0) <= 9.0;
}

// ---------------------------------------------------------------- spectrum
// Eigenvalues of the s x s Gram A (row stride s4), s <= 128, in one block:
//  1. Householder reduction to a symmetric tridiagonal T (diagonal d, off-
//     diagonal e), in LDS: step k maps column k below the diagonal onto its
//     first entry with H = I - beta v v^T (v0 = x0 - alpha, alpha = -sign(x0)
//     ||x||, so v0 has no cancellation) applied to the trailing block as
//     A <- A - v w^T - w v^T, p = beta A v, w = p - (beta / 2)(v . p) v.  A
//     column already zero below its first entry is left alone (H = I).
//  2. The j-th smallest eigenvalue of T by multisection on Sturm counts
//     (count(x) = number of negative pivots of T - x I = number of eigenvalues
//     below x): a group of K lanes evaluates K interior points of the current
//     interval and keeps the subinterval where the count passes j, from the
//     Gershgorin interval down to 4 ulp of ||T||.
// Both steps are backward stable: the eigenvalues carry an absolute error of a
// few ulp of the largest, as the Gram itself does.  Every sum has a fixed
// order, so results are reproducible.
// sigma[k] = sqrt(max(lambda, 0)) in descending order; r_eff = sum lambda^+ /
// max lambda (0 for the zero matrix).
constexpr int kEigThreads = 512;

// Sum over lanes of wave 0 of v (a butterfly; lane 0's order is fixed).
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// G = false: the s x s matrix (s <= 128) is copied into LDS.  G = true
// (128 < s <= 256): the reduction works in place on the Gram matrix in the
// workspace (512 KiB at most, L2-resident), the block's barriers ordering its
// global reads and writes as they order the LDS ones.  NT threads: 512 for
// s <= 64, else 1024 (more lanes per row and more multisection points per
// eigenvalue pay once the rows are long).
template <bool G, int NT>
__global__ __launch_bounds__(NT) void k_mx_eig(int s, int s4, double* A, double* sigma, double* r_eff) {
  constexpr int SM = G ? kMaxShort : kEigLdsMax;
  constexpr int TPR = NT / SM;  // lanes per row of the matrix-vector products
  __shared__ double M_lds[G ? 1 : SM * (SM + 1)];
  __shared__ double s_v[SM], s_w[SM], s_d[SM], s_e[SM], s_e2[SM], s_lam[SM];
  __shared__ double s_beta, s_k, s_lo, s_hi, s_tn, s_piv;
  __shared__ int s_bad;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  // row stride: padded to an odd count in LDS (columns of M are read across lanes)
  const int ms = G ? s4 : s + 1;
  double* M = G ? A : M_lds;
  if constexpr (!G)
    for (int e = t; e < s * s; e += NT) M[(e / s) * ms + e % s] = A[(e / s) * s4 + e % s];
  __syncthreads();

  // 1. tridiagonal reduction
  for (int k = 0; k + 2 < s; ++k) {
    const int r0 = k + 1, L = s - r0;  // trailing block rows / cols [r0, s), L >= 2
    if (wave == 0) {
      double x2 = 0.0;  // sum of x_i^2 below the first entry (lane i: i, i + 64, ...)
      for (int i = lane; i < L; i += 64)
        if (i >= 1) x2 += M[(r0 + i) * ms + k] * M[(r0 + i) * ms + k];
      x2 = wave_sum(x2);
      if (lane == 0) {
        const double x0 = M[r0 * ms + k];
        s_d[k] = M[k * ms + k];
        if (x2 == 0.0) {  // already reduced
          s_e[k] = x0;
          s_beta = 0.0;
        } else {
          const double nx = sqrt(x0 * x0 + x2);
          const double alpha = x0 >= 0.0 ? -nx : nx;
          const double v0 = x0 - alpha;
          s_e[k] = alpha;
          s_v[0] = v0;
          s_beta = 2.0 / (x2 + v0 * v0);
        }
      }
    }
    for (int i = 1 + t; i < L; i += NT) s_v[i] = M[(r0 + i) * ms + k];
    __syncthreads();
    const double beta = s_beta;
    if (beta == 0.0) {  // uniform; the barrier keeps the next step's writes of s_beta behind every read
      __syncthreads();
      continue;
    }
    // p = beta A22 v: TPR lanes per row, strided columns, combined in a fixed order
    {
      const int i = t / TPR, u = t % TPR;
      double acc = 0.0;
      if (i < L)
        for (int j = u; j < L; j += TPR) acc += M[(r0 + i) * ms + r0 + j] * s_v[j];
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) acc += __shfl_xor(acc, o);
      if (i < L && u == 0) s_w[i] = beta * acc;
    }
    __syncthreads();
    if (wave == 0) {
      double vp = 0.0;
      for (int i = lane; i < L; i += 64) vp += s_v[i] * s_w[i];
      vp = wave_sum(vp);
      if (lane == 0) s_k = 0.5 * beta * vp;
    }
    __syncthreads();
    // A22 -= v w^T + w v^T with w = p - K v formed on the fly (s_w holds p)
    const double kk = s_k;
    for (int e = t; e < L * L; e += NT) {
      const int i = e / L, j = e % L;
      const double vi = s_v[i], vj = s_v[j];
      const double wi = s_w[i] - kk * vi, wj = s_w[j] - kk * vj;
      M[(r0 + i) * ms + r0 + j] -= vi * wj + wi * vj;
    }
    __syncthreads();
  }
  if (t == 0) {
    if (s >= 2) {
      s_d[s - 2] = M[(s - 2) * ms + s - 2];
      s_e[s - 2] = M[(s - 1) * ms + s - 2];
    }
    s_d[s - 1] = M[(s - 1) * ms + s - 1];
    // Gershgorin interval, ||T|| and the smallest pivot magnitude
    double lo = 0.0, hi = 0.0, emax = 0.0;
    // sum of |entries|: non-finite exactly when a NaN or an infinity in W reached
    // the tridiagonal matrix (a finite Gram stays far below the float64 range)
    double mag = 0.0;
    for (int i = 0; i < s; ++i) {
      const double rad = (i > 0 ? fabs(s_e[i - 1]) : 0.0) + (i + 1 < s ? fabs(s_e[i]) : 0.0);
      mag += fabs(s_d[i]) + rad;
      lo = i == 0 || s_d[i] - rad < lo ? s_d[i] - rad : lo;
      hi = i == 0 || s_d[i] + rad > hi ? s_d[i] + rad : hi;
      if (i + 1 < s) {
        s_e2[i] = s_e[i] * s_e[i];
        emax = s_e2[i] > emax ? s_e2[i] : emax;
      }
    }
    const bool finite = isfinite(mag);
    const double tn = fabs(lo) > fabs(hi) ? fabs(lo) : fabs(hi);
    const double piv = DBL_MIN * (emax > 1.0 ? emax : 1.0);
    const double pad = 2.1 * (DBL_EPSILON * tn * s + 2.0 * piv);
    s_lo = lo - pad;
    s_hi = hi + pad;
    s_tn = finite ? tn : 0.0;  // no search on a non-finite matrix
    s_piv = piv;
    s_bad = !finite;
  }
  __syncthreads();

  // 2. multisection: group g of K lanes finds the g-th smallest eigenvalue
  {
    int K = 64;
    while (K > 1 && K * s > NT) K >>= 1;
    const int g = t / K, u = t % K;
    const double tn = s_tn, piv = s_piv;
    if (g < s) {
      double lam = 0.0;
      if (tn > 0.0) {
        double a = s_lo, b = s_hi;
        const double tol = 4.0 * DBL_EPSILON * tn;
        const int sh = lane - u;  // the group's first lane in the wave
        for (int it = 0; it < 200 && b - a > tol; ++it) {
          const double step = (b - a) / (K + 1);
          const double x = a + step * (u + 1);
          // Sturm count: q_i = d_i - x - e_{i-1}^2 / q_{i-1}, with the quotient from the
          // hardware reciprocal and one Newton step (|q| >= piv keeps it finite)
          int c = 0;
          double q = s_d[0] - x;
          if (fabs(q) < piv) q = -piv;
          c += q < 0.0;
          for (int i0 = 1; i0 < s; i0 += 4) {
            double dd[4], ee[4];
#pragma unroll
            for (int u2 = 0; u2 < 4; ++u2) {
              const int i = i0 + u2 < s ? i0 + u2 : s - 1;
              dd[u2] = s_d[i];
              ee[u2] = s_e2[i - 1];
            }
#pragma unroll
            for (int u2 = 0; u2 < 4; ++u2) {
              if (i0 + u2 < s) {
                const double r0 = __builtin_amdgcn_rcp(q);
                const double rq = fma(r0, fma(-q, r0, 1.0), r0);
                q = dd[u2] - x - ee[u2] * rq;
                if (fabs(q) < piv) q = -piv;
                c += q < 0.0;
              }
            }
          }
          // the first point with more than g eigenvalues below it closes the interval
          const uint64_t m = (__ballot(c > g) >> sh) & (K == 64 ? ~0ull : ((1ull << K) - 1));
          if (m == 0) {
            a = a + step * K;
          } else {
            const int f = __builtin_ctzll(m);
            const double nb = a + step * (f + 1);
            if (f > 0) a = a + step * f;
            b = nb;
          }
        }
        lam = 0.5 * (a + b);
      }
      if (u == 0) s_lam[g] = lam;
    }
  }
  __syncthreads();
  if (s_bad) {  // uniform: every output is NaN
    for (int i = t; i < s; i += NT) sigma[i] = __builtin_nan("");
    if (t == 0) r_eff[0] = __builtin_nan("");
    return;
  }
  // descending order by rank (ties by index)
  for (int i = t; i < s; i += NT) {
    const double li = s_lam[i];
    int rank = 0;
    for (int j = 0; j < s; ++j) {
      const double lj = s_lam[j];
      rank += (lj > li) || (lj == li && j < i);
    }
    sigma[rank] = sqrt(li > 0.0 ? li : 0.0);
  }
  if (t == 0) {
    double tot = 0.0, top = 0.0;
    for (int i = 0; i < s; ++i) {
      const double l = s_lam[i] > 0.0 ? s_lam[i] : 0.0;
      tot += l;
      top = l > top ? l : top;
    }
    r_eff[0] = top > 0.0 ? tot / top : 0.0;
  }
}

// ---------------------------------------------------------------- host
size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct Plan {
  Dims d;
  size_t off_x, off_part, off_a, off_b, off_scal, bytes;
};

bool shape_ok(int64_t p, int64_t q, int max_short) {
  const int64_t s = p < q ? p : q, L = p < q ? q : p;
  return s >= 1 && s <= max_short && L <= kMaxLong;
}

Plan make_plan(int p, int q) {
  Plan P{};
  Dims& d = P.d;
  d.tall = p >= q;
  d.L = d.tall ? p : q;
  d.s = d.tall ? q : p;
  d.s4 = (d.s + 3) & ~3;
  d.q = q;
  d.b_lds = d.s4 * d.s4 <= 8192;
  d.fuse_b = d.s4 <= 64;
  const int room = kLdsDoubles - (d.b_lds ? d.s4 * d.s4 : 0);
  // the Gram pass also keeps up to 4096 doubles of row-group sums beside the tile
  int sub = (room - 4096) / (d.s4 + 1);
  sub = sub > 512 ? 512 : sub;
  sub = sub >= 16 ? sub & ~15 : (sub >= 1 ? sub : 1);
  d.sub = sub;
  // Chunks: at least one per 64 rows and one per 2^18 multiply-adds of the
  // row update (L s4^2 in all), at most 256, partial Grams capped at 64 MiB.
  // Fewer chunks make the ordered reduction short; more make each block short.
  const int64_t cap = (int64_t)(64u << 20) / ((int64_t)d.s4 * d.s4 * 8);
  const int64_t by_rows = (d.L + 63) / 64;
  const int64_t by_work = ((int64_t)d.L * d.s4 * d.s4 + (1 << 18) - 1) >> 18;
  int64_t nch = by_rows > by_work ? by_rows : by_work;
  nch = nch > 256 ? 256 : nch;
  if (nch > cap) nch = cap > 0 ? cap : 1;
  const int64_t ch = (d.L + nch - 1) / nch;
  d.ch = (int)ch;
  d.nch = (int)((d.L + ch - 1) / ch);
  size_t off = 0;
  P.off_x = off;
  off += align256((size_t)d.L * d.s4 * 8);
  P.off_part = off;
  off += align256((size_t)d.nch * d.s4 * d.s4 * 8);
  P.off_a = off;
  off += align256((size_t)d.s4 * d.s4 * 8);
  P.off_b = off;
  off += align256((size_t)d.s4 * d.s4 * 8);
  P.off_scal = off;
  off += 256;
  P.bytes = off;
  return P;
}

using resbm_host::aligned;
using resbm_host::launch_status;
using resbm_host::overlap;

int32_t check_ws(const Plan& P, const void* ws, size_t ws_bytes) {
  if (!ws) return RESBM_E_NULL;
  if (!aligned(ws, 256)) return RESBM_E_ALIGN;
  if (ws_bytes < P.bytes) return RESBM_E_WORKSPACE;
  return RESBM_OK;
}

// Load, then `steps` Newton-Schulz steps (at least one launch set; steps == 0
// runs one with coefficients (1, 0, 0), i.e. X_0 itself), the last one in
// output mode MODE_OUT.
template <int MODE_OUT>
void run_ns(const Plan& P, char* ws, RowArgs g, int steps, double a, double b, double c, hipStream_t st) {
  const Dims& d = P.d;
  g.X = (double*)(ws + P.off_x);
  g.part = (double*)(ws + P.off_part);
  g.B = (const double*)(ws + P.off_b);
  g.scal = (const double*)(ws + P.off_scal);
  double* A = (double*)(ws + P.off_a);
  double* B = (double*)(ws + P.off_b);
  double* scal = (double*)(ws + P.off_scal);
  const dim3 grid(d.nch), blk(kThreads);
  hipLaunchKernelGGL(k_mx_rows<kLoad>, grid, blk, 0, st, d, g);
  const int n = steps > 0 ? steps : 1;
  if (steps == 0) { a = 1.0; b = 0.0; c = 0.0; }
  const int ne = d.s4 * d.s4;
  if (small_ok(d.s4, n, a)) {
    // X_n = U R, R from the short-side recurrence: the row pass with a = 0 and
    // B = R, read from the workspace (scal[0] = 1)
    hipLaunchKernelGGL(k_mx_reduce, dim3((ne + kThreads - 1) / kThreads), blk, 0, st, ne, d.nch,
                       (const double*)g.part, A);
    const int nt = (d.s4 + 15) / 16;
    auto small = nt <= 1 ? k_mx_small<1> : nt == 2 ? k_mx_small<2> : nt == 3 ? k_mx_small<3> : k_mx_small<4>;
    hipLaunchKernelGGL(small, dim3(1), dim3(kSmallThreads), 0, st, d.s4, (const double*)A, n, a, b, c, B, scal);
    Dims d2 = d;
    d2.fuse_b = 0;
    RowArgs gi = g;
    gi.a = 0.0;
    hipLaunchKernelGGL(k_mx_rows<MODE_OUT>, grid, blk, 0, st, d2, gi);
    return;
  }
  for (int i = 0; i < n; ++i) {
    hipLaunchKernelGGL(k_mx_reduce, dim3((ne + kThreads - 1) / kThreads), blk, 0, st, ne, d.nch,
                       (const double*)g.part, A);
    if (!d.fuse_b)
      hipLaunchKernelGGL(k_mx_poly, dim3((d.s4 + 15) / 16), blk, 0, st, d.s4, (const double*)A, B, scal,
                         (int)(i == 0), b, c);
    RowArgs gi = g;
    gi.A = A;
    gi.first = i == 0;
    gi.a = a;
    gi.cb = b;
    gi.cc = c;
    if (i + 1 < n)
      hipLaunchKernelGGL(k_mx_rows<kStep>, grid, blk, 0, st, d, gi);
    else
      hipLaunchKernelGGL(k_mx_rows<MODE_OUT>, grid, blk, 0, st, d, gi);
  }
}

}  // namespace resbm_mx

using namespace resbm_mx;

extern "C" {

size_t resbm_matrix_workspace_bytes(int32_t p, int32_t q) {
  if (!shape_ok(p, q, kMaxShort)) return 0;
  return make_plan(p, q).bytes;
}

int32_t resbm_newton_schulz(int32_t p, int32_t q, const float* G, float* O, int32_t steps, double a, double b,
                            double c, void* ws, size_t ws_bytes, void* stream) {
  if (!shape_ok(p, q, kMaxShort) || steps < 0 || steps > kMaxSteps) return RESBM_E_SHAPE;
  if (!G || !O) return RESBM_E_NULL;
  const Plan P = make_plan(p, q);
  const int32_t w = check_ws(P, ws, ws_bytes);
  if (w != RESBM_OK) return w;
  if (!aligned(G, 4) || !aligned(O, 4)) return RESBM_E_ALIGN;
  const size_t bm = (size_t)p * q * 4;
  if (overlap(O, bm, G, bm) || overlap(ws, P.bytes, G, bm) || overlap(ws, P.bytes, O, bm)) return RESBM_E_ALIAS;
  RowArgs g{};
  g.src = G;
  g.out = O;
  run_ns<kOutO>(P, (char*)ws, g, steps, a, b, c, (hipStream_t)stream);
  return launch_status();
}

int32_t resbm_muon_update(int32_t p, int32_t q, float* W, const float* G, float* M, double lr, double momentum,
                          double weight_decay, double scale, int32_t nesterov, int32_t steps, double a, double b,
                          double c, void* ws, size_t ws_bytes, void* stream) {
  if (!shape_ok(p, q, kMaxShort) || steps < 0 || steps > kMaxSteps) return RESBM_E_SHAPE;
  if (!W || !G) return RESBM_E_NULL;
  const Plan P = make_plan(p, q);
  const int32_t w = check_ws(P, ws, ws_bytes);
  if (w != RESBM_OK) return w;
  if (!aligned(W, 4) || !aligned(G, 4) || (M && !aligned(M, 4))) return RESBM_E_ALIGN;
  const size_t bm = (size_t)p * q * 4;
  if (overlap(W, bm, G, bm) || overlap(W, bm, M, bm) || overlap(G, bm, M, bm) || overlap(ws, P.bytes, W, bm) ||
      overlap(ws, P.bytes, G, bm) || overlap(ws, P.bytes, M, bm))
    return RESBM_E_ALIAS;
  RowArgs g{};
  g.src = G;
  g.mom = M;
  g.mu = momentum;
  g.nesterov = nesterov ? 1 : 0;
  g.out = W;
  g.lr = lr;
  // a negative scale selects the cited method's default, 0.2 sqrt(max(p, q))
  g.scale = scale < 0.0 ? 0.2 * sqrt((double)(p > q ? p : q)) : scale;
  g.wd = weight_decay;
  run_ns<kOutW>(P, (char*)ws, g, steps, a, b, c, (hipStream_t)stream);
  return launch_status();
}

int32_t resbm_spectrum(int32_t p, int32_t q, const float* W, double* sigma, double* r_eff, void* ws,
                       size_t ws_bytes, void* stream) {
  if (!shape_ok(p, q, kMaxShort)) return RESBM_E_SHAPE;
  if (!W || !sigma || !r_eff) return RESBM_E_NULL;
  const Plan P = make_plan(p, q);
  const int32_t w = check_ws(P, ws, ws_bytes);
  if (w != RESBM_OK) return w;
  if (!aligned(W, 4) || !aligned(sigma, 8) || !aligned(r_eff, 8)) return RESBM_E_ALIGN;
  const size_t bm = (size_t)p * q * 4, bs = (size_t)P.d.s * 8;
  if (overlap(sigma, bs, r_eff, 8) || overlap(ws, P.bytes, W, bm) || overlap(ws, P.bytes, sigma, bs) ||
      overlap(ws, P.bytes, r_eff, 8) || overlap(sigma, bs, W, bm) || overlap(r_eff, 8, W, bm))
    return RESBM_E_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  char* wsc = (char*)ws;
  RowArgs g{};
  g.X = (double*)(wsc + P.off_x);
  g.part = (double*)(wsc + P.off_part);
  g.src = W;
  const Dims& d = P.d;
  hipLaunchKernelGGL(k_mx_rows<kLoad>, dim3(d.nch), dim3(kThreads), 0, st, d, g);
  const int ne = d.s4 * d.s4;
  double* A = (double*)(wsc + P.off_a);
  hipLaunchKernelGGL(k_mx_reduce, dim3((ne + kThreads - 1) / kThreads), dim3(kThreads), 0, st, ne, d.nch,
                     (const double*)g.part, A);
  constexpr int NT1 = kEigThreads, NT2 = 2 * kEigThreads;
  if (d.s <= 64)
    hipLaunchKernelGGL((k_mx_eig<false, NT1>), dim3(1), dim3(NT1), 0, st, d.s, d.s4, A, sigma, r_eff);
  else if (d.s <= kEigLdsMax)
    hipLaunchKernelGGL((k_mx_eig<false, NT2>), dim3(1), dim3(NT2), 0, st, d.s, d.s4, A, sigma, r_eff);
  else
    hipLaunchKernelGGL((k_mx_eig<true, NT2>), dim3(1), dim3(NT2), 0, st, d.s, d.s4, A, sigma, r_eff);
  return launch_status();
}

}  // extern "C"
