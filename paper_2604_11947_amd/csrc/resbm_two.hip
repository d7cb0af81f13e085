// HIP kernels of the two-linears-per-side bottleneck and of the encoder fused
// into the FFN output projection, for gfx950, and their C ABI.
//
// Paper: ResBM, Sec. 3.2 (encoder and decoder each two linear layers with a
// non-linearity between them; encoder at the end of stage l, decoder at the
// start of stage l+1, only b crosses the boundary), Eq. 2 and Eq. 5 (the
// encoder's skip keeps columns [0, r) of the attention output).  With the
// intermediate width m:
//     encoder  u = z W1,  b = x_attn P^id + phi(u) W2
//     decoder  v = b W3,  z~ = phi(v) W4
// and the backward steps are the adjoints of these maps.
//
// Every step is one launch of a single matrix-core GEMM kernel, C = A B over
// bf16 operands with float32 accumulation, whose two template switches say
// which of A and B is stored K-contiguous.  The steps differ only in a prologue
// (phi applied to the A operand while it is staged into LDS) and an epilogue
// (bf16 or float32 store, multiplication by phi'(X) of a saved pre-activation,
// addition of identity-path columns, a split-K partial sum, or the encoder's
// contraction of the output tile).  The n x m products (2 T n m flops each)
// are matrix-core bound; the r-wide ones stream a T x m tensor and are memory
// bound.
//
// A block computes a BM x BN tile of C in 64-deep stages, double buffered in
// LDS with one barrier per stage and the next stage's loads in flight during
// the current stage's products.  256 x 256 tiles load their operands straight
// into LDS (buffer loads with an LDS destination); the smaller ones go through
// registers (where the phi prologue is applied).  Every wave multiplies its
// (16 FM) x (16 FN) sub-tile with v_mfma_f32_16x16x32_bf16.  The B operand takes the instruction's first slot,
// so a lane's accumulator holds four consecutive columns of one output row and
// stores them with one 8-byte (bf16) or 16-byte (float32) store.
// K-contiguous operands are staged as [rows][64] and read as 16-byte chunks;
// the others as [64][rows] and read transposed with ds_read_b64_tr_b16.
// Split-K partial sums are added in split order by a second kernel, so every
// result is reproducible bit for bit.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "resbm.h"
#include "resbm_buffer.hpp"
#include "resbm_host.hpp"
#include "resbm_mfma.hpp"

namespace resbm2 {

using resbm::bf16x4;
using resbm::bf16x8;
using resbm::bld16;
using resbm::bld8;
using resbm::bst16;
using resbm::bst8;
using resbm::f32x4;
using resbm::kMaxRange;
using resbm::kOOB;
using resbm::make_rsrc;
using resbm::rsrc_t;

constexpr int KT = 64;  // K depth of one stage

enum Epi : int {
  kEpiBf16 = 0,   // C = rne(acc)
  kEpiF32 = 1,    // C = acc (float32)
  kEpiDphi = 2,   // C = rne(acc * phi'(X))   (X: saved pre-activation, same shape as C)
  kEpiAdd = 3,    // C = rne(acc + X) on columns < x_cols, rne(acc) elsewhere
  kEpiPart = 4,   // partial[split] = acc (float32, M x N contiguous per split)
  kEpiBf16Phi = 5,  // C = rne(acc) and D = rne(phi(acc)) (a pre-activation and its activation)
  kEpiEncode = 6,   // C = rne(acc) (the FFN output z) and D[tile column][row] = C_tile W_e[tile rows]
};

struct GemmArgs {
  int M, N, K;
  const void* A; int64_t lda; int64_t a_bytes;
  const void* B; int64_t ldb; int64_t b_bytes;
  void* C; int64_t ldc; int64_t c_bytes;
  const void* X; int64_t ldx; int64_t x_bytes; int x_cols;
  void* D; int64_t ldd; int64_t d_bytes;
  int kc;  // K per split (a multiple of KT); gridDim.z splits
};

// SiLU, a sigmoid(a) with sigmoid(a) = 1 / (1 + 2^(-a log2 e)) from the
// hardware exp2 and reciprocal (about 1 ulp each).
__device__ __forceinline__ float silu(float a) {
  return a * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-a * 1.44269504088896341f));
}

// SiLU on 8 bf16 values, each result rounded to bf16 (the operand the next
// product consumes).
__device__ __forceinline__ uint4 silu8(uint4 v) {
  bf16x8 h = __builtin_bit_cast(bf16x8, v);
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (__bf16)silu((float)h[e]);
  return __builtin_bit_cast(uint4, h);
}

// Column permutation of a [KT][I] tile (I a multiple of 128) that is read with
// ds_read_b64_tr_b16: the low four bits of the 8-element chunk index are XORed
// with 2 (row % 4 + 4 ((row / 8) % 2)).  One transposed read of 32 lanes touches
// two adjacent chunks in each of 8 rows (r0 .. r0 + 3 and r0 + 8 .. r0 + 11);
// the XOR values are 8 distinct even numbers, so the 16 chunks land on 16
// distinct 16-byte bank slots.  Chunks stay in their row and 256-byte window,
// so whole-row copies stay conflict-free too.  (An XOR with the row's low four
// bits leaves two rows of each such read on the same banks.)
__device__ __forceinline__ int tr_col(int row, int col) {
  const int f = ((row & 3) | ((row >> 1) & 4)) << 1;
  return ((((col >> 3) ^ f) & 15) | ((col >> 3) & ~15)) << 3 | (col & 7);
}

// Column permutation of a K-contiguous [I][64] tile: the chunk index is XORed
// with (row / 2) % 8.  dma_tile inverts it when it stages such a tile.
__device__ __forceinline__ int kc_col(int row, int col) {
  return ((((col >> 3) ^ (row >> 1)) & 7) << 3) | (col & 7);
}

// Position of element (row, col) in a staged tile.  K-contiguous operands are
// staged [I][64] (row = index along M or N, col = k); the others [64][I]
// (row = k, col = index), I = 32, 64 or a multiple of 128.
template <bool KC, int I>
__device__ __forceinline__ int tile_pos(int row, int col) {
  if constexpr (KC) {
    static_assert(KT == 64, "kc_col permutes the 8 chunks of a 64-element row");
    return row * KT + kc_col(row, col);
  } else if constexpr (I % 128 == 0) {
    return row * I + tr_col(row, col);
  } else {
    return row * I + resbm::tile_col<I>(row, col);
  }
}

// Operand fragment for 16 indices starting at i0 and the 32-deep K step kk of
// the staged tile: lane (row16, grp) receives Op[i0 + row16][32 kk + 8 grp + e].
template <bool KC, int I>
__device__ __forceinline__ bf16x8 frag(const __bf16* tile, int i0, int kk, int row16, int grp) {
  if constexpr (KC) {
    return __builtin_bit_cast(bf16x8,
                              *reinterpret_cast<const uint4*>(tile + tile_pos<true, I>(i0 + row16, 32 * kk + 8 * grp)));
  } else {
    // Two ds_read_b64_tr_b16: within a 16-lane group, lane j addresses row
    // 32 kk + 8 grp + 4 q + j / 4, columns i0 + 4 (j % 4) .. + 3, and lane i
    // collects four consecutive rows of column i0 + i.
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    s16x4 h[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int row = 32 * kk + 8 * grp + 4 * q + (row16 >> 2);
      const __bf16* p = tile + tile_pos<false, I>(row, i0 + 4 * (row16 & 3));
      h[q] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
    }
    return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){h[0][0], h[0][1], h[0][2], h[0][3],
                                                                                 h[1][0], h[1][1], h[1][2], h[1][3]});
  }
}

// One operand of a GEMM stage: which 16-byte chunks a thread moves from global
// memory into the staged tile.  NI = extent along M or N (for range checks).
template <bool KC, int I, int NTH>
struct Operand {
  static constexpr int CHUNKS = I * KT / 8;
  static constexpr int PER = CHUNKS / NTH;
  static_assert(CHUNKS % NTH == 0, "tile chunks must divide over the block");
  uint4 r[PER];

  // Chunk c covers 8 elements: K-contiguous (row = c / 8 along I, k = 8 (c % 8));
  // otherwise (row = c / (I / 8) along k, index = 8 (c % (I / 8))).
  __device__ __forceinline__ void load(rsrc_t src, int64_t ld, int i0, int NI, int k0, int kend, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = tid + NTH * p;
      int idx, k;
      if constexpr (KC) {
        idx = i0 + c / 8;
        k = k0 + 8 * (c % 8);
      } else {
        k = k0 + c / (I / 8);
        idx = i0 + 8 * (c % (I / 8));
      }
      const bool ok = idx < NI && k < kend;
      const int64_t off = KC ? ((int64_t)idx * ld + k) * 2 : ((int64_t)k * ld + idx) * 2;
      r[p] = bld16(src, ok ? (uint32_t)off : kOOB);
    }
  }
  template <bool PHI>
  __device__ __forceinline__ void put(__bf16* tile, int tid) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = tid + NTH * p;
      const int row = KC ? c / 8 : c / (I / 8);
      const int col = KC ? 8 * (c % 8) : 8 * (c % (I / 8));
      *reinterpret_cast<uint4*>(tile + tile_pos<KC, I>(row, col)) = PHI ? silu8(r[p]) : r[p];
    }
  }
};

// Direct-to-LDS staging of one operand tile (buffer loads with the LDS
// destination): wave w of NW moves the 1 KiB blocks p NW + w of the tile, lane l
// filling bytes [16 l, 16 l + 16) of its block, so each lane fetches the chunk
// whose swizzled position that is (both swizzles are XORs, their own inverse).
// Out-of-range chunks are fetched at kOOB and land as zeros.
template <bool KC, int I, int NW>
__device__ __forceinline__ void dma_tile(rsrc_t src, int64_t ld, int i0, int NI, int k0, int kend, __bf16* tile,
                                         int wave, int lane) {
  static_assert(KC || I % 128 == 0, "direct staging of a k-major tile needs rows of a multiple of 128");
  constexpr int BLOCKS = I * KT * 2 / 1024;
  static_assert(BLOCKS % NW == 0, "tile blocks must divide over the waves");
#pragma unroll
  for (int p = 0; p < BLOCKS / NW; ++p) {
    const int blk = p * NW + wave;
    const int o = blk * 1024 + lane * 16;
    int idx, k;
    if constexpr (KC) {
      const int row = o >> 7, pc = (o >> 4) & 7;
      idx = i0 + row;
      k = k0 + 8 * ((pc ^ (row >> 1)) & 7);  // kc_col's XOR
    } else {
      const int row = o / (I * 2), pc = (o >> 4) % (I / 8);
      const int f = ((row & 3) | ((row >> 1) & 4)) << 1;  // tr_col's XOR
      k = k0 + row;
      idx = i0 + 8 * (((pc ^ f) & 15) | (pc & ~15));
    }
    const bool ok = idx < NI && k < kend;
    const int64_t off = KC ? ((int64_t)idx * ld + k) * 2 : ((int64_t)k * ld + idx) * 2;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (__attribute__((address_space(3))) void*)(tile + blk * 512), 16,
                                             ok ? (uint32_t)off : kOOB, 0, 0, 0);
  }
}

// Block index -> tile index.  Consecutive blocks are dispatched to the eight
// XCDs in turn; each XCD is given a contiguous range of tiles, and tile indices
// run along N first, so the tiles resident on one XCD share the rows of A (the
// token stream in the T-row products) through its L2.
__device__ __forceinline__ int xcd_tile(int id, int nb) {
  const int x = id & 7, li = id >> 3;
  return x * (nb >> 3) + min(x, nb & 7) + li;
}

// Fragment-ordered hi/lo bf16 copy of a row-major float32 matrix W (rows x
// cols, row stride ld) for the B slot of a contraction over its rows: fragment
// f = ks * nc + cb, lane (row16, grp) holds W[32 ks + 8 grp + e][16 cb + row16]
// (zeros outside the matrix); per fragment 1 KiB of hi parts, then 1 KiB of lo
// parts.  One block of 64 lanes per fragment.
__global__ __launch_bounds__(64) void k_frag_prep(const float* __restrict__ W, int rows, int cols, int64_t ld, int nc,
                                                  __bf16* __restrict__ out) {
  const int l = threadIdx.x, row16 = l & 15, grp = l >> 4;
  const int f = blockIdx.x;
  const int ks = f / nc, cb = f % nc;
  const int c = 16 * cb + row16;
  bf16x8 hi, lo;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int j = 32 * ks + 8 * grp + e;
    const float w = (j < rows && c < cols) ? W[(int64_t)j * ld + c] : 0.0f;
    __bf16 h, q;
    resbm::split_hi_lo(w, h, q);
    hi[e] = h;
    lo[e] = q;
  }
  reinterpret_cast<bf16x8*>(out)[(int64_t)(2 * f) * 64 + l] = hi;
  reinterpret_cast<bf16x8*>(out)[(int64_t)(2 * f + 1) * 64 + l] = lo;
}

// Encoder contraction in the epilogue of the FFN output projection (z = h W_down,
// Sec. 3.2 places the encoder right after the feed-forward layer): the block's
// rounded 256 x 256 tile of z goes to LDS (its four stage buffers, 64 rows
// each), and wave w multiplies rows 32 w .. 32 w + 31 of it by the tile's 256
// rows of W_e (float32, as hi + lo bf16 fragments prepared by k_frag_prep, in
// X), writing the float32 partial sum D[tile column][row][0 .. r).  The
// partials are added in tile order by k_enc_finish.
template <int BM, int BN, int WM, int WN, int FM, int FN>
__device__ __forceinline__ void encode_epilogue(const GemmArgs& g, const f32x4 (&acc)[FM][FN], __bf16* q0,
                                                __bf16* q1, __bf16* q2, __bf16* q3, int m0, int n0) {
  static_assert(BM == 256 && BN == 256 && WM * WN == 8, "the encoder epilogue runs on 256 x 256 tiles of 8 waves");
  const int lane = threadIdx.x & 63, row16 = lane & 15, grp = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WM, wn = wave / WM;
  auto quarter = [&](int q) { return q == 0 ? q0 : (q == 1 ? q1 : (q == 2 ? q2 : q3)); };
  __syncthreads();  // every wave has finished reading the last stage
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int ml = (wm * FM + i) * 16 + row16;
    __bf16* q = quarter(ml >> 6);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nl = (wn * FN + j) * 16 + 4 * grp;
      bf16x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = (__bf16)acc[i][j][e];
      *reinterpret_cast<uint2*>(q + (ml & 63) * 256 + resbm::wide_col(ml & 63, nl)) = __builtin_bit_cast(uint2, h);
    }
  }
  __syncthreads();
  const rsrc_t rw = make_rsrc(g.X, g.x_bytes);
  const int r = g.x_cols, nt = n0 / BN, nc = (r + 63) / 64 * 4;
  const __bf16* zq = quarter(wave >> 1);
  const rsrc_t rd = make_rsrc(g.D, g.d_bytes);
  for (int jg = 0; jg < r; jg += 64) {
    f32x4 a2[2][4];
#pragma unroll
    for (int ib = 0; ib < 2; ++ib)
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) a2[ib][jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
    for (int ks = 0; ks < 8; ++ks) {
      bf16x8 zf[2], hi[4], lo[4];
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const uint32_t off = (uint32_t)((((n0 >> 5) + ks) * nc + (jg >> 4) + jb) * 2048 + lane * 16);
        hi[jb] = __builtin_bit_cast(bf16x8, bld16(rw, off));
        lo[jb] = __builtin_bit_cast(bf16x8, bld16(rw, off + 1024));
      }
#pragma unroll
      for (int ib = 0; ib < 2; ++ib) {
        const int row = 32 * (wave & 1) + 16 * ib + row16, col = 32 * ks + 8 * grp;
        zf[ib] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(zq + row * 256 + resbm::wide_col(row, col)));
      }
#pragma unroll
      for (int jb = 0; jb < 4; ++jb)
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
          a2[ib][jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo[jb], zf[ib], a2[ib][jb], 0, 0, 0);
          a2[ib][jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi[jb], zf[ib], a2[ib][jb], 0, 0, 0);
        }
    }
    // lane (row16, grp) of (ib, jb) holds D[row][jg + 16 jb + 4 grp .. + 3] of tile row 32 w + 16 ib + row16
#pragma unroll
    for (int ib = 0; ib < 2; ++ib) {
      const int t = m0 + 32 * wave + 16 * ib + row16;
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const int jj = jg + 16 * jb + 4 * grp;
        const bool ok = t < g.M && jj < r;
        const int64_t off = (((int64_t)nt * g.M + t) * r + jj) * 4;
        bst16(rd, ok ? (uint32_t)off : kOOB, __builtin_bit_cast(uint4, a2[ib][jb]));
      }
    }
  }
}

// LATE (direct staging only): the next stage's loads are issued after the
// first half of the current stage's products instead of before them, so the
// products start right after the barrier; it pays where a block's K depth is
// moderate (2-10 % at 1024 and 4096) and costs where it is long (3 % at 14336).
template <bool AK, bool BKC, int BM, int BN, int WM, int WN, int EPI, bool PHI_A, bool LATE = false>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm(GemmArgs g) {
  constexpr int NTH = 64 * WM * WN;
  constexpr int FM = BM / (16 * WM), FN = BN / (16 * WN);
  static_assert(FM * 16 * WM == BM && FN * 16 * WN == BN, "wave tiling must cover the block tile");
  // Direct-to-LDS staging for the 256 x 256 tiles without an A prologue; the
  // others stage through registers.  Four separate LDS arrays keep the stage
  // buffers distinct objects for the compiler's wait-count analysis.
  constexpr bool kDma = BM == 256 && BN == 256 && !PHI_A;
  __shared__ __attribute__((aligned(16))) __bf16 s_a0[BM * KT], s_a1[BM * KT];
  __shared__ __attribute__((aligned(16))) __bf16 s_b0[BN * KT], s_b1[BN * KT];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int row16 = lane & 15, grp = lane >> 4;
  const int wm = wave % WM, wn = wave / WM;
  const int tiles_n = (g.N + BN - 1) / BN;
  const int t = xcd_tile(blockIdx.x, gridDim.x);
  const int m0 = (t / tiles_n) * BM, n0 = (t % tiles_n) * BN;
  const int kbeg = blockIdx.z * g.kc, kend = min(g.K, kbeg + g.kc);
  const int nst = (kend - kbeg + KT - 1) / KT;

  const rsrc_t ra = make_rsrc(g.A, g.a_bytes), rb = make_rsrc(g.B, g.b_bytes);

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto products_kk = [&](const __bf16* ta, const __bf16* tb, int kk) {
    {
      bf16x8 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) fa[i] = frag<AK, BM>(ta, (wm * FM + i) * 16, kk, row16, grp);
#pragma unroll
      for (int j = 0; j < FN; ++j) fb[j] = frag<BKC, BN>(tb, (wn * FN + j) * 16, kk, row16, grp);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
    }
  };
  static_assert(KT == 64, "a stage is two 32-deep halves");
  auto products = [&](const __bf16* ta, const __bf16* tb) {
    products_kk(ta, tb, 0);
    products_kk(ta, tb, 1);
  };

  if constexpr (kDma) {
    constexpr int NW = WM * WN;
    auto stage = [&](int s, __bf16* a, __bf16* b) {
      dma_tile<AK, BM, NW>(ra, g.lda, m0, g.M, kbeg + s * KT, kend, a, wave, lane);
      dma_tile<BKC, BN, NW>(rb, g.ldb, n0, g.N, kbeg + s * KT, kend, b, wave, lane);
    };
    // Stage s + 1 streams into the other buffers while stage s is multiplied;
    // a stage is complete once every wave has seen its own loads land.
    auto step = [&](int s, const __bf16* a, const __bf16* b, __bf16* na, __bf16* nb) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if constexpr (LATE) {
        products_kk(a, b, 0);
        if (s + 1 < nst) stage(s + 1, na, nb);
        products_kk(a, b, 1);
      } else {
        if (s + 1 < nst) stage(s + 1, na, nb);
        products(a, b);
      }
    };
    if (nst > 0) stage(0, s_a0, s_b0);
    for (int s = 0; s < nst; s += 2) {
      step(s, s_a0, s_b0, s_a1, s_b1);
      if (s + 1 < nst) step(s + 1, s_a1, s_b1, s_a0, s_b0);
    }
  } else {
    Operand<AK, BM, NTH> opa;
    Operand<BKC, BN, NTH> opb;
    if (nst > 0) {
      opa.load(ra, g.lda, m0, g.M, kbeg, kend, tid);
      opb.load(rb, g.ldb, n0, g.N, kbeg, kend, tid);
      opa.template put<PHI_A>(s_a0, tid);
      opb.template put<false>(s_b0, tid);
    }
    __syncthreads();
    for (int s = 0; s < nst; ++s) {
      const bool more = s + 1 < nst;
      if (more) {
        opa.load(ra, g.lda, m0, g.M, kbeg + (s + 1) * KT, kend, tid);
        opb.load(rb, g.ldb, n0, g.N, kbeg + (s + 1) * KT, kend, tid);
      }
      products(s & 1 ? s_a1 : s_a0, s & 1 ? s_b1 : s_b0);
      if (more) {
        opa.template put<PHI_A>(s & 1 ? s_a0 : s_a1, tid);
        opb.template put<false>(s & 1 ? s_b0 : s_b1, tid);
      }
      __syncthreads();
    }
  }

  // Epilogue: lane (row16, grp) of tile (i, j) holds C[m][n .. n + 3].
  const rsrc_t rc = make_rsrc(g.C, g.c_bytes);
  const rsrc_t rx = make_rsrc(g.X, g.x_bytes);
  const rsrc_t rd = make_rsrc(g.D, g.d_bytes);
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + (wm * FM + i) * 16 + row16;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + (wn * FN + j) * 16 + 4 * grp;
      const bool ok = m < g.M && n < g.N;
      f32x4 v = acc[i][j];
      if constexpr (EPI == kEpiF32 || EPI == kEpiPart) {
        const int64_t off = EPI == kEpiPart ? (((int64_t)blockIdx.z * g.M + m) * g.N + n) * 4
                                            : ((int64_t)m * g.ldc + n) * 4;
        bst16(rc, ok ? (uint32_t)off : kOOB, __builtin_bit_cast(uint4, v));
      } else {
        if constexpr (EPI == kEpiDphi || EPI == kEpiAdd) {
          const bool xok = ok && (EPI == kEpiDphi || n < g.x_cols);
          const uint2 xr = bld8(rx, xok ? (uint32_t)(((int64_t)m * g.ldx + n) * 2) : kOOB);
          const bf16x4 x = __builtin_bit_cast(bf16x4, xr);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (EPI == kEpiDphi) v[e] *= resbm::silu_grad((float)x[e]);
            else v[e] += (float)x[e];
          }
        }
        bf16x4 h;
#pragma unroll
        for (int e = 0; e < 4; ++e) h[e] = (__bf16)v[e];
        bst8(rc, ok ? (uint32_t)(((int64_t)m * g.ldc + n) * 2) : kOOB, __builtin_bit_cast(uint2, h));
        if constexpr (EPI == kEpiBf16Phi) {
#pragma unroll
          for (int e = 0; e < 4; ++e) h[e] = (__bf16)silu(v[e]);  // from the float32 accumulator
          bst8(rd, ok ? (uint32_t)(((int64_t)m * g.ldd + n) * 2) : kOOB, __builtin_bit_cast(uint2, h));
        }
      }
    }
  }
  if constexpr (EPI == kEpiEncode) encode_epilogue<BM, BN, WM, WN, FM, FN>(g, acc, s_a0, s_a1, s_b0, s_b1, m0, n0);
}

// ---------------------------------------------------------------- decoder into RMSNorm + QKV
struct DqArgs {
  int T, n, N, r;
  const __bf16* b;       // T x r
  const __bf16* wdf;     // W_d fragments (k_frag_prep)
  const float* gamma;    // n
  const __bf16* W;       // n x N, row-major
  int64_t w_bytes;
  __bf16* out;           // T x N, row stride ld_out
  int64_t ld_out, out_bytes;
  float eps;
};

// out = RMSNorm(b W_d) W_qkv on 256 x 256 output tiles (8 waves of 128 x 64,
// the 64-deep stages of k_gemm).  The A operand of every stage -- 64 columns
// of z~ for the tile's 256 rows -- is rebuilt in the block instead of read:
// wave w forms rows [32 w, 32 w + 32) of it as b W_d (W_d hi and lo: two
// products per 16 x 16 piece and 32-deep k-step of r), multiplies by gamma and
// rounds to bf16 into the LDS tile; W_qkv streams in as in k_gemm.  Each wave
// also sums the squares of its rows' float32 z~ over the whole K loop; the row
// scale 1 / sqrt(mean z~^2 + eps) is applied in the epilogue (RMSNorm is a
// per-row scale of z~ gamma).  The rebuild costs 2 KS / 4 of the tile's
// products (W_d as hi + lo, KS = r / 32 rounded up).
template <int KS>
__global__ __launch_bounds__(512) void k_dec_qkv(DqArgs g) {
  constexpr int BM = 256, BN = 256, WM = 2, WN = 4, NW = 8;
  constexpr int FM = BM / (16 * WM), FN = BN / (16 * WN);
  __shared__ __attribute__((aligned(16))) __bf16 s_a0[BM * KT], s_a1[BM * KT];
  __shared__ __attribute__((aligned(16))) __bf16 s_b0[BN * KT], s_b1[BN * KT];
  __shared__ float s_ssq[BM];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int row16 = lane & 15, grp = lane >> 4;
  const int wm = wave % WM, wn = wave / WM;
  const int tiles_n = (g.N + BN - 1) / BN;
  const int t = xcd_tile(blockIdx.x, gridDim.x);
  const int m0 = (t / tiles_n) * BM, n0 = (t % tiles_n) * BN;
  const int nst = g.n / KT;
  const int nc = g.n / 16;

  const rsrc_t rw = make_rsrc(g.W, g.w_bytes);
  const rsrc_t rbr = make_rsrc(g.b + (int64_t)m0 * g.r, (int64_t)max(0, min(BM, g.T - m0)) * g.r * 2);
  const rsrc_t rwd = make_rsrc(g.wdf, (int64_t)KS * nc * 2048);
  const rsrc_t rg = make_rsrc(g.gamma, (int64_t)g.n * 4);

  // b rows of this wave's rebuild (the A slot: lane holds b[row][32 ks + 8 grp + e])
  bf16x8 bfr[2][KS];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int row = 32 * wave + 16 * rb + row16, j = 32 * ks + 8 * grp;
      bfr[rb][ks] = __builtin_bit_cast(bf16x8, bld16(rbr, j < g.r ? (uint32_t)((row * g.r + j) * 2) : kOOB));
    }
  // W_d fragments and gamma of a stage, loaded one stage ahead
  struct Wd {
    bf16x8 hi[4][KS], lo[4][KS];
    float4 gm[4];
  };
  auto load_wd = [&](Wd& w, int s) {
    const bool ok = s < nst;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int c16 = (s * KT) / 16 + cb;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int64_t f = (int64_t)ks * nc + c16;
        w.hi[cb][ks] = __builtin_bit_cast(bf16x8, bld16(rwd, ok ? (uint32_t)(((2 * f) * 64 + lane) * 16) : kOOB));
        w.lo[cb][ks] = __builtin_bit_cast(bf16x8, bld16(rwd, ok ? (uint32_t)(((2 * f + 1) * 64 + lane) * 16) : kOOB));
      }
      const uint4 gv = bld16(rg, ok ? (uint32_t)((s * KT + 16 * cb + 4 * grp) * 4) : kOOB);
      w.gm[cb] = make_float4(__builtin_bit_cast(float, gv.x), __builtin_bit_cast(float, gv.y),
                             __builtin_bit_cast(float, gv.z), __builtin_bit_cast(float, gv.w));
    }
  };
  float ssq[2] = {0.f, 0.f};
  // z~ gamma for the stage's 64 columns and the wave's 32 rows, into the A tile
  auto rebuild = [&](const Wd& w, __bf16* a) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w.hi[cb][ks], bfr[rb][ks], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w.lo[cb][ks], bfr[rb][ks], acc, 0, 0, 0);
        }
        // lane (row16, grp): z~[row][16 cb + 4 grp + v]
        const float gv[4] = {w.gm[cb].x, w.gm[cb].y, w.gm[cb].z, w.gm[cb].w};
        bf16x4 h;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          ssq[rb] = fmaf(acc[v], acc[v], ssq[rb]);
          h[v] = (__bf16)(acc[v] * gv[v]);
        }
        const int row = 32 * wave + 16 * rb + row16;
        *reinterpret_cast<uint2*>(a + tile_pos<true, BM>(row, 16 * cb + 4 * grp)) = __builtin_bit_cast(uint2, h);
      }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto products_kk = [&](const __bf16* ta, const __bf16* tb, int kk) {
    bf16x8 fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[i] = frag<true, BM>(ta, (wm * FM + i) * 16, kk, row16, grp);
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[j] = frag<false, BN>(tb, (wn * FN + j) * 16, kk, row16, grp);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
  };

  Wd wd;
  load_wd(wd, 0);
  // stage 0: its A tile and the B tile
  rebuild(wd, s_a0);
  load_wd(wd, 1);
  dma_tile<false, BN, NW>(rw, g.N, n0, g.N, 0, g.n, s_b0, wave, lane);
  auto step = [&](int s, const __bf16* a, const __bf16* b, __bf16* na, __bf16* nb) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (s + 1 < nst) {
      dma_tile<false, BN, NW>(rw, g.N, n0, g.N, (s + 1) * KT, g.n, nb, wave, lane);
      rebuild(wd, na);
      load_wd(wd, s + 2);
    }
    products_kk(a, b, 0);
    products_kk(a, b, 1);
  };
  for (int s = 0; s < nst; s += 2) {
    step(s, s_a0, s_b0, s_a1, s_b1);
    if (s + 1 < nst) step(s + 1, s_a1, s_b1, s_a0, s_b0);
  }

  // row sums of squares: the four lane groups of a row, then one writer per row
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    float v = ssq[rb];
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (grp == 0) s_ssq[32 * wave + 16 * rb + row16] = v;
  }
  __syncthreads();

  const rsrc_t ro = make_rsrc(g.out, g.out_bytes);
  const float inv_n = 1.0f / (float)g.n;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int ml = (wm * FM + i) * 16 + row16;
    const int m = m0 + ml;
    const float sc = 1.0f / sqrtf(s_ssq[ml] * inv_n + g.eps);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + (wn * FN + j) * 16 + 4 * grp;
      const bool ok = m < g.T && n < g.N;
      bf16x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = (__bf16)(acc[i][j][e] * sc);
      bst8(ro, ok ? (uint32_t)(((int64_t)m * g.ld_out + n) * 2) : kOOB, __builtin_bit_cast(uint2, h));
    }
  }
}

// out[i] = sum over s in order of part[s][i], i < count (count % 4 == 0).
__global__ __launch_bounds__(256) void k_splitk_sum(const float* __restrict__ part, int S, int64_t count,
                                                    float* __restrict__ out) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q * 4 >= count) return;
  const float4* p = reinterpret_cast<const float4*>(part) + q;
  float4 a = p[0];
  for (int s = 1; s < S; ++s) {
    const float4 b = p[(int64_t)s * (count / 4)];
    a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
  }
  reinterpret_cast<float4*>(out)[q] = a;
}

// p[i] = rne(silu(v[i])), 8 elements per thread (count % 8 == 0).
__global__ __launch_bounds__(256) void k_silu(const __bf16* __restrict__ v, int64_t count, __bf16* __restrict__ p) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q * 8 >= count) return;
  reinterpret_cast<uint4*>(p)[q] = silu8(reinterpret_cast<const uint4*>(v)[q]);
}

// a = sum over the NT column tiles, in order, of the encoder partials;
// b = rne(x_attn[:, :r] + phi(a)); a_save = a.  4 columns per thread.
__global__ __launch_bounds__(256) void k_enc_finish(int64_t T, int r, int NT, int act, const float* __restrict__ part,
                                                    const __bf16* __restrict__ x, int64_t ld_x, __bf16* __restrict__ b,
                                                    float* __restrict__ a_save) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per = r / 4;
  if (q >= T * per) return;
  const int64_t t = q / per;
  const int c = (int)(q % per) * 4;
  float4 a = *reinterpret_cast<const float4*>(part + t * r + c);
  for (int k = 1; k < NT; ++k) {
    const float4 p = *reinterpret_cast<const float4*>(part + ((int64_t)k * T + t) * r + c);
    a.x += p.x; a.y += p.y; a.z += p.z; a.w += p.w;
  }
  if (a_save) *reinterpret_cast<float4*>(a_save + t * r + c) = a;
  const bf16x4 xv = __builtin_bit_cast(bf16x4, *reinterpret_cast<const uint2*>(x + t * ld_x + c));
  const float av[4] = {a.x, a.y, a.z, a.w};
  bf16x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = (__bf16)((float)xv[e] + resbm::act_phi(av[e], act));
  *reinterpret_cast<uint2*>(b + t * r + c) = __builtin_bit_cast(uint2, o);
}

// g_x[t][0 .. r) <- rne(g_x + g_b), 4 columns per thread (r % 8 == 0).
__global__ __launch_bounds__(256) void k_skip_grad(int64_t T, int r, const __bf16* __restrict__ g_b,
                                                   __bf16* __restrict__ g_x, int64_t ld_gx) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per = r / 4;
  if (q >= T * per) return;
  const int64_t t = q / per;
  const int c = (int)(q % per) * 4;
  const bf16x4 b = __builtin_bit_cast(bf16x4, *reinterpret_cast<const uint2*>(g_b + t * r + c));
  uint2* px = reinterpret_cast<uint2*>(g_x + t * ld_gx + c);
  bf16x4 x = __builtin_bit_cast(bf16x4, *px);
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = (__bf16)((float)x[e] + (float)b[e]);
  *px = __builtin_bit_cast(uint2, x);
}

}  // namespace resbm2

// ============================================================ host side
using namespace resbm2;

namespace {

constexpr size_t kWsAlign2 = 256;
constexpr int kTargetBlocks = 256;   // split-K aims at one block per compute unit

using resbm_host::aligned;
using resbm_host::extent;
using resbm_host::ld_ok;
using resbm_host::overlap;
size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
bool shape_ok2(int64_t T, int n, int m, int r) {
  return T >= 0 && T <= (1ll << 31) && n >= 8 && n <= 65536 && n % 8 == 0 && m >= 8 && m <= 65536 && m % 8 == 0 &&
         r >= 8 && r <= n && r % 8 == 0;
}
bool fits(size_t bytes) { return bytes <= (size_t)kMaxRange; }

// Block tile shapes: 256 x 256 (8 waves of 128 x 64) for the n x m products,
// 128 x 128 (4 waves of 64 x 64) where M or N is below 256, and a narrow one
// for an r-wide output (N = r).  Products with M = r use 128 x 128; the rows
// beyond r read nothing.
enum Shape { kBig = 0, kWide = 1, kNarrow32 = 2, kNarrow64 = 3, kNarrow128 = 4 };

Shape wide_for(int M, int N) { return M >= 256 && N >= 256 ? kBig : kWide; }
Shape narrow_for(int N) { return N <= 32 ? kNarrow32 : (N <= 64 ? kNarrow64 : kNarrow128); }
int shape_bm(Shape s) { return s == kBig ? 256 : (s == kWide ? 128 : 64); }
int shape_bn(Shape s) {
  return s == kBig ? 256 : (s == kWide || s == kNarrow128 ? 128 : (s == kNarrow32 ? 32 : 64));
}

struct Split {
  int S;
  int kc;
};
// Splits of a token-deep (K = T) product: enough blocks to fill the chip, each
// split at least 4 stages deep.
Split split_for(int M, int N, int K, Shape s) {
  const int64_t tiles = (int64_t)((M + shape_bm(s) - 1) / shape_bm(s)) * ((N + shape_bn(s) - 1) / shape_bn(s));
  int64_t S = (kTargetBlocks + tiles - 1) / tiles;
  const int64_t maxS = std::max<int64_t>(1, K / (4 * KT));
  S = std::min(S, maxS);
  const int64_t per = (K + S - 1) / S;
  const int kc = (int)round_up((size_t)per, KT);
  return {(int)((K + kc - 1) / kc), kc};
}
size_t part_bytes(int M, int N, const Split& sp) {
  return sp.S > 1 ? round_up((size_t)sp.S * M * N * 4, kWsAlign2) : 0;
}

struct Plan2 {
  Split dW4, dW3, dW2, dW1;
  size_t inter;      // one T x m bf16 intermediate (phi(v), g_v or g_u)
  size_t enc_fwd, dec_fwd, dec_bwd, enc_bwd;
};
Plan2 make_plan2(int64_t T, int n, int m, int r) {
  Plan2 p;
  p.dW4 = split_for(m, n, (int)T, wide_for(m, n));
  p.dW3 = split_for(r, m, (int)T, kWide);
  p.dW2 = split_for(m, r, (int)T, narrow_for(r));
  p.dW1 = split_for(n, m, (int)T, wide_for(n, m));
  p.inter = round_up((size_t)T * m * 2, kWsAlign2);
  p.enc_fwd = p.inter;
  p.dec_fwd = p.inter;
  p.dec_bwd = 2 * p.inter + std::max(part_bytes(m, n, p.dW4), part_bytes(r, m, p.dW3));
  p.enc_bwd = p.inter + std::max(part_bytes(m, r, p.dW2), part_bytes(n, m, p.dW1));
  return p;
}

template <bool AK, bool BKC, int BM, int BN, int WM, int WN, int EPI, bool PHI, bool LATE = false>
void launch(const GemmArgs& g, int S, hipStream_t st) {
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  hipLaunchKernelGGL((k_gemm<AK, BKC, BM, BN, WM, WN, EPI, PHI, LATE>), dim3(tiles, 1, S), dim3(64 * WM * WN), 0, st,
                     g);
}

// Runs C = op(A) op(B) with the epilogue EPI and tile shape s.
template <bool AK, bool BKC, int EPI, bool PHI>
void gemm(Shape s, const GemmArgs& g, int S, hipStream_t st) {
  switch (s) {
    case kBig:
      if (std::min(g.K, g.kc) <= 4096) launch<AK, BKC, 256, 256, 2, 4, EPI, PHI, true>(g, S, st);
      else launch<AK, BKC, 256, 256, 2, 4, EPI, PHI, false>(g, S, st);
      break;
    case kWide: launch<AK, BKC, 128, 128, 2, 2, EPI, PHI>(g, S, st); break;
    case kNarrow32: launch<AK, BKC, 64, 32, 4, 1, EPI, PHI>(g, S, st); break;
    case kNarrow64: launch<AK, BKC, 64, 64, 4, 1, EPI, PHI>(g, S, st); break;
    case kNarrow128: launch<AK, BKC, 64, 128, 4, 1, EPI, PHI>(g, S, st); break;
  }
}

GemmArgs args(int M, int N, int K, const void* A, int64_t lda, size_t ab, const void* B, int64_t ldb, size_t bb,
              void* C, int64_t ldc, size_t cb) {
  GemmArgs g{};
  g.M = M; g.N = N; g.K = K;
  g.A = A; g.lda = lda; g.a_bytes = (int64_t)ab;
  g.B = B; g.ldb = ldb; g.b_bytes = (int64_t)bb;
  g.C = C; g.ldc = ldc; g.c_bytes = (int64_t)cb;
  g.kc = (int)round_up((size_t)K, KT);
  return g;
}

// A token-deep weight-gradient product (K = T): float32 result W (M x N,
// contiguous), split over tokens with the partial sums in `part` when that
// fills the chip better.
template <bool PHI>
void weight_grad(Shape s, GemmArgs g, const Split& sp, float* W, void* part, hipStream_t st) {
  if (sp.S == 1) {
    g.C = W; g.ldc = g.N; g.c_bytes = (int64_t)g.M * g.N * 4;
    gemm<false, false, kEpiF32, PHI>(s, g, 1, st);
    return;
  }
  g.C = part; g.c_bytes = (int64_t)sp.S * g.M * g.N * 4; g.kc = sp.kc;
  gemm<false, false, kEpiPart, PHI>(s, g, sp.S, st);
  const int64_t count = (int64_t)g.M * g.N;
  hipLaunchKernelGGL(k_splitk_sum, dim3((unsigned)((count / 4 + 255) / 256)), dim3(256), 0, st, (const float*)part,
                     sp.S, count, W);
}


int32_t check_ws(size_t need, const void* ws, size_t ws_bytes) {
  if (need == 0) return RESBM_OK;
  if (!ws) return RESBM_E_NULL;
  if (!aligned(ws, kWsAlign2)) return RESBM_E_ALIGN;
  return ws_bytes < need ? RESBM_E_WORKSPACE : RESBM_OK;
}

}  // namespace

extern "C" {

size_t resbm2_workspace_bytes(int64_t T, int32_t n, int32_t m, int32_t r) {
  if (!shape_ok2(T, n, m, r) || T == 0) return 0;
  const Plan2 p = make_plan2(T, n, m, r);
  return std::max(std::max(p.enc_fwd, p.dec_fwd), std::max(p.dec_bwd, p.enc_bwd));
}

int32_t resbm2_encode_fwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act, const void* x_attn, int64_t ld_x,
                          const void* z, int64_t ld_z, const void* W1, const void* W2, void* b, void* u, void* ws,
                          size_t ws_bytes, void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (!shape_ok2(T, n, m, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const bool silu = act == RESBM_ACT_SILU;
  const Plan2 p = make_plan2(T, n, m, r);
  const size_t need = silu ? p.enc_fwd : 0;
  int32_t e = check_ws(need, ws, ws_bytes);
  if (e) return e;
  if (!x_attn || !z || !W1 || !W2 || !b || !u) return RESBM_E_NULL;
  if (!ld_ok(ld_x, n) || !ld_ok(ld_z, n)) return RESBM_E_SHAPE;
  if (!aligned(x_attn, 16) || !aligned(z, 16) || !aligned(W1, 16) || !aligned(W2, 16) || !aligned(b, 16) ||
      !aligned(u, 16))
    return RESBM_E_ALIGN;
  const size_t bx = extent(T, n, ld_x, 2), bz = extent(T, n, ld_z, 2), bw1 = (size_t)n * m * 2,
               bw2 = (size_t)m * r * 2, bb = (size_t)T * r * 2, bu = (size_t)T * m * 2;
  if (!fits(bx) || !fits(bz) || !fits(bu) || !fits(bw1)) return RESBM_E_SHAPE;
  if (overlap(b, bb, x_attn, bx) || overlap(b, bb, z, bz) || overlap(b, bb, W1, bw1) || overlap(b, bb, W2, bw2) ||
      overlap(u, bu, x_attn, bx) || overlap(u, bu, z, bz) || overlap(u, bu, W1, bw1) || overlap(u, bu, W2, bw2) ||
      overlap(u, bu, b, bb) || overlap(ws, need, x_attn, bx) || overlap(ws, need, z, bz) ||
      overlap(ws, need, W1, bw1) || overlap(ws, need, W2, bw2) || overlap(ws, need, b, bb) ||
      overlap(ws, need, u, bu))
    return RESBM_E_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  const int Ti = (int)T;
  // u = z W1  (A = z, K-contiguous; B = W1 [n][m], m-contiguous), and with SiLU
  // also phi(u) (workspace), formed from the float32 accumulator
  GemmArgs g = args(Ti, m, n, z, ld_z, bz, W1, m, bw1, u, m, bu);
  if (silu) {
    g.D = ws; g.ldd = m; g.d_bytes = (int64_t)bu;
    gemm<true, false, kEpiBf16Phi, false>(wide_for(Ti, m), g, 1, st);
  } else {
    gemm<true, false, kEpiBf16, false>(wide_for(Ti, m), g, 1, st);
  }
  // b = x_attn[:, :r] + phi(u) W2
  g = args(Ti, r, m, silu ? ws : u, m, bu, W2, r, bw2, b, r, bb);
  g.X = x_attn; g.ldx = ld_x; g.x_bytes = (int64_t)bx; g.x_cols = r;
  gemm<true, false, kEpiAdd, false>(narrow_for(r), g, 1, st);
  return resbm_host::launch_status();
}

int32_t resbm2_decode_fwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act, const void* b, const void* W3,
                          const void* W4, void* z_tilde, int64_t ld_zt, void* v, void* ws, size_t ws_bytes,
                          void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (!shape_ok2(T, n, m, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const bool silu = act == RESBM_ACT_SILU;
  const Plan2 p = make_plan2(T, n, m, r);
  const size_t need = silu ? p.dec_fwd : 0;
  int32_t e = check_ws(need, ws, ws_bytes);
  if (e) return e;
  if (!b || !W3 || !W4 || !z_tilde || !v) return RESBM_E_NULL;
  if (!ld_ok(ld_zt, n)) return RESBM_E_SHAPE;
  if (!aligned(b, 16) || !aligned(W3, 16) || !aligned(W4, 16) || !aligned(z_tilde, 16) || !aligned(v, 16))
    return RESBM_E_ALIGN;
  const size_t bb = (size_t)T * r * 2, bw3 = (size_t)r * m * 2, bw4 = (size_t)m * n * 2,
               bzt = extent(T, n, ld_zt, 2), bv = (size_t)T * m * 2;
  if (!fits(bzt) || !fits(bv) || !fits(bw4)) return RESBM_E_SHAPE;
  if (overlap(z_tilde, bzt, b, bb) || overlap(z_tilde, bzt, W3, bw3) || overlap(z_tilde, bzt, W4, bw4) ||
      overlap(v, bv, b, bb) || overlap(v, bv, W3, bw3) || overlap(v, bv, W4, bw4) || overlap(v, bv, z_tilde, bzt) ||
      overlap(ws, need, b, bb) || overlap(ws, need, W3, bw3) || overlap(ws, need, W4, bw4) ||
      overlap(ws, need, z_tilde, bzt) || overlap(ws, need, v, bv))
    return RESBM_E_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  const int Ti = (int)T;
  // v = b W3, and with SiLU also phi(v) (workspace), formed from the float32 accumulator
  GemmArgs g = args(Ti, m, r, b, r, bb, W3, m, bw3, v, m, bv);
  if (silu) {
    g.D = ws; g.ldd = m; g.d_bytes = (int64_t)bv;
    gemm<true, false, kEpiBf16Phi, false>(wide_for(Ti, m), g, 1, st);
  } else {
    gemm<true, false, kEpiBf16, false>(wide_for(Ti, m), g, 1, st);
  }
  // z~ = phi(v) W4
  g = args(Ti, n, m, silu ? ws : v, m, bv, W4, n, bw4, z_tilde, ld_zt, bzt);
  gemm<true, false, kEpiBf16, false>(wide_for(Ti, n), g, 1, st);
  return resbm_host::launch_status();
}

int32_t resbm2_decode_bwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act, const void* b, const void* v,
                          const void* g_zt, int64_t ld_gzt, const void* g_id, int64_t ld_gid, const void* W3,
                          const void* W4, void* g_b, float* dW3, float* dW4, void* ws, size_t ws_bytes,
                          void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (!shape_ok2(T, n, m, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan2 p = make_plan2(T, n, m, r);
  int32_t e = check_ws(p.dec_bwd, ws, ws_bytes);
  if (e) return e;
  if (!b || !v || !g_zt || !W3 || !W4 || !g_b || !dW3 || !dW4) return RESBM_E_NULL;
  if (!ld_ok(ld_gzt, n) || (g_id && !ld_ok(ld_gid, n))) return RESBM_E_SHAPE;
  if (!aligned(b, 16) || !aligned(v, 16) || !aligned(g_zt, 16) || (g_id && !aligned(g_id, 16)) ||
      !aligned(W3, 16) || !aligned(W4, 16) || !aligned(g_b, 16) || !aligned(dW3, 16) || !aligned(dW4, 16))
    return RESBM_E_ALIGN;
  const size_t bb = (size_t)T * r * 2, bv = (size_t)T * m * 2, bg = extent(T, n, ld_gzt, 2),
               bid = g_id ? extent(T, n, ld_gid, 2) : 0, bw3 = (size_t)r * m * 2, bw4 = (size_t)m * n * 2,
               bd3 = (size_t)r * m * 4, bd4 = (size_t)m * n * 4;
  if (!fits(bg) || !fits(bid) || !fits(bv) || !fits(bw4) || !fits(p.dec_bwd)) return RESBM_E_SHAPE;
  const void* ins[] = {b, v, g_zt, g_id, W3, W4};
  const size_t inb[] = {bb, bv, bg, bid, bw3, bw4};
  void* outs[] = {g_b, dW3, dW4, ws};
  const size_t outb[] = {bb, bd3, bd4, p.dec_bwd};
  for (int o = 0; o < 4; ++o) {
    for (int i = 0; i < 6; ++i)
      if (overlap(outs[o], outb[o], ins[i], inb[i])) return RESBM_E_ALIAS;
    for (int o2 = o + 1; o2 < 4; ++o2)
      if (overlap(outs[o], outb[o], outs[o2], outb[o2])) return RESBM_E_ALIAS;
  }
  hipStream_t st = (hipStream_t)stream;
  const int Ti = (int)T;
  char* w = (char*)ws;
  void* g_v = w;
  void* pv = w + p.inter;
  void* part = w + 2 * p.inter;
  const bool silu = act == RESBM_ACT_SILU;
  // g_v = (g_zt W4^T) * phi'(v)   (B(k, j) = W4[j][k]: K-contiguous)
  GemmArgs g = args(Ti, m, n, g_zt, ld_gzt, bg, W4, n, bw4, g_v, m, bv);
  if (silu) {
    g.X = v; g.ldx = m; g.x_bytes = (int64_t)bv;
    gemm<true, true, kEpiDphi, false>(wide_for(Ti, m), g, 1, st);
  } else {
    gemm<true, true, kEpiBf16, false>(wide_for(Ti, m), g, 1, st);
  }
  // dW4 = phi(v)^T g_zt   (A(i, k) = phi(v)[k][i], B(k, j) = g_zt[k][j]); phi(v) formed once
  if (silu) {
    const int64_t cnt = T * m;
    hipLaunchKernelGGL(k_silu, dim3((unsigned)((cnt / 8 + 255) / 256)), dim3(256), 0, st, (const __bf16*)v, cnt,
                       (__bf16*)pv);
  }
  g = args(m, n, Ti, silu ? pv : v, m, bv, g_zt, ld_gzt, bg, nullptr, 0, 0);
  weight_grad<false>(wide_for(m, n), g, p.dW4, dW4, part, st);
  // dW3 = b^T g_v
  g = args(r, m, Ti, b, r, bb, g_v, m, bv, nullptr, 0, 0);
  weight_grad<false>(kWide, g, p.dW3, dW3, part, st);
  // g_b = g_v W3^T + g_id[:, :r]
  g = args(Ti, r, m, g_v, m, bv, W3, m, bw3, g_b, r, bb);
  if (g_id) {
    g.X = g_id; g.ldx = ld_gid; g.x_bytes = (int64_t)bid; g.x_cols = r;
    gemm<true, true, kEpiAdd, false>(narrow_for(r), g, 1, st);
  } else {
    gemm<true, true, kEpiBf16, false>(narrow_for(r), g, 1, st);
  }
  return resbm_host::launch_status();
}

int32_t resbm2_encode_bwd(int64_t T, int32_t n, int32_t m, int32_t r, int32_t act, const void* z, int64_t ld_z,
                          const void* u, const void* g_b, const void* W1, const void* W2, void* g_z, int64_t ld_gz,
                          void* g_x, int64_t ld_gx, float* dW1, float* dW2, void* ws, size_t ws_bytes,
                          void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (!shape_ok2(T, n, m, r)) return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const Plan2 p = make_plan2(T, n, m, r);
  int32_t e = check_ws(p.enc_bwd, ws, ws_bytes);
  if (e) return e;
  if (!z || !u || !g_b || !W1 || !W2 || !g_z || !dW1 || !dW2) return RESBM_E_NULL;
  if (!ld_ok(ld_z, n) || !ld_ok(ld_gz, n) || (g_x && !ld_ok(ld_gx, n))) return RESBM_E_SHAPE;
  if (!aligned(z, 16) || !aligned(u, 16) || !aligned(g_b, 16) || !aligned(W1, 16) || !aligned(W2, 16) ||
      !aligned(g_z, 16) || (g_x && !aligned(g_x, 16)) || !aligned(dW1, 16) || !aligned(dW2, 16))
    return RESBM_E_ALIGN;
  const bool fused = g_x == g_z;
  if (fused && ld_gx != ld_gz) return RESBM_E_ALIAS;
  const size_t bz = extent(T, n, ld_z, 2), bu = (size_t)T * m * 2, bgb = (size_t)T * r * 2,
               bw1 = (size_t)n * m * 2, bw2 = (size_t)m * r * 2, bgz = extent(T, n, ld_gz, 2),
               bgx = (g_x && !fused) ? extent(T, n, ld_gx, 2) : 0, bd1 = (size_t)n * m * 4,
               bd2 = (size_t)m * r * 4;
  if (!fits(bz) || !fits(bu) || !fits(bgz) || !fits(bgx) || !fits(bw1) || !fits(p.enc_bwd)) return RESBM_E_SHAPE;
  const void* ins[] = {z, u, g_b, W1, W2};
  const size_t inb[] = {bz, bu, bgb, bw1, bw2};
  void* outs[] = {g_z, fused ? nullptr : g_x, dW1, dW2, ws};
  const size_t outb[] = {bgz, bgx, bd1, bd2, p.enc_bwd};
  for (int o = 0; o < 5; ++o) {
    for (int i = 0; i < 5; ++i)
      if (overlap(outs[o], outb[o], ins[i], inb[i])) return RESBM_E_ALIAS;
    for (int o2 = o + 1; o2 < 5; ++o2)
      if (overlap(outs[o], outb[o], outs[o2], outb[o2])) return RESBM_E_ALIAS;
  }
  hipStream_t st = (hipStream_t)stream;
  const int Ti = (int)T;
  char* w = (char*)ws;
  void* g_u = w;
  void* part = w + p.inter;
  const bool silu = act == RESBM_ACT_SILU;
  // g_u = (g_b W2^T) * phi'(u)   (B(k, j) = W2[j][k]: K-contiguous)
  GemmArgs g = args(Ti, m, r, g_b, r, bgb, W2, r, bw2, g_u, m, bu);
  if (silu) {
    g.X = u; g.ldx = m; g.x_bytes = (int64_t)bu;
    gemm<true, true, kEpiDphi, false>(wide_for(Ti, m), g, 1, st);
  } else {
    gemm<true, true, kEpiBf16, false>(wide_for(Ti, m), g, 1, st);
  }
  // dW2 = phi(u)^T g_b
  g = args(m, r, Ti, u, m, bu, g_b, r, bgb, nullptr, 0, 0);
  if (silu) weight_grad<true>(narrow_for(r), g, p.dW2, dW2, part, st);
  else weight_grad<false>(narrow_for(r), g, p.dW2, dW2, part, st);
  // dW1 = z^T g_u
  g = args(n, m, Ti, z, ld_z, bz, g_u, m, bu, nullptr, 0, 0);
  weight_grad<false>(wide_for(n, m), g, p.dW1, dW1, part, st);
  // g_z = g_u W1^T (+ g_b on columns [0, r) when g_x is g_z)   (B(k, j) = W1[j][k])
  g = args(Ti, n, m, g_u, m, bu, W1, m, bw1, g_z, ld_gz, bgz);
  if (fused) {
    g.X = g_b; g.ldx = r; g.x_bytes = (int64_t)bgb; g.x_cols = r;
    gemm<true, true, kEpiAdd, false>(wide_for(Ti, n), g, 1, st);
  } else {
    gemm<true, true, kEpiBf16, false>(wide_for(Ti, n), g, 1, st);
    if (g_x) {
      const int64_t cnt = T * (r / 4);
      hipLaunchKernelGGL(k_skip_grad, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0, st, T, r,
                         (const __bf16*)g_b, (__bf16*)g_x, ld_gx);
    }
  }
  return resbm_host::launch_status();
}

// Workspace of the fused encoder: the float32 partial sums (one T x r slice per
// 256 columns of z), then the W_e fragments (k_frag_prep: 256-row tiles, r
// rounded up to 64 columns).
static size_t ffn_part_bytes(int64_t T, int n, int r) {
  return round_up((size_t)((n + 255) / 256) * (size_t)T * r * 4, kWsAlign2);
}
static size_t ffn_frag_count(int n, int r) { return (size_t)((n + 255) / 256 * 8) * (size_t)((r + 63) / 64 * 4); }

size_t resbm_ffn_encode_workspace_bytes(int64_t T, int32_t n, int32_t r) {
  if (T <= 0 || n < 8 || n > 65536 || n % 8 || r < 8 || r > n || r % 8) return 0;
  return ffn_part_bytes(T, n, r) + round_up(ffn_frag_count(n, r) * 2048, kWsAlign2);
}

int32_t resbm_ffn_encode_fwd(int64_t T, int32_t d_ff, int32_t n, int32_t r, int32_t act, const void* h, int64_t ld_h,
                             const void* W_down, const void* x_attn, int64_t ld_x, const float* W_e, void* z,
                             int64_t ld_z, void* b, float* a_save, void* ws, size_t ws_bytes, void* stream) {
  if (act != RESBM_ACT_IDENTITY && act != RESBM_ACT_SILU) return RESBM_E_ACT;
  if (T < 0 || T > (1ll << 31) || d_ff < 8 || d_ff > 262144 || d_ff % 8 || n < 8 || n > 65536 || n % 8 || r < 8 ||
      r > n || r % 8)
    return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const size_t need = resbm_ffn_encode_workspace_bytes(T, n, r);
  int32_t e = check_ws(need, ws, ws_bytes);
  if (e) return e;
  if (!h || !W_down || !x_attn || !W_e || !z || !b) return RESBM_E_NULL;
  if (!ld_ok(ld_h, d_ff) || !ld_ok(ld_x, n) || !ld_ok(ld_z, n)) return RESBM_E_SHAPE;
  if (!aligned(h, 16) || !aligned(W_down, 16) || !aligned(x_attn, 16) || !aligned(W_e, 16) || !aligned(z, 16) ||
      !aligned(b, 16) || (a_save && !aligned(a_save, 16)))
    return RESBM_E_ALIGN;
  const size_t bh = extent(T, d_ff, ld_h, 2), bwd = (size_t)d_ff * n * 2, bx = extent(T, n, ld_x, 2),
               bwe = (size_t)n * r * 4, bz = extent(T, n, ld_z, 2), bb = (size_t)T * r * 2,
               ba = a_save ? (size_t)T * r * 4 : 0;
  if (!fits(bh) || !fits(bwd) || !fits(bz) || !fits(need)) return RESBM_E_SHAPE;
  const void* ins[] = {h, W_down, x_attn, W_e};
  const size_t inb[] = {bh, bwd, bx, bwe};
  void* outs[] = {z, b, a_save, ws};
  const size_t outb[] = {bz, bb, ba, need};
  for (int o = 0; o < 4; ++o) {
    for (int i = 0; i < 4; ++i)
      if (overlap(outs[o], outb[o], ins[i], inb[i])) return RESBM_E_ALIAS;
    for (int o2 = o + 1; o2 < 4; ++o2)
      if (overlap(outs[o], outb[o], outs[o2], outb[o2])) return RESBM_E_ALIAS;
  }
  hipStream_t st = (hipStream_t)stream;
  // W_e fragments, then z = h W_down with the encoder partials in the epilogue
  const size_t pb = ffn_part_bytes(T, n, r), nf = ffn_frag_count(n, r);
  char* wf = (char*)ws + pb;
  hipLaunchKernelGGL(k_frag_prep, dim3((unsigned)nf), dim3(64), 0, st, W_e, n, r, (int64_t)r, (r + 63) / 64 * 4,
                     (__bf16*)wf);
  GemmArgs g = args((int)T, n, d_ff, h, ld_h, bh, W_down, n, bwd, z, ld_z, bz);
  g.X = wf; g.x_cols = r; g.x_bytes = (int64_t)(nf * 2048);
  g.D = ws; g.d_bytes = (int64_t)pb;
  launch<true, false, 256, 256, 2, 4, kEpiEncode, false>(g, 1, st);
  const int64_t cnt = T * (r / 4);
  hipLaunchKernelGGL(k_enc_finish, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0, st, T, r, (n + 255) / 256, act,
                     (const float*)ws, (const __bf16*)x_attn, ld_x, (__bf16*)b, a_save);
  return resbm_host::launch_status();
}

size_t resbm_decode_qkv_workspace_bytes(int32_t n, int32_t r) {
  if (n < 64 || n > 65536 || n % 64 || r < 8 || r > 64 || r % 8) return 0;
  return round_up((size_t)((r + 31) / 32) * (n / 16) * 2048, kWsAlign2);
}

int32_t resbm_decode_qkv_fwd(int64_t T, int32_t n, int32_t r, int32_t N, const void* b, const float* W_d,
                             const float* gamma, const void* W_qkv, float eps, void* out, int64_t ld_out, void* ws,
                             size_t ws_bytes, void* stream) {
  if (T < 0 || T > (1ll << 31) - 256 || n < 64 || n > 65536 || n % 64 || r < 8 || r > 64 || r % 8 || N < 8 ||
      N > 262144 || N % 8 || !(eps >= 0.0f))
    return RESBM_E_SHAPE;
  if (T == 0) return RESBM_OK;
  const size_t need = resbm_decode_qkv_workspace_bytes(n, r);
  int32_t e = check_ws(need, ws, ws_bytes);
  if (e) return e;
  if (!b || !W_d || !gamma || !W_qkv || !out) return RESBM_E_NULL;
  if (!ld_ok(ld_out, N)) return RESBM_E_SHAPE;
  if (!aligned(b, 16) || !aligned(W_d, 16) || !aligned(gamma, 16) || !aligned(W_qkv, 16) || !aligned(out, 16))
    return RESBM_E_ALIGN;
  const size_t bb = (size_t)T * r * 2, bwd = (size_t)r * n * 4, bg = (size_t)n * 4, bw = (size_t)n * N * 2,
               bo = extent(T, N, ld_out, 2);
  if (!fits(bw) || !fits(bo) || !fits(bb)) return RESBM_E_SHAPE;
  const void* ins[] = {b, W_d, gamma, W_qkv};
  const size_t inb[] = {bb, bwd, bg, bw};
  for (int i = 0; i < 4; ++i)
    if (overlap(out, bo, ins[i], inb[i]) || overlap(ws, need, ins[i], inb[i])) return RESBM_E_ALIAS;
  if (overlap(out, bo, ws, need)) return RESBM_E_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  const int KS = (r + 31) / 32;
  hipLaunchKernelGGL(k_frag_prep, dim3((unsigned)(KS * (n / 16))), dim3(64), 0, st, W_d, r, n, (int64_t)n, n / 16,
                     (__bf16*)ws);
  DqArgs g{};
  g.T = (int)T; g.n = n; g.N = N; g.r = r;
  g.b = (const __bf16*)b; g.wdf = (const __bf16*)ws; g.gamma = gamma;
  g.W = (const __bf16*)W_qkv; g.w_bytes = (int64_t)bw;
  g.out = (__bf16*)out; g.ld_out = ld_out; g.out_bytes = (int64_t)bo;
  g.eps = eps;
  const unsigned tiles = (unsigned)(((T + 255) / 256) * ((N + 255) / 256));
  if (KS == 1)
    hipLaunchKernelGGL(k_dec_qkv<1>, dim3(tiles), dim3(512), 0, st, g);
  else
    hipLaunchKernelGGL(k_dec_qkv<2>, dim3(tiles), dim3(512), 0, st, g);
  return resbm_host::launch_status();
}

}  // extern "C"
