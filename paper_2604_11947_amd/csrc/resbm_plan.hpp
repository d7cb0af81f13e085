// Tiling plan of the four boundary ops.  The tile shapes are constexpr
// functions shared by the kernels (template arguments) and the host (grid
// sizes, workspace), so the two can never disagree.
#pragma once

#include <stddef.h>
#include <stdint.h>

// Launch-shape targets, in waves (or workgroups) per compute unit.
#ifndef RESBM_DF_WAVES_PER_CU
#define RESBM_DF_WAVES_PER_CU 4
#endif
#ifndef RESBM_DB_WG_PER_CU
#define RESBM_DB_WG_PER_CU 1
#endif
#ifndef RESBM_EB_BLOCKS_PER_CU
#define RESBM_EB_BLOCKS_PER_CU 1
#endif
#ifndef RESBM_EF_MT_SMALL_R
#define RESBM_EF_MT_SMALL_R 4
#endif

// The hardware hands consecutive blocks of a grid to the 8 XCDs in turn.  The
// streaming kernels with 2-D grids (decode_bwd, encode_bwd) put the token
// dimension first, so that each XCD sees every column range rather than one
// narrow column strip of every row; encode_fwd blocks start their walk over
// the columns at rotated stages.
#ifndef RESBM_XCD_SPREAD
#define RESBM_XCD_SPREAD 1
#endif
#ifndef RESBM_DF_TOKEN_FASTEST
#define RESBM_DF_TOKEN_FASTEST 1
#endif

namespace resbm {

constexpr int kNumCU = 256;          // MI355X compute units (8 XCDs x 32)
constexpr size_t kWsAlign = 256;

// ---- encode_fwd: a block owns 16*MT tokens; its KW waves split the n-contraction.
// 64 tokens per block up to r = 64 (at r = 64: 55 -> 46 us at n = 4096, T = 16384),
// 32 up to r = 128 (at r = 128: 116 -> 90 us; every block reads all of W_e's
// fragments, so more tokens per block mean less L2 traffic), 16 beyond (32 was
// slower at r = 256).
constexpr int ef_mt(int NT) { return NT <= 2 ? RESBM_EF_MT_SMALL_R : (NT <= 4 ? 4 : (NT <= 8 ? 2 : 1)); }
// k-steps of 32 columns per wave and stage: two up to r = 64, so that a stage
// row is 512 bytes (at r = 64: 51 -> 41 us with the 64-token blocks)
constexpr int ef_u(int NT) { return NT <= 4 ? 2 : 1; }
// encode_fwd up to RESBM_EF_WE_LDS j-tiles of r (bf16 build): each wave splits
// its own rows of W_e into hi / lo bf16 planes in LDS and reads the fragments
// back transposed, instead of reading fragments that a prologue kernel
// prepared (that kernel costs a fixed ~4.5 us per call, whatever its size).
// Every block repeats the split, on one wave per SIMD: at r = 16 the kernel
// runs 25.7 us against 24.3 + 4.5 (prologue); at r = 32 31.6 against
// 26.7 + 4.4, so r = 32 keeps the prologue.
#ifndef RESBM_EF_WE_LDS
#define RESBM_EF_WE_LDS 1
#endif
constexpr bool ef_we_lds(int NT) { return !RESBM_IO_F32_BUILD && NT <= RESBM_EF_WE_LDS; }
#ifndef RESBM_EF_KW
#define RESBM_EF_KW 4
#endif
constexpr int ef_kw(int NT) { return 8 * 16 * ef_mt(NT) * (16 * NT + 4) * 4 <= 73728 ? RESBM_EF_KW : 4; }

// ---- decode_fwd: a wave owns 16*CT columns and walks a token range.
// Four column tiles up to r = 128 (at r = 128: 69 -> 45 us), two beyond (at
// r = 256: 236 -> 128 us); the g_z pass of encode_bwd follows the same shape.
#ifndef RESBM_DF_CT_W4
#define RESBM_DF_CT_W4 4
#endif
#ifndef RESBM_DF_CT_W8
#define RESBM_DF_CT_W8 2
#endif
#ifndef RESBM_DF_WAVES_PER_CU_WIDE
#define RESBM_DF_WAVES_PER_CU_WIDE 4
#endif
constexpr int df_ct(int KS) { return KS <= 2 ? 4 : (KS <= 4 ? RESBM_DF_CT_W4 : RESBM_DF_CT_W8); }
constexpr int df_waves_per_cu(int KS) { return KS <= 2 ? RESBM_DF_WAVES_PER_CU : RESBM_DF_WAVES_PER_CU_WIDE; }

// ---- decode_bwd: 8 waves x 64 columns per block, JT j-tiles (16 of r each) per pass.
#ifndef RESBM_DB_WAVES
#define RESBM_DB_WAVES 8
#endif
constexpr int kDbWaves = RESBM_DB_WAVES;
constexpr int kDbWC = 512 / kDbWaves;  // a block spans 512 columns (1 KiB of a bf16 row)
constexpr int db_jt(int NT) { return NT < 4 ? NT : 4; }

// ---- encode_bwd: blocks of CW x TW waves; a wave owns 16*CT columns, a block
// step covers 32*TW tokens (g_z is written by the decode_fwd expand kernel).
// Workspace: the dW_e partials of the token groups, then g_h (split) for g_z.
// a 256-column block up to r = 64 (at r = 64: 127 -> 112 us for the op); the
// float32 build's tiles are twice as large and keep 128 columns up to r = 128
#if RESBM_IO_F32_BUILD
constexpr int eb_ct(int KS) { return KS <= 1 ? 4 : (KS <= 4 ? 2 : 1); }
#else
// 128 columns beyond r = 64 (at r = 128, with two token waves: 351 -> 219 us
// for the op; at r = 256: 867 -> 696 us)
constexpr int eb_ct(int KS) { return KS <= 2 ? 4 : 2; }
#endif
#ifndef RESBM_EB_CW
#define RESBM_EB_CW 4
#endif
constexpr int eb_cw(int) { return RESBM_EB_CW; }
#ifndef RESBM_EB_TW
#define RESBM_EB_TW 2
#endif
// two token waves up to r = 128; at r = 256 the g_h tiles of two would not fit LDS
constexpr int eb_tw(int KS) { return KS <= 4 ? RESBM_EB_TW : 1; }

// ---- wide rank: above r = 64 (more than four 16-column tiles of r) the ops
// switch to the row / token contraction kernels and the expand kernel with
// block-shared inputs.
#ifndef RESBM_WIDE_NT
#define RESBM_WIDE_NT 5
#endif
constexpr int kWideNT = RESBM_WIDE_NT;
// the expand kernel with block-shared input rows from this many 32-deep k-steps of r
#ifndef RESBM_EXPAND_WIDE_KS
#define RESBM_EXPAND_WIDE_KS 3
#endif
constexpr int kExpandWideKS = RESBM_EXPAND_WIDE_KS;
// encode_bwd's g_z pass (three products per k-step, split input) takes it from
// this many k-steps: at r = 64 the g_z pass ran 157 -> 129 us (n = 8192, 32768
// tokens) and 51 -> 42 us (n = 4096, 16384 tokens) on it, where decode_fwd's
// pass (two products) ran slower (93 -> 123 us, 29 -> 37 us)
#ifndef RESBM_EXPAND_WIDE_KS_GZ
#define RESBM_EXPAND_WIDE_KS_GZ 2
#endif
constexpr int kExpandWideKSGZ = RESBM_EXPAND_WIDE_KS_GZ;
constexpr int tw_ntw(int NT) { return (NT + 3) / 4; }  // j-tiles per wave (four waves split r)
// wide row contraction: ring of weight-fragment registers (2, 4 or 8 k-steps;
// fragments are loaded ring - 1 k-steps ahead)
#ifndef RESBM_RW_RING
#define RESBM_RW_RING 4
#endif
constexpr int kRwRing = RESBM_RW_RING;
// largest token-step multiplier of the wide token contraction (1: 32-token steps)
#ifndef RESBM_TW_TSM
#define RESBM_TW_TSM 2
#endif
// tokens of the streamed matrix the wide token contraction has in flight
#ifndef RESBM_TW_XTOK
#define RESBM_TW_XTOK 128
#endif
// Row contraction of the wide path (k_rowc_wide).  A block of rw_waves waves
// owns rw_tok(NT) tokens and one of rw_rh(NT) groups of j-tiles; each wave owns
// rw_ntw j-tiles of its group.  Eight waves from RESBM_RW_WAVES8_NT j-tiles per
// group on (two per SIMD; one block per CU
// leaves a four-wave block one wave per SIMD, with nothing to cover its loads
// and barriers): 330 / 524 us at r = 128 / 256 against 339 / 528 with four.
// From RESBM_RW_SPLIT_NT j-tiles on, 128-token blocks split r in two halves:
// each block then reads half of the weight fragments for twice the tokens.
#ifndef RESBM_RW_WAVES8_NT
#define RESBM_RW_WAVES8_NT 5
#endif
#ifndef RESBM_RW_SPLIT_NT
#define RESBM_RW_SPLIT_NT 12
#endif
constexpr int rw_rh(int NT) { return NT >= RESBM_RW_SPLIT_NT ? 2 : 1; }
constexpr int rw_waves(int NT) { return (NT + rw_rh(NT) - 1) / rw_rh(NT) >= RESBM_RW_WAVES8_NT ? 8 : 4; }
constexpr int rw_tok(int NT) { return 64 * rw_rh(NT); }
constexpr int rw_ntw(int NT) {
  return ((NT + rw_rh(NT) - 1) / rw_rh(NT) + rw_waves(NT) - 1) / rw_waves(NT);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
inline size_t align_ws(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }
inline int64_t clamp64(int64_t v, int64_t lo, int64_t hi) { return v < lo ? lo : (v > hi ? hi : v); }

struct Plan {
  int64_t T;
  int n, r;
  int RP, NT;   // r rounded up to 16 (tiles of the r-wide side)
  int KP, KS;   // r rounded up to 32 (steps of a contraction over r)

  int ef_mt, ef_kw, ef_nblk;
  size_t ef_wf_off, ef_ws;

  int df_ct, df_nstrips, df_nwg, df_tpg, df_ngrp;

  int db_jt, db_njg, db_ncg, db_TB, db_ntg;
  size_t db_gbp_off, db_dwp_off, db_ws;

  int eb_ct, eb_bc, eb_ncb, eb_TB, eb_ntg;
  size_t eb_dwp_off, eb_gh_off, eb_ws;

  bool wide;                    // NT >= kWideNT
  int rw_nblk;                  // row contraction: blocks (see rw_tok, rw_rh)
  int tw_ncb, tw_ntg, tw_TB;    // token contraction: 128-column blocks x token groups of tw_TB tokens
  size_t db_wf_off;             // decode_bwd (wide): W_d fragments

  size_t ws_total;
};

inline bool shape_ok(int n, int r) {
  return n >= 64 && n <= 65536 && n % 64 == 0 && r >= 4 && r % 4 == 0 && r <= 256 && r <= n;
}

inline Plan make_plan(int64_t T, int n, int r) {
  Plan p{};
  p.T = T; p.n = n; p.r = r;
  p.RP = (int)round_up(r, 16); p.NT = p.RP / 16;
  p.KP = (int)round_up(r, 32); p.KS = p.KP / 32;
  const int64_t Tm = T > 0 ? T : 1;

  // ---- encode_fwd: fragment-ordered hi/lo copy of W_e in the workspace
  p.ef_mt = ef_mt(p.NT);
  p.ef_kw = ef_kw(p.NT);
  p.ef_nblk = (int)ceil_div(Tm, 16 * p.ef_mt);
  p.ef_wf_off = 0;
  p.ef_ws = align_ws((size_t)n * p.RP * 4);

  // ---- decode_fwd
  p.df_ct = df_ct(p.KS);
  p.df_nstrips = n / (16 * p.df_ct);
  p.df_nwg = (int)ceil_div(p.df_nstrips, 4);
  {
    const int64_t ntile = ceil_div(Tm, 16);
    const int64_t g = clamp64(ceil_div((int64_t)df_waves_per_cu(p.KS) * kNumCU, (int64_t)p.df_nwg * 4), 1, ntile);
    p.df_tpg = (int)(16 * ceil_div(ntile, g));
    // a token group's output rows lie in one buffer descriptor (32-bit byte
    // offsets): at most 1 GiB of dense rows per group
    const int64_t cap = (((int64_t)1 << 30) / ((int64_t)n * 4)) / 16 * 16;
    if (p.df_tpg > cap) p.df_tpg = (int)(cap < 16 ? 16 : cap);
    p.df_ngrp = (int)ceil_div(Tm, p.df_tpg);
  }

  // ---- decode_bwd: g_b partials per column group, dW_d partials per token group
  p.db_jt = db_jt(p.NT);
  p.db_njg = (int)ceil_div(p.NT, p.db_jt);
  p.db_ncg = (int)ceil_div(n, kDbWaves * kDbWC);
  {
    const int64_t nstep = ceil_div(Tm, 32);
    const int64_t g = clamp64(ceil_div((int64_t)RESBM_DB_WG_PER_CU * kNumCU, (int64_t)p.db_ncg * p.db_njg), 1, nstep);
    p.db_TB = (int)(32 * ceil_div(nstep, g));
    p.db_ntg = (int)ceil_div(Tm, p.db_TB);
  }
  p.db_gbp_off = 0;
  const size_t gbp = align_ws((size_t)p.db_ncg * Tm * p.RP * 4);
  p.db_dwp_off = gbp;
  p.db_ws = gbp + align_ws((size_t)p.db_ntg * p.RP * n * 4);

  // ---- encode_bwd: dW_e partials per token group
  p.eb_ct = eb_ct(p.KS);
  p.eb_bc = eb_cw(p.KS) * 16 * p.eb_ct;
  p.eb_ncb = (int)ceil_div(n, p.eb_bc);
  {
    const int64_t ts = 32 * eb_tw(p.KS);
    const int64_t nstep = ceil_div(Tm, ts);
    const int64_t g = clamp64(ceil_div((int64_t)RESBM_EB_BLOCKS_PER_CU * kNumCU, p.eb_ncb), 1, nstep);
    p.eb_TB = (int)(ts * ceil_div(nstep, g));
    p.eb_ntg = (int)ceil_div(Tm, p.eb_TB);
  }
  p.eb_dwp_off = 0;
  p.eb_gh_off = align_ws((size_t)p.eb_ntg * n * p.RP * 4);
  p.eb_ws = p.eb_gh_off + align_ws((size_t)Tm * r * 4);  // g_h, split into two bf16 planes (or one fp32)

  // ---- wide rank: decode_bwd = row contraction (g_b) + token contraction (dW_d
  // partials) + their ordered sum; encode_bwd = g_h + token contraction (dW_e
  // partials) + expand (g_z, with the ordered sums riding along)
  p.wide = p.NT >= kWideNT;
  if (p.wide) {
    // 64-token blocks; or, with r split in two, 128-token blocks in runs of 16:
    // the two halves of a token group 8 blocks apart, on one XCD
    const int64_t rw_ntg = ceil_div(Tm, rw_tok(p.NT));
    p.rw_nblk = (int)(rw_rh(p.NT) == 1 ? rw_ntg : 16 * ceil_div(rw_ntg, 8));
    p.tw_ncb = (int)ceil_div(n, 128);
    const int64_t nstep = ceil_div(Tm, 32);
    const int64_t g = clamp64(ceil_div((int64_t)kNumCU, p.tw_ncb), 1, nstep);
    p.tw_TB = (int)(32 * ceil_div(nstep, g));
    p.tw_ntg = (int)ceil_div(Tm, p.tw_TB);
    p.db_wf_off = 0;
    p.db_gbp_off = 0;
    p.db_dwp_off = align_ws((size_t)n * p.RP * 4);
    p.db_ws = p.db_dwp_off + align_ws((size_t)p.tw_ntg * p.RP * n * 4);
    p.eb_ntg = p.tw_ntg;
    p.eb_dwp_off = 0;
    p.eb_gh_off = align_ws((size_t)p.tw_ntg * n * p.RP * 4);
    p.eb_ws = p.eb_gh_off + align_ws((size_t)Tm * r * 4);
  }

  size_t m = p.ef_ws;
  if (p.db_ws > m) m = p.db_ws;
  if (p.eb_ws > m) m = p.eb_ws;
  p.ws_total = m;
  return p;
}

}  // namespace resbm
