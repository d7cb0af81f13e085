// Host-side tiling plan of the four boundary ops.  The same plan sizes the
// workspace (resbm_workspace_bytes) and drives the launches, so the two can
// never disagree.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace resbm {

constexpr int kNumCU = 256;          // MI355X compute units (8 XCDs x 32)
constexpr size_t kWsAlign = 256;

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
inline size_t align_ws(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }

struct Plan {
  int64_t T;
  int n, r;
  int RP, NT;   // r rounded up to 16 (output tiles of the r-wide side)
  int KP, KS;   // r rounded up to 32 (contraction steps over r)

  // encode_fwd: waves own 16*MT tokens, blockIdx.y splits the n-contraction.
  int ef_MT, ef_tpb, ef_nblk, ef_S, ef_kspl;
  size_t ef_wf_off, ef_part_off, ef_ws;

  // decode_fwd: waves own a strip of 16*CT columns, blockIdx.y a token range.
  int df_CT, df_nstrips, df_nwg, df_tpg, df_ngrp;

  // decode_bwd: 8 waves x 64 columns per block, JT j-tiles per pass.
  int db_JT, db_njg, db_ncg, db_TB, db_ntg;
  size_t db_gbp_off, db_dwp_off, db_ws;

  // encode_bwd: 4 waves x 16*CT columns per block, blockIdx.y a token range.
  int eb_CT, eb_ncg, eb_TB, eb_ntg;
  size_t eb_dwp_off, eb_ws;

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
  const int nks = n / 32;
  const int64_t Tm = T > 0 ? T : 1;

  // ---- encode_fwd
  p.ef_MT = p.NT <= 2 ? 4 : (p.NT <= 4 ? 2 : 1);
  p.ef_tpb = 4 * 16 * p.ef_MT;
  p.ef_nblk = (int)ceil_div(Tm, p.ef_tpb);
  {
    int64_t waves0 = (int64_t)p.ef_nblk * 4;
    int64_t S = ceil_div(8 * kNumCU, waves0);
    int64_t smax = nks / 4 > 0 ? nks / 4 : 1;   // at least 4 k-steps per split
    if (S > smax) S = smax;
    if (S < 1) S = 1;
    p.ef_kspl = (int)ceil_div(nks, S);
    p.ef_S = (int)ceil_div(nks, p.ef_kspl);
  }
  p.ef_wf_off = 0;
  size_t wf_bytes = align_ws((size_t)n * p.RP * 4);
  p.ef_part_off = wf_bytes;
  size_t part_bytes = p.ef_S > 1 ? align_ws((size_t)p.ef_S * Tm * p.RP * 4) : 0;
  p.ef_ws = wf_bytes + part_bytes;

  // ---- decode_fwd
  p.df_CT = p.KS <= 2 ? 4 : (p.KS <= 4 ? 2 : 1);
  p.df_nstrips = n / (16 * p.df_CT);
  p.df_nwg = (int)ceil_div(p.df_nstrips, 4);
  {
    int64_t ntile = ceil_div(Tm, 16);
    int64_t g = ceil_div(8 * kNumCU, (int64_t)p.df_nwg * 4);
    if (g > ntile) g = ntile;
    if (g < 1) g = 1;
    p.df_tpg = (int)(16 * ceil_div(ntile, g));
    p.df_ngrp = (int)ceil_div(Tm, p.df_tpg);
  }

  // ---- decode_bwd
  p.db_JT = p.NT < 4 ? p.NT : 4;
  p.db_njg = (int)ceil_div(p.NT, p.db_JT);
  p.db_ncg = (int)ceil_div(n, 8 * 64);
  {
    int64_t nstep = ceil_div(Tm, 32);
    int64_t g = ceil_div(kNumCU, (int64_t)p.db_ncg * p.db_njg);
    if (g > nstep) g = nstep;
    if (g < 1) g = 1;
    p.db_TB = (int)(32 * ceil_div(nstep, g));
    p.db_ntg = (int)ceil_div(Tm, p.db_TB);
  }
  p.db_gbp_off = 0;
  size_t gbp = align_ws((size_t)p.db_ncg * Tm * p.RP * 4);
  p.db_dwp_off = gbp;
  p.db_ws = gbp + align_ws((size_t)p.db_ntg * p.RP * n * 4);

  // ---- encode_bwd
  p.eb_CT = p.KS <= 2 ? 4 : (p.KS <= 4 ? 2 : 1);
  p.eb_ncg = (int)ceil_div(n, 4 * 16 * p.eb_CT);
  {
    int64_t nstep = ceil_div(Tm, 32);
    int64_t g = ceil_div(2 * kNumCU, (int64_t)p.eb_ncg);
    if (g > nstep) g = nstep;
    if (g < 1) g = 1;
    p.eb_TB = (int)(32 * ceil_div(nstep, g));
    p.eb_ntg = (int)ceil_div(Tm, p.eb_TB);
  }
  p.eb_dwp_off = 0;
  p.eb_ws = align_ws((size_t)p.eb_ntg * n * p.RP * 4);

  size_t m = p.ef_ws;
  if (p.db_ws > m) m = p.db_ws;
  if (p.eb_ws > m) m = p.eb_ws;
  p.ws_total = m;
  return p;
}

}  // namespace resbm
