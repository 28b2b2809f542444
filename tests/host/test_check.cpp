// Host-only test of the argument validation and workspace layout (no GPU).
#include <cassert>
#include <cmath>
#include <cstdio>
#include <string>

#include "../../paper_2602_01219_amd/csrc/check.hpp"

static mita_cfg_t base() {
  mita_cfg_t c{};
  c.B = 2; c.H = 12; c.N = 16384; c.d = 64; c.grid_h = 128; c.grid_w = 128;
  c.M = 128; c.lm_h = 8; c.lm_w = 16; c.k = 512; c.s = 1; c.use_shared = 1; c.use_routed = 1;
  c.dtype = MITA_BF16; c.scale = 0.f; c.flags = 0;
  return c;
}

#define EXPECT(expr, code)                                                     \
  do {                                                                         \
    mita_cfg_t c = base();                                                     \
    expr;                                                                      \
    std::string e;                                                             \
    int got = mita::check_cfg(&c, &e);                                         \
    if (got != (code)) {                                                       \
      std::printf("FAIL %s: got %d want %d (%s)\n", #expr, got, code, e.c_str()); \
      return 1;                                                                \
    }                                                                          \
  } while (0)

int main() {
  EXPECT((void)0, MITA_OK);
  EXPECT(c.d = 96, MITA_ERR_UNSUPPORTED);
  EXPECT(c.s = 2, MITA_OK);
  EXPECT(c.s = MITA_MAX_S, MITA_OK);
  EXPECT(c.s = MITA_MAX_S + 1, MITA_ERR_UNSUPPORTED);
  EXPECT(c.s = 0, MITA_ERR_UNSUPPORTED);
  EXPECT((c.M = 2, c.lm_h = 1, c.lm_w = 2, c.s = 3), MITA_ERR_INVALID_ARG);  // s > M
  EXPECT((c.M = 2, c.lm_h = 1, c.lm_w = 2, c.s = 3, c.use_routed = 0), MITA_OK);
  EXPECT(c.dtype = 7, MITA_ERR_UNSUPPORTED);
  EXPECT(c.N = 70000, MITA_ERR_INVALID_ARG);                       // grid no longer matches
  EXPECT((c.N = 131072, c.grid_h = 256, c.grid_w = 512), MITA_ERR_UNSUPPORTED);
  EXPECT(c.k = 0, MITA_ERR_INVALID_ARG);
  EXPECT(c.k = 16385, MITA_ERR_INVALID_ARG);
  EXPECT(c.k = 16384, MITA_OK);
  EXPECT((c.M = 0, c.lm_h = 0), MITA_ERR_INVALID_ARG);
  EXPECT((c.lm_h = 4, c.lm_w = 16), MITA_ERR_INVALID_ARG);         // lm grid != M
  EXPECT((c.grid_h = 4, c.grid_w = 4096, c.lm_h = 8), MITA_ERR_INVALID_ARG);  // lm grid > token grid
  EXPECT((c.use_shared = 0, c.use_routed = 0), MITA_ERR_INVALID_ARG);
  EXPECT(c.use_shared = 2, MITA_ERR_INVALID_ARG);
  EXPECT(c.scale = -1.f, MITA_ERR_INVALID_ARG);
  EXPECT(c.flags = 0x80, MITA_ERR_INVALID_ARG);
  EXPECT(c.flags = MITA_FLAG_STAGED_GATHER, MITA_OK);
  EXPECT(c.flags = MITA_FLAG_STAGED_GATHER | MITA_FLAG_FULL_SCORES, MITA_OK);
  EXPECT(c.B = 0, MITA_ERR_INVALID_ARG);
  assert(mita::check_cfg(nullptr, nullptr) == MITA_ERR_INVALID_ARG);

  // workspace layout: aligned, non-overlapping, monotone
  mita_cfg_t c = base();
  mita::FwdLayout L = mita::forward_layout(c);
  const size_t offs[] = {L.q_lm,      L.v_lm,   L.scores, L.partial, L.idx,     L.kx,   L.vx,
                         L.expert,    L.perm,   L.offsets, L.tile_cnt, L.tile_base, L.counts, L.tile_start,
                         L.group,  L.pair_o, L.pair_lse, L.plo,    L.ccnt,   L.cand,    L.fail,    L.total};
  for (size_t i = 0; i + 1 < sizeof offs / sizeof offs[0]; ++i) {
    assert(offs[i] % 256 == 0);
    assert(offs[i] <= offs[i + 1]);
  }
  assert(L.scores - L.v_lm >= (size_t)2 * 12 * 128 * 64 * 2);
  assert(L.idx - L.partial == mita::scores_ws_bytes(c));
  assert(L.kx == L.vx && L.vx == L.expert);  // tiles absent without the staged-gather flag
  c.flags = MITA_FLAG_STAGED_GATHER;
  mita::FwdLayout L2 = mita::forward_layout(c);
  assert(L2.vx - L2.kx == (size_t)24 * 128 * 512 * 64 * 2);
  assert(mita::workspace_size(&c, MITA_WS_TOPK) == 0);
  // fused selection: sample of 1024 keys; the smallest pivot rank with
  // P(X >= r) <= 1e-9 for X ~ H(16384, 511, 1024) is 69, and the smallest
  // power-of-two cap with P(Y < 69) <= 1e-9 for Y ~ H(16384, cap, 1024) is 2048
  assert(mita::fused_select(c) && mita::sel_ns(c) == 1024 && mita::sel_cap(c) == 2048);
  assert(mita::sel_rank(c) == 69);
  assert(mita::hyper_sf(16384, 511, 1024, 69) <= mita::SEL_EPS && mita::hyper_sf(16384, 511, 1024, 68) > mita::SEL_EPS);
  assert(mita::hyper_cdf_below(16384, 2048, 1024, 69) <= mita::SEL_EPS);
  assert(mita::hyper_cdf_below(16384, 1024, 1024, 69) > mita::SEL_EPS);
  // the two tails of one law add up to 1 (X >= r or X < r)
  for (int r = 1; r < 200; r += 7) {
    const double t = mita::hyper_sf(16384, 2048, 1024, r) + mita::hyper_cdf_below(16384, 2048, 1024, r);
    assert(std::fabs(t - 1.0) < 1e-9);
  }
  assert(L2.ccnt - L2.plo == (size_t)24 * 128 * 4);
  assert(L2.cand - L2.ccnt == (size_t)24 * 128 * 32 * 4);
  assert(L2.fail - L2.cand == (size_t)24 * 128 * 32 * 512 * 8);
  assert(L2.total - L2.fail >= (size_t)(24 * 128 + 1) * 4);
  c.flags = MITA_FLAG_FULL_SCORES;
  assert(!mita::fused_select(c) && mita::forward_layout(c).plo == mita::forward_layout(c).total);
  c.flags = 0;
  c.k = 4096;  // rank 340, cap 8192
  assert(mita::fused_select(c) && mita::sel_rank(c) == 340 && mita::sel_cap(c) == 8192);
  c.k = 6000;  // rank 467 would need a cap above 8192: stored-S path
  assert(!mita::fused_select(c));
  c.grid_h = 32; c.grid_w = 32; c.N = 1024; c.k = 1024;  // the sample is the whole row: rank = k
  assert(mita::fused_select(c) && mita::sel_rank(c) == 1024 && mita::sel_cap(c) == 1024);
  c.grid_h = 32; c.grid_w = 64; c.N = 2048; c.k = 2048;  // k = N > the sample: no rank meets the bound
  assert(!mita::fused_select(c));
  c.grid_h = 256; c.grid_w = 256; c.N = 65536; c.k = 1024;  // rank 45; cap 4096 misses, 8192 meets the bound
  assert(mita::fused_select(c) && mita::sel_rank(c) == 45 && mita::sel_cap(c) == 8192);
  c.grid_h = 64; c.grid_w = 64; c.N = 4096; c.k = 256;  // rank 107, cap 1024
  assert(mita::fused_select(c) && mita::sel_rank(c) == 107 && mita::sel_cap(c) == 1024);
  // attention row lists in LDS: fp32 d = 128 tiles take 137216 bytes, so at
  // most 6656 rows fit beside them; the bf16 DMA tiles (16 KB at d = 64) leave
  // room for the longest list staged in LDS (8192 rows)
  assert(mita::list_in_lds(6656, 137216) && !mita::list_in_lds(6657, 137216));
  assert(mita::list_in_lds(8192, 16384) && !mita::list_in_lds(8193, 16384));
  assert(mita::list_in_lds(8192, 32768) && !mita::list_in_lds(8192, 163840 - 32767));
  // s > 1: (query, rank) pairs in 2 M groups; the pairs' partials and log-sum-exps
  c = base();
  c.s = 2;
  assert(mita::route_groups(c) == 256 && mita::route_items(c) == 32768 && mita::route_tiles(c) == 512);
  mita::FwdLayout L3 = mita::forward_layout(c);
  assert(L3.perm - L3.expert == (size_t)24 * 16384 * 2 * 4);
  assert(L3.tile_start - L3.counts == (size_t)24 * 256 * 4);
  assert(L3.pair_lse - L3.pair_o == (size_t)24 * 16384 * 2 * 64 * 4);
  assert(mita::workspace_size(&c, MITA_WS_ATTEND) ==
         mita::align_up((size_t)24 * 257 * 4) + (size_t)24 * 16384 * 2 * 64 * 4 + (size_t)24 * 16384 * 2 * 4);
  c.use_routed = 0;  // s does not matter without routing
  assert(!mita::multi_route(c) && mita::forward_layout(c).pair_o == mita::forward_layout(c).pair_lse);
  c = base();
  c.d = 96;
  assert(mita::workspace_size(&c, MITA_WS_FORWARD) == 0);
  std::printf("host checks ok\n");
  return 0;
}
