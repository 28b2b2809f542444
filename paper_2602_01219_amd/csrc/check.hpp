// check.hpp - host-only argument validation and workspace layout for the
// MiTA C ABI. Header-only, no HIP dependency: the host test builds it with g++.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <cmath>
#include <cstdio>
#include <string>

#include "mita.h"

namespace mita {

constexpr size_t WS_ALIGN = 256;
constexpr int ATT_TQ = 64;     // queries per attention workgroup
constexpr int ROUTE_TQ = 64;   // queries per routing tile (one wave)
constexpr int SCORE_NC = 512;  // keys per score/landmark-value workgroup chunk
// Top-k selection fused with the score pass of the forward.
constexpr int SEL_NS = 1024;   // sampled keys per landmark row (pivot estimate)
constexpr int SEL_CAP = 4096;  // most candidates the exact selection of one row takes

inline size_t align_up(size_t x) { return (x + WS_ALIGN - 1) / WS_ALIGN * WS_ALIGN; }
inline size_t elem_bytes(const mita_cfg_t &c) { return c.dtype == MITA_F32 ? 4 : 2; }
inline int64_t BH(const mita_cfg_t &c) { return (int64_t)c.B * c.H; }
inline int score_chunks(const mita_cfg_t &c) { return (c.N + SCORE_NC - 1) / SCORE_NC; }
inline int route_tiles(const mita_cfg_t &c) { return (c.N + ROUTE_TQ - 1) / ROUTE_TQ; }
inline float eff_scale(const mita_cfg_t &c) { return c.scale != 0.f ? c.scale : 1.0f / std::sqrt((float)c.d); }

inline int sel_ns(const mita_cfg_t &c) { return c.N < SEL_NS ? c.N : SEL_NS; }
// Does the forward select the top-k sets inside the score pass? Rows whose
// sample covers the whole row always fit their list; otherwise the expected
// list length, at most k + 5 sqrt(64 k) + 128 for N / ns <= 64, must stay
// inside SEL_CAP, which k <= SEL_CAP / 4 ensures.
inline bool fused_select(const mita_cfg_t &c) {
  return c.use_routed && !(c.flags & MITA_FLAG_FULL_SCORES) && (c.N <= SEL_NS || 4 * (int64_t)c.k <= SEL_CAP);
}
// Rank r of the pivot among the ns sampled scores of a row: the pivot is the
// r-th largest sample score. With the sample equal to the row, r = k exactly;
// otherwise r is the expected rank of the k-th token, k ns / N, plus five
// binomial standard deviations (and one), so that at least k tokens of the
// row score >= pivot except with negligible probability.
inline int sel_rank(const mita_cfg_t &c) {
  const int ns = sel_ns(c);
  if (ns == c.N) return c.k;
  const double f = (double)c.k * ns / c.N;
  const double sd = std::sqrt(f * (1.0 - (double)c.k / c.N));
  const int r = (int)std::ceil(f + 5.0 * sd) + 1;
  return r < ns ? r : ns;
}
// Candidates one row may list before it falls back: a power of two in
// [1024, SEL_CAP] above the count expected at the pivot rank plus six
// standard deviations (the whole row when it is shorter).
inline int sel_cap(const mita_cfg_t &c) {
  const int ns = sel_ns(c);
  const double r = sel_rank(c);
  const double bound = ns == c.N ? c.N : (r + 6.0 * std::sqrt(r)) * ((double)c.N / ns);
  int cap = 1024;
  while (cap < SEL_CAP && cap < bound) cap *= 2;
  return c.N < cap ? c.N : cap;
}

// Validate a configuration. On failure, writes a message into err.
inline int check_cfg(const mita_cfg_t *c, std::string *err) {
  char buf[256];
  auto fail = [&](int st, const char *msg) {
    if (err) *err = msg;
    return st;
  };
  if (!c) return fail(MITA_ERR_INVALID_ARG, "cfg is NULL");
  if (c->B < 1 || c->H < 1 || c->N < 1 || c->d < 1) return fail(MITA_ERR_INVALID_ARG, "B, H, N, d must be >= 1");
  if (c->dtype != MITA_F32 && c->dtype != MITA_BF16) return fail(MITA_ERR_UNSUPPORTED, "dtype must be MITA_F32 or MITA_BF16");
  if (c->d != 64 && c->d != 128) return fail(MITA_ERR_UNSUPPORTED, "d must be 64 or 128");
  if (c->s != 1) return fail(MITA_ERR_UNSUPPORTED, "only s = 1 routed expert per query is supported");
  if (c->grid_h < 1 || c->grid_w < 1 || (int64_t)c->grid_h * c->grid_w != c->N)
    return fail(MITA_ERR_INVALID_ARG, "grid_h * grid_w must equal N");
  if (c->lm_h < 1 || c->lm_w < 1 || (int64_t)c->lm_h * c->lm_w != c->M)
    return fail(MITA_ERR_INVALID_ARG, "lm_h * lm_w must equal M");
  if (c->lm_h > c->grid_h || c->lm_w > c->grid_w) return fail(MITA_ERR_INVALID_ARG, "landmark grid exceeds token grid");
  if (c->M < 1 || c->M > c->N) return fail(MITA_ERR_INVALID_ARG, "M must be in [1, N]");
  if (c->M > 1024) return fail(MITA_ERR_UNSUPPORTED, "M must be <= 1024");
  if (c->use_shared != 0 && c->use_shared != 1) return fail(MITA_ERR_INVALID_ARG, "use_shared must be 0 or 1");
  if (c->use_routed != 0 && c->use_routed != 1) return fail(MITA_ERR_INVALID_ARG, "use_routed must be 0 or 1");
  if (!c->use_shared && !c->use_routed) return fail(MITA_ERR_INVALID_ARG, "use_shared and use_routed are both 0");
  if (c->k < 1 || c->k > c->N) return fail(MITA_ERR_INVALID_ARG, "k must be in [1, N]");
  if (c->N > MITA_MAX_N) {
    snprintf(buf, sizeof buf, "N = %d exceeds the supported maximum %d", c->N, MITA_MAX_N);
    return fail(MITA_ERR_UNSUPPORTED, buf);
  }
  if (!(c->scale >= 0.f) || std::isinf(c->scale)) return fail(MITA_ERR_INVALID_ARG, "scale must be finite and >= 0");
  if (c->flags & ~(uint32_t)(MITA_FLAG_STAGED_GATHER | MITA_FLAG_FULL_SCORES))
    return fail(MITA_ERR_INVALID_ARG, "unknown flag bits");
  // Every index/offset the kernels form fits in 64-bit; int32 outputs need N and M*k in range.
  if ((int64_t)c->M * c->k > INT32_MAX) return fail(MITA_ERR_UNSUPPORTED, "M * k too large");
  return MITA_OK;
}

// Workspace layout of mita_forward (offsets in bytes; 0-sized pieces allowed).
struct FwdLayout {
  size_t q_lm, v_lm, scores, partial, idx, kx, vx, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start,
      plo, ccnt, cand, fail, total;
};

inline size_t scores_ws_bytes(const mita_cfg_t &c) {
  // per (b, h, chunk, landmark): (running max, running sum) and d accumulators
  const size_t rows = (size_t)BH(c) * score_chunks(c) * c.M;
  return align_up(rows * 2 * sizeof(float)) + align_up(rows * c.d * sizeof(float));
}
// Routing scratch: per-tile expert counts, per-tile scatter bases, per-expert
// totals and the attention work list, in that order.
inline size_t route_tiles_bytes(const mita_cfg_t &c) {
  return align_up((size_t)BH(c) * route_tiles(c) * c.M * sizeof(int32_t));
}
inline size_t route_ws_bytes(const mita_cfg_t &c) {
  return 2 * route_tiles_bytes(c) + align_up((size_t)BH(c) * c.M * sizeof(int32_t)) +
         align_up((size_t)BH(c) * (c.M + 1) * sizeof(int32_t));
}
inline size_t attend_ws_bytes(const mita_cfg_t &c) { return align_up((size_t)BH(c) * (c.M + 1) * sizeof(int32_t)); }

inline FwdLayout forward_layout(const mita_cfg_t &c) {
  FwdLayout L{};
  size_t off = 0;
  const size_t e = elem_bytes(c);
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes);
    return o;
  };
  const size_t bh = (size_t)BH(c);
  L.q_lm = take(bh * c.M * c.d * e);
  L.v_lm = take(c.use_shared ? bh * c.M * c.d * e : 0);
  L.scores = take(c.use_routed ? bh * c.M * (size_t)c.N * 4 : 0);
  L.partial = take(c.use_shared ? scores_ws_bytes(c) : 0);
  L.idx = take(c.use_routed ? bh * c.M * (size_t)c.k * 4 : 0);
  const bool staged = c.use_routed && (c.flags & MITA_FLAG_STAGED_GATHER);
  L.kx = take(staged ? bh * c.M * (size_t)c.k * c.d * e : 0);
  L.vx = take(staged ? bh * c.M * (size_t)c.k * c.d * e : 0);
  L.expert = take(c.use_routed ? bh * c.N * 4 : 0);
  L.perm = take(c.use_routed ? bh * c.N * 4 : 0);
  L.offsets = take(c.use_routed ? bh * (c.M + 1) * 4 : 0);
  L.tile_cnt = take(c.use_routed ? bh * route_tiles(c) * c.M * 4 : 0);
  L.tile_base = take(c.use_routed ? bh * route_tiles(c) * c.M * 4 : 0);
  L.counts = take(c.use_routed ? bh * c.M * 4 : 0);
  L.tile_start = take(c.use_routed ? bh * (c.M + 1) * 4 : 0);
  // fused selection: pivots, candidate counts and lists,
  // then the fallback counter followed by the fallback row list
  const bool fs = fused_select(c);
  L.plo = take(fs ? bh * c.M * 4 : 0);
  // per (row, key chunk): candidate count and a list region of SCORE_NC entries
  L.ccnt = take(fs ? bh * c.M * (size_t)score_chunks(c) * 4 : 0);
  L.cand = take(fs ? bh * c.M * (size_t)score_chunks(c) * SCORE_NC * 8 : 0);
  L.fail = take(fs ? (bh * c.M + 1) * 4 : 0);
  L.total = off;
  return L;
}

inline size_t workspace_size(const mita_cfg_t *c, int which) {
  if (check_cfg(c, nullptr) != MITA_OK) return 0;
  switch (which) {
    case MITA_WS_FORWARD: return forward_layout(*c).total;
    case MITA_WS_SCORES: return scores_ws_bytes(*c);
    case MITA_WS_TOPK: return 0;
    case MITA_WS_ROUTE: return route_ws_bytes(*c);
    case MITA_WS_ATTEND: return attend_ws_bytes(*c);
    default: return 0;
  }
}

inline bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// [a, a + na) and [b, b + nb) overlap?
inline bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
  if (!a || !b || !na || !nb) return false;
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

}  // namespace mita
