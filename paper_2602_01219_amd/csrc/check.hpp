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
constexpr int SEL_CAP = 8192;  // most candidates the exact selection of one row takes
// Per-row probability allowed for each of the two ways a row's candidate list
// can miss (too short to hold the top-k, too long for the cap), under the
// model below; such a row is still selected exactly, only slower.
constexpr double SEL_EPS = 1e-9;

// LDS one workgroup can hold on gfx950 (the whole 160 KB of a CU).
constexpr size_t LDS_BYTES = 160 * 1024;
// Longest key row list (shared plus routed rows, 4 bytes each) the attention
// stages in LDS; longer ones are read from memory.
constexpr int IDX_LDS_MAX = 8192;
// Does a row list of nlist entries fit in LDS beside a kernel's static LDS?
inline bool list_in_lds(int nlist, size_t static_bytes) {
  return nlist <= IDX_LDS_MAX && static_bytes + (size_t)nlist * 4 <= LDS_BYTES;
}

inline size_t align_up(size_t x) { return (x + WS_ALIGN - 1) / WS_ALIGN * WS_ALIGN; }
inline size_t elem_bytes(const mita_cfg_t &c) { return c.dtype == MITA_F32 ? 4 : 2; }
inline int64_t BH(const mita_cfg_t &c) { return (int64_t)c.B * c.H; }
inline int score_chunks(const mita_cfg_t &c) { return (c.N + SCORE_NC - 1) / SCORE_NC; }
// Routing items: the queries (s = 1) or the (query, rank) pairs n * s + j
// (s > 1), grouped into M groups (s = 1) or 2 M (s > 1: group e holds the
// rank-1 pairs of expert e, group M + e its other pairs).
inline int route_s(const mita_cfg_t &c) { return c.use_routed ? c.s : 1; }
inline bool multi_route(const mita_cfg_t &c) { return route_s(c) > 1; }
inline int route_items(const mita_cfg_t &c) { return c.N * route_s(c); }
inline int route_groups(const mita_cfg_t &c) { return multi_route(c) ? 2 * c.M : c.M; }
inline int route_tiles(const mita_cfg_t &c) { return (route_items(c) + ROUTE_TQ - 1) / ROUTE_TQ; }
inline float eff_scale(const mita_cfg_t &c) { return c.scale != 0.f ? c.scale : 1.0f / std::sqrt((float)c.d); }

// ---------------------------------------------------------------------------
// Plan of the fused selection. A row's pivot is the r-th largest of the
// scores at ns evenly spaced keys; the score pass lists every token scoring
// >= pivot and the exact selection runs on that list when it holds between k
// and cap entries. Model: the row's scores are exchangeable over positions, so
// the sampled positions are a uniform random ns-subset of the N tokens and,
// for any fixed set of K tokens (the row's K first in the top-k order), the
// number of samples among them is hypergeometric, X ~ H(N, K, ns).
//  - The list is shorter than k only if at least r samples lie among the
//    row's first k - 1 tokens: P = P(X >= r), K = k - 1. r is the smallest
//    rank with P <= SEL_EPS.
//  - The list is longer than cap only if fewer than r samples lie among the
//    row's first cap tokens: P = P(X < r), K = cap. cap is the smallest power
//    of two in [1024, SEL_CAP] (or N) with P <= SEL_EPS.
// Both bounds are for the exact r-th sample, which is the pivot. When the
// sample is the whole row (N <= SEL_NS) the rank is k and the list cannot
// miss. A configuration with no rank or cap meeting the bounds is not
// selected in the score pass.
// ---------------------------------------------------------------------------
inline double log_choose(double n, double x) { return std::lgamma(n + 1.0) - std::lgamma(x + 1.0) - std::lgamma(n - x + 1.0); }

// log P(X = x), X ~ H(N, K, n)
inline double hyper_log_pmf(int64_t N, int64_t K, int64_t n, int64_t x) {
  return log_choose((double)K, (double)x) + log_choose((double)(N - K), (double)(n - x)) - log_choose((double)N, (double)n);
}

// Tails of X ~ H(N, K, n), each summed from its inner end on the side of the
// mode where the terms shrink (so the first term cannot underflow while the
// rest matter); the other side is the complement.
//   upward:   P(x + 1) / P(x) = (K - x)(n - x) / ((x + 1)(N - K - n + x + 1))
//   downward: P(x - 1) / P(x) = x (N - K - n + x) / ((K - x + 1)(n - x + 1))
inline int64_t hyper_mode(int64_t N, int64_t K, int64_t n) { return (int64_t)(((double)(n + 1) * (K + 1)) / (N + 2)); }

// sum of P(x) for x >= r, r above the mode
inline double hyper_sum_up(int64_t N, int64_t K, int64_t n, int64_t r, int64_t hi) {
  double t = std::exp(hyper_log_pmf(N, K, n, r)), s = 0.0;
  for (int64_t x = r; x <= hi; ++x) {
    s += t;
    t *= (double)(K - x) * (double)(n - x) / ((double)(x + 1) * (double)(N - K - n + x + 1));
    if (t <= s * 1e-18) break;
  }
  return s;
}
// sum of P(x) for x <= r, r below the mode
inline double hyper_sum_down(int64_t N, int64_t K, int64_t n, int64_t r, int64_t lo) {
  double t = std::exp(hyper_log_pmf(N, K, n, r)), s = 0.0;
  for (int64_t x = r; x >= lo; --x) {
    s += t;
    t *= (double)x * (double)(N - K - n + x) / ((double)(K - x + 1) * (double)(n - x + 1));
    if (t <= s * 1e-18) break;
  }
  return s;
}

// P(X >= r)
inline double hyper_sf(int64_t N, int64_t K, int64_t n, int64_t r) {
  const int64_t lo = n - (N - K) > 0 ? n - (N - K) : 0, hi = K < n ? K : n;
  if (r <= lo) return 1.0;
  if (r > hi) return 0.0;
  const double p = r > hyper_mode(N, K, n) ? hyper_sum_up(N, K, n, r, hi) : 1.0 - hyper_sum_down(N, K, n, r - 1, lo);
  return p < 0.0 ? 0.0 : (p > 1.0 ? 1.0 : p);
}

// P(X < r)
inline double hyper_cdf_below(int64_t N, int64_t K, int64_t n, int64_t r) {
  const int64_t lo = n - (N - K) > 0 ? n - (N - K) : 0, hi = K < n ? K : n;
  if (r <= lo) return 0.0;
  if (r > hi) return 1.0;
  const double p = r - 1 < hyper_mode(N, K, n) ? hyper_sum_down(N, K, n, r - 1, lo) : 1.0 - hyper_sum_up(N, K, n, r, hi);
  return p < 0.0 ? 0.0 : (p > 1.0 ? 1.0 : p);
}

struct SelPlan {
  bool ok;   // the score pass can select this (N, k)
  int ns;    // sampled keys per row
  int rank;  // pivot rank among the samples
  int cap;   // longest list the exact selection takes
};

inline SelPlan make_sel_plan(int N, int k) {
  SelPlan p{false, N < SEL_NS ? N : SEL_NS, 0, 0};
  if (N <= SEL_NS) {  // the sample is the row: exact pivot, list never misses
    p.ok = true;
    p.rank = k;
    p.cap = N;
    return p;
  }
  const int64_t ns = p.ns;
  // smallest rank with P(at least r samples among the first k - 1 tokens) <= eps;
  // below the mean of that count the probability is about 1/2 or more
  int64_t r = (int64_t)std::floor((double)(k - 1) * ns / N) + 1;
  while (r <= ns && hyper_sf(N, k - 1, ns, r) > SEL_EPS) ++r;
  if (r > ns) return p;
  p.rank = (int)r;
  for (int64_t cap = 1024; cap <= SEL_CAP; cap *= 2) {
    if (cap >= N) {
      p.cap = N;
      p.ok = true;
      return p;
    }
    if (hyper_cdf_below(N, cap, ns, r) <= SEL_EPS) {
      p.cap = (int)cap;
      p.ok = true;
      return p;
    }
  }
  return p;
}

// The plan of cfg's (N, k), remembered per thread for the last (N, k) seen.
inline SelPlan sel_plan(const mita_cfg_t &c) {
  thread_local int last_n = -1, last_k = -1;
  thread_local SelPlan last{};
  if (c.N != last_n || c.k != last_k) {
    last = make_sel_plan(c.N, c.k);
    last_n = c.N;
    last_k = c.k;
  }
  return last;
}

// Does the forward select the top-k sets inside the score pass?
inline bool fused_select(const mita_cfg_t &c) {
  return c.use_routed && !(c.flags & MITA_FLAG_FULL_SCORES) && sel_plan(c).ok;
}
inline int sel_ns(const mita_cfg_t &c) { return sel_plan(c).ns; }
inline int sel_rank(const mita_cfg_t &c) { return sel_plan(c).rank; }
inline int sel_cap(const mita_cfg_t &c) { return sel_plan(c).cap; }

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
  if (c->s < 1 || c->s > MITA_MAX_S) return fail(MITA_ERR_UNSUPPORTED, "s must be in [1, MITA_MAX_S]");
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
  if (c->use_routed && c->s > c->M) return fail(MITA_ERR_INVALID_ARG, "s must not exceed M");
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
      group, pair_o, pair_lse, plo, ccnt, cand, fail, total;
};

inline size_t scores_ws_bytes(const mita_cfg_t &c) {
  // per (b, h, chunk, landmark): (running max, running sum) and d accumulators
  const size_t rows = (size_t)BH(c) * score_chunks(c) * c.M;
  return align_up(rows * 2 * sizeof(float)) + align_up(rows * c.d * sizeof(float));
}
// Routing scratch: per-tile group counts, per-tile scatter bases, per-group
// totals, the attention work list and (s > 1) the group of every pair, in
// that order.
inline size_t route_tiles_bytes(const mita_cfg_t &c) {
  return align_up((size_t)BH(c) * route_tiles(c) * route_groups(c) * sizeof(int32_t));
}
inline size_t route_counts_bytes(const mita_cfg_t &c) {
  return align_up((size_t)BH(c) * route_groups(c) * sizeof(int32_t));
}
inline size_t route_start_bytes(const mita_cfg_t &c) {
  return align_up((size_t)BH(c) * (route_groups(c) + 1) * sizeof(int32_t));
}
inline size_t route_group_bytes(const mita_cfg_t &c) {
  return multi_route(c) ? align_up((size_t)BH(c) * route_items(c) * sizeof(int32_t)) : 0;
}
inline size_t route_ws_bytes(const mita_cfg_t &c) {
  return 2 * route_tiles_bytes(c) + route_counts_bytes(c) + route_start_bytes(c) + route_group_bytes(c);
}
// s > 1: the fp32 partial result and the log-sum-exp (log2 units) of every pair
inline size_t pair_out_bytes(const mita_cfg_t &c) {
  return multi_route(c) ? align_up((size_t)BH(c) * route_items(c) * c.d * sizeof(float)) : 0;
}
inline size_t pair_lse_bytes(const mita_cfg_t &c) {
  return multi_route(c) ? align_up((size_t)BH(c) * route_items(c) * sizeof(float)) : 0;
}
// attention scratch: the work list, then (s > 1) the pair partials
inline size_t attend_ws_bytes(const mita_cfg_t &c) {
  return route_start_bytes(c) + pair_out_bytes(c) + pair_lse_bytes(c);
}

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
  const size_t items = (size_t)route_items(c), groups = (size_t)route_groups(c);
  L.expert = take(c.use_routed ? bh * items * 4 : 0);
  L.perm = take(c.use_routed ? bh * items * 4 : 0);
  L.offsets = take(c.use_routed ? bh * (groups + 1) * 4 : 0);
  L.tile_cnt = take(c.use_routed ? bh * route_tiles(c) * groups * 4 : 0);
  L.tile_base = take(c.use_routed ? bh * route_tiles(c) * groups * 4 : 0);
  L.counts = take(c.use_routed ? bh * groups * 4 : 0);
  L.tile_start = take(c.use_routed ? bh * (groups + 1) * 4 : 0);
  L.group = take(route_group_bytes(c));
  L.pair_o = take(pair_out_bytes(c));
  L.pair_lse = take(pair_lse_bytes(c));
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

// Workspace of mita_backward: the forward's layout (its recomputation
// fills the landmarks, landmark values, score-pass partials, top-k sets and
// routing), then the landmark rows' log-sum-exp and the fp32 gradient
// buffers.
struct BwdLayout {
  FwdLayout f;
  size_t lse_lm, dq_direct, dk_acc, dv_acc, dq_lm_acc, dv_lm_acc, q_lse, q_D, stage_k, stage_v, inv_start, inv_slot,
      dv_lm16, D_lm, total;
};

inline BwdLayout backward_layout(const mita_cfg_t &c) {
  BwdLayout L{};
  L.f = forward_layout(c);
  size_t off = L.f.total;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes);
    return o;
  };
  const size_t bh = (size_t)BH(c), nd = bh * c.N * c.d * 4, md = bh * c.M * c.d * 4;
  L.lse_lm = take(bh * c.M * 4);
  L.dq_direct = take(nd);
  L.dk_acc = take(nd);
  L.dv_acc = take(nd);
  L.dq_lm_acc = take(md);
  L.dv_lm_acc = take(md);
  L.q_lse = take(bh * c.N * 4);
  L.q_D = take(bh * c.N * 4);
  const size_t stage = c.use_routed ? bh * c.M * (size_t)c.k * c.d * 4 : 0;
  L.stage_k = take(stage);
  L.stage_v = take(stage);
  L.inv_start = take(c.use_routed ? bh * (c.N + 1) * 4 : 0);
  L.inv_slot = take(c.use_routed ? bh * c.M * (size_t)c.k * 4 : 0);
  // the landmark values' gradient in bf16 and each landmark row's dV~ . V~
  L.dv_lm16 = take(c.use_shared ? bh * c.M * c.d * 2 : 0);
  L.D_lm = take(c.use_shared ? bh * c.M * 4 : 0);
  L.total = off;
  return L;
}

// Workspace of mita_landmarks_tome (the merge rounds' buffers, TomeBufs order).
struct TomeLayout {
  size_t S0, S1, cnt0, cnt1, rep0, rep1, X, score, match, sel, merged, alive, pos, total;
};

inline TomeLayout tome_layout(const mita_cfg_t &c) {
  TomeLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes);
    return o;
  };
  const size_t bh = (size_t)BH(c), n = (size_t)c.N, h = (n + 1) / 2;
  L.S0 = take(bh * n * c.d * 8);
  L.S1 = take(bh * n * c.d * 8);
  L.cnt0 = take(bh * n * 4);
  L.cnt1 = take(bh * n * 4);
  L.rep0 = take(bh * n * 4);
  L.rep1 = take(bh * n * 4);
  L.X = take(bh * n * c.d * 4);
  L.score = take(bh * h * 4);
  L.match = take(bh * h * 4);
  L.sel = take(bh * h * 4);
  L.merged = take(bh * h * 4);
  L.alive = take(bh * n * 4);
  L.pos = take(bh * (n + 1) * 4);
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
    case MITA_WS_BACKWARD: return c->s == 1 || !c->use_routed ? backward_layout(*c).total : 0;
    case MITA_WS_TOME: return tome_layout(*c).total;
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
