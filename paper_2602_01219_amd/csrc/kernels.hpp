// kernels.hpp - launchers of the MiTA HIP kernels (host side declarations).
// Every launcher only enqueues on `st`; shapes were validated by the caller.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mita.h"

namespace mita {

// Per-launch timing of mita_forward_timed: every launcher calls
// launched(kernel, st) right after enqueueing a kernel. It records an event on
// st behind the launch when a timed forward is being enqueued on this thread
// (nothing otherwise) and returns hipGetLastError().
hipError_t launched(const char *kernel, hipStream_t st);

// Landmark pooling (Sec. 3.2; Algorithm 1 AdaptiveAvgPool): q [BH,N,d] -> q_lm [BH,M,d].
// If zero_counts (zero_cursor) is not NULL its BH*M entries are set to 0
// (routing totals; the forward's placement cursors).
hipError_t launch_pool(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *zero_counts, int32_t *zero_cursor,
                       hipStream_t st);

// Set n int32 entries to 0.
hipError_t launch_zero(int32_t *p, int64_t n, hipStream_t st);
// The same for two arrays in one launch (either may be NULL or empty).
hipError_t launch_zero2(int32_t *p, int64_t n, int32_t *p2, int64_t n2, hipStream_t st);

// Buffers of the top-k selection fused with the score pass (rows = BH*M).
struct SelectBufs {
  uint32_t *plo;        // [rows] pivot keys
  uint32_t *ccnt;       // [rows, chunks] candidates listed per key chunk
  uint2 *cand;          // [rows, chunks, SCORE_NC] (unscaled dot bits, token index) lists
  uint32_t *fail_cnt;   // rows that fall back to the full score row
  int32_t *fail_list;   // [rows] their row numbers
  int ns, cap, rank;
  // non-null when the sample is the whole row (ns == N): the pivot launch
  // writes the top-k sets here itself, the score pass lists nothing and the
  // finish selects nothing (direct selection)
  int32_t *idx;
};

// Scores S = fl(q_lm . k) * scale (optional) and landmark values (optional):
// split over key chunks, partials in `partial`, merged into v_lm. With sel,
// the candidates of the fused selection are listed instead of storing S
// (launch_select_pivots must have run) and the landmark-value merge is left to
// launch_select_finish.
hipError_t launch_scores(const mita_cfg_t &c, const void *q_lm, const void *k, const void *v, float *scores,
                         void *v_lm, void *partial, const SelectBufs *sel, hipStream_t st);

// Fused selection, before the score pass: sampled scores, per-row pivots;
// zeroes the candidate and fallback counters.
hipError_t launch_select_pivots(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sel,
                                hipStream_t st);

// Fused selection, after the score pass: exact top-k from the candidate
// lists into idx; rows whose list is unusable get their score row recomputed
// into S (same arithmetic as the score pass) and the exact top-k of it. With
// v_lm, also merges the score pass's landmark-value partials into v_lm (the
// score pass then leaves that merge out).
hipError_t launch_select_finish(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sel,
                                float *S, int32_t *idx, const void *partial, void *v_lm, hipStream_t st);

// Score rows of the listed landmark rows only (fallback of the fused selection).
hipError_t launch_scores_rows(const mita_cfg_t &c, const void *q_lm, const void *k, float *S,
                              const uint32_t *nrows, const int32_t *rows, hipStream_t st);

// Exact per-row top-k of fp32 scores [rows, N] -> ascending int32 indices [rows, k].
// With nrows/rows != NULL only the *nrows rows listed in rows are processed.
hipError_t launch_topk(const mita_cfg_t &c, const float *scores, int32_t *idx, hipStream_t st,
                       const uint32_t *nrows = nullptr, const int32_t *rows = nullptr);

// Expert tiles k_x/v_x [BH,M,k,d] from idx [BH,M,k].
hipError_t launch_gather(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                         hipStream_t st);

// Routing: expert [BH,N], per-tile counts and bases, offsets [BH,M+1], perm [BH,N],
// attention work list tile_start [BH,M+1]. counts [BH,M] must be zero on entry.
// With s > 1: expert [BH,N,s], the pairs' groups in group [BH,N*s], perm [BH,N*s],
// offsets and tile_start [BH,2M+1], counts [BH,2M] (zeroed here).
hipError_t launch_route(const mita_cfg_t &c, const void *q, const void *q_lm, int32_t *expert, int32_t *perm,
                        int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base, int32_t *counts,
                        int32_t *tile_start, int32_t *group, hipStream_t st);

// The finish of the fused selection (launch_select_finish: top-k into idx,
// fallback rows, landmark-value merge into v_lm when given) together with the
// routing (launch_route), in two combined launches; with logits_done the
// routing logits (expert, counts) were formed by launch_pivots_logits and the
// first launch runs the selection's finish rows alone.
hipError_t launch_select_route(const mita_cfg_t &c, const void *q, const void *q_lm, const void *k,
                               const SelectBufs &sel, float *S, int32_t *idx, const void *partial, void *v_lm,
                               int32_t *expert, int32_t *perm, int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base,
                               int32_t *counts, int32_t *tile_start, bool logits_done, hipStream_t st);

// Whether launch_pivots_logits serves this configuration (bf16, sample in LDS).
bool pivots_with_logits(const mita_cfg_t &c, const SelectBufs &sel);
// The sampled scores and pivots (launch_select_pivots) and the routing
// logits (expert [BH,N] and counts [BH,M], which must be zero on entry) in one
// launch.
hipError_t launch_pivots_logits(const mita_cfg_t &c, const void *q, const void *q_lm, const void *k,
                                const SelectBufs &sel, int32_t *expert, int32_t *counts, hipStream_t st);

// Attention work list from offsets: tile_start [BH, M+1].
hipError_t launch_worklist(const mita_cfg_t &c, const int32_t *offsets, int32_t *tile_start, hipStream_t st);

// MiTA attention (Eq. mita). With idx != NULL the routed keys are read in place
// from k/v rows idx[b,h,e,:]; otherwise from the expert tiles kx/vx. With
// s > 1 the pairs' partials go to pair_o [BH,N*s,d] / pair_lse [BH,N*s] and a
// combine launch merges them into o.
hipError_t launch_attend(const mita_cfg_t &c, const void *q, const void *q_lm, const void *v_lm, const void *kv_k,
                         const void *kv_v, const int32_t *idx, const int32_t *perm, const int32_t *offsets,
                         const int32_t *tile_start, void *o, float *pair_o, float *pair_lse, hipStream_t st);

// Random-selection landmarks: q_lm[bh, i] = q[bh, sel[bh, i]] (NaN row for an
// index outside [0, N)).
hipError_t launch_select_landmarks(const mita_cfg_t &c, const void *q, const int32_t *sel, void *q_lm,
                                   hipStream_t st);

// Backward pass (gradients with the top-k sets and routing held fixed).
// Inputs: the forward's tensors and the state its recomputation left in the
// workspace; accumulators zeroed beforehand.
struct BwdBufs {
  const void *q, *k, *v, *o, *dO;  // [BH, N, d]
  const void *q_lm, *v_lm;         // [BH, M, d]
  const int32_t *idx, *perm, *offsets, *tile_start;
  const void *part_ml;             // score-pass partials (max, sum) per key chunk
  float *lse_lm;                   // [BH, M] (written)
  float *dq_direct;                // [BH, N, d] (written)
  float *dk_acc, *dv_acc;          // [BH, N, d] (zeroed)
  float *dq_lm_acc, *dv_lm_acc;    // [BH, M, d] (zeroed)
  float *q_lse, *q_D;              // [BH, N] per-query log-sum-exp and dO . o (written)
  float *stage_k, *stage_v;        // [BH, M, k, d] per-expert sums of the routed keys (written)
  int32_t *inv_start, *inv_slot;   // inverse index of the top-k sets: [BH, N + 1], [BH, M * k]
  void *dv_lm16;                   // [BH, M, d] bf16 copy of the landmark values' gradient
  float *D_lm;                     // [BH, M] dV~ . V~ per landmark row
  void *dq, *dk, *dv;              // [BH, N, d] outputs (io type)
};
hipError_t launch_backward(const mita_cfg_t &c, const BwdBufs &b, hipStream_t st);

// Exclusive scan of n int32 counts per head (cnt [BH, n]) into start [BH, n + 1].
hipError_t launch_scan_counts(const int32_t *cnt, int32_t *start, int n, int64_t bh, hipStream_t st);

// Token merging as landmark extraction: q_lm [BH, M, d]; assign [BH, N] (the
// landmark of every token) when not NULL. Buffers of the merge rounds:
struct TomeBufs {
  int64_t *S[2];           // [BH, N, d] member sums of the current tokens (fixed point), ping-pong
  int32_t *cnt[2];         // [BH, N] member counts
  int32_t *rep[2];         // [BH, N] every token's current position
  float *X;                // [BH, N, d] unit vectors of the sums
  float *score;            // [BH, ceil(N / 2)] edge scores
  int32_t *match, *sel, *merged;  // [BH, ceil(N / 2)]
  int32_t *alive, *pos;    // [BH, N], [BH, N + 1]
};
hipError_t launch_tome(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *assign, const TomeBufs &b,
                       hipStream_t st);

}  // namespace mita
