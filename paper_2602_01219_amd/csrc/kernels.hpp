// kernels.hpp - launchers of the MiTA HIP kernels (host side declarations).
// Every launcher only enqueues on `st`; shapes were validated by the caller.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mita.h"

namespace mita {

// Landmark pooling (Sec. 3.2; Algorithm 1 AdaptiveAvgPool): q [BH,N,d] -> q_lm [BH,M,d].
// If zero_counts is not NULL its BH*M entries are set to 0 (routing totals).
hipError_t launch_pool(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *zero_counts, hipStream_t st);

// Set n int32 entries to 0.
hipError_t launch_zero(int32_t *p, int64_t n, hipStream_t st);

// Scores S = fl(q_lm . k) * scale (optional) and landmark values (optional):
// split over key chunks, partials in `partial`, merged into v_lm.
hipError_t launch_scores(const mita_cfg_t &c, const void *q_lm, const void *k, const void *v, float *scores,
                         void *v_lm, void *partial, hipStream_t st);

// Exact per-row top-k of fp32 scores [rows, N] -> ascending int32 indices [rows, k].
hipError_t launch_topk(const mita_cfg_t &c, const float *scores, int32_t *idx, hipStream_t st);

// Expert tiles k_x/v_x [BH,M,k,d] from idx [BH,M,k].
hipError_t launch_gather(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                         hipStream_t st);

// Routing: expert [BH,N], per-tile counts and bases, offsets [BH,M+1], perm [BH,N],
// attention work list tile_start [BH,M+1]. counts [BH,M] must be zero on entry.
hipError_t launch_route(const mita_cfg_t &c, const void *q, const void *q_lm, int32_t *expert, int32_t *perm,
                        int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base, int32_t *counts,
                        int32_t *tile_start, hipStream_t st);

// Attention work list from offsets: tile_start [BH, M+1].
hipError_t launch_worklist(const mita_cfg_t &c, const int32_t *offsets, int32_t *tile_start, hipStream_t st);

// MiTA attention (Eq. mita). With idx != NULL the routed keys are read in place
// from k/v rows idx[b,h,e,:]; otherwise from the expert tiles kx/vx.
hipError_t launch_attend(const mita_cfg_t &c, const void *q, const void *q_lm, const void *v_lm, const void *kv_k,
                         const void *kv_v, const int32_t *idx, const int32_t *perm, const int32_t *offsets,
                         const int32_t *tile_start, void *o, hipStream_t st);

}  // namespace mita
