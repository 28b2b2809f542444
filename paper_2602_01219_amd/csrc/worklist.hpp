// worklist.hpp - the attention work list: which 64 queries (of one expert
// group) a workgroup of an attention kernel takes.
#pragma once
#include "cdna4.hpp"
#include "check.hpp"

namespace mita {

// Work-list tiles are spread so that each XCD takes a contiguous range of
// the (head, tile) slots, head-major: with at least 8 heads an XCD works
// through whole heads, one at a time, so the head's K and V rows are fetched
// into that XCD's L2 only (spread by tile within each head, every XCD needed
// a share of every head's rows, about three times the K / V fetches at the
// 16K-token shape); consecutive tiles, usually of one expert, share the L2
// too. Workgroups go to the 8 XCDs round robin by linear index L (x fastest),
// so slot f = (L % 8) * C + L / 8, C = slots / 8, covers head f / T and tile
// f % T of that head, T = the grid's x extent (a multiple of 8).
constexpr int NXCD = 8;

// Slot of workgroup L in a grid of NXCD * C workgroups whose slots the XCDs
// take in contiguous ranges of C (XCD x: slots [x C, (x + 1) C)).
__device__ __forceinline__ int xcd_slot(int L, int C) { return (L % NXCD) * C + L / NXCD; }

// The workgroup's head bh, queries [q_begin, q_end) (positions in perm) and
// their group e (of G), from the work list; false for a workgroup past its
// end. Without ROUTED, bh keeps the caller's value and the workgroup takes
// queries 64 blockIdx.x onwards.
template <bool ROUTED>
__device__ __forceinline__ bool attend_queries(const int32_t *__restrict__ tile_start,
                                               const int32_t *__restrict__ offsets, int64_t &bh, int N, int M,
                                               int &e, int &q_begin, int &q_end) {
  e = 0;
  if (ROUTED) {
    const int T = (int)gridDim.x;
    const int64_t L = (int64_t)blockIdx.y * T + blockIdx.x;
    const int64_t C = (int64_t)T * gridDim.y / NXCD;
    const int64_t f = (L % NXCD) * C + L / NXCD;
    bh = f / T;
    const int t = (int)(f % T);
    const int32_t *ts = tile_start + bh * (M + 1);
    const int ntl = ts[M];
    if (t >= ntl) return false;
    int lo = 0, hi = M - 1;  // largest e with ts[e] <= t
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (ts[mid] <= t)
        lo = mid;
      else
        hi = mid - 1;
    }
    e = lo;
    const int32_t *of = offsets + bh * (M + 1);
    q_begin = of[e] + (t - ts[e]) * ATT_TQ;
    q_end = min(of[e + 1], q_begin + ATT_TQ);
  } else {
    q_begin = (int)blockIdx.x * ATT_TQ;
    if (q_begin >= N) return false;
    q_end = min(N, q_begin + ATT_TQ);
  }
  return true;
}

}  // namespace mita
