// worklist.hpp - the attention work list: which 64 queries (of one expert
// group) a workgroup of an attention kernel takes.
#pragma once
#include "cdna4.hpp"
#include "check.hpp"

namespace mita {

// Work-list tiles are spread so that consecutive tiles (usually of the same
// expert) run on the same XCD and share its L2: with 8 XCDs taking workgroups
// round robin, x -> (xcd = x % 8, slot = x / 8) covers tile xcd * C + slot,
// C = ceil(tiles / 8); the grid's x extent is a multiple of 8.
constexpr int NXCD = 8;

// The workgroup's queries [q_begin, q_end) (positions in perm) and their
// group e (of G), from the work list; false for a workgroup past its end.
template <bool ROUTED>
__device__ __forceinline__ bool attend_queries(const int32_t *__restrict__ tile_start,
                                               const int32_t *__restrict__ offsets, int64_t bh, int N, int M, int &e,
                                               int &q_begin, int &q_end) {
  e = 0;
  if (ROUTED) {
    const int32_t *ts = tile_start + bh * (M + 1);
    const int ntl = ts[M];
    const int C = (ntl + NXCD - 1) / NXCD;
    const int slot = (int)blockIdx.x / NXCD;
    const int t = ((int)blockIdx.x % NXCD) * C + slot;
    if (slot >= C || t >= ntl) return false;
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
