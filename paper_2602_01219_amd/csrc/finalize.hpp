// finalize.hpp - the finish of the fused top-k selection for one landmark
// row (Eq. top-k): exact top-k from the row's candidate lists, the row's
// landmark-value merge; used by the finalize kernel and by the launch that
// runs it together with the routing logits.
#pragma once
#include "cdna4.hpp"
#include "flash.hpp"
#include "check.hpp"
#include "sample.hpp"

namespace mita {

// ---------------------------------------------------------------------------
// Exact top-k from the candidate lists: one workgroup per landmark row. The
// order is that of the composite C = key * 2^32 + (2^32 - 1 - index), larger
// first; composites are distinct, so exactly k tokens have C >= C_k, the k-th
// largest. The row's chunk regions are packed into LDS (token order kept);
// radix rounds over a 256-bin histogram of the current composite range (each
// round shrinks the range by 2^8) run until at most 64 candidates remain,
// which one wave ranks directly; an ordered scan then writes the tokens with
// C >= C_k.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t composite(uint2 e) {
  return ((uint64_t)e.x << 32) | (uint64_t)(0xffffffffu - e.y);
}

constexpr int MAX_CHUNKS = MITA_MAX_N / SCORE_NC;

template <typename T, int D, int CAP, bool MERGE> struct FinalizeLds {
  float red[MERGE ? 256 / D : 1][3][D];
  uint2 lst[CAP];
  uint32_t pre[MAX_CHUNKS + 1];
  uint32_t hist[256];
  uint32_t wsum[2][4];
  uint64_t wred[2][4];
  uint64_t rem[64];
  uint64_t bc64;
  uint32_t bc[3];
};

template <typename T, int D, int CAP, bool MERGE>
__device__ __forceinline__ void finalize_row(FinalizeLds<T, D, CAP, MERGE> &sh, int64_t row,
                                             const uint2 *__restrict__ cand, const uint32_t *__restrict__ ccnt,
                                             int32_t *__restrict__ idx, uint32_t *__restrict__ fail_cnt,
                                             int32_t *__restrict__ fail_list, int k, int cap, int nch,
                                             const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                             T *__restrict__ v_lm, int M, float scale) {
  auto &red = sh.red;
  auto &lst = sh.lst;
  auto &pre = sh.pre;
  auto &hist = sh.hist;
  auto &wsum = sh.wsum;
  auto &wred = sh.wred;
  auto &rem = sh.rem;
  auto &bc64 = sh.bc64;
  auto &bc = sh.bc;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  // the landmark-value partials are loaded first; the merge uses them last
  LandmarkMerge<T, D> lmm;
  if (MERGE) lmm.prefetch(part_ml, part_o, row / M, (int)(row % M), M, nch);

  // chunk counts -> exclusive prefix (nch <= 256: one chunk per thread)
  const uint32_t cc = tid < nch ? ccnt[row * nch + tid] : 0u;
  const uint32_t wincl = wave_inclusive_scan(cc);
  if (lane == 63) wsum[0][w] = wincl;
  __syncthreads();
  uint32_t before = 0, total = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    before += i < w ? wsum[0][i] : 0u;
    total += wsum[0][i];
  }
  if (tid <= nch) pre[tid] = before + wincl - cc;
  if (total < (uint32_t)k || total > (uint32_t)cap) {  // uniform
    if (tid == 0) fail_list[atomicAdd(fail_cnt, 1u)] = (int32_t)row;
    if (MERGE) lmm.finish(part_ml, part_o, v_lm, row / M, (int)(row % M), M, nch, red);
    return;
  }
  __syncthreads();
  // compaction into LDS, with the composite range of the list: wave w copies
  // chunks w, w + 4, ..., lane j taking entries j, j + 64, ...; the first 64
  // entries of CU chunks are loaded together before any is stored
  const int L = (int)total;
  uint64_t lo = ~0ull, hi = 0ull;
  auto put = [&](uint2 e, uint32_t at) {
    // listed as the bits of the unscaled dot: the score is fl(dot * scale)
    const uint2 x = make_uint2(score_key(__uint_as_float(e.x) * scale), e.y);
    lst[at] = x;
    const uint64_t c = composite(x);
    lo = c < lo ? c : lo;
    hi = c > hi ? c : hi;
  };
  constexpr int CU = 4;
  const uint2 *crow = cand + row * nch * (int64_t)SCORE_NC;
  for (int c0 = w; c0 < nch; c0 += 4 * CU) {
    uint2 e[CU];
    uint32_t b[CU], n[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const int c = c0 + 4 * u;
      b[u] = c < nch ? pre[c] : 0u;
      n[u] = c < nch ? pre[c + 1] - b[u] : 0u;
      e[u] = (uint32_t)lane < n[u] ? crow[(int64_t)c * SCORE_NC + lane] : make_uint2(0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < CU; ++u)
      if ((uint32_t)lane < n[u]) put(e[u], b[u] + lane);
#pragma unroll
    for (int u = 0; u < CU; ++u)
      for (uint32_t j = lane + 64; j < n[u]; j += 64) put(crow[(int64_t)(c0 + 4 * u) * SCORE_NC + j], b[u] + j);
  }
  lo = wave_min_u64(lo);
  hi = wave_max_u64(hi);
  if (lane == 0) {
    wred[0][w] = lo;
    wred[1][w] = hi;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    lo = wred[0][i] < lo ? wred[0][i] : lo;
    hi = wred[1][i] > hi ? wred[1][i] : hi;
  }
  uint32_t need = (uint32_t)k, inrange = (uint32_t)L;
  uint64_t ck = 0;
  while (true) {
    if (lo == hi) {  // a single composite left
      ck = lo;
      break;
    }
    if (inrange <= 64u) {
      if (tid == 0) bc[0] = 0u;
      __syncthreads();
      for (int i = tid; i < L; i += 256) {
        const uint64_t c = composite(lst[i]);
        if (c >= lo && c <= hi) {
          const uint32_t s = atomicAdd(&bc[0], 1u);
          if (s < 64u) rem[s] = c;
        }
      }
      __syncthreads();
      if (w == 0) {
        const uint64_t mine = lane < (int)inrange ? rem[lane] : 0ull;
        uint32_t rank = 0;
        for (uint32_t j = 0; j < inrange; ++j) rank += rem[j] > mine;
        if (lane < (int)inrange && rank == need - 1u) bc64 = mine;
      }
      __syncthreads();
      ck = bc64;
      break;
    }
    const uint64_t span = hi - lo;
    const int bits = 64 - __clzll((long long)span);
    const int shift = bits > 8 ? bits - 8 : 0;
    hist[tid] = 0u;
    __syncthreads();
    for (int i = tid; i < L; i += 256) {
      const uint64_t c = composite(lst[i]);
      if (c >= lo && c <= hi) atomicAdd(&hist[(uint32_t)((c - lo) >> shift)], 1u);
    }
    __syncthreads();
    // thread t takes bin 255 - t: the scan runs from the top bin down
    const uint32_t cnt = hist[255 - tid];
    const uint32_t incl = wave_inclusive_scan(cnt);
    if (lane == 63) wsum[1][w] = incl;
    __syncthreads();
    uint32_t ab = incl - cnt;
#pragma unroll
    for (int i = 0; i < 4; ++i) ab += i < w ? wsum[1][i] : 0u;
    if (ab < need && need <= ab + cnt) {
      bc[0] = (uint32_t)(255 - tid);
      bc[1] = ab;
      bc[2] = cnt;
    }
    __syncthreads();
    const uint32_t b = bc[0];
    need -= bc[1];
    inrange = bc[2];
    lo += (uint64_t)b << shift;
    const uint64_t width = (1ull << shift) - 1ull;
    if (hi - lo > width) hi = lo + width;
    __syncthreads();  // bc and hist are rewritten by the next round
  }

  // ordered output: the list is in ascending token order; thread t takes
  // entries [t E, t E + E) and one block scan places its selected ones
  int32_t *out = idx + row * (int64_t)k;
  const int E = (L + 255) / 256;
  const int i0 = tid * E, i1 = min(L, i0 + E);
  uint32_t nsel = 0;
  for (int i = i0; i < i1; ++i) nsel += composite(lst[i]) >= ck;
  const uint32_t sincl = wave_inclusive_scan(nsel);
  if (lane == 63) wsum[0][w] = sincl;  // wsum[0] was last read before the compaction
  __syncthreads();
  uint32_t at = sincl - nsel;
#pragma unroll
  for (int j = 0; j < 4; ++j) at += j < w ? wsum[0][j] : 0u;
  for (int i = i0; i < i1; ++i) {
    const uint2 e = lst[i];
    if (composite(e) >= ck) {
      if (at < (uint32_t)k) out[at] = (int32_t)e.y;
      ++at;
    }
  }
  if (MERGE) lmm.finish(part_ml, part_o, v_lm, row / M, (int)(row % M), M, nch, red);
}

// ---------------------------------------------------------------------------
// The same finish by one wave per row, for lists of at most SEL_NS entries
// and at most 64 key chunks (no barriers; a workgroup takes four rows):
// the chunk regions are packed into LDS in token order, the keys (score_key
// of the scaled dot) read back 16 per lane (entry j = lane + 64 m, key 0
// past the list), the k-th largest key K found exactly by pivot_of, and an
// ordered scan over the entries writes every token with a key above K and,
// in token order, as many with key K as the set still needs: the tokens with
// composite >= C_k, in ascending order, as finalize_row writes them.
// ---------------------------------------------------------------------------
struct FinalizeWaveLds {
  uint2 lst[SEL_NS];
  uint32_t scratch[384];  // pivot_of's histogram and slots
};

template <typename T, int D, bool MERGE>
__device__ __forceinline__ void finalize_row_wave(FinalizeWaveLds &sh, int64_t row, const uint2 *__restrict__ cand,
                                                  const uint32_t *__restrict__ ccnt, int32_t *__restrict__ idx,
                                                  uint32_t *__restrict__ fail_cnt, int32_t *__restrict__ fail_list,
                                                  int k, int cap, int nch, const float2 *__restrict__ part_ml,
                                                  const float *__restrict__ part_o, T *__restrict__ v_lm, int M,
                                                  float scale) {
  const int lane = threadIdx.x & 63;
  // the landmark-value partials are loaded first; the merge uses them last
  constexpr int DL = D / 64;  // dimensions per lane
  LandmarkMerge1<D> lmm[DL];
  if (MERGE)
#pragma unroll
    for (int u = 0; u < DL; ++u) lmm[u].prefetch(part_ml, part_o, row / M, (int)(row % M), M, nch, lane + 64 * u);
  // chunk counts -> exclusive prefix (nch <= 64: one chunk per lane)
  const uint32_t cc = lane < nch ? ccnt[row * nch + lane] : 0u;
  const uint32_t incl = wave_inclusive_scan(cc);
  const uint32_t total = (uint32_t)__shfl((int)incl, 63);
  const uint32_t excl = incl - cc;
  if (total >= (uint32_t)k && total <= (uint32_t)cap) {
    // the list into LDS, the first 64 entries of four chunks loaded before any is stored
    const uint2 *crow = cand + row * nch * (int64_t)SCORE_NC;
    for (int c0 = 0; c0 < nch; c0 += 4) {
      uint2 e[4];
      uint32_t n[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + u < nch ? c0 + u : 0;
        n[u] = c0 + u < nch ? (uint32_t)__shfl((int)cc, c) : 0u;
        b[u] = (uint32_t)__shfl((int)excl, c);
        e[u] = (uint32_t)lane < n[u] ? crow[(int64_t)c * SCORE_NC + lane] : make_uint2(0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if ((uint32_t)lane < n[u]) sh.lst[b[u] + lane] = make_uint2(score_key(__uint_as_float(e[u].x) * scale), e[u].y);
        for (uint32_t j = lane + 64; j < n[u]; j += 64) {
          const uint2 x = crow[(int64_t)(c0 + u) * SCORE_NC + j];
          sh.lst[b[u] + j] = make_uint2(score_key(__uint_as_float(x.x) * scale), x.y);
        }
      }
    }
    uint32_t v[PIVOT_PER];
    int32_t ix[PIVOT_PER];
#pragma unroll
    for (int m = 0; m < PIVOT_PER; ++m) {
      const uint32_t j = (uint32_t)(lane + 64 * m);
      const uint2 x = j < total ? sh.lst[j] : make_uint2(0u, 0u);
      v[m] = x.x;
      ix[m] = (int32_t)x.y;
    }
    const uint32_t K = pivot_of(v, sh.scratch, k);
    uint32_t gt = 0;
#pragma unroll
    for (int m = 0; m < PIVOT_PER; ++m) gt += v[m] > K ? 1u : 0u;
    const uint32_t need_eq = (uint32_t)k - wave_sum_u32(gt);  // >= 1: K is the k-th largest
    int32_t *out = idx + row * (int64_t)k;
    uint32_t taken = 0, eq_seen = 0;
#pragma unroll
    for (int m = 0; m < PIVOT_PER; ++m) {
      const uint64_t be = __ballot(v[m] == K);
      const bool take = v[m] > K || (v[m] == K && eq_seen + lanes_below(be) < need_eq);
      const uint64_t bt = __ballot(take);
      if (take) out[taken + lanes_below(bt)] = ix[m];
      taken += (uint32_t)__popcll(bt);
      eq_seen += (uint32_t)__popcll(be);
    }
  } else if (lane == 0) {
    fail_list[atomicAdd(fail_cnt, 1u)] = (int32_t)row;
  }
  if (MERGE)
#pragma unroll
    for (int u = 0; u < DL; ++u)
      v_lm[row * D + lane + 64 * u] =
          from_f32<T>(lmm[u].finish(part_ml, part_o, row / M, (int)(row % M), M, nch, lane + 64 * u));
}

}  // namespace mita
