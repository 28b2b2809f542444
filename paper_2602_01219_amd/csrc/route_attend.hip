// route_attend.hip - routing of queries to landmarks and the MiTA attention.
#include <climits>
#include <type_traits>

#include "cdna4.hpp"
#include "flash.hpp"
#include "kernels.hpp"
#include "check.hpp"
#include "scores.hpp"
#include "topk_row.hpp"
#include "finalize.hpp"
#include "sample.hpp"
#include "worklist.hpp"

namespace mita {

// ---------------------------------------------------------------------------
// Routing logits and argmax (Sec. 3.2: logits Q^T Q_lm, rank-1 expert;
// Algorithm 1 ArgMax). Workgroup = 4 waves, wave = one 64-query routing tile
// (4 column groups of 16 queries). The landmarks are staged in LDS 64 at a
// time; each wave forms L^T = Q_lm Q^T on MFMA one 16-landmark block at a
// time, every landmark fragment serving its 4 query groups, and keeps a
// lane-local running (max, argmax) with strict '>' in increasing landmark
// order, then merges the four lane groups of each query column preferring
// the lower landmark on equal values. Each wave also counts its tile's
// queries per expert and adds them to the per-expert totals (zeroed
// beforehand).
// ---------------------------------------------------------------------------
constexpr int ROUTE_LB = 64;  // landmarks staged in LDS per step

template <typename T, int D> struct RouteLds {
  static constexpr int VE = 16 / (int)sizeof(T);
  static constexpr int LSTR = D + VE;  // padded landmark row (elements)
  static constexpr int BYTES = ROUTE_LB * LSTR * (int)sizeof(T);
};

// Workgroup (bx, by) of the routing grid (NWV waves, one 64-query tile
// each); lms: RouteLds<T, D>::BYTES of LDS, cnt: NWV M words of LDS.
template <typename T, int D, bool TILES = true, int NWV = 4>
__device__ __forceinline__ void route_logits_body(T *lms, uint32_t *cnt, int bx, int by, const T *__restrict__ q,
                                                  const T *__restrict__ q_lm, int32_t *__restrict__ expert,
                                                  int32_t *__restrict__ tile_cnt, int32_t *__restrict__ counts, int N,
                                                  int M, float scale, int ntiles) {
  constexpr int VE = RouteLds<T, D>::VE;
  constexpr int LSTR = RouteLds<T, D>::LSTR;
  const int64_t bh = by;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int tile = bx * NWV + w;
  uint32_t *wc = cnt + w * M;
  for (int i = lane; i < M; i += 64) wc[i] = 0u;
  Frag<T> qf[4][D / 32];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int n = tile * ROUTE_TQ + c * 16 + p;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (n < N)
        qf[c][ks].load(q + (bh * N + n) * D + ks * 32 + g * 8);
      else
        qf[c][ks].zero();
    }
  }
  const T *lmb = q_lm + bh * (int64_t)M * D;
  float best[4];
  int arg[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    best[c] = -INFINITY;
    arg[c] = 0;
  }
  for (int l0 = 0; l0 < M; l0 += ROUTE_LB) {
    const int nl = min(ROUTE_LB, M - l0);
    __syncthreads();
    for (int ch = threadIdx.x; ch < ROUTE_LB * (D / VE); ch += 64 * NWV) {
      const int r = ch / (D / VE), cc = ch % (D / VE);
      uint4 x = make_uint4(0, 0, 0, 0);
      if (r < nl) x = *reinterpret_cast<const uint4 *>(lmb + (int64_t)(l0 + r) * D + cc * VE);
      *reinterpret_cast<uint4 *>(lms + r * LSTR + cc * VE) = x;
    }
    __syncthreads();
    if (tile >= ntiles) continue;
    for (int sb = 0; sb < nl; sb += 16) {
      f32x4 acc[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<T> a;
        a.load(lms + (sb + p) * LSTR + ks * 32 + g * 8);
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = mma(a, qf[c][ks], acc[c]);
      }
      // running argmax, branch-free (selects); the first maximum is kept, and
      // landmarks are visited in increasing order, so ties go to the lower one
      const bool full = sb + 16 <= nl;
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int lmi = l0 + sb + 4 * g + r;
          const float val = acc[c][r] * scale;
          const bool up = (full || lmi < M) && val > best[c];
          best[c] = up ? val : best[c];
          arg[c] = up ? lmi : arg[c];
        }
    }
  }
  if (tile >= ntiles) return;  // no workgroup barriers below
  // merge the four lane groups of each query column (lower landmark wins ties)
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float ob = __shfl_xor(best[c], o);
      const int oa = __shfl_xor(arg[c], o);
      if (ob > best[c] || (ob == best[c] && oa < arg[c])) {
        best[c] = ob;
        arg[c] = oa;
      }
    }
    const int n = tile * ROUTE_TQ + c * 16 + p;
    if (g == 0 && n < N) {
      expert[bh * N + n] = arg[c];
      atomicAdd(&wc[arg[c]], 1u);
    }
  }
  int32_t *tc = TILES ? tile_cnt + (bh * ntiles + tile) * (int64_t)M : nullptr;
  for (int i = lane; i < M; i += 64) {
    const uint32_t x = wc[i];
    if (TILES) tc[i] = (int32_t)x;
    if (x) atomicAdd(&counts[bh * M + i], (int32_t)x);  // integer sums: order-independent
  }
}

template <typename T, int D>
__global__ __launch_bounds__(BLOCK) void route_logits_kernel(const T *__restrict__ q, const T *__restrict__ q_lm,
                                                             int32_t *__restrict__ expert,
                                                             int32_t *__restrict__ tile_cnt,
                                                             int32_t *__restrict__ counts, int N, int M,
                                                             float scale, int ntiles) {
  __shared__ __align__(16) T lms[RouteLds<T, D>::BYTES / sizeof(T)];
  extern __shared__ uint32_t cnt[];  // [4][M]
  route_logits_body<T, D>(lms, cnt, (int)blockIdx.x, (int)blockIdx.y, q, q_lm, expert, tile_cnt, counts, N, M, scale,
                          ntiles);
}

// ---------------------------------------------------------------------------
// Routing to S > 1 experts (Sec. 3.2: e_j(q), the rank-j expert under the
// logits Q^T Q_lm). The logits are formed as in route_logits_body; each lane
// keeps the S best (logit, landmark) pairs of the landmarks it sees, ordered
// by larger logit, then lower landmark (a NaN logit counts as -inf). The
// four lane groups of a query column then merge their lists: S rounds, each
// taking the best head among the four lists (the owner's list advances;
// landmarks are distinct, so the owner is unique). Writes expert[n * S + j]
// and the pair's group: expert for j = 0, M + expert otherwise.
// ---------------------------------------------------------------------------
template <int S> struct TopS {
  float v[S];
  int a[S];
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int j = 0; j < S; ++j) {
      v[j] = -INFINITY;
      a[j] = INT_MAX;  // sorts after every landmark
    }
  }
  // insertion in order: (x, i) moves down the list past every entry it beats
  __device__ __forceinline__ void insert(float x, int i) {
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const bool up = x > v[j] || (x == v[j] && i < a[j]);
      const float tv = v[j];
      const int ta = a[j];
      v[j] = up ? x : v[j];
      a[j] = up ? i : a[j];
      x = up ? tv : x;
      i = up ? ta : i;
    }
  }
  __device__ __forceinline__ void head(int h, float &x, int &i) const {
    x = -INFINITY;
    i = INT_MAX;
#pragma unroll
    for (int j = 0; j < S; ++j) {
      x = h == j ? v[j] : x;
      i = h == j ? a[j] : i;
    }
  }
};

template <typename T, int D, int S>
__global__ __launch_bounds__(BLOCK) void route_tops_kernel(const T *__restrict__ q, const T *__restrict__ q_lm,
                                                           int32_t *__restrict__ expert, int32_t *__restrict__ group,
                                                           int N, int M, float scale, int ntq) {
  constexpr int VE = RouteLds<T, D>::VE;
  constexpr int LSTR = RouteLds<T, D>::LSTR;
  __shared__ __align__(16) T lms[RouteLds<T, D>::BYTES / sizeof(T)];
  const int64_t bh = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int tile = blockIdx.x * 4 + w;
  Frag<T> qf[4][D / 32];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int n = tile * ROUTE_TQ + c * 16 + p;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (tile < ntq && n < N)
        qf[c][ks].load(q + (bh * N + n) * D + ks * 32 + g * 8);
      else
        qf[c][ks].zero();
    }
  }
  const T *lmb = q_lm + bh * (int64_t)M * D;
  TopS<S> top[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) top[c].init();
  for (int l0 = 0; l0 < M; l0 += ROUTE_LB) {
    const int nl = min(ROUTE_LB, M - l0);
    __syncthreads();
    for (int ch = threadIdx.x; ch < ROUTE_LB * (D / VE); ch += BLOCK) {
      const int r = ch / (D / VE), cc = ch % (D / VE);
      uint4 x = make_uint4(0, 0, 0, 0);
      if (r < nl) x = *reinterpret_cast<const uint4 *>(lmb + (int64_t)(l0 + r) * D + cc * VE);
      *reinterpret_cast<uint4 *>(lms + r * LSTR + cc * VE) = x;
    }
    __syncthreads();
    if (tile >= ntq) continue;
    for (int sb = 0; sb < nl; sb += 16) {
      f32x4 acc[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<T> a;
        a.load(lms + (sb + p) * LSTR + ks * 32 + g * 8);
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = mma(a, qf[c][ks], acc[c]);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int lmi = l0 + sb + 4 * g + r;
          float val = acc[c][r] * scale;
          val = val != val ? -INFINITY : val;
          if (lmi < l0 + nl) top[c].insert(val, lmi);
        }
    }
  }
  if (tile >= ntq) return;  // no workgroup barriers below
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int n = tile * ROUTE_TQ + c * 16 + p;
    int h = 0;
#pragma unroll
    for (int j = 0; j < S; ++j) {
      float x;
      int i;
      top[c].head(h, x, i);
      float bx = x;
      int bi = i;
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float ox = __shfl_xor(bx, o);
        const int oi = __shfl_xor(bi, o);
        if (ox > bx || (ox == bx && oi < bi)) {
          bx = ox;
          bi = oi;
        }
      }
      h += i == bi ? 1 : 0;
      if (g == 0 && n < N) {
        const int64_t at = (bh * N + n) * S + j;
        expert[at] = bi;
        group[at] = j == 0 ? bi : M + bi;
      }
    }
  }
}

// Per-tile group counts of the routing items (one wave per 64-item tile):
// tile_cnt[tile][g] and the per-group totals (zeroed beforehand).
// cnt: 4 G words of LDS.
__global__ __launch_bounds__(256) void pair_count_kernel(const int32_t *__restrict__ group,
                                                         int32_t *__restrict__ tile_cnt,
                                                         int32_t *__restrict__ counts, int NP, int G, int ntiles) {
  extern __shared__ uint32_t cnt[];
  const int64_t bh = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + w;
  uint32_t *wc = cnt + w * G;
  for (int i = lane; i < G; i += 64) wc[i] = 0u;
  __syncthreads();
  const int item = tile * ROUTE_TQ + lane;
  if (tile < ntiles && item < NP) atomicAdd(&wc[group[bh * NP + item]], 1u);
  __syncthreads();
  if (tile >= ntiles) return;
  int32_t *tc = tile_cnt + (bh * ntiles + tile) * (int64_t)G;
  for (int i = lane; i < G; i += 64) {
    const uint32_t x = wc[i];
    tc[i] = (int32_t)x;
    if (x) atomicAdd(&counts[bh * G + i], (int32_t)x);
  }
}

// Block-wide exclusive scan of one value per thread (NT threads); returns the
// exclusive prefix, *total gets the sum.
template <int NT> __device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t *wsum, uint32_t *total) {
  constexpr int NW = NT / 64;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t incl = wave_inclusive_scan(x);
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t s = wsum[i];
    before += i < w ? s : 0u;
    all += s;
  }
  __syncthreads();
  *total = all;
  return before + incl - x;
}

// Block-wide sum of one value per thread (256 threads).
__device__ __forceinline__ uint32_t block_sum256(uint32_t x, uint32_t *wsum) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  x = wave_sum_u32(x);
  if (lane == 0) wsum[w] = x;
  __syncthreads();
  const uint32_t t = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  return t;
}

// Offsets and scatter bases (Algorithm 1 BinCount of the argmax and CumSum).
// One workgroup per (b*h, block of SCAN_EB experts): offsets[e] = sum of the
// sizes of experts before e, the attention work list tile_start[e] = sum of
// ceil(size / 64) before e, and tile_base[tile][e] = offsets[e] + the queries
// of expert e in earlier routing tiles (an exclusive scan over tiles). 256
// tiles at a time are staged in LDS as [tile][expert] (each thread reads its
// tile's SCAN_EB consecutive counts); wave w then scans experts 4w .. 4w+3,
// lane l taking tiles 4l .. 4l+3, and the bases go back through LDS so each
// thread writes its tile's row.
constexpr int SCAN_EB = 16;

struct ScanLds {
  uint32_t cnt[256][SCAN_EB + 1];
  uint32_t wsum[2][4];
  uint32_t eoff[SCAN_EB];
};

// Workgroup (bx, by) of the scan grid (ceil(M / SCAN_EB), BH).
__device__ __forceinline__ void route_scan_body(ScanLds &sh, int bx, int by, const int32_t *__restrict__ tile_cnt,
                                                const int32_t *__restrict__ counts, int32_t *__restrict__ tile_base,
                                                int32_t *__restrict__ offsets, int32_t *__restrict__ tile_start,
                                                int ntiles, int M, int N) {
  auto &cnt = sh.cnt;
  auto &wsum = sh.wsum;
  auto &eoff = sh.eoff;
  const int e0 = bx * SCAN_EB;
  const int ne = min(SCAN_EB, M - e0);
  const int64_t bh = by;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int32_t *cn = counts + bh * M;

  // exclusive prefixes of the expert sizes (and of their tile counts) at e0 .. e0+ne-1
  uint32_t a = 0, t = 0;
  for (int i = tid; i < e0; i += 256) {
    const uint32_t c = (uint32_t)cn[i];
    a += c;
    t += (c + ATT_TQ - 1) / ATT_TQ;
  }
  uint32_t off = block_sum256(a, wsum[0]);
  uint32_t ts = block_sum256(t, wsum[1]);
  if (tid == 0) {
    for (int j = 0; j < ne; ++j) {
      const uint32_t c = (uint32_t)cn[e0 + j];
      eoff[j] = off;
      offsets[bh * (M + 1) + e0 + j] = (int32_t)off;
      tile_start[bh * (M + 1) + e0 + j] = (int32_t)ts;
      off += c;
      ts += (c + ATT_TQ - 1) / ATT_TQ;
    }
    if (e0 + ne == M) {
      offsets[bh * (M + 1) + M] = (int32_t)off;
      tile_start[bh * (M + 1) + M] = (int32_t)ts;
    }
  }
  __syncthreads();
  // running totals of wave w's experts 4w .. 4w+3 over the tiles done so far
  uint32_t carry[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) carry[q] = 4 * w + q < ne ? eoff[4 * w + q] : 0u;
  const int32_t *tc = tile_cnt + bh * ntiles * (int64_t)M + e0;
  int32_t *tb = tile_base + bh * ntiles * (int64_t)M + e0;
  for (int t0 = 0; t0 < ntiles; t0 += 256) {
    const int tt = t0 + tid;
    // all SCAN_EB loads issued before any is used: addresses clamped into the
    // tile row's expert block (always valid), values masked afterwards
    const int64_t trow = (int64_t)(tt < ntiles ? tt : 0) * M;
    uint32_t c[SCAN_EB];
#pragma unroll
    for (int j = 0; j < SCAN_EB; ++j) c[j] = (uint32_t)tc[trow + min(j, ne - 1)];
#pragma unroll
    for (int j = 0; j < SCAN_EB; ++j) cnt[tid][j] = tt < ntiles && j < ne ? c[j] : 0u;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = 4 * w + q;
      uint32_t v[4], part = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[i] = cnt[4 * lane + i][j];
        part += v[i];
      }
      const uint32_t incl = wave_inclusive_scan(part);
      uint32_t run = carry[q] + incl - part;
      carry[q] += (uint32_t)__shfl((int)incl, 63);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t c = v[i];
        v[i] = run;
        run += c;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) cnt[4 * lane + i][j] = v[i];  // only this wave touches column j
    }
    __syncthreads();
    if (tt < ntiles)
      for (int j = 0; j < ne; ++j) tb[(int64_t)tt * M + j] = (int32_t)cnt[tid][j];
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void route_scan_kernel(const int32_t *__restrict__ tile_cnt,
                                                         const int32_t *__restrict__ counts,
                                                         int32_t *__restrict__ tile_base,
                                                         int32_t *__restrict__ offsets,
                                                         int32_t *__restrict__ tile_start, int ntiles, int M,
                                                         int N) {
  __shared__ ScanLds sh;
  route_scan_body(sh, (int)blockIdx.x, (int)blockIdx.y, tile_cnt, counts, tile_base, offsets, tile_start, ntiles, M,
                  N);
}

// Stable grouping (Algorithm 1 ArgSort of the argmax): within a 64-query tile
// (one wave), a query's rank among earlier queries of the same expert comes
// from matching expert ids bit by bit with ballots.
__device__ __forceinline__ void route_scatter_body(int bx, int by, const int32_t *__restrict__ expert,
                                                   const int32_t *__restrict__ tile_base, int32_t *__restrict__ perm,
                                                   int N, int M, int ntiles, int ebits) {
  const int64_t bh = by;
  const int tile = bx * 4 + (threadIdx.x >> 6);
  if (tile >= ntiles) return;
  const int n = tile * ROUTE_TQ + (threadIdx.x & 63);
  const bool valid = n < N;
  const int e = valid ? expert[bh * N + n] : 0;
  uint64_t same = __ballot(valid);
  for (int b = 0; b < ebits; ++b) {
    const bool bit = (e >> b) & 1;
    const uint64_t ones = __ballot(bit);
    same &= bit ? ones : ~ones;
  }
  if (valid) {
    const int pos = tile_base[(bh * ntiles + tile) * (int64_t)M + e] + (int)lanes_below(same);
    perm[bh * N + pos] = n;
  }
}

constexpr int SCATTER_TPW = 4;  // 64-query tiles per wave of the forward's scatter

// Grouping without a stable order inside an expert (the forward's own
// routing: the attention gives each query the same result whatever its
// position in the grouping, so any order within an expert gives the same
// output). Workgroup (bx, by) of the scatter grid: the head's expert sizes
// become offsets (a block scan every workgroup of the head does for itself,
// into LDS; workgroup 0 of the head also writes offsets and the attention
// work list tile_start); each wave takes, per 64-query tile and expert among
// the tile's queries, one block of positions with one atomic add on that
// expert's cursor (zeroed by the pooling) and places the queries there in
// lane order. A workgroup covers 4 * SCATTER_TPW tiles.
// pre: M + 1 words of LDS, wsum: 4 words.
__device__ __forceinline__ void route_scatter_place_body(uint32_t *pre, uint32_t *wsum, int bx, int by,
                                                         const int32_t *__restrict__ expert,
                                                         const int32_t *__restrict__ counts,
                                                         int32_t *__restrict__ cursor, int32_t *__restrict__ perm,
                                                         int32_t *__restrict__ offsets,
                                                         int32_t *__restrict__ tile_start, int N, int M, int ntiles,
                                                         int ebits) {
  constexpr int EPT = (1024 + 255) / 256;  // experts per thread (M <= 1024)
  const int64_t bh = by;
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave's queries (SCATTER_TPW tiles of 64) and their experts first:
  // the blocks of positions are taken (one atomic add per expert among a
  // tile's 64) while the sizes are scanned, so the two latencies overlap
  int ej[SCATTER_TPW], rel[SCATTER_TPW], leader[SCATTER_TPW], nj[SCATTER_TPW];
  bool vj[SCATTER_TPW];
  uint64_t same[SCATTER_TPW];
#pragma unroll
  for (int j = 0; j < SCATTER_TPW; ++j) {
    const int tile = (bx * SCATTER_TPW + j) * 4 + (tid >> 6);
    nj[j] = tile * ROUTE_TQ + lane;
    vj[j] = tile < ntiles && nj[j] < N;
    ej[j] = vj[j] ? expert[bh * N + nj[j]] : 0;
  }
  uint32_t sz[EPT], a = 0, t = 0;
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int x = tid * EPT + u;
    sz[u] = x < M ? (uint32_t)counts[bh * M + x] : 0u;
  }
#pragma unroll
  for (int j = 0; j < SCATTER_TPW; ++j) {
    uint64_t sm = __ballot(vj[j]);
    for (int b = 0; b < ebits; ++b) {
      const bool bit = (ej[j] >> b) & 1;
      const uint64_t ones = __ballot(bit);
      sm &= bit ? ones : ~ones;
    }
    same[j] = sm;
    leader[j] = vj[j] ? __ffsll((unsigned long long)sm) - 1 : lane;
    rel[j] = 0;
    if (vj[j] && lane == leader[j]) rel[j] = atomicAdd(&cursor[bh * M + ej[j]], __popcll(sm));
  }
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    a += sz[u];
    t += (sz[u] + ATT_TQ - 1) / ATT_TQ;
  }
  uint32_t atot, ttot;
  uint32_t off = block_exclusive_scan<256>(a, wsum, &atot);
  uint32_t ts = bx == 0 ? block_exclusive_scan<256>(t, wsum, &ttot) : 0u;  // uniform for the workgroup
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int x = tid * EPT + u;
    if (x < M) {
      pre[x] = off;
      if (bx == 0) {
        offsets[bh * (M + 1) + x] = (int32_t)off;
        tile_start[bh * (M + 1) + x] = (int32_t)ts;
      }
    }
    off += sz[u];
    ts += (sz[u] + ATT_TQ - 1) / ATT_TQ;
  }
  if (bx == 0 && tid == 0) {
    offsets[bh * (M + 1) + M] = (int32_t)atot;
    tile_start[bh * (M + 1) + M] = (int32_t)ttot;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < SCATTER_TPW; ++j) {
    int base = (vj[j] && lane == leader[j]) ? (int)pre[ej[j]] + rel[j] : 0;
    base = __shfl(base, leader[j]);
    if (vj[j]) perm[bh * N + base + (int)lanes_below(same[j])] = nj[j];
  }
}

__global__ __launch_bounds__(256) void route_scatter_kernel(const int32_t *__restrict__ expert,
                                                            const int32_t *__restrict__ tile_base,
                                                            int32_t *__restrict__ perm, int N, int M, int ntiles,
                                                            int ebits) {
  route_scatter_body((int)blockIdx.x, (int)blockIdx.y, expert, tile_base, perm, N, M, ntiles, ebits);
}

// ---------------------------------------------------------------------------
// The finish of the fused selection and the routing, which do not depend on
// each other, share launches, so that the latency-bound selection work and
// the routing work fill one another's idle time and the fallback steps (which
// normally have nothing to do) cost no launch of their own:
//   finalize_logits_kernel: selection finalize rows | routing logits;
//   topk_scatter_kernel:    fallback rows (scored in full, then their top-k)
//                           | routing placement and scatter.
// Here the queries of an expert are grouped without a stable order (see
// route_scatter_place_body); mita_route keeps the stable grouping.
// The routing part's 2-D grid is flattened (x fastest). LDS is one buffer
// that either part lays out for itself.
// ---------------------------------------------------------------------------
// WAVE: finish rows by finalize_row_wave, four per workgroup.
template <typename T, int D, int CAP, bool MERGE, bool WAVE> struct FinalizeLogitsLds {
  static constexpr int F = WAVE ? 4 * (int)sizeof(FinalizeWaveLds) : (int)sizeof(FinalizeLds<T, D, CAP, MERGE>);
  static constexpr int BYTES = F > RouteLds<T, D>::BYTES ? F : RouteLds<T, D>::BYTES;
};

// Finalize rows and routing workgroups interleave one to one while both last,
// so the two kinds run side by side.
template <typename T, int D, int CAP, bool MERGE, bool WAVE>
__global__ __launch_bounds__(BLOCK) void finalize_logits_kernel(
    const uint2 *__restrict__ cand, const uint32_t *__restrict__ ccnt, int32_t *__restrict__ idx,
    uint32_t *__restrict__ fail_cnt, int32_t *__restrict__ fail_list, int k, int cap, int nch,
    const float2 *__restrict__ part_ml, const float *__restrict__ part_o, T *__restrict__ v_lm, int nF,
    const T *__restrict__ q, const T *__restrict__ q_lm, int32_t *__restrict__ expert, int32_t *__restrict__ tile_cnt,
    int32_t *__restrict__ counts, int N, int M, float scale, int ntiles, int route_x, int nR, int64_t nrows) {
  __shared__ __align__(16) char buf[FinalizeLogitsLds<T, D, CAP, MERGE, WAVE>::BYTES];
  extern __shared__ uint32_t cnt[];  // routing: [4][M]
  const int b = (int)blockIdx.x, lo = min(nF, nR);
  bool fin;
  int i;
  if (b < 2 * lo) {
    fin = (b & 1) == 0;
    i = b >> 1;
  } else {
    fin = nF > nR;
    i = b - lo;
  }
  if (fin) {
    if constexpr (WAVE) {
      const int w = (int)threadIdx.x >> 6;
      const int64_t row = (int64_t)i * 4 + w;
      if (row < nrows)  // the whole wave
        finalize_row_wave<T, D, MERGE>(reinterpret_cast<FinalizeWaveLds *>(buf)[w], row, cand, ccnt, idx, fail_cnt,
                                       fail_list, k, cap, nch, part_ml, part_o, v_lm, M, scale);
    } else {
      finalize_row<T, D, CAP, MERGE>(*reinterpret_cast<FinalizeLds<T, D, CAP, MERGE> *>(buf), i, cand, ccnt, idx,
                                     fail_cnt, fail_list, k, cap, nch, part_ml, part_o, v_lm, M, scale);
    }
    return;
  }
  route_logits_body<T, D, false>(reinterpret_cast<T *>(buf), cnt, i % route_x, i / route_x, q, q_lm, expert, tile_cnt, counts,
                          N, M, scale, ntiles);
}

// ---------------------------------------------------------------------------
// bf16: the sampled scores and pivots and the routing logits (independent of
// each other) share one launch of 16-wave workgroups: the few sample
// workgroups are latency-bound and leave CUs idle, which the routing
// workgroups (sixteen 64-query tiles each) fill. Workgroups [0, nSp) take
// the nS sample slots (x fastest, spread over the XCDs by xcd_slot so that a
// head's blocks share an L2; slots past nS exit), the rest the routing grid;
// LDS is one buffer that either part lays out for itself.
// ---------------------------------------------------------------------------
template <typename T, int D> struct SampleLogitsLds {
  static constexpr int A = 16 * SP_PITCH * (int)sizeof(uint32_t);
  static constexpr int BYTES = A > RouteLds<T, D>::BYTES ? A : RouteLds<T, D>::BYTES;
};

template <typename T, int D>
__global__ __launch_bounds__(1024) void sample_logits_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                             uint32_t *__restrict__ plo,
                                                             uint32_t *__restrict__ fail_cnt, int ns, int r,
                                                             int sample_x, int nS, int nSp, const T *__restrict__ q,
                                                             int32_t *__restrict__ expert,
                                                             int32_t *__restrict__ counts, int N, int M, float scale,
                                                             int ntiles, int route_x) {
  __shared__ __align__(16) char buf[SampleLogitsLds<T, D>::BYTES];
  extern __shared__ uint32_t cnt[];  // routing: [16][M]
  const int b = (int)blockIdx.x;
  if (b < nSp) {  // nSp = nS rounded up to whole XCD ranges (xcd_slot)
    const int f = xcd_slot(b, nSp / NXCD);
    if (f >= nS) return;
    sample_pivot_body<T, D, 16>(reinterpret_cast<uint32_t(*)[SP_PITCH]>(buf), f % sample_x, f / sample_x, q_lm, k,
                                plo, fail_cnt, N, M, ns, r, scale);
    return;
  }
  const int i = b - nSp;
  route_logits_body<T, D, false, 16>(reinterpret_cast<T *>(buf), cnt, i % route_x, i / route_x, q, q_lm, expert,
                                     nullptr, counts, N, M, scale, ntiles);
}

// Workgroups [0, nT) take the fallback rows: each scores its rows in full
// with the score pass's own arithmetic (one key chunk at a time), then
// selects their top-k from those rows (the barrier between orders the stores
// before the reads: the waves of a workgroup share one L1); the rest scatter.
template <typename T, int D, int CAP, bool VEC> struct TopkScatterLds {
  static constexpr int A = (int)sizeof(TopkSmem<CAP>);
  static constexpr int B = 2 * TileDims<T, D>::K_ELEMS * (int)sizeof(T);  // two K tiles
  static constexpr int BYTES = A > B ? A : B;
};

template <typename T, int D, int CAP, bool VEC>
__global__ __launch_bounds__(256) void topk_scatter_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                           float *__restrict__ S, float scale, int nchunks,
                                                           int32_t *__restrict__ idx, int kk,
                                                           const uint32_t *__restrict__ nrows,
                                                           const int32_t *__restrict__ rows, int nT,
                                                           const int32_t *__restrict__ expert,
                                                           const int32_t *__restrict__ counts,
                                                           int32_t *__restrict__ cursor, int32_t *__restrict__ perm,
                                                           int32_t *__restrict__ offsets,
                                                           int32_t *__restrict__ tile_start, int N, int M, int ntiles,
                                                           int ebits, int scat_x) {
  __shared__ __align__(16) char buf[TopkScatterLds<T, D, CAP, VEC>::BYTES];
  const int b = (int)blockIdx.x;
  if (b < nT) {
    const uint32_t nr = *nrows;
    const SelectArgs none{nullptr, nullptr, nullptr};
    for (uint32_t f = (uint32_t)b; f < nr; f += (uint32_t)nT) {
      const int row = rows[f];
      const int lm = row % M;
      for (int chunk = 0; chunk < nchunks; ++chunk) {
        __syncthreads();  // the previous use of the LDS is done
        score_chunk<T, D, true, false, false>(reinterpret_cast<T *>(buf), nullptr, q_lm, k, nullptr, S, nullptr,
                                              nullptr, none, N, M, scale, chunk, nchunks, lm / 64, row / M, lm);
      }
      __syncthreads();  // the row's scores are stored and visible to the workgroup
      topk_row<CAP, VEC, 0>(*reinterpret_cast<TopkSmem<CAP> *>(buf), nullptr, S + (int64_t)row * N,
                            idx + (int64_t)row * kk, N, kk);
    }
    return;
  }
  const int rb = b - nT;
  uint32_t *pre = reinterpret_cast<uint32_t *>(buf);
  __shared__ uint32_t wsum[4];
  route_scatter_place_body(pre, wsum, rb % scat_x, rb / scat_x, expert, counts, cursor, perm, offsets, tile_start,
                           N, M, ntiles, ebits);
}

// Attention work list: tile_start[e] = sum over e' < e of ceil(size(e') / 64),
// tile_start[G] = total tiles, for G <= 2048 groups. 1024 threads, two
// consecutive groups each.
__global__ __launch_bounds__(1024) void worklist_kernel(const int32_t *__restrict__ offsets,
                                                        int32_t *__restrict__ tile_start, int G) {
  __shared__ uint32_t wsum[16];
  const int64_t bh = blockIdx.x;
  const int e0 = 2 * threadIdx.x;
  const int32_t *of = offsets + bh * (G + 1);
  uint32_t nt[2] = {0u, 0u};
#pragma unroll
  for (int u = 0; u < 2; ++u)
    if (e0 + u < G) nt[u] = (uint32_t)((of[e0 + u + 1] - of[e0 + u] + ATT_TQ - 1) / ATT_TQ);
  uint32_t all;
  const uint32_t before = block_exclusive_scan<1024>(nt[0] + nt[1], wsum, &all);
  int32_t *ts = tile_start + bh * (G + 1);
  if (e0 < G) ts[e0] = (int32_t)before;
  if (e0 + 1 < G) ts[e0 + 1] = (int32_t)(before + nt[0]);
  if (threadIdx.x == 0) ts[G] = (int32_t)all;
}

// ---------------------------------------------------------------------------
// MiTA attention (Eq. mita with s = 1): each query attends, in one online
// softmax, over the shared expert (keys q_lm, values v_lm; Eq. shared-expert)
// and the k keys of its routed expert (Eq. mita-expert). Workgroup = 64
// queries of one expert, taken from the routing work list (Algorithm 1's
// varlen grouping); outputs are scattered back to token order. Wave w owns
// queries 32 (w / 2) .. + 31 and the key half w % 2 of every 64-key tile, so
// each wave reads half of each staged tile; the two waves of a query half
// merge their partial softmax states through LDS at the end (log-sum-exp),
// each finishing one of the two 16-query groups. Tiles are staged through
// registers; this kernel serves fp32 inputs, and bf16 ones whose key row list
// is too long for LDS (bf16 with the list in LDS goes to attend16_kernel).
// With ROUTED, routed keys come from the expert tiles, or straight from the
// K/V rows listed in idx (FUSED: the gather of Eq. gather done in place; with
// IDX_LDS the expert's index list is staged in LDS first).
// The softmax is order-independent, so the full 64-key tiles (shared, then
// routed) run first in a software-pipelined loop: tiles double-buffered in
// LDS, the next tile's loads in flight while the current one is multiplied,
// one barrier per tile, no masking. The partial tiles of either expert (when
// M or k is not a multiple of 64) follow, masked.
// Work-list tiles are spread over the XCDs (attend_queries, worklist.hpp).
// ---------------------------------------------------------------------------

// Static LDS of the attention kernels (their double-buffered tiles); the key
// row list comes on top as dynamic LDS when it is staged there.
template <typename T, int D> constexpr size_t attend_tiles_lds() {
  return 2 * (size_t)(TileDims<T, D>::K_ELEMS + TileDims<T, D>::V_ELEMS) * sizeof(T);
}
template <int D> constexpr size_t attend16_tiles_lds() { return 4 * (size_t)DmaTile<D, 32>::BYTES; }
// query groups per wave of attend16_kernel
template <int D> constexpr int ATT16_GROUPS = D == 64 ? 2 : 1;


template <typename T, int D, bool SHARED, bool ROUTED, bool FUSED, bool IDX_LDS, bool MULTI>
__global__ __launch_bounds__(BLOCK) void attend_kernel(const T *__restrict__ q, const T *__restrict__ q_lm,
                                                       const T *__restrict__ v_lm, const T *__restrict__ rk,
                                                       const T *__restrict__ rv, const int32_t *__restrict__ idx,
                                                       const int32_t *__restrict__ perm,
                                                       const int32_t *__restrict__ offsets,
                                                       const int32_t *__restrict__ tile_start, T *__restrict__ o,
                                                       int N, int M, int k, float scale, int s,
                                                       float *__restrict__ pair_o, float *__restrict__ pair_lse) {
  using TD = TileDims<T, D>;
  // tiles staged through registers (K row-major, V transposed, padded rows)
  constexpr int KBYTES = TD::K_ELEMS * (int)sizeof(T);
  constexpr int TBYTES = (int)attend_tiles_lds<T, D>() / 2;
  static_assert(TBYTES == KBYTES + TD::V_ELEMS * (int)sizeof(T), "one K tile and one V^T tile per buffer");
  __shared__ __align__(16) char tiles0[TBYTES];
  __shared__ __align__(16) char tiles1[TBYTES];
  auto Ks = [&](int b) { return reinterpret_cast<T *>(b ? tiles1 : tiles0); };
  auto Vt = [&](int b) { return reinterpret_cast<T *>((b ? tiles1 : tiles0) + KBYTES); };
  extern __shared__ uint32_t sidx[];  // with IDX_LDS: byte offsets of the M + k key rows
  int64_t bh = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;

  int e = 0, q_begin, q_end;
  if (!attend_queries<ROUTED>(tile_start, offsets, bh, N, MULTI ? 2 * M : M, e, q_begin, q_end)) return;  // uniform
  // MULTI (s > 1): the items are (query, rank) pairs; group e < M holds rank-1
  // pairs of expert e (these also take the shared expert), group M + e the
  // other pairs of expert e
  const bool with_sh = SHARED && (!MULTI || e < M);
  if (MULTI && e >= M) e -= M;
  const int NP = MULTI ? N * s : N;

  // full tiles: nA shared, then nB routed; partial ones: pA shared rows, pB routed rows
  const int nA = with_sh ? M / TK : 0, pA = with_sh ? M % TK : 0;
  const int nB = ROUTED ? k / TK : 0, pB = ROUTED ? k % TK : 0;
  const int nfull = nA + nB;
  const T *sh_k = q_lm + bh * (int64_t)M * D, *sh_v = v_lm + bh * (int64_t)M * D;
  const T *rkb, *rvb;
  const int32_t *gidx = nullptr;
  if (FUSED) {
    rkb = rk + bh * (int64_t)N * D;
    rvb = rv + bh * (int64_t)N * D;
    gidx = idx + (bh * M + e) * (int64_t)k;
  } else {
    rkb = rk + (bh * M + e) * (int64_t)k * D;
    rvb = rv + (bh * M + e) * (int64_t)k * D;
  }
  // With IDX_LDS, one row list in LDS covers every key: entries [0, M) are
  // the shared rows (identity), entries [M, M + k) the routed rows (the
  // expert's index list, or identity into its tile), each as the byte offset
  // of the row. Every tile then loads through the same code, its base pointer
  // picked by a scalar select and each row addressed by a 32-bit offset.
  const uint32_t *rows = nullptr;
  constexpr uint32_t ROWB = D * sizeof(T);
  if (IDX_LDS) {
    const int nsh = with_sh ? M : 0;
    for (int i = threadIdx.x; i < nsh; i += BLOCK) sidx[i] = (uint32_t)i * ROWB;
    if (ROUTED)
      for (int i = threadIdx.x; i < k; i += BLOCK) sidx[nsh + i] = (uint32_t)(FUSED ? gidx[i] : i) * ROWB;
    __syncthreads();
    rows = sidx;
  }
  const int rbase = with_sh ? M : 0;  // list offset of the routed rows
  auto tile_base = [&](int i, const T *&kb, const T *&vb, int &off) {
    const bool sh = i < nA;
    kb = sh ? sh_k : rkb;
    vb = sh ? sh_v : rvb;
    off = sh ? i * TK : rbase + (i - nA) * TK;
  };

  const int qh = w >> 1, kh = w & 1;  // query half, key half
  // a wave whose 32 queries all lie past the tile's end (the last tile of an
  // expert is usually partial) still stages tiles and meets the barriers but
  // skips the arithmetic
  const bool wave_busy = q_begin + qh * 32 < q_end;
  bool qvalid[2];
  int token[2], item[2];
  Frag<T> qf[2][D / 32];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int qi = q_begin + qh * 32 + c * 16 + p;
    qvalid[c] = qi < q_end;
    item[c] = qvalid[c] ? (ROUTED ? perm[bh * NP + qi] : qi) : 0;
    token[c] = MULTI ? item[c] / s : item[c];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (qvalid[c])
        qf[c][ks].load(q + (bh * N + token[c]) * D + ks * 32 + g * 8);
      else
        qf[c][ks].zero();
    }
  }
  const float sl2 = scale * LOG2E;
  wait_loads();  // the query fragments are in registers before the pipelined loop
  Online2<D> st;
  st.init();

  TileRegs<T, D> Ra;
  if (IDX_LDS) {
    // one tile ahead: tile i + 1 is loaded into registers while tile i is
    // multiplied, then stored to the other LDS buffer; the loop is unrolled
    // by two so that both buffers have fixed LDS addresses
    const T *kb, *vb;
    int off;
    auto step = [&](int i, const T *Kc, const T *Vc, T *Kn, T *Vn) {
      const bool more = i + 1 < nfull;
      if (more) {
        tile_base(i + 1, kb, vb, off);
        Ra.load_full_off(kb, vb, rows + off);
      }
      if (wave_busy) half_tile_attend<T, D>(st, Kc, Vc, kh, qf, 32, sl2);
      if (more) Ra.store(Kn, Vn);
      __syncthreads();
    };
    if (nfull > 0) {
      tile_base(0, kb, vb, off);
      Ra.load_full_off(kb, vb, rows + off);
      Ra.store(Ks(0), Vt(0));
    }
    __syncthreads();
    int i = 0;
    for (; i + 1 < nfull; i += 2) {
      step(i, Ks(0), Vt(0), Ks(1), Vt(1));
      step(i + 1, Ks(1), Vt(1), Ks(0), Vt(0));
    }
    if (i < nfull) step(i, Ks(0), Vt(0), Ks(1), Vt(1));
  } else {
    // long index lists stay in memory: one register set, one tile ahead
    for (int i = 0; i < nfull; ++i) {
      if (i == 0) {
        if (i < nA)
          Ra.load_full(sh_k, sh_v, nullptr);
        else
          Ra.load_full(rkb, rvb, FUSED ? gidx : nullptr);
        Ra.store(Ks(0), Vt(0));
        __syncthreads();
      }
      const int buf = i & 1;
      if (i + 1 < nfull) {
        const int j = i + 1;
        if (j < nA)
          Ra.load_full(sh_k + (int64_t)j * TK * D, sh_v + (int64_t)j * TK * D, nullptr);
        else if (FUSED)
          Ra.load_full(rkb, rvb, gidx + (j - nA) * TK);
        else
          Ra.load_full(rkb + (int64_t)(j - nA) * TK * D, rvb + (int64_t)(j - nA) * TK * D, nullptr);
      }
      if (wave_busy) half_tile_attend<T, D>(st, Ks(buf), Vt(buf), kh, qf, 32, sl2);
      if (i + 1 < nfull) Ra.store(Ks(buf ^ 1), Vt(buf ^ 1));
      __syncthreads();
    }
  }
  // partial tiles (masked)
  for (int part = 0; part < 2; ++part) {
    const int nr = part == 0 ? pA : pB;
    if (nr == 0) continue;  // uniform
    if (part == 0) {
      Ra.load(sh_k + (int64_t)nA * TK * D, sh_v + (int64_t)nA * TK * D, nullptr, nr);
    } else if (IDX_LDS) {
      Ra.load_off(rkb, rvb, rows + rbase + nB * TK, nr);
    } else if (FUSED) {
      Ra.load(rkb, rvb, gidx + nB * TK, nr);
    } else {
      Ra.load(rkb + (int64_t)nB * TK * D, rvb + (int64_t)nB * TK * D, nullptr, nr);
    }
    Ra.store(Ks(0), Vt(0));
    __syncthreads();
    const int nh = min(32, nr - 32 * kh);  // keys of this wave's half
    if (wave_busy && nh > 0) half_tile_attend<T, D, true>(st, Ks(0), Vt(0), kh, qf, nh, sl2);
    __syncthreads();
  }

  // merge the two key halves: wave (qh, kh) finishes query group kh and hands
  // group 1 - kh to its partner (qh, 1 - kh) through LDS (the tile buffers
  // are free after the last barrier: o values in one, m and l in the other);
  // a half that saw no key has m = -inf, l = 0
  constexpr int XN = D / 4;  // o values per lane
  static_assert(sizeof(tiles0) >= sizeof(float) * 4 * XN * 64 && sizeof(tiles1) >= sizeof(float) * 4 * 2 * 64,
                "exchange buffers");
  float *xb = reinterpret_cast<float *>(tiles0);
  float *xm = reinterpret_cast<float *>(tiles1);
  // The two key halves are combined in a fixed order (half 0, then half 1)
  // whichever wave does it, so a query's result does not depend on the
  // column group it was given (with fused multiply-adds, a * b + c * d and
  // c * d + a * b can round differently). The key half is a compile-time
  // constant in each branch (it is uniform over the wave), so no selects.
  auto hand_over = [&](auto khc) {
    constexpr int KH = decltype(khc)::value;
    float *mine = xb + w * XN * 64 + lane;
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) mine[(db * 4 + r) * 64] = st.o[1 - KH][db][r];
    xm[w * 128 + lane] = st.mval(1 - KH);
    xm[w * 128 + 64 + lane] = st.l(1 - KH);
  };
  auto finish = [&](auto khc) {
    constexpr int KH = decltype(khc)::value;
    if (!qvalid[KH]) return;
    const float *theirs = xb + (w ^ 1) * XN * 64 + lane;
    const float m_mine = st.mval(KH), m_theirs = xm[(w ^ 1) * 128 + lane];
    const float l_mine = st.l(KH), l_theirs = xm[(w ^ 1) * 128 + 64 + lane];
    const float m0 = KH ? m_theirs : m_mine, m1 = KH ? m_mine : m_theirs;  // halves 0 and 1
    const float mm = fmaxf(m0, m1);
    const float a0 = __builtin_amdgcn_exp2f(m0 - mm), a1 = __builtin_amdgcn_exp2f(m1 - mm);
    // explicit fused multiply-adds: the two branches must round alike
    const float l = __builtin_fmaf(KH ? l_mine : l_theirs, a1, (KH ? l_theirs : l_mine) * a0);
    const float inv = __builtin_amdgcn_rcpf(l);
    const float s0 = a0 * inv, s1 = a1 * inv;
    if constexpr (MULTI) {
      // the pair's normalised partial and its log-sum-exp (log2 units)
      float *prow = pair_o + (bh * NP + item[KH]) * D;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        float vals[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float om = st.o[KH][db][r], ot = theirs[(db * 4 + r) * 64];
          vals[r] = __builtin_fmaf(KH ? om : ot, s1, (KH ? ot : om) * s0);
        }
        *reinterpret_cast<float4 *>(prow + db * 16 + 4 * g) = *reinterpret_cast<const float4 *>(vals);
      }
      if (g == 0) pair_lse[bh * NP + item[KH]] = mm + __log2f(l);
      return;
    }
    T *orow = o + (bh * N + token[KH]) * D;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      T vals[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float om = st.o[KH][db][r], ot = theirs[(db * 4 + r) * 64];
        vals[r] = from_f32<T>(__builtin_fmaf(KH ? om : ot, s1, (KH ? ot : om) * s0));
      }
      T *dst = orow + db * 16 + 4 * g;
      if (sizeof(T) == 2)
        *reinterpret_cast<uint2 *>(dst) = *reinterpret_cast<const uint2 *>(vals);
      else
        *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(vals);
    }
  };
  const bool k1 = __builtin_amdgcn_readfirstlane(kh) != 0;  // uniform over the wave
  if (k1)
    hand_over(std::integral_constant<int, 1>{});
  else
    hand_over(std::integral_constant<int, 0>{});
  __syncthreads();
  if (k1)
    finish(std::integral_constant<int, 1>{});
  else
    finish(std::integral_constant<int, 0>{});
}

// ---------------------------------------------------------------------------
// Attention with whole 16-query groups per wave (bf16, key row list in LDS).
// The workgroup takes the same 64 queries as attend_kernel; each of its
// 4 / NG waves owns NG groups of 16 of them and every key, so nothing is
// merged across waves. The keys come in 32-row tiles (K and V: 8 KB at
// d = 64) by LDS DMA, double buffered with one barrier per tile. Each K / V
// fragment read from LDS serves the wave's NG groups (NG MFMAs): with NG = 2
// the LDS reads per MFMA are half those of NG = 1, and the two groups' MFMA
// chains are independent.
// ---------------------------------------------------------------------------
// d = 64, one group per wave: registers for seven waves per SIMD (seven
// workgroups of 16 + 2.5 KB LDS fit a CU at M + k = 640); two groups per
// wave: four waves per SIMD (eight two-wave workgroups per CU)
#define ATTEND16_OCCUPANCY __attribute__((amdgpu_waves_per_eu(NG == 2 ? 4 : (D == 64 ? 7 : 4))))

template <int D, bool SHARED, bool ROUTED, bool FUSED, bool MULTI, int NG>
__global__ __launch_bounds__(256 / NG) ATTEND16_OCCUPANCY void attend16_kernel(
    const bf16_t *__restrict__ q, const bf16_t *__restrict__ q_lm, const bf16_t *__restrict__ v_lm,
    const bf16_t *__restrict__ rk, const bf16_t *__restrict__ rv, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ perm, const int32_t *__restrict__ offsets, const int32_t *__restrict__ tile_start,
    bf16_t *__restrict__ o, int N, int M, int k, float scale, int s, float *__restrict__ pair_o,
    float *__restrict__ pair_lse) {
  constexpr int NW = 4 / NG;  // waves per workgroup
  constexpr int NT = 64 * NW;
  static_assert(NG * NW == 4 && NG * NW * 16 == ATT_TQ, "64 queries per workgroup");
  using DT = DmaTile<D, TK32, NW>;
  static_assert(attend16_tiles_lds<D>() == 4 * DT::BYTES, "two buffers of one K and one V tile");
  // two separate arrays (see attend_kernel): K then V of one tile each
  __shared__ __align__(16) char tiles0[2 * DT::BYTES];
  __shared__ __align__(16) char tiles1[2 * DT::BYTES];
  auto Ks = [&](int b) { return reinterpret_cast<bf16_t *>(b ? tiles1 : tiles0); };
  auto Vt = [&](int b) { return reinterpret_cast<bf16_t *>((b ? tiles1 : tiles0) + DT::BYTES); };
  extern __shared__ uint32_t sidx[];  // byte offsets of the M + k key rows
  int64_t bh = blockIdx.y;
  // the wave index as a scalar, so that the wave's busy count and the
  // softmax state's flags are scalar too (no exec-masked branches around the
  // tile)
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  int e, q_begin, q_end;
  if (!attend_queries<ROUTED>(tile_start, offsets, bh, N, MULTI ? 2 * M : M, e, q_begin, q_end)) return;  // uniform
  // MULTI (s > 1): (query, rank) pairs; group e < M: rank-1 pairs of expert e
  // (with the shared expert), group M + e: the other pairs of expert e
  const bool with_sh = SHARED && (!MULTI || e < M);
  if (MULTI && e >= M) e -= M;
  const int NP = MULTI ? N * s : N;

  // full 32-row tiles: nA shared, then nB routed; partial ones: pA, pB rows
  const int nA = with_sh ? M / TK32 : 0, pA = with_sh ? M % TK32 : 0;
  const int nB = ROUTED ? k / TK32 : 0, pB = ROUTED ? k % TK32 : 0;
  const int nfull = nA + nB;
  const bf16_t *sh_k = q_lm + bh * (int64_t)M * D, *sh_v = v_lm + bh * (int64_t)M * D;
  const bf16_t *rkb, *rvb;
  const int32_t *gidx = nullptr;
  if (FUSED) {
    rkb = rk + bh * (int64_t)N * D;
    rvb = rv + bh * (int64_t)N * D;
    gidx = idx + (bh * M + e) * (int64_t)k;
  } else {
    rkb = rk + (bh * M + e) * (int64_t)k * D;
    rvb = rv + (bh * M + e) * (int64_t)k * D;
  }
  constexpr uint32_t ROWB = D * sizeof(bf16_t);
  const int nsh = with_sh ? M : 0;
  for (int i = threadIdx.x; i < nsh; i += NT) sidx[i] = (uint32_t)i * ROWB;
  if (ROUTED)
    for (int i = threadIdx.x; i < k; i += NT) sidx[nsh + i] = (uint32_t)(FUSED ? gidx[i] : i) * ROWB;
  __syncthreads();
  const uint32_t *rows = sidx;
  auto tile_base = [&](int i, const bf16_t *&kb, const bf16_t *&vb, int &off) {
    const bool sh = i < nA;
    kb = sh ? sh_k : rkb;
    vb = sh ? sh_v : rvb;
    off = sh ? i * TK32 : nsh + (i - nA) * TK32;
  };

  // this wave's groups: group c holds queries q_begin + 16 (NG w + c) + p;
  // the groups with queries come first (nbusy of them); a wave with none
  // still stages tiles and meets the barriers but skips the arithmetic
  int qi[NG];
  bool qvalid[NG];
  Frag<bf16_t> qf[NG][D / 32];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    qi[c] = q_begin + 16 * (NG * w + c) + p;
    qvalid[c] = qi[c] < q_end;
    const int item = qvalid[c] ? (ROUTED ? perm[bh * NP + qi[c]] : qi[c]) : 0;
    const int token = MULTI ? item / s : item;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (qvalid[c])
        qf[c][ks].load(q + (bh * N + token) * D + ks * 32 + g * 8);
      else
        qf[c][ks].zero();
    }
  }
  int nbusy = 0;
#pragma unroll
  for (int c = 0; c < NG; ++c) nbusy += q_begin + 16 * (NG * w + c) < q_end ? 1 : 0;
  DmaLane<D, TK32, NW> dl;
  dl.init(w, lane);
  const bf16_t *kb, *vb;
  int off;

  // the score MFMAs take q * scale * log2 e (rounded to bf16)
  const float sl2 = scale * LOG2E;
#pragma unroll
  for (int c = 0; c < NG; ++c)
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      float x[8];
      unpack16(qf[c][ks].v, x, (const bf16_t *)nullptr);
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] *= sl2;
      qf[c][ks].from_f32(x);
    }
  Att16Addr<D> ad;
  ad.init();
  Att16<D> st[NG];
  wait_loads();
  __syncthreads();
  // step i: the DMA of tile i + 1 into the other buffer is issued, tile i is
  // multiplied, then the wave waits for its DMA and the workgroup meets.
  // Tile i lives in buffer i & 1; the loop is unrolled by two (fixed buffer
  // addresses). The first tile's column maxima are the references for every
  // later tile: no per-tile check, so the loop carries no branch (a branch
  // that redefines the softmax state makes the compiler move the state
  // between two register sets on every tile). A wave runs the loop of its
  // number of busy groups (none: the same steps without the arithmetic), so
  // no loop branches on it either. If some weight then overflowed (a later
  // score above the first tile's maximum by more than about 2^7 in log2
  // units), the whole workgroup runs its tiles once more with the reference
  // check on every tile.
  auto issue_next = [&](int i, bf16_t *Kn, bf16_t *Vn) {
    if (i + 1 < nfull) {
      tile_base(i + 1, kb, vb, off);
      dma_tile_lane<D, TK32, NW>(Kn, Vn, kb, vb, rows + off, dl);
    }
  };
  // mode 0: no arithmetic; 1: fixed references; 2: reference check per tile;
  // NGB busy groups
  auto run_tiles = [&](auto mode_c, auto ngb_c) {
    constexpr int MODE = decltype(mode_c)::value;
    constexpr int NGB = decltype(ngb_c)::value;
    auto tile = [&](const bf16_t *__restrict__ Kc, const bf16_t *__restrict__ Vc, bool first, int nv, auto masked_c) {
      constexpr bool MK = decltype(masked_c)::value;
      if (MODE == 0 || NGB == 0) return;
      if (first)
        att16_first<D, MK, NGB>(st, Kc, Vc, ad, qf, nv);
      else if (MODE == 1)
        att16_plain<D, MK, NGB>(st, Kc, Vc, ad, qf, nv);
      else
        att16_next<D, MK, NGB>(st, Kc, Vc, ad, qf, nv);
    };
    auto step = [&](int i, const bf16_t *__restrict__ Kc, const bf16_t *__restrict__ Vc, bf16_t *__restrict__ Kn,
                    bf16_t *__restrict__ Vn) {
      issue_next(i, Kn, Vn);
      // the DMA is issued before the tile's arithmetic: the scheduler would
      // otherwise sink it to the end of the step, right before its wait
      __builtin_amdgcn_sched_barrier(0);
      tile(Kc, Vc, false, TK32, std::false_type{});
      wait_loads();
      __syncthreads();
    };
    if (nfull > 0) {
      dma_tile_lane<D, TK32, NW>(Ks(0), Vt(0), nA > 0 ? sh_k : rkb, nA > 0 ? sh_v : rvb,
                                 rows + (nA > 0 ? 0 : nsh), dl);
      wait_loads();
      __syncthreads();
      issue_next(0, Ks(1), Vt(1));
      __builtin_amdgcn_sched_barrier(0);
      tile(Ks(0), Vt(0), true, TK32, std::false_type{});
      wait_loads();
      __syncthreads();
      int i = 1;
      for (; i + 1 < nfull; i += 2) {
        step(i, Ks(1), Vt(1), Ks(0), Vt(0));
        step(i + 1, Ks(0), Vt(0), Ks(1), Vt(1));
      }
      if (i < nfull) step(i, Ks(1), Vt(1), Ks(0), Vt(0));
    }
    // partial tiles (masked)
    for (int part = 0; part < 2; ++part) {
      const int nr = part == 0 ? pA : pB;
      if (nr == 0) continue;  // uniform
      if (part == 0)
        dma_tile<D, false, TK32, NW>(Ks(0), Vt(0), sh_k, sh_v, rows + nA * TK32, nr);
      else
        dma_tile<D, false, TK32, NW>(Ks(0), Vt(0), rkb, rvb, rows + nsh + nB * TK32, nr);
      wait_loads();
      __syncthreads();
      tile(Ks(0), Vt(0), nfull == 0 && (part == 0 || pA == 0), nr, std::true_type{});
      __syncthreads();
    }
  };
  auto run_busy = [&](auto mode_c) {
    if (NG == 2 && nbusy == 2)
      run_tiles(mode_c, std::integral_constant<int, NG>{});
    else if (nbusy >= 1)
      run_tiles(mode_c, std::integral_constant<int, 1>{});
    else
      run_tiles(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});
  };
  run_busy(std::integral_constant<int, 1>{});
  // A query whose weights all stayed finite is written now; if any query of
  // the workgroup overflowed, the workgroup runs its tiles again with the
  // reference check on every tile and those queries are written from that
  // run (each query's result thus depends only on its own column).
  uint32_t *redo = sidx + nsh + (ROUTED ? k : 0);  // one word past the row list
  if (threadIdx.x == 0) *redo = 0u;
  __syncthreads();
  bool done[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    done[c] = true;
    if (c < nbusy) {
      done[c] = att16_finite<D>(st[c]);
      if (__ballot(!done[c]) && lane == 0) atomicOr(redo, 1u);
    }
  }
  auto write_out = [&](int c) {
    const float lsum = att16_sum<D>(st[c]);
    const float inv = __builtin_amdgcn_rcpf(lsum);
    // the token is read again (the barriers in between keep the compiler
    // from reusing the first read), so no address stays live across the
    // tile loop
    const int tok = ROUTED ? perm[bh * NP + qi[c]] : qi[c];
    if constexpr (MULTI) {
      // the pair's normalised partial and its log-sum-exp (log2 units; the
      // scores were pre-scaled by log2 e, the reference is -nm)
      float *prow = pair_o + (bh * NP + tok) * D;
#pragma unroll
      for (int db = 0; db < D / 16; ++db)
        *reinterpret_cast<float4 *>(prow + db * 16 + 4 * g) =
            make_float4(st[c].o[db][0] * inv, st[c].o[db][1] * inv, st[c].o[db][2] * inv, st[c].o[db][3] * inv);
      if (g == 0) pair_lse[bh * NP + tok] = __log2f(lsum) - st[c].nm[0];
      return;
    }
    bf16_t *orow = o + (bh * N + tok) * D;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      bf16_t vals[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) vals[r] = from_f32<bf16_t>(st[c].o[db][r] * inv);
      *reinterpret_cast<uint2 *>(orow + db * 16 + 4 * g) = *reinterpret_cast<const uint2 *>(vals);
    }
  };
#pragma unroll
  for (int c = 0; c < NG; ++c)
    if (qvalid[c] && done[c]) write_out(c);
  __syncthreads();
  if (*redo) {  // uniform for the workgroup
    run_busy(std::integral_constant<int, 2>{});
#pragma unroll
    for (int c = 0; c < NG; ++c)
      if (qvalid[c] && !done[c]) write_out(c);
  }
}

// ---------------------------------------------------------------------------
// s > 1: the s partial results of every query (the rank-1 one including the
// shared expert) merged by their log-sum-exp (Sec. 3.2: expert-wise attention
// combined by online softmax): o = sum_j w_j o_j / sum_j w_j with
// w_j = 2^(lse_j - max_j lse_j), j in rank order. One thread per 4 dims.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void combine_kernel(const float *__restrict__ pair_o,
                                                      const float *__restrict__ pair_lse, T *__restrict__ o,
                                                      int64_t nq, int s) {
  constexpr int C = D / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n = t / C;
  const int c = (int)(t % C);
  if (n >= nq) return;
  float lse[MITA_MAX_S];
  float L = -INFINITY;
#pragma unroll
  for (int j = 0; j < MITA_MAX_S; ++j) {
    lse[j] = j < s ? pair_lse[n * s + j] : -INFINITY;
    L = fmaxf(L, lse[j]);
  }
  float den = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < MITA_MAX_S; ++j) {
    if (j >= s) break;
    const float w = __builtin_amdgcn_exp2f(lse[j] - L);
    const float4 x = *reinterpret_cast<const float4 *>(pair_o + (n * s + j) * D + 4 * c);
    den += w;
    acc[0] = __builtin_fmaf(w, x.x, acc[0]);
    acc[1] = __builtin_fmaf(w, x.y, acc[1]);
    acc[2] = __builtin_fmaf(w, x.z, acc[2]);
    acc[3] = __builtin_fmaf(w, x.w, acc[3]);
  }
  const float inv = 1.f / den;
  T vals[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) vals[r] = from_f32<T>(acc[r] * inv);
  T *dst = o + n * D + 4 * c;
  if (sizeof(T) == 2)
    *reinterpret_cast<uint2 *>(dst) = *reinterpret_cast<const uint2 *>(vals);
  else
    *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(vals);
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t route_t(const mita_cfg_t &c, const void *q, const void *q_lm, int32_t *expert, int32_t *perm,
                          int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base, int32_t *counts,
                          int32_t *tile_start, hipStream_t st) {
  const int nt = route_tiles(c);
  const unsigned bh = (unsigned)BH(c);
  hipLaunchKernelGGL((route_logits_kernel<T, D>), dim3((nt + 3) / 4, bh), dim3(BLOCK), 4 * c.M * sizeof(uint32_t),
                     st, (const T *)q, (const T *)q_lm, expert, tile_cnt, counts, c.N, c.M, eff_scale(c), nt);
  hipError_t err = launched("route_logits_kernel", st);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(route_scan_kernel, dim3((c.M + SCAN_EB - 1) / SCAN_EB, bh), dim3(256), 0, st, tile_cnt, counts,
                     tile_base, offsets, tile_start, nt, c.M, c.N);
  if ((err = launched("route_scan_kernel", st)) != hipSuccess) return err;
  int ebits = 0;
  while ((1 << ebits) < c.M) ++ebits;
  hipLaunchKernelGGL(route_scatter_kernel, dim3((nt + 3) / 4, bh), dim3(256), 0, st, expert, tile_base, perm, c.N,
                     c.M, nt, ebits);
  return launched("route_scatter_kernel", st);
}

// s > 1: top-s logits, per-tile pair counts, then the stable scan and
// scatter of route_t over the N s pairs and 2 M groups.
template <typename T, int D, int S>
static hipError_t route_multi_t(const mita_cfg_t &c, const void *q, const void *q_lm, int32_t *expert, int32_t *group,
                                int32_t *perm, int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base,
                                int32_t *counts, int32_t *tile_start, hipStream_t st) {
  const int G = route_groups(c), NP = route_items(c), nt = route_tiles(c);
  const int ntq = (c.N + ROUTE_TQ - 1) / ROUTE_TQ;
  const unsigned bh = (unsigned)BH(c);
  hipError_t err = launch_zero(counts, (int64_t)bh * G, st);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((route_tops_kernel<T, D, S>), dim3((ntq + 3) / 4, bh), dim3(BLOCK), 0, st, (const T *)q,
                     (const T *)q_lm, expert, group, c.N, c.M, eff_scale(c), ntq);
  if ((err = launched("route_tops_kernel", st)) != hipSuccess) return err;
  hipLaunchKernelGGL(pair_count_kernel, dim3((nt + 3) / 4, bh), dim3(256), 4 * (size_t)G * sizeof(uint32_t), st, group,
                     tile_cnt, counts, NP, G, nt);
  if ((err = launched("pair_count_kernel", st)) != hipSuccess) return err;
  hipLaunchKernelGGL(route_scan_kernel, dim3((G + SCAN_EB - 1) / SCAN_EB, bh), dim3(256), 0, st, tile_cnt, counts,
                     tile_base, offsets, tile_start, nt, G, NP);
  if ((err = launched("route_scan_kernel", st)) != hipSuccess) return err;
  int ebits = 0;
  while ((1 << ebits) < G) ++ebits;
  hipLaunchKernelGGL(route_scatter_kernel, dim3((nt + 3) / 4, bh), dim3(256), 0, st, group, tile_base, perm, NP, G, nt,
                     ebits);
  return launched("route_scatter_kernel", st);
}

template <typename T, int D>
static hipError_t route_multi_s(const mita_cfg_t &c, const void *q, const void *q_lm, int32_t *expert, int32_t *group,
                                int32_t *perm, int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base,
                                int32_t *counts, int32_t *tile_start, hipStream_t st) {
  static_assert(MITA_MAX_S == 4, "one instance per s");
  switch (c.s) {
    case 2: return route_multi_t<T, D, 2>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
    case 3: return route_multi_t<T, D, 3>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
    default: return route_multi_t<T, D, 4>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
  }
}

hipError_t launch_route(const mita_cfg_t &c, const void *q, const void *q_lm, int32_t *expert, int32_t *perm,
                        int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base, int32_t *counts,
                        int32_t *tile_start, int32_t *group, hipStream_t st) {
  if (multi_route(c)) {
    if (c.dtype == MITA_F32)
      return c.d == 64 ? route_multi_s<float, 64>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st)
                       : route_multi_s<float, 128>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
    return c.d == 64 ? route_multi_s<bf16_t, 64>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st)
                     : route_multi_s<bf16_t, 128>(c, q, q_lm, expert, group, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
  }
  if (c.dtype == MITA_F32)
    return c.d == 64 ? route_t<float, 64>(c, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, st)
                     : route_t<float, 128>(c, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
  return c.d == 64 ? route_t<bf16_t, 64>(c, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, st)
                   : route_t<bf16_t, 128>(c, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, st);
}

template <typename T, int D, int CAP, bool MERGE, bool WAVE>
static hipError_t select_route_t(const mita_cfg_t &c, const void *q, const void *q_lm, const void *k,
                                 const SelectBufs &sb, float *S, int32_t *idx, const void *partial, void *v_lm,
                                 int32_t *expert, int32_t *perm, int32_t *offsets, int32_t *tile_cnt,
                                 int32_t *tile_base, int32_t *counts, int32_t *tile_start, bool logits_done,
                                 hipStream_t st) {
  const int nt = route_tiles(c);
  const int bh = (int)BH(c);
  const int nch = score_chunks(c);
  const int64_t rows = (int64_t)bh * c.M;
  const float2 *ml = (const float2 *)partial;
  const float *po = MERGE ? (const float *)((const char *)partial + align_up((size_t)rows * nch * sizeof(float2)))
                          : nullptr;
  // with the logits formed beside the sampled scores, the finish rows run
  // alone; with the sets written by the pivot launch (direct selection) the
  // routing logits do
  const int route_x = (nt + 3) / 4;
  const int nF = sb.idx ? 0 : (int)(WAVE ? (rows + 3) / 4 : rows), nR = logits_done ? 0 : route_x * bh;
  if (nF + nR == 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL((finalize_logits_kernel<T, D, CAP, MERGE, WAVE>), dim3((unsigned)(nF + nR)), dim3(BLOCK),
                     nR ? 4 * c.M * sizeof(uint32_t) : 0, st, sb.cand, sb.ccnt, idx, sb.fail_cnt, sb.fail_list, c.k, sb.cap,
                     nch, ml, po, (T *)v_lm, nF, (const T *)q, (const T *)q_lm, expert, tile_cnt, counts, c.N, c.M,
                     eff_scale(c), nt, route_x, nR, rows);
  hipError_t err = launched("finalize_logits_kernel", st);
  if (err != hipSuccess) return err;
  // the fallback workgroups of the last launch (listed rows, scored in full and selected)
  // (few: the rows normally all pass and these workgroups exit at once; each
  // takes rows b, b + nT, ... when some do not)
  const int nT = (int)(rows < 64 ? rows : 64);
  int32_t *cursor = tile_base;  // the placement cursors live in the (here unused) tile_base buffer
  const int scat_x = (nt + 4 * SCATTER_TPW - 1) / (4 * SCATTER_TPW);
  const int nS = scat_x * bh;
  int ebits = 0;
  while ((1 << ebits) < c.M) ++ebits;
  constexpr int TCAP = 512;
  if (c.N % 4 == 0)
    hipLaunchKernelGGL((topk_scatter_kernel<T, D, TCAP, true>), dim3((unsigned)(nT + nS)), dim3(256), 0, st,
                       (const T *)q_lm, (const T *)k, S, eff_scale(c), nch, idx, c.k, sb.fail_cnt, sb.fail_list, nT,
                       expert, counts, cursor, perm, offsets, tile_start, c.N, c.M, nt, ebits, scat_x);
  else
    hipLaunchKernelGGL((topk_scatter_kernel<T, D, TCAP, false>), dim3((unsigned)(nT + nS)), dim3(256), 0, st,
                       (const T *)q_lm, (const T *)k, S, eff_scale(c), nch, idx, c.k, sb.fail_cnt, sb.fail_list, nT,
                       expert, counts, cursor, perm, offsets, tile_start, c.N, c.M, nt, ebits, scat_x);
  return launched("topk_scatter_kernel", st);
}

template <typename T, int D>
static hipError_t select_route_n(const mita_cfg_t &c, const void *q, const void *q_lm, const void *k,
                                 const SelectBufs &sb, float *S, int32_t *idx, const void *partial, void *v_lm,
                                 int32_t *expert, int32_t *perm, int32_t *offsets, int32_t *tile_cnt,
                                 int32_t *tile_base, int32_t *counts, int32_t *tile_start, bool logits_done,
                                 hipStream_t st) {
#define MITA_SR(CAP, MG, W)                                                                                      \
  return select_route_t<T, D, CAP, MG, W>(c, q, q_lm, k, sb, S, idx, partial, v_lm, expert, perm, offsets, tile_cnt, \
                                          tile_base, counts, tile_start, logits_done, st)
  // lists of at most SEL_NS entries over at most 64 chunks: one wave per row
  const bool wave = sb.cap <= SEL_NS && score_chunks(c) <= 64;
  if (v_lm) {
    if (wave) MITA_SR(SEL_NS, true, true);
    if (sb.cap <= 1024) MITA_SR(1024, true, false);
    if (sb.cap <= 2048) MITA_SR(2048, true, false);
    if (sb.cap <= 4096) MITA_SR(4096, true, false);
    MITA_SR(SEL_CAP, true, false);
  }
  if (wave) MITA_SR(SEL_NS, false, true);
  if (sb.cap <= 1024) MITA_SR(1024, false, false);
  if (sb.cap <= 2048) MITA_SR(2048, false, false);
  if (sb.cap <= 4096) MITA_SR(4096, false, false);
  MITA_SR(SEL_CAP, false, false);
#undef MITA_SR
}

hipError_t launch_select_route(const mita_cfg_t &c, const void *q, const void *q_lm, const void *k,
                               const SelectBufs &sb, float *S, int32_t *idx, const void *partial, void *v_lm,
                               int32_t *expert, int32_t *perm, int32_t *offsets, int32_t *tile_cnt, int32_t *tile_base,
                               int32_t *counts, int32_t *tile_start, bool logits_done, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? select_route_n<float, 64>(c, q, q_lm, k, sb, S, idx, partial, v_lm, expert, perm, offsets,
                                                 tile_cnt, tile_base, counts, tile_start, logits_done, st)
                     : select_route_n<float, 128>(c, q, q_lm, k, sb, S, idx, partial, v_lm, expert, perm, offsets,
                                                  tile_cnt, tile_base, counts, tile_start, logits_done, st);
  return c.d == 64 ? select_route_n<bf16_t, 64>(c, q, q_lm, k, sb, S, idx, partial, v_lm, expert, perm, offsets,
                                                tile_cnt, tile_base, counts, tile_start, logits_done, st)
                   : select_route_n<bf16_t, 128>(c, q, q_lm, k, sb, S, idx, partial, v_lm, expert, perm, offsets,
                                                 tile_cnt, tile_base, counts, tile_start, logits_done, st);
}

// The routing logits go beside the sampled scores when the selection's
// finish rows hold long lists (cap above 2048 entries: 32 KB and more of LDS
// per row), which would leave the routing workgroups that share their launch
// few slots per CU; with shorter lists the finish launch serves them better
// (at 16K tokens, M = 128, k = 512: 63.9 us against 75.4 for the pivots and
// the finish together).
bool pivots_with_logits(const mita_cfg_t &c, const SelectBufs &sb) {
  return c.dtype == MITA_BF16 && sb.ns <= SEL_NS && sb.cap > 2048;
}

hipError_t launch_pivots_logits(const mita_cfg_t &c, const void *q, const void *q_lm, const void *k,
                                const SelectBufs &sb, int32_t *expert, int32_t *counts, hipStream_t st) {
  if (!pivots_with_logits(c, sb)) return hipErrorInvalidValue;
  const int bh = (int)BH(c);
  const int sample_x = (c.M + 15) / 16, nS = sample_x * bh, nSp = NXCD * ((nS + NXCD - 1) / NXCD);
  const int nt = route_tiles(c), route_x = (nt + 15) / 16, nR = route_x * bh;
  const dim3 grid((unsigned)(nSp + nR));
  const size_t dyn = 16 * (size_t)c.M * sizeof(uint32_t);
  if (c.d == 64)
    hipLaunchKernelGGL((sample_logits_kernel<bf16_t, 64>), grid, dim3(1024), dyn, st, (const bf16_t *)q_lm,
                       (const bf16_t *)k, sb.plo, sb.fail_cnt, sb.ns, sb.rank, sample_x, nS, nSp, (const bf16_t *)q, expert,
                       counts, c.N, c.M, eff_scale(c), nt, route_x);
  else
    hipLaunchKernelGGL((sample_logits_kernel<bf16_t, 128>), grid, dim3(1024), dyn, st, (const bf16_t *)q_lm,
                       (const bf16_t *)k, sb.plo, sb.fail_cnt, sb.ns, sb.rank, sample_x, nS, nSp, (const bf16_t *)q, expert,
                       counts, c.N, c.M, eff_scale(c), nt, route_x);
  return launched("sample_logits_kernel", st);
}

hipError_t launch_worklist(const mita_cfg_t &c, const int32_t *offsets, int32_t *tile_start, hipStream_t st) {
  hipLaunchKernelGGL(worklist_kernel, dim3((unsigned)BH(c)), dim3(1024), 0, st, offsets, tile_start, route_groups(c));
  return launched("worklist_kernel", st);
}

template <typename T, int D, bool SH, bool RT, bool FU, bool MU>
static hipError_t attend_t3(const mita_cfg_t &c, const void *q, const void *q_lm, const void *v_lm, const void *rk,
                            const void *rv, const int32_t *idx, const int32_t *perm, const int32_t *offsets,
                            const int32_t *tile_start, void *o, float *pair_o, float *pair_lse, hipStream_t st) {
  // routed: at most ceil(items / 64) + groups tiles (each group adds at most
  // one partial tile), rounded up to a multiple of the XCD count for the tile
  // spreading
  int tiles = (route_items(c) + ATT_TQ - 1) / ATT_TQ;
  if (RT) tiles = (tiles + route_groups(c) + NXCD - 1) / NXCD * NXCD;
  const dim3 grid((unsigned)tiles, (unsigned)BH(c));
  const int nlist = (SH ? c.M : 0) + (RT ? c.k : 0);
  const int s = route_s(c);
  hipError_t err = hipSuccess;
  bool done = false;
  // the row list is staged in LDS when it and the kernel's tiles fit
  if constexpr (sizeof(T) == 2) {
    // bf16: lists of up to IDX_LDS_MAX - 1 rows (and the kernel's rerun flag)
    // beside the 16 / 32 KB DMA tiles
    if (list_in_lds(nlist + 1, attend16_tiles_lds<D>())) {
      // d = 64: two query groups per wave, two waves; d = 128: one group, four
      constexpr int NG = ATT16_GROUPS<D>;
      hipLaunchKernelGGL((attend16_kernel<D, SH, RT, FU, MU, NG>), grid, dim3(256 / NG),
                         (size_t)(nlist + 1) * sizeof(int32_t),
                         st, (const bf16_t *)q, (const bf16_t *)q_lm, (const bf16_t *)v_lm, (const bf16_t *)rk,
                         (const bf16_t *)rv, idx, perm, offsets, tile_start, (bf16_t *)o, c.N, c.M, c.k, eff_scale(c), s,
                         pair_o, pair_lse);
      err = launched("attend16_kernel", st);
      done = true;
    }
  } else {
    if (list_in_lds(nlist, attend_tiles_lds<T, D>())) {
      hipLaunchKernelGGL((attend_kernel<T, D, SH, RT, FU, true, MU>), grid, dim3(BLOCK), (size_t)nlist * sizeof(int32_t),
                         st, (const T *)q, (const T *)q_lm, (const T *)v_lm, (const T *)rk, (const T *)rv, idx, perm,
                         offsets, tile_start, (T *)o, c.N, c.M, c.k, eff_scale(c), s, pair_o, pair_lse);
      err = launched("attend_kernel", st);
      done = true;
    }
  }
  if (!done) {
    // the row list stays in memory
    hipLaunchKernelGGL((attend_kernel<T, D, SH, RT, FU, false, MU>), grid, dim3(BLOCK), 0, st, (const T *)q,
                       (const T *)q_lm, (const T *)v_lm, (const T *)rk, (const T *)rv, idx, perm, offsets, tile_start,
                       (T *)o, c.N, c.M, c.k, eff_scale(c), s, pair_o, pair_lse);
    err = launched("attend_kernel", st);
  }
  if (!MU || err != hipSuccess) return err;
  const int64_t nq = BH(c) * c.N;
  const int64_t threads = nq * (D / 4);
  hipLaunchKernelGGL((combine_kernel<T, D>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, pair_o,
                     pair_lse, (T *)o, nq, s);
  return launched("combine_kernel", st);
}

template <typename T, int D, bool MU>
static hipError_t attend_m(const mita_cfg_t &c, const void *q, const void *q_lm, const void *v_lm, const void *rk,
                           const void *rv, const int32_t *idx, const int32_t *perm, const int32_t *offsets,
                           const int32_t *tile_start, void *o, float *po, float *pl, hipStream_t st) {
  if (idx) {
    if (c.use_shared) return attend_t3<T, D, true, true, true, MU>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
    return attend_t3<T, D, false, true, true, MU>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
  }
  if (c.use_shared) return attend_t3<T, D, true, true, false, MU>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
  return attend_t3<T, D, false, true, false, MU>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
}

template <typename T, int D>
static hipError_t attend_t(const mita_cfg_t &c, const void *q, const void *q_lm, const void *v_lm, const void *rk,
                           const void *rv, const int32_t *idx, const int32_t *perm, const int32_t *offsets,
                           const int32_t *tile_start, void *o, float *po, float *pl, hipStream_t st) {
  if (!c.use_routed)
    return attend_t3<T, D, true, false, false, false>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
  if (multi_route(c)) return attend_m<T, D, true>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
  return attend_m<T, D, false>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, po, pl, st);
}

hipError_t launch_attend(const mita_cfg_t &c, const void *q, const void *q_lm, const void *v_lm, const void *rk,
                         const void *rv, const int32_t *idx, const int32_t *perm, const int32_t *offsets,
                         const int32_t *tile_start, void *o, float *pair_o, float *pair_lse, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? attend_t<float, 64>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, pair_o, pair_lse, st)
                     : attend_t<float, 128>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, pair_o, pair_lse, st);
  return c.d == 64 ? attend_t<bf16_t, 64>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, pair_o, pair_lse, st)
                   : attend_t<bf16_t, 128>(c, q, q_lm, v_lm, rk, rv, idx, perm, offsets, tile_start, o, pair_o, pair_lse, st);
}

}  // namespace mita
