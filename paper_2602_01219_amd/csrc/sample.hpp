// sample.hpp - the sampled scores and pivots of the fused top-k selection
// (Eq. top-k): each landmark row is scored against ns evenly spaced keys with
// the score pass's tile arithmetic, and its pivot is taken from those
// samples; used by the pivot launch and by the launch that runs it together
// with the routing logits.
#pragma once
#include "cdna4.hpp"
#include "flash.hpp"
#include "check.hpp"

namespace mita {

// Token index of sample j of ns: the middle of the j-th of ns equal parts of
// [0, N). Distinct and below N for ns <= N; equal to j when ns == N.
__device__ __forceinline__ int sample_pos(int j, int N, int ns) {
  return (int)(((2 * (int64_t)j + 1) * N) / (2 * (int64_t)ns));
}

// Bin of a 256-bin histogram (hist[0..255], counted from the top bin down)
// holding the need-th item, for one wave: returns the bin, *above = items in
// higher bins. need must be in [1, total].
__device__ __forceinline__ int wave_find_bin(const uint32_t *hist, uint32_t need, uint32_t *above) {
  const int lane = threadIdx.x & 63;
  uint32_t c[4], sum = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    c[q] = hist[255 - 4 * lane - q];
    sum += c[q];
  }
  const uint32_t incl = wave_inclusive_scan(sum);
  const uint32_t excl = incl - sum;
  int bin = -1;
  uint32_t ab = 0;
  if (excl < need && need <= incl) {
    uint32_t acc = excl;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (bin < 0) {
        if (acc + c[q] >= need)
          bin = 255 - 4 * lane - q;
        else
          acc += c[q];
      }
    }
    ab = acc;
  }
  const uint64_t m = __ballot(bin >= 0);
  const int src = __ffsll((unsigned long long)m) - 1;
  *above = (uint32_t)__shfl((int)ab, src);
  return __shfl(bin, src);
}

// ---------------------------------------------------------------------------
// Pivot of one landmark row from its ns (<= SEL_NS) sampled keys, held by one
// wave: lane l holds keys 4 l + 256 i + (0..3) in v[4 i .. 4 i + 3], 0 marking
// a slot past ns (no score has key 0). The pivot is the exact r-th largest
// sampled key, found in two steps:
//  1. a 256-bin LDS histogram over the VALUE range [fmin, fmax] of the row's
//     samples (bin = floor((x - fmin) * 255.5 / (fmax - fmin)), a
//     non-decreasing function of the key, so every key in a higher bin is
//     larger than every key in a lower one) gives the bin holding the r-th
//     largest and the number of samples above it. Linear bins keep the
//     counts per bin small for bell-shaped scores (bins by key bits would put
//     a third of the samples into the one bin of a binade, and its LDS
//     atomics would serialise);
//  2. that bin's keys (at most 64 of them) are compacted into one register
//     per lane and an MSB-first bisection over the 32 key bits, counting by
//     ballots, finds the exact rank among them.
// Rows whose samples span a non-finite range or crowd more than 64 into the
// bin (clustered scores) take the bisection over all samples instead.
// Uses words 0..383 of the LDS row at `lds`.
// ---------------------------------------------------------------------------
constexpr int PIVOT_PER = SEL_NS / 64;

// need-th largest of the keys x, one per lane (0 = none); 1 <= need <= count
// of nonzero keys. Bit b of the result is set iff at least `need` keys reach
// the result's higher bits with b set.
__device__ __forceinline__ uint32_t wave_kth_key(uint32_t x, uint32_t need) {
  uint32_t t = 0;
#pragma unroll
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    if ((uint32_t)__popcll(__ballot(x >= c)) >= need) t = c;
  }
  return t;
}
// The same over P keys per lane.
template <int P>
__device__ __forceinline__ uint32_t wave_kth_key(const uint32_t (&x)[P], uint32_t need) {
  uint32_t t = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    uint32_t n = 0;
#pragma unroll
    for (int i = 0; i < P; ++i) n += (uint32_t)__popcll(__ballot(x[i] >= c));
    if (n >= need) t = c;
  }
  return t;
}

__device__ __forceinline__ uint32_t pivot_of(const uint32_t (&v)[PIVOT_PER], uint32_t *lds, int r) {
  const int lane = threadIdx.x & 63;
  uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
  for (int i = 0; i < PIVOT_PER; ++i) {
    if (v[i]) mn = min(mn, v[i]);
    mx = max(mx, v[i]);
  }
  const uint32_t kmin = wave_min_u32(mn), kmax = wave_max_u32(mx);
  if (kmin == kmax) return kmin;  // all samples equal
  const float fmin = key_to_float(kmin), span = key_to_float(kmax) - fmin;
  const float inv = 255.5f / span;
  if (!(span < INFINITY) || !(inv < INFINITY)) return wave_kth_key(v, (uint32_t)r);
  // (x - fmin) <= span after rounding, so (x - fmin) * inv < 256: bins 0..255;
  // empty slots go to words 256 + lane (distinct, never read as counts)
  uint32_t bin[PIVOT_PER];
#pragma unroll
  for (int q = 0; q < 4; ++q) lds[lane + 64 * q] = 0u;
#pragma unroll
  for (int i = 0; i < PIVOT_PER; ++i) {
    const uint32_t b = min((uint32_t)((key_to_float(v[i]) - fmin) * inv), 255u);
    bin[i] = v[i] ? b : 256u + (uint32_t)lane;
    atomicAdd(lds + bin[i], 1u);
  }
  uint32_t above;
  const uint32_t b = (uint32_t)wave_find_bin(lds, (uint32_t)r, &above);
  const uint32_t cnt = lds[b];
  if (cnt > 64u) return wave_kth_key(v, (uint32_t)r);
  uint32_t *slot = lds + 320;
  uint32_t base = 0;
#pragma unroll
  for (int i = 0; i < PIVOT_PER; ++i) {
    const uint64_t m = __ballot(bin[i] == b);
    if (bin[i] == b) slot[base + lanes_below(m)] = v[i];
    base += (uint32_t)__popcll(m);
  }
  return wave_kth_key((uint32_t)lane < cnt ? slot[lane] : 0u, (uint32_t)r - above);
}

// ---------------------------------------------------------------------------
// Sampled scores and pivots in one launch. Workgroup = NW waves over 16
// landmark rows of one head (one MFMA column block); wave w scores them
// against the sampled keys [SEL_NS/NW w, SEL_NS/NW (w + 1)) in tiles of 64,
// the A fragments loaded straight from the sampled key rows (tile arithmetic
// as in the score pass, so the same values), keys = score_key(fl(dot) * scale)
// into LDS; then wave w takes the pivots of rows 16/NW w .. 16/NW (w + 1) - 1,
// its histogram and compaction slots in the first 384 words of its own row's
// keys once they are in registers (the wave's LDS accesses are in order). Workgroup (0, 0) also
// zeroes the fallback counter.
// ---------------------------------------------------------------------------
constexpr int SP_PITCH = SEL_NS + 4;  // keys per LDS row: rows start 4 banks apart

// Workgroup (bx, by) of the sample grid (16 landmarks of head by); keys: 16
// LDS rows of SP_PITCH words.
// With idx (only when the sample is the whole row, ns == N, and r == kk)
// the rows' top-kk sets are written too, in ascending token order: every key
// above the pivot and, in token order, as many keys equal to it as the set
// still needs (the order of the top-k: larger score first, lower index first
// among equal scores).
template <typename T, int D, int NW>
__device__ __forceinline__ void sample_pivot_body(uint32_t (*keys)[SP_PITCH], int bx, int by,
                                                  const T *__restrict__ q_lm, const T *__restrict__ k,
                                                  uint32_t *__restrict__ plo, uint32_t *__restrict__ fail_cnt, int N,
                                                  int M, int ns, int r, float scale, int32_t *__restrict__ idx = nullptr,
                                                  int kk = 0) {
  static_assert(16 % NW == 0 && SEL_NS % (NW * TK) == 0, "sample/pivot split");
  constexpr int PERW = SEL_NS / NW;  // samples per wave
  constexpr int RPW = 16 / NW;       // rows per wave
  const int64_t bh = by;
  const int lm0 = bx * 16;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  if (bx == 0 && by == 0 && threadIdx.x == 0) *fail_cnt = 0;
  Frag<T> qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    if (lm0 + p < M)
      qf[ks].load(q_lm + (bh * M + lm0 + p) * D + ks * 32 + g * 8);
    else
      qf[ks].zero();
  }
  const T *kb_ = k + bh * (int64_t)N * D;
  for (int j0 = w * PERW; j0 < min(ns, (w + 1) * PERW); j0 += TK) {
    // the tile's A fragments, all loads issued before the first is used
    Frag<T> a[4][D / 32];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int j = j0 + kb * 16 + p;  // A row p of block kb: sample j
      const int64_t pos = j < ns ? sample_pos(j, N, ns) : 0;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) a[kb][ks].load(kb_ + pos * D + ks * 32 + g * 8);
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) acc = mma(a[kb][ks], qf[ks], acc);
      // lane (g, p) holds samples j0 + 16 kb + 4 g + (0..3) of row p
      const int jb = j0 + kb * 16 + 4 * g;
      uint32_t key[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) key[q] = jb + q < ns ? score_key(acc[q] * scale) : 0u;
      *reinterpret_cast<uint4 *>(&keys[p][jb]) = make_uint4(key[0], key[1], key[2], key[3]);
    }
  }
  // slots past ns stay 0 (below every key) for the selection
  for (int j = ns + (int)threadIdx.x; j < SEL_NS; j += 64 * NW)
#pragma unroll
    for (int row = 0; row < 16; ++row) keys[row][j] = 0u;
  __syncthreads();
  for (int q = 0; q < RPW; ++q) {
    const int rl = RPW * w + q;
    if (lm0 + rl >= M) break;  // uniform for the wave; no workgroup barriers below
    uint32_t v[PIVOT_PER];
#pragma unroll
    for (int i = 0; i < PIVOT_PER / 4; ++i) {
      const uint4 x = *reinterpret_cast<const uint4 *>(&keys[rl][256 * i + 4 * lane]);
      v[4 * i] = x.x;
      v[4 * i + 1] = x.y;
      v[4 * i + 2] = x.z;
      v[4 * i + 3] = x.w;
    }
    const uint32_t lo = pivot_of(v, &keys[rl][0], r);
    if (lane == 0) plo[bh * M + lm0 + rl] = lo;
    if (idx) {
      // the row's keys back in LDS (pivot_of used its first words)
#pragma unroll
      for (int i = 0; i < PIVOT_PER / 4; ++i)
        *reinterpret_cast<uint4 *>(&keys[rl][256 * i + 4 * lane]) = make_uint4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
      uint32_t gt = 0;
#pragma unroll
      for (int i = 0; i < PIVOT_PER; ++i) gt += v[i] > lo ? 1u : 0u;
      const uint32_t need_eq = (uint32_t)kk - wave_sum_u32(gt);  // >= 1: lo is the kk-th largest
      int32_t *out = idx + (bh * M + lm0 + rl) * (int64_t)kk;
      uint32_t taken = 0, eq_seen = 0;
      for (int j0 = 0; j0 < ns; j0 += 64) {
        const int j = j0 + lane;
        const uint32_t key = j < ns ? keys[rl][j] : 0u;  // 0 lies below every key
        const uint64_t be = __ballot(key == lo);
        const bool take = key > lo || (key == lo && eq_seen + lanes_below(be) < need_eq);
        const uint64_t bt = __ballot(take);
        if (take) out[taken + lanes_below(bt)] = j;
        taken += (uint32_t)__popcll(bt);
        eq_seen += (uint32_t)__popcll(be);
      }
    }
  }
}

}  // namespace mita
