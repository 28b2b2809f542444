// select.hip - the top-k selection of the forward (Eq. top-k), fused with the
// landmark-key score pass so that the M x N score matrix is never stored.
//
//   1-2. sample_pivot_kernel: the scores of every landmark against ns evenly
//      spaced keys, as order-preserving keys (the same tile arithmetic as the
//      score pass, so the same values), kept in LDS; per landmark row, the
//      pivot = the r-th largest sampled key. r is chosen on the host so that
//      at least k and far fewer than `cap` tokens of the row score >= pivot,
//      except with negligible probability (r = k exactly when the sample is
//      the whole row).
//   3. the score pass lists every token scoring >= pivot (score bits, token
//      index), in token order, in one region per (row, key chunk).
//   4. finalize_kernel: with k <= count <= cap the list holds the row's whole
//      top-k, since every token left out scores below the pivot, which the
//      k-th listed score reaches. The row's regions are packed into LDS, an
//      exact radix select over the composite (score key, -index) finds the
//      k-th token of the order (larger score first, lower index first among
//      equal scores), and an ordered scan writes the selected indices, which
//      the list already holds in ascending order. A row whose count is out of
//      range goes to a fallback list.
//   5. fallback rows: the score pass recomputes the full score row and the
//      exact top-k kernel selects from it.
// The sets equal those of the exact top-k over the stored score rows.
#include "cdna4.hpp"
#include "flash.hpp"
#include "kernels.hpp"
#include "check.hpp"
#include "finalize.hpp"

namespace mita {

namespace {

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

}  // namespace

// ---------------------------------------------------------------------------
// Pivot of one landmark row from its ns (<= SEL_NS) sampled keys, held by one
// wave: lane l holds keys 4 l + 256 i + (0..3) in v[4 i .. 4 i + 3], 0 marking
// a slot past ns (no score has key 0, so it lies below every range). Radix
// rounds over a 256-bin LDS histogram of the current key range (bins span
// (hi - lo + 1) / 256 keys, so each round shrinks the range by 2^8) narrow
// down on the r-th largest sample; after two rounds the lower edge of the bin
// holding it is taken. That edge is at most the r-th largest sample, so at
// least r samples are >= pivot, and its bin spans at most 2^16 keys (a
// relative step of 2^-7 within one binade), which lists only a few more
// tokens than the exact sample statistic would.
// ---------------------------------------------------------------------------
constexpr int PIVOT_PER = SEL_NS / 64;

static __device__ __forceinline__ uint32_t pivot_of(const uint32_t (&v)[PIVOT_PER], uint32_t *hist, int r) {
  const int lane = threadIdx.x & 63;
  uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
  for (int i = 0; i < PIVOT_PER; ++i) {
    if (v[i]) mn = min(mn, v[i]);
    mx = max(mx, v[i]);
  }
  uint32_t lo = wave_min_u32(mn), hi = wave_max_u32(mx);
  uint32_t need = (uint32_t)r;
  for (int round = 0; round < 2 && lo < hi; ++round) {
    const uint32_t span = hi - lo;
    const int bits = 32 - __clz((int)span);
    const int shift = bits > 8 ? bits - 8 : 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) hist[lane + 64 * q] = 0u;
#pragma unroll
    for (int i = 0; i < PIVOT_PER; ++i)
      if (v[i] >= lo && v[i] <= hi) atomicAdd(hist + ((v[i] - lo) >> shift), 1u);
    uint32_t above;
    const int b = wave_find_bin(hist, need, &above);
    need -= above;
    lo += (uint32_t)b << shift;
    const uint32_t width = (1u << shift) - 1u;
    if (hi - lo > width) hi = lo + width;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// Sampled scores and pivots in one launch. Workgroup = NW waves over 16
// landmark rows of one head (one MFMA column block); wave w scores them
// against the sampled keys [SEL_NS/NW w, SEL_NS/NW (w + 1)) in tiles of 64,
// the A fragments loaded straight from the sampled key rows (tile arithmetic
// as in the score pass, so the same values), keys = score_key(fl(dot) * scale)
// into LDS; then wave w takes the pivots of rows 16/NW w .. 16/NW (w + 1) - 1,
// its histogram in the first 256 words of its own row's keys once they are in
// registers (the wave's LDS accesses are in order). Workgroup (0, 0) also
// zeroes the fallback counter.
// ---------------------------------------------------------------------------
constexpr int SP_PITCH = SEL_NS + 4;  // keys per LDS row: rows start 4 banks apart

template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) void sample_pivot_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                               uint32_t *__restrict__ plo,
                                                               uint32_t *__restrict__ fail_cnt, int N, int M, int ns,
                                                               int r, float scale) {
  static_assert(16 % NW == 0 && SEL_NS % (NW * TK) == 0, "sample/pivot split");
  constexpr int PERW = SEL_NS / NW;  // samples per wave
  constexpr int RPW = 16 / NW;       // rows per wave
  __shared__ __align__(16) uint32_t keys[16][SP_PITCH];
  const int64_t bh = blockIdx.y;
  const int lm0 = blockIdx.x * 16;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *fail_cnt = 0;
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
  }
}

template <typename T, int D, int CAP, bool MERGE>
__global__ __launch_bounds__(256) void finalize_kernel(const uint2 *__restrict__ cand,
                                                       const uint32_t *__restrict__ ccnt, int32_t *__restrict__ idx,
                                                       uint32_t *__restrict__ fail_cnt,
                                                       int32_t *__restrict__ fail_list, int k, int cap, int nch,
                                                       const float2 *__restrict__ part_ml,
                                                       const float *__restrict__ part_o, T *__restrict__ v_lm, int M) {
  __shared__ FinalizeLds<T, D, CAP, MERGE> sh;
  finalize_row<T, D, CAP, MERGE>(sh, blockIdx.x, cand, ccnt, idx, fail_cnt, fail_list, k, cap, nch, part_ml, part_o,
                                 v_lm, M);
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t sample_pivot_t(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb,
                                 hipStream_t st) {
  // bf16: one sample tile and one row per wave (16 waves); fp32 (more
  // registers per fragment): four waves, four tiles and four rows each
  constexpr int NW = sizeof(T) == 2 ? 16 : 4;
  const dim3 grid((unsigned)((c.M + 15) / 16), (unsigned)BH(c));
  hipLaunchKernelGGL((sample_pivot_kernel<T, D, NW>), grid, dim3(64 * NW), 0, st, (const T *)q_lm, (const T *)k,
                     sb.plo, sb.fail_cnt, c.N, c.M, sb.ns, sb.rank, eff_scale(c));
  return launched("sample_pivot_kernel", st);
}

hipError_t launch_select_pivots(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb,
                                hipStream_t st) {
  if (sb.ns > SEL_NS) return hipErrorInvalidValue;  // the workgroup holds SEL_NS keys per row
  if (c.dtype == MITA_F32)
    return c.d == 64 ? sample_pivot_t<float, 64>(c, q_lm, k, sb, st) : sample_pivot_t<float, 128>(c, q_lm, k, sb, st);
  return c.d == 64 ? sample_pivot_t<bf16_t, 64>(c, q_lm, k, sb, st) : sample_pivot_t<bf16_t, 128>(c, q_lm, k, sb, st);
}

// The finalize kernel alone (one workgroup per landmark row).
static hipError_t launch_select_finalize(const mita_cfg_t &c, const SelectBufs &sb, int32_t *idx, const void *partial,
                                  void *v_lm, hipStream_t st) {
  const unsigned rows = (unsigned)(BH(c) * c.M);
  const int nch = score_chunks(c);
  const float2 *ml = (const float2 *)partial;
  const float *po = v_lm ? (const float *)((const char *)partial + align_up((size_t)BH(c) * nch * c.M * sizeof(float2)))
                         : nullptr;
#define MITA_FINALIZE(TT, DD, CAP, MG)                                                                          \
  hipLaunchKernelGGL((finalize_kernel<TT, DD, CAP, MG>), dim3(rows), dim3(256), 0, st, sb.cand, sb.ccnt, idx,   \
                     sb.fail_cnt, sb.fail_list, c.k, sb.cap, nch, ml, po, (TT *)v_lm, c.M)
#define MITA_FINALIZE_CAP(TT, DD, MG)     \
  if (sb.cap <= 1024)                     \
    MITA_FINALIZE(TT, DD, 1024, MG);      \
  else if (sb.cap <= 2048)                \
    MITA_FINALIZE(TT, DD, 2048, MG);      \
  else if (sb.cap <= 4096)                \
    MITA_FINALIZE(TT, DD, 4096, MG);      \
  else                                    \
    MITA_FINALIZE(TT, DD, SEL_CAP, MG);
  if (!v_lm) {
    MITA_FINALIZE_CAP(float, 64, false)
  } else if (c.dtype == MITA_F32) {
    if (c.d == 64) {
      MITA_FINALIZE_CAP(float, 64, true)
    } else {
      MITA_FINALIZE_CAP(float, 128, true)
    }
  } else {
    if (c.d == 64) {
      MITA_FINALIZE_CAP(bf16_t, 64, true)
    } else {
      MITA_FINALIZE_CAP(bf16_t, 128, true)
    }
  }
#undef MITA_FINALIZE_CAP
#undef MITA_FINALIZE
  return launched("finalize_kernel", st);
}

hipError_t launch_select_finish(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb, float *S,
                                int32_t *idx, const void *partial, void *v_lm, hipStream_t st) {
  hipError_t e = launch_select_finalize(c, sb, idx, partial, v_lm, st);
  if (e != hipSuccess) return e;
  if ((e = launch_scores_rows(c, q_lm, k, S, sb.fail_cnt, sb.fail_list, st)) != hipSuccess) return e;
  return launch_topk(c, S, idx, st, sb.fail_cnt, sb.fail_list);
}

}  // namespace mita
