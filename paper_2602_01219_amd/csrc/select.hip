// select.hip - the top-k selection of the forward (Eq. top-k), fused with the
// landmark-key score pass so that the M x N score matrix is never stored.
//
//   1. sample_kernel: the scores of every landmark against ns evenly spaced
//      keys, as order-preserving keys (the same tile arithmetic as the score
//      pass, so the same values).
//   2. pivot_kernel: per landmark row, the pivot = the r-th largest sampled
//      key. r is chosen on the host so that at least k and far fewer than
//      `cap` tokens of the row score >= pivot, except with negligible
//      probability (r = k exactly when the sample is the whole row).
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
// Sampled scores. Workgroup = 4 waves x 16 landmarks over SAMPLE_NC sampled
// keys, tiles of 64 gathered into LDS; keys = score_key(fl(dot) * scale).
// Workgroup (0, 0, 0) also zeroes the fallback counter.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(BLOCK) void sample_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                       uint32_t *__restrict__ samp, uint32_t *__restrict__ fail_cnt,
                                                       int N, int M, int ns, float scale) {
  using TD = TileDims<T, D>;
  __shared__ __align__(16) T Ks[TD::K_ELEMS];
  __shared__ int32_t pos[TK];
  const int64_t bh = blockIdx.z;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int lm0 = (blockIdx.y * 4 + w) * 16;
  const int lm = lm0 + p;
  const int64_t row = bh * M + lm;
  if (blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0) *fail_cnt = 0;

  Frag<T> qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    if (lm < M)
      qf[ks].load(q_lm + row * D + ks * 32 + g * 8);
    else
      qf[ks].zero();
  }
  const T *kb_ = k + bh * (int64_t)N * D;
  const int j_begin = blockIdx.x * SAMPLE_NC, j_end = min(ns, j_begin + SAMPLE_NC);
  for (int j0 = j_begin; j0 < j_end; j0 += TK) {
    const int nvalid = min(TK, j_end - j0);
    __syncthreads();
    if (threadIdx.x < TK) pos[threadIdx.x] = (int)threadIdx.x < nvalid ? sample_pos(j0 + threadIdx.x, N, ns) : 0;
    __syncthreads();
    load_k_tile<T, D>(Ks, kb_, pos, nvalid);
    __syncthreads();
    if (lm0 >= M) continue;
    f32x4 acc[4];
    tile_scores<T, D>(acc, Ks, qf);
    if (lm < M) {
      uint32_t *srow = samp + row * (int64_t)ns + j0;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int j = kb * 16 + 4 * g;
        uint32_t key[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) key[r] = score_key(acc[kb][r] * scale);
        if ((ns & 3) == 0 && j + 3 < nvalid) {
          *reinterpret_cast<uint4 *>(srow + j) = make_uint4(key[0], key[1], key[2], key[3]);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (j + r < nvalid) srow[j + r] = key[r];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Pivots: one wave per landmark row, its ns (<= SEL_NS) sampled keys in
// registers. Radix rounds over a 256-bin LDS histogram of the current key
// range (bins span (hi - lo + 1) / 256 keys, so each round shrinks the range
// by 2^8) narrow down on the r-th largest sample; after two rounds the lower
// edge of the bin holding it is taken. That edge is at most the r-th largest
// sample, so at least r samples are >= pivot, and its bin spans at most
// 2^16 keys (a relative step of 2^-7 within one binade), which lists only a
// few more tokens than the exact sample statistic would.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pivot_kernel(const uint32_t *__restrict__ samp, uint32_t *__restrict__ plo,
                                                    int64_t rows, int ns, int r) {
  constexpr int PER = SEL_NS / 64;
  __shared__ uint32_t hist_all[4][256];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;  // a whole wave; no workgroup barriers below
  uint32_t *hist = hist_all[w];
  const uint32_t *s = samp + row * (int64_t)ns;
  // lane l holds keys 4 l + 256 i + (0..3); 0 marks a slot past ns (no score
  // has key 0, so it lies below every range)
  uint32_t v[PER];
  if ((ns & 255) == 0) {
#pragma unroll
    for (int i = 0; i < PER / 4; ++i) {
      uint4 x = make_uint4(0u, 0u, 0u, 0u);
      if (256 * i < ns) x = *reinterpret_cast<const uint4 *>(s + 256 * i + 4 * lane);
      v[4 * i] = x.x;
      v[4 * i + 1] = x.y;
      v[4 * i + 2] = x.z;
      v[4 * i + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int j = 256 * (i / 4) + 4 * lane + (i % 4);
      v[i] = j < ns ? s[j] : 0u;
    }
  }
  uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
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
    for (int i = 0; i < PER; ++i)
      if (v[i] >= lo && v[i] <= hi) atomicAdd(hist + ((v[i] - lo) >> shift), 1u);
    uint32_t above;
    const int b = wave_find_bin(hist, need, &above);
    need -= above;
    lo += (uint32_t)b << shift;
    const uint32_t width = (1u << shift) - 1u;
    if (hi - lo > width) hi = lo + width;
  }
  if (lane == 0) plo[row] = lo;
}

// One workgroup per landmark row.
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
static hipError_t sample_t(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb, hipStream_t st) {
  dim3 grid((sb.ns + SAMPLE_NC - 1) / SAMPLE_NC, (c.M + 63) / 64, (unsigned)BH(c));
  hipLaunchKernelGGL((sample_kernel<T, D>), grid, dim3(BLOCK), 0, st, (const T *)q_lm, (const T *)k, sb.samp,
                     sb.fail_cnt, c.N, c.M, sb.ns, eff_scale(c));
  return hipGetLastError();
}

hipError_t launch_select_pivots(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb,
                                hipStream_t st) {
  hipError_t e;
  if (c.dtype == MITA_F32)
    e = c.d == 64 ? sample_t<float, 64>(c, q_lm, k, sb, st) : sample_t<float, 128>(c, q_lm, k, sb, st);
  else
    e = c.d == 64 ? sample_t<bf16_t, 64>(c, q_lm, k, sb, st) : sample_t<bf16_t, 128>(c, q_lm, k, sb, st);
  if (e != hipSuccess) return e;
  const int64_t rows = BH(c) * c.M;
  hipLaunchKernelGGL(pivot_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, sb.samp, sb.plo, rows, sb.ns,
                     sb.rank);
  return hipGetLastError();
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
  return hipGetLastError();
}

hipError_t launch_select_finish(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb, float *S,
                                int32_t *idx, const void *partial, void *v_lm, hipStream_t st) {
  hipError_t e = launch_select_finalize(c, sb, idx, partial, v_lm, st);
  if (e != hipSuccess) return e;
  if ((e = launch_scores_rows(c, q_lm, k, S, sb.fail_cnt, sb.fail_list, st)) != hipSuccess) return e;
  return launch_topk(c, S, idx, st, sb.fail_cnt, sb.fail_list);
}

}  // namespace mita
