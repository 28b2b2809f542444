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
//   3. the score pass lists every token scoring >= pivot (bits of its
//      unscaled dot, token index), in token order, in one region per (row,
//      key chunk); the finish scales the dots as every score is scaled.
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
#include "sample.hpp"
#include "worklist.hpp"

namespace mita {

// One workgroup per (16 landmarks, head) slot, slots spread over the XCDs in
// contiguous ranges (xcd_slot): a head's landmark blocks share an XCD, so
// its sampled key rows are fetched into one L2 instead of one per block.
template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) void sample_pivot_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                               uint32_t *__restrict__ plo,
                                                               uint32_t *__restrict__ fail_cnt, int N, int M, int ns,
                                                               int r, float scale, int nbx, int nslots,
                                                               int32_t *__restrict__ idx, int kk) {
  __shared__ __align__(16) uint32_t keys[16][SP_PITCH];
  const int f = xcd_slot((int)blockIdx.x, (int)gridDim.x / NXCD);
  if (f >= nslots) return;  // the whole workgroup
  sample_pivot_body<T, D, NW>(keys, f % nbx, f / nbx, q_lm, k, plo, fail_cnt, N, M, ns, r, scale, idx, kk);
}

template <typename T, int D, int CAP, bool MERGE>
__global__ __launch_bounds__(256) void finalize_kernel(const uint2 *__restrict__ cand,
                                                       const uint32_t *__restrict__ ccnt, int32_t *__restrict__ idx,
                                                       uint32_t *__restrict__ fail_cnt,
                                                       int32_t *__restrict__ fail_list, int k, int cap, int nch,
                                                       const float2 *__restrict__ part_ml,
                                                       const float *__restrict__ part_o, T *__restrict__ v_lm, int M,
                                                       float scale) {
  __shared__ FinalizeLds<T, D, CAP, MERGE> sh;
  finalize_row<T, D, CAP, MERGE>(sh, blockIdx.x, cand, ccnt, idx, fail_cnt, fail_list, k, cap, nch, part_ml, part_o,
                                 v_lm, M, scale);
}

// The same with one wave per row (lists of at most SEL_NS, at most 64 chunks).
template <typename T, int D, bool MERGE>
__global__ __launch_bounds__(256) void finalize_wave_kernel(const uint2 *__restrict__ cand,
                                                            const uint32_t *__restrict__ ccnt,
                                                            int32_t *__restrict__ idx, uint32_t *__restrict__ fail_cnt,
                                                            int32_t *__restrict__ fail_list, int k, int cap, int nch,
                                                            const float2 *__restrict__ part_ml,
                                                            const float *__restrict__ part_o, T *__restrict__ v_lm,
                                                            int M, float scale, int64_t nrows) {
  __shared__ FinalizeWaveLds sh[4];
  const int w = (int)threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= nrows) return;  // the whole wave
  finalize_row_wave<T, D, MERGE>(sh[w], row, cand, ccnt, idx, fail_cnt, fail_list, k, cap, nch, part_ml, part_o,
                                 v_lm, M, scale);
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
  const int nbx = (c.M + 15) / 16, nslots = nbx * (int)BH(c);
  const dim3 grid((unsigned)(NXCD * ((nslots + NXCD - 1) / NXCD)));
  hipLaunchKernelGGL((sample_pivot_kernel<T, D, NW>), grid, dim3(64 * NW), 0, st, (const T *)q_lm, (const T *)k,
                     sb.plo, sb.fail_cnt, c.N, c.M, sb.ns, sb.rank, eff_scale(c), nbx, nslots, sb.idx, c.k);
  return launched("sample_pivot_kernel", st);
}

hipError_t launch_select_pivots(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb,
                                hipStream_t st) {
  if (sb.ns > SEL_NS) return hipErrorInvalidValue;  // the workgroup holds SEL_NS keys per row
  if (sb.idx && (sb.ns != c.N || sb.rank != c.k)) return hipErrorInvalidValue;  // direct sets need the whole row
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
                     sb.fail_cnt, sb.fail_list, c.k, sb.cap, nch, ml, po, (TT *)v_lm, c.M, eff_scale(c))
#define MITA_FINALIZE_WAVE(TT, DD, MG)                                                                          \
  hipLaunchKernelGGL((finalize_wave_kernel<TT, DD, MG>), dim3((rows + 3) / 4), dim3(256), 0, st, sb.cand, sb.ccnt, \
                     idx, sb.fail_cnt, sb.fail_list, c.k, sb.cap, nch, ml, po, (TT *)v_lm, c.M, eff_scale(c),      \
                     (int64_t)rows)
  // lists of at most SEL_NS entries over at most 64 chunks: one wave per row
  const bool wave = sb.cap <= SEL_NS && nch <= 64;
#define MITA_FINALIZE_CAP(TT, DD, MG)     \
  if (wave)                               \
    MITA_FINALIZE_WAVE(TT, DD, MG);       \
  else if (sb.cap <= 1024)                \
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
#undef MITA_FINALIZE_WAVE
#undef MITA_FINALIZE
  return launched(wave ? "finalize_wave_kernel" : "finalize_kernel", st);
}

hipError_t launch_select_finish(const mita_cfg_t &c, const void *q_lm, const void *k, const SelectBufs &sb, float *S,
                                int32_t *idx, const void *partial, void *v_lm, hipStream_t st) {
  if (sb.idx) return hipSuccess;  // the pivot launch wrote the sets; nothing is listed
  hipError_t e = launch_select_finalize(c, sb, idx, partial, v_lm, st);
  if (e != hipSuccess) return e;
  if ((e = launch_scores_rows(c, q_lm, k, S, sb.fail_cnt, sb.fail_list, st)) != hipSuccess) return e;
  return launch_topk(c, S, idx, st, sb.fail_cnt, sb.fail_list);
}

}  // namespace mita
