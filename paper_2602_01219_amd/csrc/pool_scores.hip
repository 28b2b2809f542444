// pool_scores.hip - landmark pooling, landmark-key scores with landmark
// values, and the expert-tile gather.
#include "cdna4.hpp"
#include "flash.hpp"
#include "kernels.hpp"
#include "check.hpp"
#include "scores.hpp"

namespace mita {

// ---------------------------------------------------------------------------
// Landmark queries (Sec. 3.2: average pooling over uniformly spaced windows;
// Algorithm 1 AdaptiveAvgPool; 2-D windows per Tab. A1). One workgroup per
// (b*h, landmark); threads read 16-byte chunks of the window's token rows
// (consecutive threads -> consecutive bytes), accumulate in fp32, then reduce
// over the token slots through LDS.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void pool_kernel(const T *__restrict__ q, T *__restrict__ q_lm,
                                                   int32_t *__restrict__ zero_counts, int32_t *__restrict__ zero_cursor,
                                                   int N, int gh, int gw, int lh, int lw) {
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr int CPT = D / VE;   // chunks per token row
  constexpr int P = 256 / CPT;  // token slots
  __shared__ float red[P][D + 1];
  const int i = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int M = lh * lw;
  const int a = i / lw, b = i % lw;
  const int r0 = (int)(((int64_t)a * gh) / lh), r1 = (int)(((int64_t)(a + 1) * gh + lh - 1) / lh);
  const int c0 = (int)(((int64_t)b * gw) / lw), c1 = (int)(((int64_t)(b + 1) * gw + lw - 1) / lw);
  const int cols = c1 - c0, count = (r1 - r0) * cols;
  if (zero_counts && threadIdx.x == 0) zero_counts[bh * M + i] = 0;
  if (zero_cursor && threadIdx.x == 0) zero_cursor[bh * M + i] = 0;
  const int ch = threadIdx.x % CPT, slot = threadIdx.x / CPT;
  float acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  const T *base = q + bh * (int64_t)N * D;
  constexpr int U = 4;  // token rows per thread loaded before any is summed
  for (int t0 = slot; t0 < count; t0 += U * P) {
    uint4 u[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int t = t0 + j * P;
      u[j] = make_uint4(0u, 0u, 0u, 0u);
      if (t < count) {
        const int r = r0 + t / cols, c = c0 + t % cols;
        u[j] = *reinterpret_cast<const uint4 *>(base + ((int64_t)r * gw + c) * D + ch * VE);
      }
    }
#pragma unroll
    for (int j = 0; j < U; ++j) {
      float x[VE];
      unpack16(u[j], x, (const T *)nullptr);
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[e] += x[e];
    }
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) red[slot][ch * VE + e] = acc[e];
  __syncthreads();
  // the P slot sums of each column: NQ partial sums per column (one per
  // thread), then their sum
  constexpr int NQ = 256 / D, PQ = P / NQ;
  static_assert(NQ >= 1 && P % NQ == 0, "pool reduction layout");
  const int col = threadIdx.x % D, part_i = threadIdx.x / D;
  float part = 0.f;
#pragma unroll
  for (int j = 0; j < PQ; ++j) part += red[part_i * PQ + j][col];
  __syncthreads();
  red[part_i][col] = part;
  __syncthreads();
  if (threadIdx.x < D) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NQ; ++j) s += red[j][threadIdx.x];
    q_lm[(bh * M + i) * D + threadIdx.x] = from_f32<T>(s / (float)count);
  }
}

// The same pooling for small windows (at most SMALL_WINDOW tokens): one wave
// per landmark row, four rows per workgroup; lane = (token slot, 16-byte
// chunk), the slots summed across lanes (sum order: each slot's tokens in
// order, then the slots pairwise).
constexpr int SMALL_WINDOW = 32;

template <typename T, int D>
__global__ __launch_bounds__(256) void pool_small_kernel(const T *__restrict__ q, T *__restrict__ q_lm,
                                                         int32_t *__restrict__ zero_counts,
                                                         int32_t *__restrict__ zero_cursor, int N, int gh, int gw,
                                                         int lh, int lw, int64_t rows) {
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr int CPT = D / VE;  // chunks per token row
  constexpr int PS = 64 / CPT;  // token slots per wave
  static_assert(PS >= 1 && 64 % CPT == 0, "whole token rows per wave");
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;  // the whole wave; no barriers below
  const int M = lh * lw;
  const int64_t bh = row / M;
  const int i = (int)(row % M);
  const int a = i / lw, b = i % lw;
  const int r0 = (int)(((int64_t)a * gh) / lh), r1 = (int)(((int64_t)(a + 1) * gh + lh - 1) / lh);
  const int c0 = (int)(((int64_t)b * gw) / lw), c1 = (int)(((int64_t)(b + 1) * gw + lw - 1) / lw);
  const int cols = c1 - c0, count = (r1 - r0) * cols;
  if (zero_counts && lane == 0) zero_counts[row] = 0;
  if (zero_cursor && lane == 0) zero_cursor[row] = 0;
  const int ch = lane % CPT, slot = lane / CPT;
  float acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  const T *base = q + bh * (int64_t)N * D;
  for (int t = slot; t < count; t += PS) {
    const int r = r0 + t / cols, c = c0 + t % cols;
    float x[VE];
    unpack16(*reinterpret_cast<const uint4 *>(base + ((int64_t)r * gw + c) * D + ch * VE), x, (const T *)nullptr);
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] += x[e];
  }
#pragma unroll
  for (int o = CPT; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] += __shfl_xor(acc[e], o);
  if (slot == 0) {
    T out[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) out[e] = from_f32<T>(acc[e] / (float)count);
    *reinterpret_cast<uint4 *>(q_lm + row * D + ch * VE) = *reinterpret_cast<const uint4 *>(out);
  }
}

// The bf16 d=64 pass holds 3 waves per SIMD (at most 168 VGPRs).
#define SCORES_OCCUPANCY __attribute__((amdgpu_waves_per_eu(sizeof(T) == 2 && D == 64 ? 3 : (sizeof(T) == 2 ? 2 : 1))))

template <typename T, int D, bool WRITE_S, bool DO_V, bool SELECT>
__global__ __launch_bounds__(BLOCK) SCORES_OCCUPANCY void scores_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                       const T *__restrict__ v, float *__restrict__ S,
                                                       float2 *__restrict__ part_ml, float *__restrict__ part_o,
                                                       SelectArgs sel, int N, int M, float scale) {
  using TD = TileDims<T, D>;
  __shared__ __align__(16) T Ks[2][TD::K_ELEMS];
  __shared__ __align__(16) T Vt[DO_V ? 2 : 1][DO_V ? TD::V_ELEMS : 1];
  score_chunk<T, D, WRITE_S, DO_V, SELECT>(&Ks[0][0], &Vt[0][0], q_lm, k, v, S, part_ml, part_o, sel, N, M, scale,
                                           blockIdx.x, gridDim.x, blockIdx.y, blockIdx.z, -1);
}

// The bf16 score pass with landmark values on the DMA tiles (score16_chunk):
// NW waves of NG landmark groups each; three waves per SIMD with four-wave
// workgroups (two scratch spills outside the tile loop).
template <int D, int NG, int NW, bool WRITE_S, bool SELECT>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW == 4 ? 3 : 2))) void scores16_kernel(
    const bf16_t *__restrict__ q_lm, const bf16_t *__restrict__ k, const bf16_t *__restrict__ v,
    float *__restrict__ S, float2 *__restrict__ part_ml, float *__restrict__ part_o, SelectArgs sel, int N, int M,
    float scale) {
  using DT = DmaTile<D, TK32, NW>;
  // the two tile buffers (K then V each) as separate arrays
  __shared__ __align__(16) char tiles0[2 * DT::BYTES];
  __shared__ __align__(16) char tiles1[2 * DT::BYTES];
  score16_chunk<D, NG, NW, WRITE_S, SELECT>(tiles0, tiles1, q_lm, k, v, S, part_ml, part_o, sel, N, M, scale,
                                            (int)blockIdx.x, (int)gridDim.x, (int)blockIdx.y, (int64_t)blockIdx.z);
}

// Score rows of listed landmark rows (fallback of the fused selection).
template <typename T, int D>
__global__ __launch_bounds__(BLOCK) void scores_rows_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                            float *__restrict__ S, const uint32_t *__restrict__ nrows,
                                                            const int32_t *__restrict__ rows, int N, int M,
                                                            float scale, int nchunks) {
  using TD = TileDims<T, D>;
  __shared__ __align__(16) T Ks[2][TD::K_ELEMS];
  scores_rows_body<T, D>(&Ks[0][0], (int)blockIdx.x, (int)gridDim.x, q_lm, k, S, nrows, rows, N, M, scale, nchunks);
}

// Log-sum-exp merge of the per-chunk landmark-value partials, one thread per
// (landmark row, dimension) (the same merge, in the same order, as the fused
// selection's finish applies to a row with a whole workgroup).
template <typename T, int D>
__global__ __launch_bounds__(256) void merge_kernel(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                                    T *__restrict__ v_lm, int M, int nchunks, int64_t rows) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = t / D;
  if (row >= rows) return;
  const int dim = (int)(t % D);
  v_lm[row * D + dim] =
      from_f32<T>(merge_landmark_value_1<D>(part_ml, part_o, row / M, (int)(row % M), M, nchunks, dim));
}

// ---------------------------------------------------------------------------
// Expert tiles (Eq. gather): one 16-byte chunk per thread, rows of k_x / v_x
// written contiguously, source rows read through idx.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(256) void gather_kernel(const T *__restrict__ k, const T *__restrict__ v,
                                                     const int32_t *__restrict__ idx, T *__restrict__ kx,
                                                     T *__restrict__ vx, int64_t rows, int N, int Mk) {
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr int CPR = D / VE;
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= rows * CPR) return;
  const int64_t row = c / CPR;
  const int ch = (int)(c % CPR);
  const int64_t bh = row / Mk;
  const int64_t src = bh * N + idx[row];
  const uint4 a = *reinterpret_cast<const uint4 *>(k + src * D + ch * VE);
  const uint4 b = *reinterpret_cast<const uint4 *>(v + src * D + ch * VE);
  *reinterpret_cast<uint4 *>(kx + row * D + ch * VE) = a;
  *reinterpret_cast<uint4 *>(vx + row * D + ch * VE) = b;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t pool_t(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *zc, int32_t *zcur,
                         hipStream_t st) {
  // the largest window: its most rows times its most columns
  int wr = 0, wc = 0;
  for (int a = 0; a < c.lm_h; ++a)
    wr = std::max(wr, (int)(((int64_t)(a + 1) * c.grid_h + c.lm_h - 1) / c.lm_h - ((int64_t)a * c.grid_h) / c.lm_h));
  for (int b = 0; b < c.lm_w; ++b)
    wc = std::max(wc, (int)(((int64_t)(b + 1) * c.grid_w + c.lm_w - 1) / c.lm_w - ((int64_t)b * c.grid_w) / c.lm_w));
  if ((int64_t)wr * wc <= SMALL_WINDOW) {
    const int64_t rows = BH(c) * c.M;
    hipLaunchKernelGGL((pool_small_kernel<T, D>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, (const T *)q,
                       (T *)q_lm, zc, zcur, c.N, c.grid_h, c.grid_w, c.lm_h, c.lm_w, rows);
    return launched("pool_small_kernel", st);
  }
  dim3 grid(c.M, (unsigned)BH(c));
  hipLaunchKernelGGL((pool_kernel<T, D>), grid, dim3(256), 0, st, (const T *)q, (T *)q_lm, zc, zcur, c.N, c.grid_h,
                     c.grid_w, c.lm_h, c.lm_w);
  return launched("pool_kernel", st);
}

hipError_t launch_pool(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *zc, int32_t *zcur, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? pool_t<float, 64>(c, q, q_lm, zc, zcur, st) : pool_t<float, 128>(c, q, q_lm, zc, zcur, st);
  return c.d == 64 ? pool_t<bf16_t, 64>(c, q, q_lm, zc, zcur, st) : pool_t<bf16_t, 128>(c, q, q_lm, zc, zcur, st);
}

// Random-selection landmarks (Tab. A1, landmark extraction): row i of slice
// bh is the query of token sel[bh, i]; one thread per 16-byte chunk. An index
// outside [0, N) is not read and gives a row of NaN.
template <typename T, int D>
__global__ __launch_bounds__(256) void select_landmarks_kernel(const T *__restrict__ q, const int32_t *__restrict__ sel,
                                                               T *__restrict__ q_lm, int N, int M, int64_t rows) {
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr int C = D / VE;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = t / C;
  const int c = (int)(t % C);
  if (row >= rows) return;
  const int64_t bh = row / M;
  const int src = sel[row];
  uint4 x;
  if (src >= 0 && src < N) {
    x = *reinterpret_cast<const uint4 *>(q + (bh * N + src) * D + c * VE);
  } else {
    const uint32_t nan = sizeof(T) == 4 ? 0x7fc00000u : 0x7fc07fc0u;
    x = make_uint4(nan, nan, nan, nan);
  }
  *reinterpret_cast<uint4 *>(q_lm + row * D + c * VE) = x;
}

template <typename T, int D>
static hipError_t select_landmarks_t(const mita_cfg_t &c, const void *q, const int32_t *sel, void *q_lm,
                                     hipStream_t st) {
  const int64_t rows = BH(c) * c.M;
  const int64_t threads = rows * (D * (int64_t)sizeof(T) / 16);
  hipLaunchKernelGGL((select_landmarks_kernel<T, D>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st,
                     (const T *)q, sel, (T *)q_lm, c.N, c.M, rows);
  return launched("select_landmarks_kernel", st);
}

hipError_t launch_select_landmarks(const mita_cfg_t &c, const void *q, const int32_t *sel, void *q_lm,
                                   hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? select_landmarks_t<float, 64>(c, q, sel, q_lm, st)
                     : select_landmarks_t<float, 128>(c, q, sel, q_lm, st);
  return c.d == 64 ? select_landmarks_t<bf16_t, 64>(c, q, sel, q_lm, st)
                   : select_landmarks_t<bf16_t, 128>(c, q, sel, q_lm, st);
}

// Zeroes p[0, n) and (when p2 is given) p2[0, n2): one launch for both.
__global__ __launch_bounds__(256) void zero_kernel(int32_t *__restrict__ p, int64_t n, int32_t *__restrict__ p2,
                                                   int64_t n2) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
  if (p2 && i < n2) p2[i] = 0;
}

hipError_t launch_zero(int32_t *p, int64_t n, hipStream_t st) { return launch_zero2(p, n, nullptr, 0, st); }

hipError_t launch_zero2(int32_t *p, int64_t n, int32_t *p2, int64_t n2, hipStream_t st) {
  if (!p || n <= 0) {  // the second array alone, or nothing
    p = p2;
    n = n2;
    p2 = nullptr;
    n2 = 0;
  }
  if (!p || n <= 0) return hipSuccess;
  if (!p2) n2 = 0;
  const int64_t m = n > n2 ? n : n2;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, st, p, n, p2, n2);
  return launched("zero_kernel", st);
}

template <typename T, int D>
static hipError_t scores_t(const mita_cfg_t &c, const void *q_lm, const void *k, const void *v, float *S, void *v_lm,
                           void *partial, const SelectBufs *sb, hipStream_t st) {
  const int nch = score_chunks(c);
  dim3 grid(nch, (c.M + 63) / 64, (unsigned)BH(c));
  float2 *ml = (float2 *)partial;
  float *po = v_lm ? (float *)((char *)partial + align_up((size_t)BH(c) * nch * c.M * sizeof(float2))) : nullptr;
  const float sc = eff_scale(c);
  const SelectArgs sel = sb ? SelectArgs{sb->plo, sb->ccnt, sb->cand} : SelectArgs{nullptr, nullptr, nullptr};
  const T *ql = (const T *)q_lm, *kk = (const T *)k, *vv = (const T *)v;
  // bf16, d = 128, with landmark values: every such pass (selection, stored
  // scores or values alone) runs score16_chunk, so their landmark values
  // agree. (At d = 64 the 64-key register-staged tiles of score_chunk are
  // faster: per 32-key tile the listing's fixed steps weigh twice as much
  // against the smaller products.)
  if constexpr (sizeof(T) == 2 && D == 128) {
    if (v_lm) {
      constexpr int NG = 1;
      const bool narrow = c.M <= 32 * NG;  // two waves cover the landmarks
      const int per = 16 * NG * (narrow ? 2 : 4);
      const dim3 g16(nch, (c.M + per - 1) / per, (unsigned)BH(c));
      const bf16_t *qb = (const bf16_t *)q_lm, *kb = (const bf16_t *)k, *vb = (const bf16_t *)v;
#define MITA_SCORES16(NW, W, SEL)                                                                                  \
  hipLaunchKernelGGL((scores16_kernel<D, NG, NW, W, SEL>), g16, dim3(64 * NW), 0, st, qb, kb, vb, S, ml, po, sel, \
                     c.N, c.M, sc)
      if (narrow) {
        if (sb)
          MITA_SCORES16(2, false, true);
        else if (S)
          MITA_SCORES16(2, true, false);
        else
          MITA_SCORES16(2, false, false);
      } else {
        if (sb)
          MITA_SCORES16(4, false, true);
        else if (S)
          MITA_SCORES16(4, true, false);
        else
          MITA_SCORES16(4, false, false);
      }
#undef MITA_SCORES16
      hipError_t e = launched("scores16_kernel", st);
      if (e != hipSuccess || sb) return e;  // with sel the merge runs in the selection's finish
      hipLaunchKernelGGL((merge_kernel<T, D>), dim3((unsigned)((BH(c) * c.M * D + 255) / 256)), dim3(256), 0, st, ml,
                         po, (T *)v_lm, c.M, nch, (int64_t)BH(c) * c.M);
      return launched("merge_kernel", st);
    }
  }
#define MITA_SCORES(W, V, SEL) \
  hipLaunchKernelGGL((scores_kernel<T, D, W, V, SEL>), grid, dim3(BLOCK), 0, st, ql, kk, vv, S, ml, po, sel, c.N, c.M, sc)
  if (sb) {
    if (v_lm)
      MITA_SCORES(false, true, true);
    else
      MITA_SCORES(false, false, true);
  } else if (S && v_lm) {
    MITA_SCORES(true, true, false);
  } else if (S) {
    MITA_SCORES(true, false, false);
  } else if (v_lm) {
    MITA_SCORES(false, true, false);
  } else {
    return hipSuccess;
  }
#undef MITA_SCORES
  hipError_t e = launched("scores_kernel", st);
  if (e != hipSuccess || !v_lm || sb) return e;  // with sel the merge runs in the selection's finish
  hipLaunchKernelGGL((merge_kernel<T, D>), dim3((unsigned)((BH(c) * c.M * D + 255) / 256)), dim3(256), 0, st, ml, po,
                     (T *)v_lm, c.M, nch, (int64_t)BH(c) * c.M);
  return launched("merge_kernel", st);
}

hipError_t launch_scores(const mita_cfg_t &c, const void *q_lm, const void *k, const void *v, float *S, void *v_lm,
                         void *partial, const SelectBufs *sel, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? scores_t<float, 64>(c, q_lm, k, v, S, v_lm, partial, sel, st)
                     : scores_t<float, 128>(c, q_lm, k, v, S, v_lm, partial, sel, st);
  return c.d == 64 ? scores_t<bf16_t, 64>(c, q_lm, k, v, S, v_lm, partial, sel, st)
                   : scores_t<bf16_t, 128>(c, q_lm, k, v, S, v_lm, partial, sel, st);
}

template <typename T, int D>
static hipError_t scores_rows_t(const mita_cfg_t &c, const void *q_lm, const void *k, float *S, const uint32_t *nrows,
                                const int32_t *rows, hipStream_t st) {
  // a fixed grid walks the (row, chunk) items; with no listed rows every
  // workgroup exits at once
  const int nch = score_chunks(c);
  const int64_t most = BH(c) * c.M * (int64_t)nch;
  const unsigned grid = (unsigned)(most < 1024 ? most : 1024);
  hipLaunchKernelGGL((scores_rows_kernel<T, D>), dim3(grid), dim3(BLOCK), 0, st, (const T *)q_lm, (const T *)k, S,
                     nrows, rows, c.N, c.M, eff_scale(c), nch);
  return launched("scores_rows_kernel", st);
}

hipError_t launch_scores_rows(const mita_cfg_t &c, const void *q_lm, const void *k, float *S, const uint32_t *nrows,
                              const int32_t *rows, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? scores_rows_t<float, 64>(c, q_lm, k, S, nrows, rows, st)
                     : scores_rows_t<float, 128>(c, q_lm, k, S, nrows, rows, st);
  return c.d == 64 ? scores_rows_t<bf16_t, 64>(c, q_lm, k, S, nrows, rows, st)
                   : scores_rows_t<bf16_t, 128>(c, q_lm, k, S, nrows, rows, st);
}

template <typename T, int D>
static hipError_t gather_t(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                           hipStream_t st) {
  constexpr int CPR = D / (16 / (int)sizeof(T));
  const int64_t rows = BH(c) * c.M * (int64_t)c.k;
  const int64_t blocks = (rows * CPR + 255) / 256;
  hipLaunchKernelGGL((gather_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, st, (const T *)k, (const T *)v, idx,
                     (T *)kx, (T *)vx, rows, c.N, c.M * c.k);
  return launched("gather_kernel", st);
}

hipError_t launch_gather(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                         hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? gather_t<float, 64>(c, k, v, idx, kx, vx, st) : gather_t<float, 128>(c, k, v, idx, kx, vx, st);
  return c.d == 64 ? gather_t<bf16_t, 64>(c, k, v, idx, kx, vx, st) : gather_t<bf16_t, 128>(c, k, v, idx, kx, vx, st);
}

}  // namespace mita
