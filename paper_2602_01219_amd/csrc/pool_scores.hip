// pool_scores.hip - landmark pooling, landmark-key scores with landmark
// values, and the expert-tile gather.
#include "cdna4.hpp"
#include "flash.hpp"
#include "kernels.hpp"
#include "check.hpp"

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
                                                   int32_t *__restrict__ zero_counts, int N, int gh, int gw, int lh,
                                                   int lw) {
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
  const int ch = threadIdx.x % CPT, slot = threadIdx.x / CPT;
  float acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  const T *base = q + bh * (int64_t)N * D;
  for (int t = slot; t < count; t += P) {
    const int r = r0 + t / cols, c = c0 + t % cols;
    const uint4 u = *reinterpret_cast<const uint4 *>(base + ((int64_t)r * gw + c) * D + ch * VE);
    float x[VE];
    unpack16(u, x, (const T *)nullptr);
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] += x[e];
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) red[slot][ch * VE + e] = acc[e];
  __syncthreads();
  if (threadIdx.x < D) {
    float s = 0.f;
    for (int j = 0; j < P; ++j) s += red[j][threadIdx.x];
    q_lm[(bh * M + i) * D + threadIdx.x] = from_f32<T>(s / (float)count);
  }
}

// ---------------------------------------------------------------------------
// Scores and landmark values. Workgroup = 4 waves x 16 landmarks over one
// chunk of SCORE_NC keys, key tiles of 64 staged in LDS (K row-major, V
// transposed). Each wave forms S^T for its landmarks on MFMA, optionally
// writes S = fl(dot) * scale (fp32, landmark-major), and runs an online
// softmax with P V on MFMA for the landmark values (Eq. landmark-value: the
// softmax runs over the keys of each landmark). Per-chunk partials (running
// max in log2 units, running sum, unnormalised accumulator) go to `partial`.
// ---------------------------------------------------------------------------
template <typename T, int D, bool WRITE_S, bool DO_V>
__global__ __launch_bounds__(BLOCK) void scores_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                       const T *__restrict__ v, float *__restrict__ S,
                                                       float2 *__restrict__ part_ml, float *__restrict__ part_o,
                                                       int N, int M, float scale) {
  using TD = TileDims<T, D>;
  __shared__ __align__(16) T Ks[TD::K_ELEMS];
  __shared__ __align__(16) T Vt[DO_V ? TD::V_ELEMS : 1];
  const int chunk = blockIdx.x, nchunks = gridDim.x;
  const int64_t bh = blockIdx.z;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int lm0 = (blockIdx.y * 4 + w) * 16;
  const bool active = lm0 < M;
  const int lm = lm0 + p;
  const T *kb_ = k + bh * (int64_t)N * D;
  const T *vb_ = v + bh * (int64_t)N * D;

  Frag<T> qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    if (lm < M)
      qf[ks].load(q_lm + (bh * M + lm) * D + ks * 32 + g * 8);
    else
      qf[ks].zero();
  }
  Online<D> st;
  st.init();
  const float sl2 = scale * LOG2E;
  const int key_begin = chunk * SCORE_NC, key_end = min(N, key_begin + SCORE_NC);
  for (int k0 = key_begin; k0 < key_end; k0 += TK) {
    const int nvalid = min(TK, key_end - k0);
    __syncthreads();
    load_kv_tile<T, D, DO_V>(Ks, Vt, kb_ + (int64_t)k0 * D, vb_ + (int64_t)k0 * D, nullptr, nvalid);
    __syncthreads();
    if (!active) continue;
    f32x4 acc[4];
    tile_scores<T, D>(acc, Ks, qf);
    if (WRITE_S && lm < M) {
      float *srow = S + (bh * M + lm) * (int64_t)N + k0;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int key = kb * 16 + 4 * g;
        if (key + 3 < nvalid) {
          *reinterpret_cast<float4 *>(srow + key) =
              make_float4(acc[kb][0] * scale, acc[kb][1] * scale, acc[kb][2] * scale, acc[kb][3] * scale);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (key + r < nvalid) srow[key + r] = acc[kb][r] * scale;
        }
      }
    }
    if (DO_V) tile_softmax_pv<T, D>(st, acc, Vt, nvalid, sl2);
  }
  if (!DO_V || !active) return;
  const float l = column_sum(st.l);
  if (lm < M) {
    const int64_t row = (bh * nchunks + chunk) * M + lm;
    if (g == 0) part_ml[row] = make_float2(st.m, l);
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
      *reinterpret_cast<float4 *>(part_o + row * D + db * 16 + 4 * g) =
          make_float4(st.o[db][0], st.o[db][1], st.o[db][2], st.o[db][3]);
  }
}

// Log-sum-exp merge of the per-chunk landmark-value partials (online softmax
// across chunks, in one pass: the loads do not depend on the running state,
// so they stay in flight). 256 threads = 256 / D landmarks x D dimensions.
template <typename T, int D>
__global__ __launch_bounds__(256) void merge_kernel(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                                    T *__restrict__ v_lm, int M, int nchunks) {
  constexpr int LPB = 256 / D;
  const int lm = blockIdx.x * LPB + threadIdx.x / D, dim = threadIdx.x % D;
  const int64_t bh = blockIdx.y;
  if (lm >= M) return;
  float mx = -INFINITY, L = 0.f, acc = 0.f;
#pragma unroll 8
  for (int c = 0; c < nchunks; ++c) {
    const int64_t row = (bh * nchunks + c) * M + lm;
    const float2 ml = part_ml[row];
    const float o = part_o[row * D + dim];
    const float m_new = fmaxf(mx, ml.x);
    const float a = __builtin_amdgcn_exp2f(mx - m_new), b = __builtin_amdgcn_exp2f(ml.x - m_new);
    L = L * a + ml.y * b;
    acc = acc * a + o * b;
    mx = m_new;
  }
  v_lm[(bh * M + lm) * D + dim] = from_f32<T>(acc / L);
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
static hipError_t pool_t(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *zc, hipStream_t st) {
  dim3 grid(c.M, (unsigned)BH(c));
  hipLaunchKernelGGL((pool_kernel<T, D>), grid, dim3(256), 0, st, (const T *)q, (T *)q_lm, zc, c.N, c.grid_h,
                     c.grid_w, c.lm_h, c.lm_w);
  return hipGetLastError();
}

hipError_t launch_pool(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *zc, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? pool_t<float, 64>(c, q, q_lm, zc, st) : pool_t<float, 128>(c, q, q_lm, zc, st);
  return c.d == 64 ? pool_t<bf16_t, 64>(c, q, q_lm, zc, st) : pool_t<bf16_t, 128>(c, q, q_lm, zc, st);
}

__global__ __launch_bounds__(256) void zero_kernel(int32_t *__restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

hipError_t launch_zero(int32_t *p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t scores_t(const mita_cfg_t &c, const void *q_lm, const void *k, const void *v, float *S, void *v_lm,
                           void *partial, hipStream_t st) {
  const int nch = score_chunks(c);
  dim3 grid(nch, (c.M + 63) / 64, (unsigned)BH(c));
  float2 *ml = (float2 *)partial;
  float *po = (float *)((char *)partial + align_up((size_t)BH(c) * nch * c.M * sizeof(float2)));
  const float sc = eff_scale(c);
  if (S && v_lm)
    hipLaunchKernelGGL((scores_kernel<T, D, true, true>), grid, dim3(BLOCK), 0, st, (const T *)q_lm, (const T *)k,
                       (const T *)v, S, ml, po, c.N, c.M, sc);
  else if (S)
    hipLaunchKernelGGL((scores_kernel<T, D, true, false>), grid, dim3(BLOCK), 0, st, (const T *)q_lm, (const T *)k,
                       (const T *)v, S, ml, po, c.N, c.M, sc);
  else if (v_lm)
    hipLaunchKernelGGL((scores_kernel<T, D, false, true>), grid, dim3(BLOCK), 0, st, (const T *)q_lm, (const T *)k,
                       (const T *)v, S, ml, po, c.N, c.M, sc);
  else
    return hipSuccess;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !v_lm) return e;
  constexpr int LPB = 256 / D;
  hipLaunchKernelGGL((merge_kernel<T, D>), dim3((c.M + LPB - 1) / LPB, (unsigned)BH(c)), dim3(256), 0, st, ml, po,
                     (T *)v_lm, c.M, nch);
  return hipGetLastError();
}

hipError_t launch_scores(const mita_cfg_t &c, const void *q_lm, const void *k, const void *v, float *S, void *v_lm,
                         void *partial, hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? scores_t<float, 64>(c, q_lm, k, v, S, v_lm, partial, st)
                     : scores_t<float, 128>(c, q_lm, k, v, S, v_lm, partial, st);
  return c.d == 64 ? scores_t<bf16_t, 64>(c, q_lm, k, v, S, v_lm, partial, st)
                   : scores_t<bf16_t, 128>(c, q_lm, k, v, S, v_lm, partial, st);
}

template <typename T, int D>
static hipError_t gather_t(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                           hipStream_t st) {
  constexpr int CPR = D / (16 / (int)sizeof(T));
  const int64_t rows = BH(c) * c.M * (int64_t)c.k;
  const int64_t blocks = (rows * CPR + 255) / 256;
  hipLaunchKernelGGL((gather_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, st, (const T *)k, (const T *)v, idx,
                     (T *)kx, (T *)vx, rows, c.N, c.M * c.k);
  return hipGetLastError();
}

hipError_t launch_gather(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                         hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? gather_t<float, 64>(c, k, v, idx, kx, vx, st) : gather_t<float, 128>(c, k, v, idx, kx, vx, st);
  return c.d == 64 ? gather_t<bf16_t, 64>(c, k, v, idx, kx, vx, st) : gather_t<bf16_t, 128>(c, k, v, idx, kx, vx, st);
}

}  // namespace mita
