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
// transposed). Each wave forms S^T for its landmarks on MFMA and, per mode:
//  - WRITE_S: writes S = fl(dot) * scale (fp32, landmark-major);
//  - SELECT: lists the keys whose score is >= the row's pivot, in ascending
//    token order, in the (row, chunk) region of the candidate lists (score
//    bits, token index) and writes the region's count. In a tile a
//    landmark's 64 keys sit in 4 lanes (lane group g holds keys
//    16 kb + 4 g + r): per 16-key block kb, a scan over the 4 lanes of
//    per-block counts packed in bytes gives each candidate its position, and
//    a running count carries over the tiles of the chunk (no atomics);
//  - DO_V: runs an online softmax with P V on MFMA for the landmark values
//    (Eq. landmark-value: the softmax runs over the keys of each landmark);
//    per-chunk partials (running max in log2 units, running sum,
//    unnormalised accumulator) go to `partial`.
// only_lm >= 0 restricts the S write to that landmark (the arithmetic of
// every score is the same whichever rows are written).
// ---------------------------------------------------------------------------
struct SelectArgs {
  const uint32_t *plo;  // [rows] pivot keys
  uint32_t *ccnt;       // [rows, chunks] candidates listed
  uint2 *cand;          // [rows, chunks, SCORE_NC] (score bits, token index)
};

template <typename T, int D, bool WRITE_S, bool DO_V, bool SELECT>
__device__ __forceinline__ void score_chunk(T *__restrict__ Ks, T *__restrict__ Vt, const T *__restrict__ q_lm,
                                            const T *__restrict__ k, const T *__restrict__ v, float *__restrict__ S,
                                            float2 *__restrict__ part_ml, float *__restrict__ part_o,
                                            const SelectArgs &sel, int N, int M, float scale, int chunk, int nchunks,
                                            int lmblock, int64_t bh, int only_lm) {
  // Ks / Vt: two tile buffers each, K_ELEMS / V_ELEMS apart (Vt unused without DO_V)
  using TD = TileDims<T, D>;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int lm0 = (lmblock * 4 + w) * 16;
  const bool active = lm0 < M && (only_lm < 0 || (only_lm >= lm0 && only_lm < lm0 + 16));
  const int lm = lm0 + p;
  const int64_t row = bh * M + lm;
  const T *kb_ = k + bh * (int64_t)N * D;
  const T *vb_ = DO_V ? v + bh * (int64_t)N * D : nullptr;

  Frag<T> qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    if (lm < M)
      qf[ks].load(q_lm + row * D + ks * 32 + g * 8);
    else
      qf[ks].zero();
  }
  // SELECT: a score x is listed iff score_key(x) >= plo, i.e. x >= key_to_float(plo)
  // for x not NaN (the key order is the float order with -0 == +0), and for
  // NaN (ranked as -inf) iff the pivot is -inf. plo = 0xffffffff (no row)
  // gives a NaN bound that lists nothing.
  float piv = 0.f;
  bool nan_in = false;
  if (SELECT) {
    const uint32_t plo = lm < M ? sel.plo[row] : 0xffffffffu;
    piv = key_to_float(plo);
    nan_in = plo == ordered_key(-INFINITY);
  }
  const bool write_row = WRITE_S && lm < M && (only_lm < 0 || lm == only_lm);
  uint32_t listed = 0;  // SELECT: candidates of this landmark listed so far in the chunk
  // SELECT: the candidate regions of this wave's landmarks start here (the
  // wave index is uniform; readfirstlane lets the compiler keep it scalar)
  char *cand_w = nullptr;
  if (SELECT) {
    const int lmw = (lmblock * 4 + __builtin_amdgcn_readfirstlane(w)) * 16;
    cand_w = reinterpret_cast<char *>(sel.cand + ((bh * M + lmw) * nchunks + chunk) * (int64_t)SCORE_NC);
  }
  wait_loads();  // landmark fragments and pivot are in registers before the pipelined loop
  Online<D> st;
  st.init();
  const float sl2 = scale * LOG2E;
  const int key_begin = chunk * SCORE_NC, key_end = min(N, key_begin + SCORE_NC);
  const int ntile = (key_end - key_begin + TK - 1) / TK;

  // key tiles double-buffered in LDS: the next tile's loads are in flight
  // while the current one is used, one barrier per tile
  TileRegs<T, D, DO_V> R;
  R.load(kb_ + (int64_t)key_begin * D, DO_V ? vb_ + (int64_t)key_begin * D : nullptr, nullptr,
         min(TK, key_end - key_begin));
  R.store(Ks, Vt);
  __syncthreads();
  for (int t = 0; t < ntile; ++t) {
    const int buf = t & 1;
    T *Kc = Ks + buf * TD::K_ELEMS, *Vc = DO_V ? Vt + buf * TD::V_ELEMS : Vt;
    const int k0 = key_begin + t * TK;
    const int nvalid = min(TK, key_end - k0);
    if (t + 1 < ntile)
      R.load(kb_ + (int64_t)(k0 + TK) * D, DO_V ? vb_ + (int64_t)(k0 + TK) * D : nullptr, nullptr,
             min(TK, key_end - k0 - TK));
    // The tile's global stores (S or candidates) are issued after the next
    // tile's LDS store: on gfx9 one counter tracks loads and stores, so the
    // wait for the prefetched loads would otherwise also wait for them.
    f32x4 acc[4];
    uint32_t m[4] = {0u, 0u, 0u, 0u}, pos = 0u, tot = 0u;
    if (active) {
      tile_scores<T, D>(acc, Kc, qf);
      if (SELECT) {
        // per-kb candidate bits m[kb] (bit r); per-kb counts in bytes
        if (nvalid == TK && !__ballot(nan_in)) {  // full tile, no -inf pivot in the wave
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) m[kb] |= (acc[kb][r] * scale >= piv) ? 1u << r : 0u;
        } else {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float x = acc[kb][r] * scale;
              const bool c = x >= piv || (nan_in && x != x);
              if (c && kb * 16 + 4 * g + r < nvalid) m[kb] |= 1u << r;
            }
        }
        uint32_t packed = 0;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) packed |= (uint32_t)__popc(m[kb]) << (8 * kb);
        // inclusive scan over the lane groups of landmark p (bytes stay below 17)
        uint32_t incl = packed;
        uint32_t y = (uint32_t)__shfl_up((int)incl, 16);
        if (g >= 1) incl += y;
        y = (uint32_t)__shfl_up((int)incl, 32);
        if (g >= 2) incl += y;
        tot = (uint32_t)__shfl((int)incl, 48 + p);  // per-kb totals of the landmark
        // byte kb of pos: candidates of the landmark before this lane's block kb
        pos = (incl - packed) + (tot << 8) + (tot << 16) + (tot << 24);
      }
      if (DO_V) tile_softmax_pv<T, D>(st, acc, Vc, nvalid, sl2);
    }
    if (t + 1 < ntile) R.store(Ks + (buf ^ 1) * TD::K_ELEMS, DO_V ? Vt + (buf ^ 1) * TD::V_ELEMS : Vt);
    if (active && write_row) {
      float *srow = S + row * (int64_t)N + k0;
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
    if (SELECT && active) {
      // a lane's candidates of block kb take consecutive entries; addresses
      // are a 32-bit byte offset from the wave's base (its 16 landmarks'
      // regions of this chunk)
      const uint32_t lane_off = ((uint32_t)p * (uint32_t)nchunks * SCORE_NC + listed) * 8u;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if (!__ballot(m[kb] != 0u)) continue;  // no candidate of this block in the wave
        uint32_t at = lane_off + ((pos >> (8 * kb)) & 255u) * 8u;
        const uint32_t ib = (uint32_t)(k0 + kb * 16 + 4 * g);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (m[kb] & (1u << r)) {
            *reinterpret_cast<uint2 *>(cand_w + at) = make_uint2(__float_as_uint(acc[kb][r] * scale), ib + r);
            at += 8u;
          }
      }
      listed += (tot * 0x01010101u) >> 24;
    }
    __syncthreads();
  }
  if (SELECT && active && lm < M && g == 0) sel.ccnt[row * nchunks + chunk] = listed;
  if (!DO_V || !active) return;
  const float l = st.l();
  if (lm < M) {
    const int64_t prow = (bh * nchunks + chunk) * M + lm;
    if (g == 0) part_ml[prow] = make_float2(st.m, l);
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
      *reinterpret_cast<float4 *>(part_o + prow * D + db * 16 + 4 * g) =
          make_float4(st.o[db][0], st.o[db][1], st.o[db][2], st.o[db][3]);
  }
}

template <typename T, int D, bool WRITE_S, bool DO_V, bool SELECT>
__global__ __launch_bounds__(BLOCK) void scores_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                       const T *__restrict__ v, float *__restrict__ S,
                                                       float2 *__restrict__ part_ml, float *__restrict__ part_o,
                                                       SelectArgs sel, int N, int M, float scale) {
  using TD = TileDims<T, D>;
  __shared__ __align__(16) T Ks[2][TD::K_ELEMS];
  __shared__ __align__(16) T Vt[DO_V ? 2 : 1][DO_V ? TD::V_ELEMS : 1];
  score_chunk<T, D, WRITE_S, DO_V, SELECT>(&Ks[0][0], &Vt[0][0], q_lm, k, v, S, part_ml, part_o, sel, N, M, scale,
                                           blockIdx.x, gridDim.x, blockIdx.y, blockIdx.z, -1);
}

// Score rows of listed landmark rows (fallback of the fused selection): work
// item = (listed row, key chunk); each item recomputes the row's 64-landmark
// block exactly as the score pass does and writes that row only.
template <typename T, int D>
__global__ __launch_bounds__(BLOCK) void scores_rows_kernel(const T *__restrict__ q_lm, const T *__restrict__ k,
                                                            float *__restrict__ S, const uint32_t *__restrict__ nrows,
                                                            const int32_t *__restrict__ rows, int N, int M,
                                                            float scale, int nchunks) {
  using TD = TileDims<T, D>;
  __shared__ __align__(16) T Ks[2][TD::K_ELEMS];
  const int64_t items = (int64_t)*nrows * nchunks;
  const SelectArgs none{nullptr, nullptr, nullptr};
  for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
    const int row = rows[it / nchunks];
    const int chunk = (int)(it % nchunks);
    const int lm = row % M;
    __syncthreads();  // the previous item's last reads of Ks are done
    score_chunk<T, D, true, false, false>(&Ks[0][0], nullptr, q_lm, k, nullptr, S, nullptr, nullptr, none, N, M,
                                          scale, chunk, nchunks, lm / 64, row / M, lm);
  }
}

// Log-sum-exp merge of the per-chunk landmark-value partials, one workgroup
// per landmark row (the same merge, in the same order, as the fused
// selection's finish applies).
template <typename T, int D>
__global__ __launch_bounds__(256) void merge_kernel(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                                    T *__restrict__ v_lm, int M, int nchunks) {
  __shared__ float red[256 / D][3][D];
  merge_landmark_value<T, D>(part_ml, part_o, v_lm, blockIdx.y, blockIdx.x, M, nchunks, red);
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
                           void *partial, const SelectBufs *sb, hipStream_t st) {
  const int nch = score_chunks(c);
  dim3 grid(nch, (c.M + 63) / 64, (unsigned)BH(c));
  float2 *ml = (float2 *)partial;
  float *po = v_lm ? (float *)((char *)partial + align_up((size_t)BH(c) * nch * c.M * sizeof(float2))) : nullptr;
  const float sc = eff_scale(c);
  const SelectArgs sel = sb ? SelectArgs{sb->plo, sb->ccnt, sb->cand} : SelectArgs{nullptr, nullptr, nullptr};
  const T *ql = (const T *)q_lm, *kk = (const T *)k, *vv = (const T *)v;
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
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !v_lm || sb) return e;  // with sel the merge runs in the selection's finish
  hipLaunchKernelGGL((merge_kernel<T, D>), dim3((unsigned)c.M, (unsigned)BH(c)), dim3(256), 0, st, ml, po, (T *)v_lm,
                     c.M, nch);
  return hipGetLastError();
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
  return hipGetLastError();
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
  return hipGetLastError();
}

hipError_t launch_gather(const mita_cfg_t &c, const void *k, const void *v, const int32_t *idx, void *kx, void *vx,
                         hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? gather_t<float, 64>(c, k, v, idx, kx, vx, st) : gather_t<float, 128>(c, k, v, idx, kx, vx, st);
  return c.d == 64 ? gather_t<bf16_t, 64>(c, k, v, idx, kx, vx, st) : gather_t<bf16_t, 128>(c, k, v, idx, kx, vx, st);
}

}  // namespace mita
