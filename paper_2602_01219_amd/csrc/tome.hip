// tome.hip - token merging as landmark extraction (Tab. A1 lists ToMe among
// the landmark extractions; bipartite soft matching, applied in rounds until
// M tokens remain).
//
// A round over the current sequence of n merged tokens (each the mean of its
// original tokens' queries, in sequence order):
//   1. A = the tokens at even positions, B = those at odd positions;
//   2. each A token's match is the B token of largest cosine similarity
//      (lower B position on ties), its edge score that similarity;
//   3. the r = min(n - M, |A|) edges of largest score (lower A position on
//      ties) merge: each of those A tokens joins its match;
//   4. the survivors (unmerged A tokens and all B tokens) keep their order.
// The landmarks are the final tokens' means, in sequence order.
//
// The member sums of the current tokens are kept in 64-bit fixed point
// (2^-32 units): merging adds them with integer atomic adds, which give the
// same sums in any order, so every round's decisions (and the landmarks) do
// not depend on the order in which the hardware runs the adds. Similarities
// are fp32 dot products (MFMA) of the fp32 unit vectors of the sums.
#include <utility>

#include "cdna4.hpp"
#include "check.hpp"
#include "flash.hpp"
#include "kernels.hpp"

namespace mita {

constexpr double TOME_ONE = 4294967296.0;  // fixed-point unit of the member sums

// Fixed-point value of x (rounded to nearest; |x| must stay below 2^31 per sum).
__device__ __forceinline__ int64_t tome_fix(float x) { return (int64_t)__double2ll_rn((double)x * TOME_ONE); }

template <typename T>
__global__ __launch_bounds__(256) void tome_init_kernel(const T *__restrict__ q, int64_t *__restrict__ S,
                                                        int32_t *__restrict__ cnt, int32_t *__restrict__ rep,
                                                        int64_t rows, int D, int N) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rows * D) return;
  S[t] = tome_fix(to_f32<T>(q[t]));
  if (t % D == 0) {
    const int64_t row = t / D;
    cnt[row] = 1;
    rep[row] = (int32_t)(row % N);
  }
}

// Unit vectors of the current tokens' sums (fp32; a zero sum gives zeros).
// One wave per row.
template <int D>
__global__ __launch_bounds__(256) void tome_norm_kernel(const int64_t *__restrict__ S, float *__restrict__ X, int n,
                                                        int N, int64_t rows) {
  constexpr int PER = D / 64;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t bh = r / n, j = r % n;
  const int64_t *src = S + (bh * N + j) * D;
  double v[PER], ss = 0.0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    v[i] = (double)src[lane + 64 * i];
    ss += v[i] * v[i];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  const double inv = ss > 0.0 ? 1.0 / sqrt(ss) : 0.0;
  float *dst = X + (bh * N + j) * D;
#pragma unroll
  for (int i = 0; i < PER; ++i) dst[lane + 64 * i] = (float)(v[i] * inv);
}

// Each A token's best B token: A row a is X row 2a, B row b is X row 2b + 1.
// Workgroup = 4 waves, wave = 64 A rows (4 column groups of 16); the B rows
// are staged in LDS 64 at a time and scored on MFMA (S^T = B A^T); each lane
// keeps a running (max, argmax) with strict '>' in increasing b, then the four
// lane groups of a column merge, preferring the lower b on equal values.
template <int D>
__global__ __launch_bounds__(256) void tome_match_kernel(const float *__restrict__ X, float *__restrict__ score,
                                                         int32_t *__restrict__ match, int n, int N, int nA_tiles) {
  constexpr int LSTR = D + 4;
  __shared__ __align__(16) float lms[64 * LSTR];
  const int64_t bh = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int tile = blockIdx.x * 4 + w;
  const int nA = (n + 1) / 2, nB = n / 2;
  const float *Xb = X + bh * (int64_t)N * D;
  Frag<float> af[4][D / 32];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int a = tile * 64 + c * 16 + p;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (tile < nA_tiles && a < nA)
        af[c][ks].load(Xb + (int64_t)(2 * a) * D + ks * 32 + g * 8);
      else
        af[c][ks].zero();
    }
  }
  float best[4];
  int arg[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    best[c] = -INFINITY;
    arg[c] = 0;
  }
  for (int b0 = 0; b0 < nB; b0 += 64) {
    const int nl = min(64, nB - b0);
    __syncthreads();
    for (int ch = threadIdx.x; ch < 64 * (D / 4); ch += 256) {
      const int r = ch / (D / 4), cc = ch % (D / 4);
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (r < nl) x = *reinterpret_cast<const float4 *>(Xb + (int64_t)(2 * (b0 + r) + 1) * D + cc * 4);
      *reinterpret_cast<float4 *>(lms + r * LSTR + cc * 4) = x;
    }
    __syncthreads();
    if (tile >= nA_tiles) continue;
    for (int sb = 0; sb < nl; sb += 16) {
      f32x4 acc[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<float> bf;
        bf.load(lms + (sb + p) * LSTR + ks * 32 + g * 8);
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = mma(bf, af[c][ks], acc[c]);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int b = b0 + sb + 4 * g + r;
          const float val = acc[c][r];
          const bool up = sb + 4 * g + r < nl && val > best[c];
          best[c] = up ? val : best[c];
          arg[c] = up ? b : arg[c];
        }
    }
  }
  if (tile >= nA_tiles) return;  // no workgroup barriers below
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
    const int a = tile * 64 + c * 16 + p;
    if (g == 0 && a < nA) {
      score[bh * nA + a] = best[c];
      match[bh * nA + a] = arg[c];
    }
  }
}

// merged[a] = 1 for the r selected A tokens (zeroed beforehand)
__global__ __launch_bounds__(256) void tome_flag_kernel(const int32_t *__restrict__ sel, int32_t *__restrict__ merged,
                                                        int r, int nA, int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t bh = t / r;
  merged[bh * nA + sel[t]] = 1;
}

// alive[j] = 1 for the survivors of the round
__global__ __launch_bounds__(256) void tome_alive_kernel(const int32_t *__restrict__ merged, int32_t *__restrict__ alive,
                                                         int n, int nA, int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t bh = t / n;
  const int j = (int)(t % n);
  alive[t] = (j & 1) || !merged[bh * nA + j / 2] ? 1 : 0;
}

// survivors' sums and counts to their new positions
__global__ __launch_bounds__(256) void tome_copy_kernel(const int64_t *__restrict__ S, const int32_t *__restrict__ cnt,
                                                        const int32_t *__restrict__ alive,
                                                        const int32_t *__restrict__ pos, int64_t *__restrict__ S2,
                                                        int32_t *__restrict__ cnt2, int n, int N, int D,
                                                        int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t row = t / D;
  const int dd = (int)(t % D);
  const int64_t bh = row / n;
  const int j = (int)(row % n);
  if (!alive[bh * n + j]) return;
  const int np = pos[bh * (n + 1) + j];
  S2[(bh * N + np) * D + dd] = S[(bh * N + j) * D + dd];
  if (dd == 0) cnt2[bh * N + np] = cnt[bh * N + j];
}

// each merged A token's sums and count added to its match's new row
// (integer adds: the result does not depend on their order)
__global__ __launch_bounds__(256) void tome_add_kernel(const int64_t *__restrict__ S, const int32_t *__restrict__ cnt,
                                                       const int32_t *__restrict__ sel,
                                                       const int32_t *__restrict__ match,
                                                       const int32_t *__restrict__ pos, int64_t *__restrict__ S2,
                                                       int32_t *__restrict__ cnt2, int r, int n, int nA, int N, int D,
                                                       int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t e = t / D;
  const int dd = (int)(t % D);
  const int64_t bh = e / r;
  const int a = sel[e];
  const int jb = 2 * match[bh * nA + a] + 1;
  const int np = pos[bh * (n + 1) + jb];
  atomicAdd(reinterpret_cast<unsigned long long *>(S2 + (bh * N + np) * D + dd),
            (unsigned long long)S[(bh * N + 2 * a) * D + dd]);
  if (dd == 0) atomicAdd(cnt2 + bh * N + np, cnt[bh * N + 2 * a]);
}

// every original token's current position
__global__ __launch_bounds__(256) void tome_rep_kernel(const int32_t *__restrict__ rep,
                                                       const int32_t *__restrict__ merged,
                                                       const int32_t *__restrict__ match,
                                                       const int32_t *__restrict__ pos, int32_t *__restrict__ rep2,
                                                       int n, int nA, int N, int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t bh = t / N;
  int j = rep[t];
  if (!(j & 1) && merged[bh * nA + j / 2]) j = 2 * match[bh * nA + j / 2] + 1;
  rep2[t] = pos[bh * (n + 1) + j];
}

// landmarks: the means of the final tokens
template <typename T>
__global__ __launch_bounds__(256) void tome_out_kernel(const int64_t *__restrict__ S, const int32_t *__restrict__ cnt,
                                                       T *__restrict__ q_lm, int M, int N, int D, int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t row = t / D;
  const int dd = (int)(t % D);
  const int64_t bh = row / M;
  const int i = (int)(row % M);
  const double v = (double)S[(bh * N + i) * D + dd] / TOME_ONE / (double)cnt[bh * N + i];
  q_lm[t] = from_f32<T>((float)v);
}

static unsigned blocks(int64_t n) { return (unsigned)((n + 255) / 256); }

template <typename T, int D>
static hipError_t tome_t(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *assign, const TomeBufs &b,
                         hipStream_t st) {
  const int N = c.N, M = c.M;
  const int64_t bh = BH(c);
  hipError_t err;
  int64_t *S = b.S[0], *S2 = b.S[1];
  int32_t *cnt = b.cnt[0], *cnt2 = b.cnt[1], *rep = b.rep[0], *rep2 = b.rep[1];
  hipLaunchKernelGGL((tome_init_kernel<T>), dim3(blocks(bh * N * D)), dim3(256), 0, st, (const T *)q, S, cnt, rep,
                     bh * N, D, N);
  if ((err = launched("tome_init_kernel", st)) != hipSuccess) return err;
  int n = N;
  while (n > M) {
    const int nA = (n + 1) / 2;
    const int r = min(n - M, nA);
    hipLaunchKernelGGL((tome_norm_kernel<D>), dim3((unsigned)((bh * n + 3) / 4)), dim3(256), 0, st, S, b.X, n, N,
                       bh * n);
    if ((err = launched("tome_norm_kernel", st)) != hipSuccess) return err;
    const int nat = (nA + 63) / 64;
    hipLaunchKernelGGL((tome_match_kernel<D>), dim3((unsigned)((nat + 3) / 4), (unsigned)bh), dim3(256), 0, st, b.X,
                       b.score, b.match, n, N, nat);
    if ((err = launched("tome_match_kernel", st)) != hipSuccess) return err;
    // the r best edges: exact top-r of each head's nA scores (ties: lower A position)
    mita_cfg_t tc = c;
    tc.N = nA;
    tc.M = 1;
    tc.k = r;
    if ((err = launch_topk(tc, b.score, b.sel, st)) != hipSuccess) return err;
    if ((err = launch_zero(b.merged, bh * nA, st)) != hipSuccess) return err;
    hipLaunchKernelGGL(tome_flag_kernel, dim3(blocks(bh * r)), dim3(256), 0, st, b.sel, b.merged, r, nA, bh * r);
    if ((err = launched("tome_flag_kernel", st)) != hipSuccess) return err;
    hipLaunchKernelGGL(tome_alive_kernel, dim3(blocks(bh * n)), dim3(256), 0, st, b.merged, b.alive, n, nA, bh * n);
    if ((err = launched("tome_alive_kernel", st)) != hipSuccess) return err;
    if ((err = launch_scan_counts(b.alive, b.pos, n, bh, st)) != hipSuccess) return err;
    hipLaunchKernelGGL(tome_copy_kernel, dim3(blocks(bh * n * D)), dim3(256), 0, st, S, cnt, b.alive, b.pos, S2, cnt2,
                       n, N, D, bh * n * D);
    if ((err = launched("tome_copy_kernel", st)) != hipSuccess) return err;
    hipLaunchKernelGGL(tome_add_kernel, dim3(blocks(bh * r * D)), dim3(256), 0, st, S, cnt, b.sel, b.match, b.pos, S2,
                       cnt2, r, n, nA, N, D, bh * r * D);
    if ((err = launched("tome_add_kernel", st)) != hipSuccess) return err;
    hipLaunchKernelGGL(tome_rep_kernel, dim3(blocks(bh * N)), dim3(256), 0, st, rep, b.merged, b.match, b.pos, rep2, n,
                       nA, N, bh * N);
    if ((err = launched("tome_rep_kernel", st)) != hipSuccess) return err;
    std::swap(S, S2);
    std::swap(cnt, cnt2);
    std::swap(rep, rep2);
    n -= r;
  }
  hipLaunchKernelGGL((tome_out_kernel<T>), dim3(blocks(bh * M * D)), dim3(256), 0, st, S, cnt, (T *)q_lm, M, N, D,
                     bh * M * D);
  if ((err = launched("tome_out_kernel", st)) != hipSuccess) return err;
  if (assign) {
    err = hipMemcpyAsync(assign, rep, (size_t)bh * N * sizeof(int32_t), hipMemcpyDeviceToDevice, st);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

hipError_t launch_tome(const mita_cfg_t &c, const void *q, void *q_lm, int32_t *assign, const TomeBufs &b,
                       hipStream_t st) {
  if (c.dtype == MITA_F32)
    return c.d == 64 ? tome_t<float, 64>(c, q, q_lm, assign, b, st) : tome_t<float, 128>(c, q, q_lm, assign, b, st);
  return c.d == 64 ? tome_t<bf16_t, 64>(c, q, q_lm, assign, b, st) : tome_t<bf16_t, 128>(c, q, q_lm, assign, b, st);
}

}  // namespace mita
