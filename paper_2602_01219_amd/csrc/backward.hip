// backward.hip - gradients of the MiTA forward with respect to q, k, v, the
// top-k sets and the routing held fixed (they are piecewise constant in the
// inputs): the attention of Eq. mita, the landmark values of Eq.
// landmark-value (itself an attention of the landmark queries over all keys)
// and the pooling of the landmark queries.
//
// Both attentions take the same kernel, bwd_kernel, in one of two modes:
//   ATT: a workgroup takes one tile of the forward's work list (64 queries
//        of one expert); its keys are the shared landmarks (keys q_lm,
//        values v_lm) and the expert's k routed rows. A first pass over the
//        keys forms each query's log-sum-exp, a second one the gradients:
//        dQ stays in registers (a query's keys are all seen here) and is
//        written once; dK and dV of each key tile, summed over the 64
//        queries, go by fp32 atomic adds to the keys' rows (token rows for
//        routed keys, landmark rows for shared ones).
//   LMV: a workgroup takes 64 landmarks (as queries) and one chunk of the
//        N keys; the upstream gradient is that of the landmark values, the
//        log-sum-exp of each landmark row comes from the score pass. dQ (the
//        landmark queries' gradient) is a partial sum over the chunk and is
//        added atomically.
// Per key tile of 32 keys, with P = softmax weights and dO the upstream
// gradient of the queries' outputs:
//   S^T = K Q^T, dP^T = V dO^T                      (keys x queries)
//   P = exp2(S^T * scale * log2 e - lse), dZ = P (dP - D), D = dO . o
//   dQ += dZ K,  dK += dZ^T Q,  dV += P^T dO        (scale applied at the end)
// All products run on MFMA (16x16 tiles over 32-long reduction steps) from
// LDS copies laid out so that every operand is read as 8 consecutive
// elements: Q and dO row-major (and, for bf16 at d = 64, transposed; else
// their columns are read element by element), the key tile row-major and
// transposed, P and dZ as [key][query] and dZ as [query][key].
// Summation orders of the atomic adds vary from run to run, so the key-side
// gradients are not bitwise reproducible (the rounding differs by a few ulp).
#include "cdna4.hpp"
#include "check.hpp"
#include "flash.hpp"
#include "kernels.hpp"
#include "worklist.hpp"

namespace mita {

constexpr int BWD_TQ = 64;  // queries per workgroup
constexpr int BWD_TK = 32;  // keys per tile
constexpr int BWD_CHUNK = 512;  // keys per workgroup of the landmark-value backward

template <typename T, int D> struct BwdLds {
  static constexpr int PAD = 16 / (int)sizeof(T);
  static constexpr bool TRANS = sizeof(T) == 2 && D == 64;  // transposed copies of Q and dO
  static constexpr int QS = D + PAD;        // [query][d]
  static constexpr int TS = BWD_TQ + PAD;   // [d][query]
  static constexpr int KS = D + PAD;        // [key][d]
  static constexpr int KTS = BWD_TK + PAD;  // [d][key]
  static constexpr int PS = BWD_TQ + PAD;   // [key][query]
  static constexpr int ZS = BWD_TK + PAD;   // [query][key]
  static constexpr int NQ = BWD_TQ * QS, NQT = TRANS ? D * TS : 1, NK = BWD_TK * KS, NKT = D * KTS,
                       NP = BWD_TK * PS, NZ = BWD_TQ * ZS;
};

// 8 elements base[(r0 + i) * stride + col], i < 8 (a column of a row-major tile).
template <typename T> __device__ __forceinline__ Frag<T> load_col(const T *base, int stride, int r0, int col);
template <> __device__ __forceinline__ Frag<bf16_t> load_col(const bf16_t *base, int stride, int r0, int col) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)base[(r0 + 2 * i) * stride + col].bits | ((uint32_t)base[(r0 + 2 * i + 1) * stride + col].bits << 16);
  Frag<bf16_t> f;
  f.v = make_uint4(w[0], w[1], w[2], w[3]);
  return f;
}
template <> __device__ __forceinline__ Frag<float> load_col(const float *base, int stride, int r0, int col) {
  Frag<float> f;
  f.a = make_float4(base[r0 * stride + col], base[(r0 + 1) * stride + col], base[(r0 + 2) * stride + col],
                    base[(r0 + 3) * stride + col]);
  f.b = make_float4(base[(r0 + 4) * stride + col], base[(r0 + 5) * stride + col], base[(r0 + 6) * stride + col],
                    base[(r0 + 7) * stride + col]);
  return f;
}

// 16 bytes of T at p as VE floats.
template <typename T> __device__ __forceinline__ void load16_f32(const T *p, float *x) {
  unpack16(*reinterpret_cast<const uint4 *>(p), x, p);
}

// Arguments of bwd_kernel (both modes).
struct BwdArgs {
  const void *q, *k, *v, *o, *dO;  // [BH, N, d] (io type)
  const void *q_lm, *v_lm;         // [BH, M, d] (io type)
  const int32_t *idx, *perm, *offsets, *tile_start;
  const float *lse_lm;     // [BH, M] landmark rows' log-sum-exp, log2 units (LMV)
  const float *dv_lm;      // [BH, M, d] gradient of the landmark values (LMV input)
  float *dq;               // [BH, N, d] ATT: the queries' direct gradient (written)
  float *dk, *dv;          // [BH, N, d] accumulators (atomic adds)
  float *dq_lm, *dv_lm_out;  // [BH, M, d] accumulators (atomic adds)
  int N, M, topk, chunk;
  float scale;
};

constexpr int BWD_ATT = 0, BWD_LMV = 1;

template <typename T, int D, int MODE, bool SHARED, bool ROUTED>
__global__ __launch_bounds__(256) void bwd_kernel(BwdArgs a) {
  using L = BwdLds<T, D>;
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr bool TRANS = L::TRANS;
  __shared__ __align__(16) T Qs[L::NQ];
  __shared__ __align__(16) T dOs[L::NQ];
  __shared__ __align__(16) T QT[L::NQT];
  __shared__ __align__(16) T dOT[L::NQT];
  __shared__ __align__(16) T Ks[L::NK];
  __shared__ __align__(16) T Vs[L::NK];
  __shared__ __align__(16) T KT[L::NKT];
  __shared__ __align__(16) T Pkq[L::NP];
  __shared__ __align__(16) T Zkq[L::NP];
  __shared__ __align__(16) T Zqk[L::NZ];
  __shared__ float Dq[BWD_TQ];
  __shared__ int32_t qrow[BWD_TQ];  // each query's row in its tensor (token or landmark), -1 if none
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 4, p = lane & 15;
  const int N = a.N, M = a.M, K = a.topk;
  const T *q = (const T *)a.q, *kk = (const T *)a.k, *vv = (const T *)a.v;
  const T *q_lm = (const T *)a.q_lm, *v_lm = (const T *)a.v_lm;

  // ---------------------------------------------------------------- queries
  int e = 0, q_begin = 0, q_end = 0, c0 = 0, c1 = 0;
  if (MODE == BWD_ATT) {
    if (!attend_queries<ROUTED>(a.tile_start, a.offsets, bh, N, M, e, q_begin, q_end)) return;  // uniform
  } else {
    const int nlb = (M + BWD_TQ - 1) / BWD_TQ;
    const int lb = (int)blockIdx.x % nlb, ch = (int)blockIdx.x / nlb;
    q_begin = lb * BWD_TQ;
    q_end = min(M, q_begin + BWD_TQ);
    c0 = ch * a.chunk;
    c1 = min(N, c0 + a.chunk);
    if (c0 >= N) return;
  }
  if (tid < BWD_TQ) {
    const int qi = q_begin + tid;
    int r = -1;
    if (qi < q_end) r = MODE == BWD_ATT ? (ROUTED ? a.perm[bh * N + qi] : qi) : qi;
    qrow[tid] = r;
  }
  __syncthreads();
  // Q and dO rows (zero for missing queries), their transposes, and D = dO . o
  {
    const T *qsrc = MODE == BWD_ATT ? q + bh * (int64_t)N * D : q_lm + bh * (int64_t)M * D;
    for (int c = tid; c < BWD_TQ * (D / VE); c += 256) {
      const int row = c / (D / VE), cc = c % (D / VE);
      const int r = qrow[row];
      uint4 xq = make_uint4(0, 0, 0, 0), xd = make_uint4(0, 0, 0, 0);
      if (r >= 0) {
        xq = *reinterpret_cast<const uint4 *>(qsrc + (int64_t)r * D + cc * VE);
        if (MODE == BWD_ATT) {
          xd = *reinterpret_cast<const uint4 *>((const T *)a.dO + (bh * N + r) * D + cc * VE);
        } else {
          float f[VE];
          const float *src = a.dv_lm + (bh * M + r) * D + cc * VE;
#pragma unroll
          for (int i = 0; i < VE; ++i) f[i] = src[i];
          T t[VE];
#pragma unroll
          for (int i = 0; i < VE; ++i) t[i] = from_f32<T>(f[i]);
          xd = *reinterpret_cast<const uint4 *>(t);
        }
      }
      *reinterpret_cast<uint4 *>(Qs + row * L::QS + cc * VE) = xq;
      *reinterpret_cast<uint4 *>(dOs + row * L::QS + cc * VE) = xd;
      if constexpr (TRANS) {
        const T *tq = reinterpret_cast<const T *>(&xq), *td = reinterpret_cast<const T *>(&xd);
#pragma unroll
        for (int i = 0; i < VE; ++i) {
          QT[(cc * VE + i) * L::TS + row] = tq[i];
          dOT[(cc * VE + i) * L::TS + row] = td[i];
        }
      }
    }
    // D: four threads per query, D / 4 dimensions each, in fp32 (the upstream
    // gradient of the landmark values in its own fp32)
    const int row = tid >> 2, part = tid & 3;
    const int r = qrow[row];
    float dsum = 0.f;
    if (r >= 0) {
#pragma unroll
      for (int c = 0; c < D / 4; c += VE) {
        const int dim = part * (D / 4) + c;
        float ov[VE], dv[VE];
        if (MODE == BWD_ATT) {
          load16_f32((const T *)a.o + (bh * N + r) * D + dim, ov);
          load16_f32((const T *)a.dO + (bh * N + r) * D + dim, dv);
        } else {
          load16_f32(v_lm + (bh * M + r) * D + dim, ov);
#pragma unroll
          for (int i = 0; i < VE; ++i) dv[i] = a.dv_lm[(bh * M + r) * D + dim + i];
        }
#pragma unroll
        for (int i = 0; i < VE; ++i) dsum = __builtin_fmaf(ov[i], dv[i], dsum);
      }
    }
    dsum += __shfl_xor(dsum, 1);
    dsum += __shfl_xor(dsum, 2);
    if (part == 0) Dq[row] = dsum;
  }
  __syncthreads();

  // ---------------------------------------------------------------- keys
  // tiles: [0, nA) shared (landmark rows), [nA, nA + nB) routed / chunk rows
  const int nA = MODE == BWD_ATT && SHARED ? (M + BWD_TK - 1) / BWD_TK : 0;
  const int nkB = MODE == BWD_ATT ? (ROUTED ? K : 0) : c1 - c0;
  const int nB = (nkB + BWD_TK - 1) / BWD_TK;
  const int ntile = nA + nB;
  const int32_t *gidx = MODE == BWD_ATT && ROUTED ? a.idx + (bh * M + e) * (int64_t)K : nullptr;
  // row of key j of tile i in its tensor; rows >= nr are padding
  auto key_row = [&](int i, int j, bool &shared_key, int &nr) -> int {
    shared_key = i < nA;
    if (shared_key) {
      nr = min(BWD_TK, M - i * BWD_TK);
      return i * BWD_TK + j;
    }
    const int b0 = (i - nA) * BWD_TK;
    nr = min(BWD_TK, nkB - b0);
    if (MODE == BWD_ATT) return j < nr ? gidx[b0 + j] : 0;
    return c0 + b0 + j;
  };
  // stage key tile i: K rows (and V rows and K^T when full)
  auto stage = [&](int i, bool with_v) {
    for (int c = tid; c < BWD_TK * (D / VE); c += 256) {
      const int j = c / (D / VE), cc = c % (D / VE);
      bool sk;
      int nr;
      const int r = key_row(i, j, sk, nr);
      uint4 xk = make_uint4(0, 0, 0, 0), xv = make_uint4(0, 0, 0, 0);
      if (j < nr) {
        const T *kb = sk ? q_lm + bh * (int64_t)M * D : kk + bh * (int64_t)N * D;
        const T *vb = sk ? v_lm + bh * (int64_t)M * D : vv + bh * (int64_t)N * D;
        xk = *reinterpret_cast<const uint4 *>(kb + (int64_t)r * D + cc * VE);
        if (with_v) xv = *reinterpret_cast<const uint4 *>(vb + (int64_t)r * D + cc * VE);
      }
      *reinterpret_cast<uint4 *>(Ks + j * L::KS + cc * VE) = xk;
      if (with_v) {
        *reinterpret_cast<uint4 *>(Vs + j * L::KS + cc * VE) = xv;
        const T *tk = reinterpret_cast<const T *>(&xk);
#pragma unroll
        for (int u = 0; u < VE; ++u) KT[(cc * VE + u) * L::KTS + j] = tk[u];
      }
    }
  };
  const float sl2 = a.scale * LOG2E;
  const int myq = 16 * w + p;  // this lane's query (column of the S^T blocks)
  const bool qok = qrow[myq] >= 0;
  // S^T blocks of the wave's 16 queries against the tile's 32 keys
  auto scores = [&](f32x4 (&s)[2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<T> A, B;
        A.load(Ks + (16 * kb + p) * L::KS + 32 * ks + 8 * g);
        B.load(Qs + myq * L::QS + 32 * ks + 8 * g);
        s[kb] = mma(A, B, s[kb]);
      }
    }
  };

  // ---------------------------------------------------------------- pass 1: lse
  float lse;
  if (MODE == BWD_ATT) {
    float m = -INFINITY, l = 0.f;
    for (int i = 0; i < ntile; ++i) {
      __syncthreads();
      stage(i, false);
      __syncthreads();
      bool sk;
      int nr;
      key_row(i, 0, sk, nr);
      f32x4 s[2];
      scores(s);
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx = 16 * kb + 4 * g + r < nr ? fmaxf(mx, s[kb][r] * sl2) : mx;
      const float mn = fmaxf(m, mx);
      float add = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          add += 16 * kb + 4 * g + r < nr ? __builtin_amdgcn_exp2f(s[kb][r] * sl2 - mn) : 0.f;
      l = (mn == -INFINITY ? 0.f : l * __builtin_amdgcn_exp2f(m - mn)) + add;
      m = mn;
    }
    // merge the four lane groups of the query's column
    const float mc = max_lane_groups(m);
    float lc = m == -INFINITY ? 0.f : l * __builtin_amdgcn_exp2f(m - mc);
    lc += __shfl_xor(lc, 16);
    lc += __shfl_xor(lc, 32);
    lse = mc + __log2f(lc);
  } else {
    lse = qok ? a.lse_lm[bh * M + q_begin + myq] : 0.f;
  }
  const float dq_row = Dq[myq];

  // ---------------------------------------------------------------- pass 2: gradients
  f32x4 dqa[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) dqa[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int NBLK = D / 16;  // dK / dV blocks per wave (D / 4 over the workgroup)
  for (int i = 0; i < ntile; ++i) {
    __syncthreads();
    stage(i, true);
    __syncthreads();
    bool sk;
    int nr;
    key_row(i, 0, sk, nr);
    f32x4 s[2], dp[2];
    scores(s);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      dp[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<T> A, B;
        A.load(Vs + (16 * kb + p) * L::KS + 32 * ks + 8 * g);
        B.load(dOs + myq * L::QS + 32 * ks + 8 * g);
        dp[kb] = mma(A, B, dp[kb]);
      }
    }
    // P and dZ of (key 16 kb + 4 g + r, query myq)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float pz[4], zz[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 16 * kb + 4 * g + r;
        const bool ok = qok && key < nr;
        const float pr = ok ? __builtin_amdgcn_exp2f(s[kb][r] * sl2 - lse) : 0.f;
        pz[r] = pr;
        zz[r] = pr * (dp[kb][r] - dq_row);
        Pkq[key * L::PS + myq] = from_f32<T>(pz[r]);
        Zkq[key * L::PS + myq] = from_f32<T>(zz[r]);
      }
      T z4[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) z4[r] = from_f32<T>(zz[r]);
      T *dst = Zqk + myq * L::ZS + 16 * kb + 4 * g;
      if (sizeof(T) == 2)
        *reinterpret_cast<uint2 *>(dst) = *reinterpret_cast<const uint2 *>(z4);
      else
        *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(z4);
    }
    __syncthreads();
    // dQ (queries 16 w + 4 g + r, dims 16 db + p) += dZ K over the tile's 32 keys
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      Frag<T> A, B;
      A.load(Zqk + myq * L::ZS + 8 * g);
      B.load(KT + (16 * db + p) * L::KTS + 8 * g);
      dqa[db] = mma(A, B, dqa[db]);
    }
    // dK = dZ^T Q and dV = P^T dO over the 64 queries (two 32-long steps):
    // block b = w * NBLK + j of D / 4: first half dK, second half dV
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      const int b = w * NBLK + j;
      const bool isv = b >= D / 8;
      const int rem = isv ? b - D / 8 : b;
      const int kb = rem / (D / 16), db = rem % (D / 16);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int qs = 0; qs < 2; ++qs) {
        Frag<T> A, B;
        A.load((isv ? Pkq : Zkq) + (16 * kb + p) * L::PS + 32 * qs + 8 * g);
        if constexpr (TRANS)
          B.load((isv ? dOT : QT) + (16 * db + p) * L::TS + 32 * qs + 8 * g);
        else
          B = load_col<T>(isv ? dOs : Qs, L::QS, 32 * qs + 8 * g, 16 * db + p);
        acc = mma(A, B, acc);
      }
      // rows: key 16 kb + 4 g + r of the tile; column: dim 16 db + p
      const float f = isv ? 1.f : a.scale;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 16 * kb + 4 * g + r;
        if (key >= nr) continue;
        bool sk2;
        int nr2;
        const int row = key_row(i, key, sk2, nr2);
        float *dst;
        if (sk)
          dst = (isv ? a.dv_lm_out : a.dq_lm) + (bh * M + row) * D;
        else
          dst = (isv ? a.dv : a.dk) + (bh * N + row) * D;
        unsafeAtomicAdd(dst + 16 * db + p, acc[r] * f);
      }
    }
  }

  // ---------------------------------------------------------------- dQ out
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qq = 16 * w + 4 * g + r;
    const int row = qrow[qq];
    if (row < 0) continue;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const float val = dqa[db][r] * a.scale;
      if (MODE == BWD_ATT)
        a.dq[(bh * N + row) * D + 16 * db + p] = val;
      else
        unsafeAtomicAdd(a.dq_lm + (bh * M + row) * D + 16 * db + p, val);
    }
  }
}

// Log-sum-exp (log2 units) of every landmark row's scores, from the score
// pass's per-chunk (max, sum) partials: one thread per row.
__global__ __launch_bounds__(256) void lse_rows_kernel(const float2 *__restrict__ part_ml, float *__restrict__ lse,
                                                       int64_t rows, int M, int nch) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= rows) return;
  const int64_t bh = t / M;
  const int lm = (int)(t % M);
  float m = -INFINITY, l = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float2 x = part_ml[(bh * nch + c) * M + lm];
    const float mn = fmaxf(m, x.x);
    if (mn == -INFINITY) continue;
    l = l * __builtin_amdgcn_exp2f(m - mn) + x.y * __builtin_amdgcn_exp2f(x.x - mn);
    m = mn;
  }
  lse[t] = m + __log2f(l);
}

// The gradients in the io type: dq = the direct part + the pooling backward
// of the landmark queries' gradient (each token of window W_i receives
// dq_lm_i / |W_i|), dk, dv from their accumulators. One thread per 4 dims.
// Along each axis a position lies in at most two adaptive windows, among
// floor(pos * g / G) - 1 .. + 1.
template <typename T, int D, bool POOL>
__global__ __launch_bounds__(256) void bwd_finish_kernel(const float *__restrict__ dq_direct,
                                                         const float *__restrict__ dq_lm,
                                                         const float *__restrict__ dk_acc,
                                                         const float *__restrict__ dv_acc, T *__restrict__ dq,
                                                         T *__restrict__ dk, T *__restrict__ dv, int64_t rows, int N,
                                                         int M, int gh, int gw, int lh, int lw) {
  constexpr int C = D / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = t / C;
  const int c = (int)(t % C);
  if (row >= rows) return;
  const int64_t bh = row / N;
  const int tok = (int)(row % N);
  const int64_t at = row * D + 4 * c;
  float4 x = *reinterpret_cast<const float4 *>(dq_direct + at);
  if (POOL) {
    const int pr = tok / gw, pc = tok % gw;
    const int ar = (int)((int64_t)pr * lh / gh), ac = (int)((int64_t)pc * lw / gw);
    for (int a = max(0, ar - 1); a <= min(lh - 1, ar + 1); ++a) {
      const int r0 = (int)((int64_t)a * gh / lh), r1 = (int)(((int64_t)(a + 1) * gh + lh - 1) / lh);
      if (pr < r0 || pr >= r1) continue;
      for (int b = max(0, ac - 1); b <= min(lw - 1, ac + 1); ++b) {
        const int s0 = (int)((int64_t)b * gw / lw), s1 = (int)(((int64_t)(b + 1) * gw + lw - 1) / lw);
        if (pc < s0 || pc >= s1) continue;
        const float inv = 1.f / (float)((r1 - r0) * (s1 - s0));
        const float4 y = *reinterpret_cast<const float4 *>(dq_lm + (bh * M + a * lw + b) * D + 4 * c);
        x.x += y.x * inv;
        x.y += y.y * inv;
        x.z += y.z * inv;
        x.w += y.w * inv;
      }
    }
  }
  const float4 yk = *reinterpret_cast<const float4 *>(dk_acc + at);
  const float4 yv = *reinterpret_cast<const float4 *>(dv_acc + at);
  auto put = [&](T *dst, float4 f) {
    T vals[4] = {from_f32<T>(f.x), from_f32<T>(f.y), from_f32<T>(f.z), from_f32<T>(f.w)};
    if (sizeof(T) == 2)
      *reinterpret_cast<uint2 *>(dst + at) = *reinterpret_cast<const uint2 *>(vals);
    else
      *reinterpret_cast<uint4 *>(dst + at) = *reinterpret_cast<const uint4 *>(vals);
  };
  put(dq, x);
  put(dk, yk);
  put(dv, yv);
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t bwd_t(const mita_cfg_t &c, const BwdBufs &b, hipStream_t st) {
  BwdArgs a{};
  a.q = b.q;
  a.k = b.k;
  a.v = b.v;
  a.o = b.o;
  a.dO = b.dO;
  a.q_lm = b.q_lm;
  a.v_lm = b.v_lm;
  a.idx = b.idx;
  a.perm = b.perm;
  a.offsets = b.offsets;
  a.tile_start = b.tile_start;
  a.lse_lm = b.lse_lm;
  a.dv_lm = b.dv_lm_acc;
  a.dq = b.dq_direct;
  a.dk = b.dk_acc;
  a.dv = b.dv_acc;
  a.dq_lm = b.dq_lm_acc;
  a.dv_lm_out = b.dv_lm_acc;
  a.N = c.N;
  a.M = c.M;
  a.topk = c.k;
  a.chunk = BWD_CHUNK;
  a.scale = eff_scale(c);
  const unsigned bh = (unsigned)BH(c);
  hipError_t err;
  if (c.use_shared) {
    const int64_t rows = BH(c) * c.M;
    hipLaunchKernelGGL(lse_rows_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, st, (const float2 *)b.part_ml,
                       b.lse_lm, rows, c.M, score_chunks(c));
    if ((err = launched("lse_rows_kernel", st)) != hipSuccess) return err;
  }
  // the attention of Eq. mita
  int tiles = (c.N + ATT_TQ - 1) / ATT_TQ;
  if (c.use_routed) tiles = (tiles + c.M + NXCD - 1) / NXCD * NXCD;
  const dim3 grid((unsigned)tiles, bh);
  if (c.use_shared && c.use_routed)
    hipLaunchKernelGGL((bwd_kernel<T, D, BWD_ATT, true, true>), grid, dim3(256), 0, st, a);
  else if (c.use_routed)
    hipLaunchKernelGGL((bwd_kernel<T, D, BWD_ATT, false, true>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((bwd_kernel<T, D, BWD_ATT, true, false>), grid, dim3(256), 0, st, a);
  if ((err = launched("bwd_attend_kernel", st)) != hipSuccess) return err;
  // the landmark values (Eq. landmark-value), once their gradient is complete
  if (c.use_shared) {
    const int nlb = (c.M + BWD_TQ - 1) / BWD_TQ, nch = (c.N + BWD_CHUNK - 1) / BWD_CHUNK;
    hipLaunchKernelGGL((bwd_kernel<T, D, BWD_LMV, true, false>), dim3((unsigned)(nlb * nch), bh), dim3(256), 0, st,
                       a);
    if ((err = launched("bwd_landmark_kernel", st)) != hipSuccess) return err;
  }
  const int64_t rows = BH(c) * c.N;
  const int64_t threads = rows * (D / 4);
  const dim3 fg((unsigned)((threads + 255) / 256));
  if (c.use_shared)
    hipLaunchKernelGGL((bwd_finish_kernel<T, D, true>), fg, dim3(256), 0, st, b.dq_direct, b.dq_lm_acc, b.dk_acc,
                       b.dv_acc, (T *)b.dq, (T *)b.dk, (T *)b.dv, rows, c.N, c.M, c.grid_h, c.grid_w, c.lm_h, c.lm_w);
  else
    hipLaunchKernelGGL((bwd_finish_kernel<T, D, false>), fg, dim3(256), 0, st, b.dq_direct, b.dq_lm_acc, b.dk_acc,
                       b.dv_acc, (T *)b.dq, (T *)b.dk, (T *)b.dv, rows, c.N, c.M, c.grid_h, c.grid_w, c.lm_h, c.lm_w);
  return launched("bwd_finish_kernel", st);
}

hipError_t launch_backward(const mita_cfg_t &c, const BwdBufs &b, hipStream_t st) {
  if (c.dtype == MITA_F32) return c.d == 64 ? bwd_t<float, 64>(c, b, st) : bwd_t<float, 128>(c, b, st);
  return c.d == 64 ? bwd_t<bf16_t, 64>(c, b, st) : bwd_t<bf16_t, 128>(c, b, st);
}

}  // namespace mita
