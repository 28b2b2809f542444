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
//        keys forms each query's log-sum-exp (kept for the key side), a
//        second one dQ, in registers (a query's keys are all seen here),
//        written once.
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
// The keys' gradients of the MiTA attention come from bwd_kv_kernel, where a
// workgroup owns 64 keys and streams the queries that attend them, so that
// dK and dV stay in registers: a routed key block of one expert sees that
// expert's queries (the per-expert sums are staged and then summed per token
// through an inverse index of the top-k sets); a block of shared keys sees a
// chunk of all queries (few atomic adds per chunk). fp32 atomic adds retire at
// a few hundred G/s on the whole chip, so a design that adds every 64-query
// tile's key gradients atomically is bound by them.
// The landmark queries' gradient and the landmark-value backward use atomic
// adds whose order varies from run to run, so dq, dk, dv are reproducible
// only to rounding (a few ulp), not bit for bit.
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
  float *q_lse, *q_D;      // [BH, N] ATT: each query's log-sum-exp (log2 units) and dO . o (written)
  const void *dv_lm16;     // [BH, M, d] bf16 copy of dv_lm (the DMA-tiled landmark-value pass)
  const float *D_lm;       // [BH, M] dv_lm . v_lm (the DMA-tiled landmark-value pass)
  int N, M, topk, chunk;
  float scale;
};

constexpr int BWD_ATT = 0, BWD_LMV = 1;

template <typename T, int D, int MODE, bool SHARED, bool ROUTED>
__global__ __launch_bounds__(256) void bwd_kernel(BwdArgs a) {
  using L = BwdLds<T, D>;
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr bool TRANS = L::TRANS;
  // the key-side tiles ([key][query] P and dZ, transposed Q and dO) serve
  // the LMV mode's dK and dV only
  constexpr bool KEYS = MODE == BWD_LMV;
  __shared__ __align__(16) T Qs[L::NQ];
  __shared__ __align__(16) T dOs[L::NQ];
  __shared__ __align__(16) T QT[KEYS ? L::NQT : 1];
  __shared__ __align__(16) T dOT[KEYS ? L::NQT : 1];
  __shared__ __align__(16) T Ks[L::NK];
  __shared__ __align__(16) T Vs[L::NK];
  __shared__ __align__(16) T KT[L::NKT];
  __shared__ __align__(16) T Pkq[KEYS ? L::NP : 1];
  __shared__ __align__(16) T Zkq[KEYS ? L::NP : 1];
  __shared__ __align__(16) T Zqk[L::NZ];
  __shared__ float Dq[BWD_TQ];
  __shared__ int32_t qrow[BWD_TQ];  // each query's row in its tensor (token or landmark), -1 if none
  int64_t bh = blockIdx.y;
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
      if constexpr (TRANS && KEYS) {
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
    if (g == 0 && qok) {
      a.q_lse[bh * N + qrow[myq]] = lse;
      a.q_D[bh * N + qrow[myq]] = Dq[myq];
    }
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
        if constexpr (KEYS) {
          Pkq[key * L::PS + myq] = from_f32<T>(pz[r]);
          Zkq[key * L::PS + myq] = from_f32<T>(zz[r]);
        }
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
    // LMV: dK = dZ^T Q and dV = P^T dO over the 64 queries (two 32-long
    // steps), block b = w * NBLK + j of D / 4: first half dK, second half dV
    // (in ATT mode the keys' gradients come from bwd_kv_kernel)
    if constexpr (KEYS)
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
        if constexpr (TRANS && KEYS)
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

// ---------------------------------------------------------------------------
// The dQ pass for bf16 with the key row list in LDS, on the forward
// attention's tile machinery (attend16_kernel): each wave owns NG 16-query
// column groups of the workgroup's 64 queries and every key; 32-key tiles by
// LDS DMA, double buffered, one barrier per tile, K and V row-major with the
// 16-byte swizzle, K^T read by ds_read_b64_tr_b16 for dQ. Per group and key
// tile (lane (g, p): keys 16 kb + 4 g + r of query p):
//   pass 1 (K tiles only): S^T = K Q^T, each lane's running (max, sum) of
//     exp2(S^T scale log2 e); the four lane groups merge into the query's
//     log-sum-exp (log2 units);
//   pass 2 (K and V tiles): P = exp2(S^T scale log2 e - lse), dP^T = V dO^T,
//     dZ = P (dP - D) (rounded to bf16 for the MFMA), dQ^T += K^T dZ^T;
// then dQ * scale, the log-sum-exp and D = dO . o (fp32, over the lane's 16
// dimensions and then the four lane groups) are written per query, as
// bwd_kernel does. S and P take the unscaled bf16 queries and an fp32
// multiply by scale log2 e, as the key-owned kernel does.
// ---------------------------------------------------------------------------
constexpr int BWD16_TK = 32;
constexpr int BWD16_LMV_CHUNK = 2048;  // keys per workgroup of the landmark queries' gradient
template <int D> constexpr int BWD16_GROUPS = D == 64 ? 2 : 1;
template <int D> constexpr size_t bwd16_tiles_lds() { return 4 * (size_t)DmaTile<D, BWD16_TK>::BYTES; }

template <int D, bool SHARED, bool ROUTED, int NG, bool LMV = false>
__global__ __launch_bounds__(256 / NG) __attribute__((amdgpu_waves_per_eu(4))) void bwd_att16_kernel(BwdArgs a) {
  constexpr int NW = 4 / NG;  // waves per workgroup
  constexpr int NT = 64 * NW;
  constexpr int TK = BWD16_TK;
  static_assert(NG * NW * 16 == BWD_TQ, "64 queries per workgroup");
  using DT = DmaTile<D, TK, NW>;
  constexpr int RB = 2 * D;  // bytes per K / V row
  __shared__ __align__(16) char tiles0[2 * DT::BYTES];
  __shared__ __align__(16) char tiles1[2 * DT::BYTES];
  auto Ks = [&](int b) { return reinterpret_cast<bf16_t *>(b ? tiles1 : tiles0); };
  auto Vt = [&](int b) { return reinterpret_cast<bf16_t *>((b ? tiles1 : tiles0) + DT::BYTES); };
  extern __shared__ uint32_t sidx[];  // byte offsets of the M + k key rows
  int64_t bh = blockIdx.y;
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int N = a.N, M = a.M, K = a.topk;
  int e = 0, q_begin, q_end, c0 = 0, nck = 0;
  if (LMV) {
    // landmark block lb (the queries) against key chunk ch
    const int nlb = (M + BWD_TQ - 1) / BWD_TQ;
    const int lb = (int)blockIdx.x % nlb, ch = (int)blockIdx.x / nlb;
    q_begin = lb * BWD_TQ;
    q_end = min(M, q_begin + BWD_TQ);
    c0 = ch * a.chunk;
    if (c0 >= N) return;  // uniform
    nck = min(N - c0, a.chunk);
  } else if (!attend_queries<ROUTED>(a.tile_start, a.offsets, bh, N, M, e, q_begin, q_end)) {
    return;  // uniform
  }
  // LMV: the chunk's keys take the place of the routed ones
  const int nrt = LMV ? nck : (ROUTED ? K : 0);
  const int nA = SHARED && !LMV ? M / TK : 0, pA = SHARED && !LMV ? M % TK : 0;
  const int nB = nrt / TK, pB = nrt % TK;
  const int nfull = nA + nB;
  const bf16_t *sh_k = (const bf16_t *)a.q_lm + bh * (int64_t)M * D;
  const bf16_t *sh_v = (const bf16_t *)a.v_lm + bh * (int64_t)M * D;
  const bf16_t *rkb = (const bf16_t *)a.k + bh * (int64_t)N * D;
  const bf16_t *rvb = (const bf16_t *)a.v + bh * (int64_t)N * D;
  const int nsh = SHARED && !LMV ? M : 0;
  for (int i = threadIdx.x; i < nsh; i += NT) sidx[i] = (uint32_t)i * RB;
  if (LMV) {
    for (int i = threadIdx.x; i < nck; i += NT) sidx[i] = (uint32_t)(c0 + i) * RB;
  } else if (ROUTED) {
    const int32_t *gidx = a.idx + (bh * M + e) * (int64_t)K;
    for (int i = threadIdx.x; i < K; i += NT) sidx[nsh + i] = (uint32_t)gidx[i] * RB;
  }
  __syncthreads();
  const uint32_t *rows = sidx;
  auto tile_base = [&](int i, const bf16_t *&kb, const bf16_t *&vb, int &off) {
    const bool sh = i < nA;
    kb = sh ? sh_k : rkb;
    vb = sh ? sh_v : rvb;
    off = sh ? i * TK : nsh + (i - nA) * TK;
  };

  // this wave's groups: group c holds queries q_begin + 16 (NG w + c) + p
  // (LMV: landmark rows of q_lm, their upstream gradient in bf16, D given)
  const bf16_t *qg = LMV ? (const bf16_t *)a.q_lm : (const bf16_t *)a.q;
  const bf16_t *dOg = LMV ? (const bf16_t *)a.dv_lm16 : (const bf16_t *)a.dO, *og = (const bf16_t *)a.o;
  const int QN = LMV ? M : N;  // rows per head of the query tensors
  int tok[NG];
  bool qvalid[NG];
  Frag<bf16_t> qf[NG][D / 32], df[NG][D / 32];
  float Dq[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    const int qi = q_begin + 16 * (NG * w + c) + p;
    qvalid[c] = qi < q_end;
    tok[c] = qvalid[c] ? (ROUTED && !LMV ? a.perm[bh * N + qi] : qi) : 0;
    float dpart = 0.f;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const int64_t at = (bh * QN + tok[c]) * D + ks * 32 + g * 8;
      if (LMV) {
        if (qvalid[c]) {
          qf[c][ks].load(qg + at);
          df[c][ks].load(dOg + at);
        } else {
          qf[c][ks].zero();
          df[c][ks].zero();
        }
      } else if (qvalid[c]) {
        qf[c][ks].load(qg + at);
        df[c][ks].load(dOg + at);
        float ov[8], dv[8];
        load16_f32(og + at, ov);
        unpack16(df[c][ks].v, dv, (const bf16_t *)nullptr);
#pragma unroll
        for (int i = 0; i < 8; ++i) dpart = __builtin_fmaf(ov[i], dv[i], dpart);
      } else {
        qf[c][ks].zero();
        df[c][ks].zero();
      }
    }
    // D = dO . o of query p: the four lane groups' parts, in a fixed order
    const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(dpart), __float_as_uint(dpart), false, false);
    const float pair = __uint_as_float(x[0]) + __uint_as_float(x[1]);
    const auto y = __builtin_amdgcn_permlane32_swap(__float_as_uint(pair), __float_as_uint(pair), false, false);
    Dq[c] = __uint_as_float(y[0]) + __uint_as_float(y[1]);
    if (LMV) Dq[c] = qvalid[c] ? a.D_lm[bh * M + tok[c]] : 0.f;
  }
  int nbusy = 0;
#pragma unroll
  for (int c = 0; c < NG; ++c) nbusy += q_begin + 16 * (NG * w + c) < q_end ? 1 : 0;
  DmaLane<D, TK, NW> dl;
  dl.init(w, lane);
  Att16Addr<D> ad;
  ad.init();
  const float sl2 = a.scale * LOG2E;
  const bf16_t *kb, *vb;
  int off;
  wait_loads();
  __syncthreads();

  // S^T of the tile for the first NGB groups, from zero
  auto scores = [&](f32x4 (&acc)[NG][2], const bf16_t *Kl, auto ngb_c) {
    constexpr int NGB = decltype(ngb_c)::value;
    const char *kbase = reinterpret_cast<const char *>(Kl);
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
      for (int c = 0; c < NGB; ++c) acc[c][kb2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<bf16_t> A;
        A.v = *reinterpret_cast<const uint4 *>(kbase + ad.k[ks] + kb2 * 16 * RB);
#pragma unroll
        for (int c = 0; c < NGB; ++c) acc[c][kb2] = mma(A, qf[c][ks], acc[c][kb2]);
      }
    }
  };
  // One sweep over the key tiles (DMA pipeline as in attend16_kernel);
  // body(Kc, Vc, nvalid, masked_c) runs each tile's arithmetic.
  auto sweep = [&](auto with_v_c, auto body) {
    constexpr bool WV = decltype(with_v_c)::value;
    auto issue = [&](int j, bf16_t *Kn, bf16_t *Vn) {
      if (j < nfull) {
        tile_base(j, kb, vb, off);
        dma_tile_lane<D, TK, NW, WV>(Kn, Vn, kb, vb, rows + off, dl);
      }
    };
    auto step = [&](int i, int b) {
      issue(i + 1, Ks(b ^ 1), Vt(b ^ 1));
      __builtin_amdgcn_sched_barrier(0);
      body(Ks(b), Vt(b), TK, std::false_type{});
      wait_loads();
      __syncthreads();
    };
    if (nfull > 0) {
      issue(0, Ks(0), Vt(0));
      wait_loads();
      __syncthreads();
      int i = 0;
      for (; i + 1 < nfull; i += 2) {
        step(i, 0);
        step(i + 1, 1);
      }
      if (i < nfull) step(i, 0);
    }
    for (int part = 0; part < 2; ++part) {
      const int nr = part == 0 ? pA : pB;
      if (nr == 0) continue;  // uniform
      if (part == 0)
        dma_tile<D, false, TK, NW, WV>(Ks(0), Vt(0), sh_k, sh_v, rows + nA * TK, nr);
      else
        dma_tile<D, false, TK, NW, WV>(Ks(0), Vt(0), rkb, rvb, rows + nsh + nB * TK, nr);
      wait_loads();
      __syncthreads();
      body(Ks(0), Vt(0), nr, std::true_type{});
      __syncthreads();
    }
  };

  // ------------------------------------------------------------ pass 1: lse
  float lm[NG], ll[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    lm[c] = -INFINITY;
    ll[c] = 0.f;
  }
  auto pass1 = [&](auto ngb_c) {
    constexpr int NGB = decltype(ngb_c)::value;
    sweep(std::false_type{}, [&](const bf16_t *Kc, const bf16_t *, int nv, auto masked_c) {
      constexpr bool MK = decltype(masked_c)::value;
      if (NGB == 0) return;
      f32x4 acc[NG][2];
      scores(acc, Kc, ngb_c);
#pragma unroll
      for (int c = 0; c < NGB; ++c) {
        float mx = -INFINITY;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            mx = (!MK || 16 * kb2 + 4 * g + r < nv) ? fmaxf(mx, acc[c][kb2][r]) : mx;
        const float mn = fmaxf(lm[c], mx * sl2);
        float add = 0.f;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            add += (!MK || 16 * kb2 + 4 * g + r < nv) ? __builtin_amdgcn_exp2f(__builtin_fmaf(acc[c][kb2][r], sl2, -mn))
                                                      : 0.f;
        ll[c] = (mn == -INFINITY ? 0.f : ll[c] * __builtin_amdgcn_exp2f(lm[c] - mn)) + add;
        lm[c] = mn;
      }
    });
  };
  // (LMV: each landmark row's log-sum-exp comes from the score pass)
  if (LMV)
    ;
  else if (NG == 2 && nbusy == 2)
    pass1(std::integral_constant<int, NG>{});
  else if (nbusy >= 1)
    pass1(std::integral_constant<int, 1>{});
  else
    pass1(std::integral_constant<int, 0>{});
  float lse[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    if (LMV) {
      lse[c] = qvalid[c] ? a.lse_lm[bh * M + tok[c]] : 0.f;
      continue;
    }
    const float mc = max_lane_groups(lm[c]);
    const float lc = lm[c] == -INFINITY ? 0.f : ll[c] * __builtin_amdgcn_exp2f(lm[c] - mc);
    const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(lc), __float_as_uint(lc), false, false);
    const float pair = __uint_as_float(x[0]) + __uint_as_float(x[1]);
    const auto y = __builtin_amdgcn_permlane32_swap(__float_as_uint(pair), __float_as_uint(pair), false, false);
    lse[c] = qvalid[c] ? mc + __log2f(__uint_as_float(y[0]) + __uint_as_float(y[1])) : 0.f;
  }

  // ------------------------------------------------------------ pass 2: dQ
  f32x4 dqa[NG][D / 16];
#pragma unroll
  for (int c = 0; c < NG; ++c)
#pragma unroll
    for (int db = 0; db < D / 16; ++db) dqa[c][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto pass2 = [&](auto ngb_c) {
    constexpr int NGB = decltype(ngb_c)::value;
    sweep(std::true_type{}, [&](const bf16_t *Kc, const bf16_t *Vc, int nv, auto masked_c) {
      constexpr bool MK = decltype(masked_c)::value;
      if (NGB == 0) return;
      f32x4 acc[NG][2], dp[NG][2];
      scores(acc, Kc, ngb_c);
      const char *vbase = reinterpret_cast<const char *>(Vc);
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
        for (int c = 0; c < NGB; ++c) dp[c][kb2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
          Frag<bf16_t> A;
          A.v = *reinterpret_cast<const uint4 *>(vbase + ad.k[ks] + kb2 * 16 * RB);
#pragma unroll
          for (int c = 0; c < NGB; ++c) dp[c][kb2] = mma(A, df[c][ks], dp[c][kb2]);
        }
      }
      Frag<bf16_t> z[NG];
#pragma unroll
      for (int c = 0; c < NGB; ++c) {
        float zz[8];
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[c][kb2][r], sl2, -lse[c]));
            if (MK && 16 * kb2 + 4 * g + r >= nv) pr = 0.f;
            zz[4 * kb2 + r] = pr * (dp[c][kb2][r] - Dq[c]);
          }
        z[c].from_f32(zz);
      }
      // dQ^T += K^T dZ^T: the K^T operand by transposing reads of the K tile
      const char *kbase = reinterpret_cast<const char *>(Kc);
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        uint2 half[2];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
          half[h2] = __builtin_bit_cast(
              uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(kbase + ad.v[db] + h2 * 16 * RB)));
        Frag<bf16_t> A;
        A.v = make_uint4(half[0].x, half[0].y, half[1].x, half[1].y);
#pragma unroll
        for (int c = 0; c < NGB; ++c) dqa[c][db] = mma(A, z[c], dqa[c][db]);
      }
    });
  };
  if (NG == 2 && nbusy == 2)
    pass2(std::integral_constant<int, NG>{});
  else if (nbusy >= 1)
    pass2(std::integral_constant<int, 1>{});
  else
    pass2(std::integral_constant<int, 0>{});

  // ------------------------------------------------------------ outputs
  if (LMV) {  // the chunk's part of the landmark queries' gradient
#pragma unroll
    for (int c = 0; c < NG; ++c) {
      if (!qvalid[c]) continue;
      float *drow = a.dq_lm + (bh * M + tok[c]) * D;
#pragma unroll
      for (int db = 0; db < D / 16; ++db)
#pragma unroll
        for (int r = 0; r < 4; ++r) unsafeAtomicAdd(drow + db * 16 + 4 * g + r, dqa[c][db][r] * a.scale);
    }
    return;
  }
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    if (!qvalid[c]) continue;
    float *drow = a.dq + (bh * N + tok[c]) * D;
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
      *reinterpret_cast<float4 *>(drow + db * 16 + 4 * g) =
          make_float4(dqa[c][db][0] * a.scale, dqa[c][db][1] * a.scale, dqa[c][db][2] * a.scale,
                      dqa[c][db][3] * a.scale);
    if (g == 0) {
      a.q_lse[bh * N + tok[c]] = lse[c];
      a.q_D[bh * N + tok[c]] = Dq[c];
    }
  }
}

// ---------------------------------------------------------------------------
// Key-owned backward of the MiTA attention: a workgroup owns KB = 64 keys
// (wave w the 16 keys 16 w ..), whose K and V fragments stay in registers,
// and streams the queries that attend them in tiles of 64, with each query's
// log-sum-exp and D = dO . o from the dQ pass. Per query tile:
//   S^T = K Q^T, dP^T = V dO^T (keys x queries, one wave's 16 keys),
//   P = exp2(S^T scale log2 e - lse), dZ = P (dP - D),
//   dK += dZ^T Q, dV += P^T dO (reduction over the tile's 64 queries; P and
//   dZ go through a per-wave LDS area to take the operand layout).
//   ROUTED: block x = (expert e, key block b); keys idx[e][64 b ..], queries
//           the expert's group (perm[offsets[e] ..]); the expert's sums are
//           written to the staging rows [e][64 b ..] (plain stores).
//   SHARED: block x = (landmark block, chunk of BWD_QCHUNK queries in token
//           order); keys q_lm / v_lm rows; the sums are added atomically to
//           the landmark rows.
// Blocks are spread over the XCDs as the attention work list is, so the key
// blocks of one expert (same queries) share an L2.
// ---------------------------------------------------------------------------
constexpr int BWD_KB = 64;
constexpr int BWD_QCHUNK = 2048;

template <typename T, int D> struct KvLds {
  static constexpr int PAD = 16 / (int)sizeof(T);
  static constexpr bool TRANS = sizeof(T) == 2 && D == 64;
  static constexpr int QS = D + PAD, TS = BWD_TQ + PAD, WS = BWD_TQ + PAD;
  static constexpr int NQ = BWD_TQ * QS, NQT = TRANS ? D * TS : 1, NW = 4 * 16 * WS;
};

struct KvArgs {
  const void *q, *k, *v, *dO, *q_lm, *v_lm;
  const int32_t *idx, *perm, *offsets;
  const float *q_lse, *q_D;   // [BH, N]
  const void *dv_lm16;        // LMV keys: [BH, M, d] bf16 gradient of the landmark values
  const float *lse_lm, *D_lm; // LMV keys: [BH, M] the landmark rows' log-sum-exp and dV~ . V~
  float *dk_acc, *dv_acc;     // LMV keys without the fused finish: [BH, N, d] accumulators (added to)
  // LMV keys with the fused finish (dk_out != NULL): the routed keys' staged
  // per-expert rows (inverse index inv_start / inv_slot, NULL without
  // routing) are summed in, and dk, dv written in bf16
  const int32_t *inv_start, *inv_slot;
  void *dk_out, *dv_out;
  float *stage_k, *stage_v;   // ROUTED: [BH, M, k, d]
  float *dq_lm, *dv_lm;       // SHARED: [BH, M, d] accumulators
  int N, M, topk, nblk;       // nblk: key blocks per expert (ROUTED) or landmark blocks (SHARED)
  int ntotal;                 // blocks with work (the grid is rounded up to a multiple of 8)
  float scale;
};

template <typename T, int D, bool ROUTED>
__global__ __launch_bounds__(256) void bwd_kv_kernel(KvArgs a) {
  using L = KvLds<T, D>;
  constexpr int VE = 16 / (int)sizeof(T);
  constexpr bool TRANS = L::TRANS;
  __shared__ __align__(16) T Qs[L::NQ];
  __shared__ __align__(16) T dOs[L::NQ];
  __shared__ __align__(16) T QT[L::NQT];
  __shared__ __align__(16) T dOT[L::NQT];
  __shared__ __align__(16) T Pw[L::NW];
  __shared__ __align__(16) T Zw[L::NW];
  __shared__ float lse_s[BWD_TQ], D_s[BWD_TQ];
  __shared__ int32_t qtok[BWD_TQ];
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, g = lane >> 4, p = lane & 15;
  const int N = a.N, M = a.M, K = a.topk;
  const T *q = (const T *)a.q, *dO = (const T *)a.dO;
  // the block, spread over the XCDs
  const int nb = (int)gridDim.x;
  const int C = (nb + NXCD - 1) / NXCD;
  const int x = ((int)blockIdx.x % NXCD) * C + (int)blockIdx.x / NXCD;
  if (x >= a.ntotal) return;  // uniform
  int e = 0, kb0, nkeys, q0, nq;
  if (ROUTED) {
    e = x / a.nblk;
    kb0 = (x % a.nblk) * BWD_KB;
    nkeys = min(BWD_KB, K - kb0);
    q0 = a.offsets[bh * (M + 1) + e];
    nq = a.offsets[bh * (M + 1) + e + 1] - q0;
  } else {
    kb0 = (x % a.nblk) * BWD_KB;
    nkeys = min(BWD_KB, M - kb0);
    q0 = (x / a.nblk) * BWD_QCHUNK;
    nq = min(BWD_QCHUNK, N - q0);
  }
  // (an expert without queries still writes its staging rows: zeros)
  // this wave's 16 keys: K and V fragments (row p of the wave's block)
  const int mykey = 16 * w + p;
  const bool kvalid = mykey < nkeys;
  int krow = 0;
  if (kvalid) krow = ROUTED ? a.idx[(bh * M + e) * (int64_t)K + kb0 + mykey] : kb0 + mykey;
  const T *kbase = ROUTED ? (const T *)a.k + bh * (int64_t)N * D : (const T *)a.q_lm + bh * (int64_t)M * D;
  const T *vbase = ROUTED ? (const T *)a.v + bh * (int64_t)N * D : (const T *)a.v_lm + bh * (int64_t)M * D;
  Frag<T> kf[D / 32], vf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    if (kvalid) {
      kf[ks].load(kbase + (int64_t)krow * D + 32 * ks + 8 * g);
      vf[ks].load(vbase + (int64_t)krow * D + 32 * ks + 8 * g);
    } else {
      kf[ks].zero();
      vf[ks].zero();
    }
  }
  const float sl2 = a.scale * LOG2E;
  f32x4 dk[D / 16], dv[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    dk[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    dv[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  T *pw = Pw + w * 16 * L::WS, *zw = Zw + w * 16 * L::WS;
  for (int t0 = 0; t0 < nq; t0 += BWD_TQ) {
    __syncthreads();
    if (tid < BWD_TQ) {
      int tok = -1;
      if (t0 + tid < nq) tok = ROUTED ? a.perm[bh * N + q0 + t0 + tid] : q0 + t0 + tid;
      qtok[tid] = tok;
      lse_s[tid] = tok >= 0 ? a.q_lse[bh * N + tok] : 0.f;
      D_s[tid] = tok >= 0 ? a.q_D[bh * N + tok] : 0.f;
    }
    __syncthreads();
    for (int c = tid; c < BWD_TQ * (D / VE); c += 256) {
      const int row = c / (D / VE), cc = c % (D / VE);
      const int tok = qtok[row];
      uint4 xq = make_uint4(0, 0, 0, 0), xd = make_uint4(0, 0, 0, 0);
      if (tok >= 0) {
        xq = *reinterpret_cast<const uint4 *>(q + (bh * N + tok) * D + cc * VE);
        xd = *reinterpret_cast<const uint4 *>(dO + (bh * N + tok) * D + cc * VE);
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
    __syncthreads();
    // P and dZ of (key 16 w + 4 g + r, query 16 qb + p) into the wave's LDS area
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f}, dp = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<T> B;
        B.load(Qs + (16 * qb + p) * L::QS + 32 * ks + 8 * g);
        s = mma(kf[ks], B, s);
        B.load(dOs + (16 * qb + p) * L::QS + 32 * ks + 8 * g);
        dp = mma(vf[ks], B, dp);
      }
      const int qq = 16 * qb + p;
      const bool qok = qtok[qq] >= 0;
      const float lq = lse_s[qq], dq = D_s[qq];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 16 * w + 4 * g + r;
        const bool ok = qok && key < nkeys;
        const float pr = ok ? __builtin_amdgcn_exp2f(s[r] * sl2 - lq) : 0.f;
        pw[(4 * g + r) * L::WS + qq] = from_f32<T>(pr);
        zw[(4 * g + r) * L::WS + qq] = from_f32<T>(pr * (dp[r] - dq));
      }
    }
    __syncthreads();
    // dK += dZ^T Q, dV += P^T dO: rows = the wave's 16 keys, columns = dims
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
#pragma unroll
      for (int qs = 0; qs < 2; ++qs) {
        Frag<T> A, B;
        A.load(zw + p * L::WS + 32 * qs + 8 * g);
        if constexpr (TRANS)
          B.load(QT + (16 * db + p) * L::TS + 32 * qs + 8 * g);
        else
          B = load_col<T>(Qs, L::QS, 32 * qs + 8 * g, 16 * db + p);
        dk[db] = mma(A, B, dk[db]);
        A.load(pw + p * L::WS + 32 * qs + 8 * g);
        if constexpr (TRANS)
          B.load(dOT + (16 * db + p) * L::TS + 32 * qs + 8 * g);
        else
          B = load_col<T>(dOs, L::QS, 32 * qs + 8 * g, 16 * db + p);
        dv[db] = mma(A, B, dv[db]);
      }
    }
  }
  // rows: key 16 w + 4 g + r of the block; column: dim 16 db + p
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int key = 16 * w + 4 * g + r;
    if (key >= nkeys) continue;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      if (ROUTED) {
        const int64_t at = ((bh * M + e) * (int64_t)K + kb0 + key) * D + 16 * db + p;
        a.stage_k[at] = dk[db][r] * a.scale;
        a.stage_v[at] = dv[db][r];
      } else {
        const int64_t at = (bh * M + kb0 + key) * D + 16 * db + p;
        unsafeAtomicAdd(a.dq_lm + at, dk[db][r] * a.scale);
        unsafeAtomicAdd(a.dv_lm + at, dv[db][r]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The key-owned backward for bf16 on the same tile machinery, with the roles
// of queries and keys exchanged: each wave owns NG 16-key column groups of
// the block's 64 keys (their K and V rows as MFMA B fragments in registers)
// and streams the block's queries in 32-row tiles (Q and dO rows by LDS
// DMA, double buffered, row-major with the 16-byte swizzle). Per group and
// query tile (lane (g, p): queries 16 qb + 4 g + r of key p):
//   S = Q K^T, dP = dO V^T; P = exp2(S scale log2 e - lse_q),
//   dZ = P (dP - D_q) (both rounded to bf16 for the MFMA);
//   dV^T += dO^T P, dK^T += Q^T dZ, with dO^T and Q^T read by transposing
//   LDS reads of the tiles (the P and dZ fragments are already the B
//   operand, in the key order of the transposing reads).
// The queries' rows, log-sum-exps and D come in chunks of QC queries
// (offsets and values staged in LDS per chunk). The sums go where
// bwd_kv_kernel puts them (staging rows, or atomic adds for the landmarks).
// ---------------------------------------------------------------------------
constexpr int KV16_QC = 512;  // queries per staged chunk
// key blocks of bwd_kv16_kernel: an expert's routed keys (its queries),
// landmark keys (a chunk of all queries), or tokens as the keys of the
// landmark values (the landmark rows as queries; each token row is owned by
// one block, so the sums are added to the accumulators without atomics)
constexpr int KV_ROUTED = 0, KV_SHARED = 1, KV_LMV = 2;

template <int D, int KM, int NG>
__device__ __forceinline__ void bwd_kv16_body(KvArgs a) {
  constexpr bool ROUTED = KM == KV_ROUTED;
  constexpr int NW = 4 / NG;
  constexpr int NT = 64 * NW;
  constexpr int TQ = BWD16_TK;  // queries per tile
  static_assert(NG * NW * 16 == BWD_KB, "64 keys per workgroup");
  using DT = DmaTile<D, TQ, NW>;
  constexpr int RB = 2 * D;
  __shared__ __align__(16) char tiles0[2 * DT::BYTES];
  __shared__ __align__(16) char tiles1[2 * DT::BYTES];
  __shared__ uint32_t qoff[KV16_QC];
  __shared__ float lse_s[KV16_QC], D_s[KV16_QC];
  auto Qt = [&](int b) { return reinterpret_cast<bf16_t *>(b ? tiles1 : tiles0); };
  auto Dt = [&](int b) { return reinterpret_cast<bf16_t *>((b ? tiles1 : tiles0) + DT::BYTES); };
  const int64_t bh = blockIdx.y;
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int N = a.N, M = a.M, K = a.topk;
  // the block, spread over the XCDs
  const int nb = (int)gridDim.x;
  const int C = (nb + NXCD - 1) / NXCD;
  const int x = ((int)blockIdx.x % NXCD) * C + (int)blockIdx.x / NXCD;
  if (x >= a.ntotal) return;  // uniform
  int e = 0, kb0, nkeys, q0, nq;
  if (KM == KV_ROUTED) {
    e = x / a.nblk;
    kb0 = (x % a.nblk) * BWD_KB;
    nkeys = min(BWD_KB, K - kb0);
    q0 = a.offsets[bh * (M + 1) + e];
    nq = a.offsets[bh * (M + 1) + e + 1] - q0;
  } else if (KM == KV_SHARED) {
    kb0 = (x % a.nblk) * BWD_KB;
    nkeys = min(BWD_KB, M - kb0);
    q0 = (x / a.nblk) * BWD_QCHUNK;
    nq = min(BWD_QCHUNK, N - q0);
  } else {
    kb0 = x * BWD_KB;
    nkeys = min(BWD_KB, N - kb0);
    q0 = 0;
    nq = M;
  }
  // (an expert without queries still writes its staging rows: zeros)
  const bool tok_keys = KM != KV_SHARED;  // keys are token rows of k, v
  const bf16_t *kbase = tok_keys ? (const bf16_t *)a.k + bh * (int64_t)N * D : (const bf16_t *)a.q_lm + bh * (int64_t)M * D;
  const bf16_t *vbase = tok_keys ? (const bf16_t *)a.v + bh * (int64_t)N * D : (const bf16_t *)a.v_lm + bh * (int64_t)M * D;
  Frag<bf16_t> kf[NG][D / 32], vf[NG][D / 32];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    const int key = 16 * (NG * w + c) + p;
    const bool kvalid = key < nkeys;
    const int krow = kvalid ? (ROUTED ? a.idx[(bh * M + e) * (int64_t)K + kb0 + key] : kb0 + key) : 0;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (kvalid) {
        kf[c][ks].load(kbase + (int64_t)krow * D + 32 * ks + 8 * g);
        vf[c][ks].load(vbase + (int64_t)krow * D + 32 * ks + 8 * g);
      } else {
        kf[c][ks].zero();
        vf[c][ks].zero();
      }
    }
  }
  f32x4 dka[NG][D / 16], dva[NG][D / 16];
#pragma unroll
  for (int c = 0; c < NG; ++c)
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      dka[c][db] = f32x4{0.f, 0.f, 0.f, 0.f};
      dva[c][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  DmaLane<D, TQ, NW> dl;
  dl.init(w, lane);
  Att16Addr<D> ad;
  ad.init();
  const float sl2 = a.scale * LOG2E;
  // the streamed queries: tokens (q, dO), or for LMV keys the landmark rows
  // (q_lm and the landmark values' gradient)
  const bf16_t *qg = KM == KV_LMV ? (const bf16_t *)a.q_lm + bh * (int64_t)M * D
                                  : (const bf16_t *)a.q + bh * (int64_t)N * D;
  const bf16_t *dOg = KM == KV_LMV ? (const bf16_t *)a.dv_lm16 + bh * (int64_t)M * D
                                   : (const bf16_t *)a.dO + bh * (int64_t)N * D;

  // one query tile: nv valid rows at chunk position j0
  auto tile = [&](const bf16_t *Qc, const bf16_t *Dc, int j0, int nv, auto masked_c) {
    constexpr bool MK = decltype(masked_c)::value;
    const char *qbase = reinterpret_cast<const char *>(Qc), *dbase = reinterpret_cast<const char *>(Dc);
    f32x4 s[NG][2], dp[NG][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
      for (int c = 0; c < NG; ++c) {
        s[c][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
        dp[c][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        Frag<bf16_t> A, B;
        A.v = *reinterpret_cast<const uint4 *>(qbase + ad.k[ks] + qb * 16 * RB);
        B.v = *reinterpret_cast<const uint4 *>(dbase + ad.k[ks] + qb * 16 * RB);
#pragma unroll
        for (int c = 0; c < NG; ++c) {
          s[c][qb] = mma(A, kf[c][ks], s[c][qb]);
          dp[c][qb] = mma(B, vf[c][ks], dp[c][qb]);
        }
      }
    }
    // the rows' log-sum-exps and D (queries 16 qb + 4 g + r of the tile)
    float lq[2][4], dq[2][4];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const float4 l4 = *reinterpret_cast<const float4 *>(&lse_s[j0 + 16 * qb + 4 * g]);
      const float4 d4 = *reinterpret_cast<const float4 *>(&D_s[j0 + 16 * qb + 4 * g]);
      lq[qb][0] = l4.x; lq[qb][1] = l4.y; lq[qb][2] = l4.z; lq[qb][3] = l4.w;
      dq[qb][0] = d4.x; dq[qb][1] = d4.y; dq[qb][2] = d4.z; dq[qb][3] = d4.w;
    }
    Frag<bf16_t> pf[NG], zf[NG];
#pragma unroll
    for (int c = 0; c < NG; ++c) {
      float pp[8], zz[8];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float pr = __builtin_amdgcn_exp2f(__builtin_fmaf(s[c][qb][r], sl2, -lq[qb][r]));
          float zr = pr * (dp[c][qb][r] - dq[qb][r]);
          // rows past the chunk's last query: their log-sum-exp and D slots
          // in LDS were not written for this chunk and may hold any bits
          // (0 * NaN would spread into every key's dK), so both weights are
          // set, not scaled, to zero
          if (MK && 16 * qb + 4 * g + r >= nv) pr = zr = 0.f;
          pp[4 * qb + r] = pr;
          zz[4 * qb + r] = zr;
        }
      pf[c].from_f32(pp);
      zf[c].from_f32(zz);
    }
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      uint2 hq[2], hd[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        hq[h2] = __builtin_bit_cast(
            uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(qbase + ad.v[db] + h2 * 16 * RB)));
        hd[h2] = __builtin_bit_cast(
            uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(dbase + ad.v[db] + h2 * 16 * RB)));
      }
      Frag<bf16_t> AQ, AD;
      AQ.v = make_uint4(hq[0].x, hq[0].y, hq[1].x, hq[1].y);
      AD.v = make_uint4(hd[0].x, hd[0].y, hd[1].x, hd[1].y);
#pragma unroll
      for (int c = 0; c < NG; ++c) {
        dva[c][db] = mma(AD, pf[c], dva[c][db]);
        dka[c][db] = mma(AQ, zf[c], dka[c][db]);
      }
    }
  };

  for (int c0 = 0; c0 < nq; c0 += KV16_QC) {
    const int nc = min(KV16_QC, nq - c0);
    __syncthreads();  // the previous chunk's tiles and arrays are done
    for (int j = threadIdx.x; j < nc; j += NT) {
      const int tok = ROUTED ? a.perm[bh * N + q0 + c0 + j] : q0 + c0 + j;
      qoff[j] = (uint32_t)tok * RB;
      lse_s[j] = KM == KV_LMV ? a.lse_lm[bh * M + tok] : a.q_lse[bh * N + tok];
      D_s[j] = KM == KV_LMV ? a.D_lm[bh * M + tok] : a.q_D[bh * N + tok];
    }
    __syncthreads();
    const int nfull = nc / TQ, part = nc % TQ;
    auto issue = [&](int j, int b) {
      if (j < nfull) dma_tile_lane<D, TQ, NW>(Qt(b), Dt(b), qg, dOg, qoff + j * TQ, dl);
    };
    auto step = [&](int i, int b) {
      issue(i + 1, b ^ 1);
      __builtin_amdgcn_sched_barrier(0);
      tile(Qt(b), Dt(b), i * TQ, TQ, std::false_type{});
      wait_loads();
      __syncthreads();
    };
    if (nfull > 0) {
      issue(0, 0);
      wait_loads();
      __syncthreads();
      int i = 0;
      for (; i + 1 < nfull; i += 2) {
        step(i, 0);
        step(i + 1, 1);
      }
      if (i < nfull) step(i, 0);
    }
    if (part > 0) {
      dma_tile<D, false, TQ, NW>(Qt(0), Dt(0), qg, dOg, qoff + nfull * TQ, part);
      wait_loads();
      __syncthreads();
      tile(Qt(0), Dt(0), nfull * TQ, part, std::true_type{});
    }
  }
  // LMV keys with the fused finish: each key's staged per-expert rows (the
  // first FS slots loaded together: the index, then every row's dims) are
  // added to the landmark-value sums, and dk, dv written in bf16
  if (KM == KV_LMV && a.dk_out) {
    constexpr int FS = 8;
    const int64_t per_head = (int64_t)M * K;
#pragma unroll
    for (int c = 0; c < NG; ++c) {
      const int key = 16 * (NG * w + c) + p;
      if (key >= nkeys) continue;
      float4 k4[D / 16], v4[D / 16];
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        k4[db] = make_float4(dka[c][db][0] * a.scale, dka[c][db][1] * a.scale, dka[c][db][2] * a.scale,
                             dka[c][db][3] * a.scale);
        v4[db] = make_float4(dva[c][db][0], dva[c][db][1], dva[c][db][2], dva[c][db][3]);
      }
      if (a.inv_start) {
        const int s0 = a.inv_start[bh * (N + 1) + kb0 + key], s1 = a.inv_start[bh * (N + 1) + kb0 + key + 1];
        const int n = s1 - s0;
        int64_t src[FS];
#pragma unroll
        for (int i = 0; i < FS; ++i) src[i] = i < n ? (bh * per_head + a.inv_slot[bh * per_head + s0 + i]) * D : 0;
        auto add = [&](int64_t sr) {
#pragma unroll
          for (int db = 0; db < D / 16; ++db) {
            const float4 yk = *reinterpret_cast<const float4 *>(a.stage_k + sr + 16 * db + 4 * g);
            const float4 yv = *reinterpret_cast<const float4 *>(a.stage_v + sr + 16 * db + 4 * g);
            k4[db].x += yk.x; k4[db].y += yk.y; k4[db].z += yk.z; k4[db].w += yk.w;
            v4[db].x += yv.x; v4[db].y += yv.y; v4[db].z += yv.z; v4[db].w += yv.w;
          }
        };
        if constexpr (D == 64) {
          // two rows' loads in flight before either is added (slot order
          // kept; the registers come from running two waves per SIMD)
          auto add2 = [&](int64_t r0, int64_t r1) {
            float4 yk[2][D / 16], yv[2][D / 16];
#pragma unroll
            for (int db = 0; db < D / 16; ++db) {
              yk[0][db] = *reinterpret_cast<const float4 *>(a.stage_k + r0 + 16 * db + 4 * g);
              yv[0][db] = *reinterpret_cast<const float4 *>(a.stage_v + r0 + 16 * db + 4 * g);
              yk[1][db] = *reinterpret_cast<const float4 *>(a.stage_k + r1 + 16 * db + 4 * g);
              yv[1][db] = *reinterpret_cast<const float4 *>(a.stage_v + r1 + 16 * db + 4 * g);
            }
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
              for (int db = 0; db < D / 16; ++db) {
                k4[db].x += yk[b][db].x; k4[db].y += yk[b][db].y; k4[db].z += yk[b][db].z; k4[db].w += yk[b][db].w;
                v4[db].x += yv[b][db].x; v4[db].y += yv[b][db].y; v4[db].z += yv[b][db].z; v4[db].w += yv[b][db].w;
              }
          };
          int i = 0;
#pragma unroll
          for (int j = 0; j < FS; j += 2)
            if (j + 1 < n) add2(src[j], src[j + 1]), i = j + 2;
          for (; i + 1 < n; i += 2)
            add2((bh * per_head + a.inv_slot[bh * per_head + s0 + i]) * D,
                 (bh * per_head + a.inv_slot[bh * per_head + s0 + i + 1]) * D);
          if (i < n) add(i < FS ? src[i] : (bh * per_head + a.inv_slot[bh * per_head + s0 + i]) * D);
        } else {
#pragma unroll
          for (int i = 0; i < FS; ++i)
            if (i < n) add(src[i]);
          for (int i = FS; i < n; ++i) add((bh * per_head + a.inv_slot[bh * per_head + s0 + i]) * D);
        }
      }
      const int64_t at = (bh * N + kb0 + key) * D + 4 * g;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        const bf16_t kb4[4] = {from_f32<bf16_t>(k4[db].x), from_f32<bf16_t>(k4[db].y), from_f32<bf16_t>(k4[db].z),
                               from_f32<bf16_t>(k4[db].w)};
        const bf16_t vb4[4] = {from_f32<bf16_t>(v4[db].x), from_f32<bf16_t>(v4[db].y), from_f32<bf16_t>(v4[db].z),
                               from_f32<bf16_t>(v4[db].w)};
        *reinterpret_cast<uint2 *>((bf16_t *)a.dk_out + at + 16 * db) = *reinterpret_cast<const uint2 *>(kb4);
        *reinterpret_cast<uint2 *>((bf16_t *)a.dv_out + at + 16 * db) = *reinterpret_cast<const uint2 *>(vb4);
      }
    }
    return;
  }
  // dK^T, dV^T: dims 16 db + 4 g + r of key p of group c
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    const int key = 16 * (NG * w + c) + p;
    if (key >= nkeys) continue;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const float4 kq = make_float4(dka[c][db][0] * a.scale, dka[c][db][1] * a.scale, dka[c][db][2] * a.scale,
                                    dka[c][db][3] * a.scale);
      const float4 vq = make_float4(dva[c][db][0], dva[c][db][1], dva[c][db][2], dva[c][db][3]);
      if (KM == KV_ROUTED) {
        const int64_t at = ((bh * M + e) * (int64_t)K + kb0 + key) * D + 16 * db + 4 * g;
        *reinterpret_cast<float4 *>(a.stage_k + at) = kq;
        *reinterpret_cast<float4 *>(a.stage_v + at) = vq;
      } else if (KM == KV_LMV) {
        const int64_t at = (bh * N + kb0 + key) * D + 16 * db + 4 * g;
        float4 k4 = kq, v4 = vq;
        const float4 ak = *reinterpret_cast<const float4 *>(a.dk_acc + at);
        const float4 av = *reinterpret_cast<const float4 *>(a.dv_acc + at);
        k4.x += ak.x; k4.y += ak.y; k4.z += ak.z; k4.w += ak.w;
        v4.x += av.x; v4.y += av.y; v4.z += av.z; v4.w += av.w;
        *reinterpret_cast<float4 *>(a.dk_acc + at) = k4;
        *reinterpret_cast<float4 *>(a.dv_acc + at) = v4;
      } else {
        const int64_t at = (bh * M + kb0 + key) * D + 16 * db + 4 * g;
        unsafeAtomicAdd(a.dq_lm + at, kq.x);
        unsafeAtomicAdd(a.dq_lm + at + 1, kq.y);
        unsafeAtomicAdd(a.dq_lm + at + 2, kq.z);
        unsafeAtomicAdd(a.dq_lm + at + 3, kq.w);
        unsafeAtomicAdd(a.dv_lm + at, vq.x);
        unsafeAtomicAdd(a.dv_lm + at + 1, vq.y);
        unsafeAtomicAdd(a.dv_lm + at + 2, vq.z);
        unsafeAtomicAdd(a.dv_lm + at + 3, vq.w);
      }
    }
  }
}

// Three waves per SIMD; the landmark-value mode at d = 64 runs two, whose
// registers hold two staged rows in flight in its finish (measured at 16384
// tokens, 12 heads, 2 batches: that pass 379 -> 353 us, while the routed pass
// with two waves went 361 -> 391 us).
template <int D, int KM, int NG>
__global__ __launch_bounds__(256 / NG) __attribute__((amdgpu_waves_per_eu(3))) void bwd_kv16_kernel(KvArgs a) {
  bwd_kv16_body<D, KM, NG>(a);
}
template <int NG>
__global__ __launch_bounds__(256 / NG) __attribute__((amdgpu_waves_per_eu(2))) void bwd_kv16_lmv64_kernel(KvArgs a) {
  bwd_kv16_body<64, KV_LMV, NG>(a);
}

// The landmark values' gradient in bf16 (the MFMA operand of the DMA-tiled
// landmark-value kernels) and each landmark row's D = dV~ . V~ (fp32): D / 8
// consecutive lanes per row, 8 dims each, their partial dots summed by a
// butterfly over those lanes.
template <int D>
__global__ __launch_bounds__(256) void lmv_prep_kernel(const float *__restrict__ dv_lm, const bf16_t *__restrict__ v_lm,
                                                       bf16_t *__restrict__ dv16, float *__restrict__ D_lm,
                                                       int64_t rows) {
  constexpr int L = D / 8;  // lanes per row (8 or 16: rows never straddle a wave)
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = t / L;
  const int c = 8 * (int)(t % L);
  float dsum = 0.f;
  if (row < rows) {
    const float4 f0 = *reinterpret_cast<const float4 *>(dv_lm + row * D + c);
    const float4 f1 = *reinterpret_cast<const float4 *>(dv_lm + row * D + c + 4);
    const float f[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
    float vv[8];
    load16_f32(v_lm + row * D + c, vv);
    bf16_t tt[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dsum = __builtin_fmaf(vv[i], f[i], dsum);
      tt[i] = from_f32<bf16_t>(f[i]);
    }
    *reinterpret_cast<uint4 *>(dv16 + row * D + c) = *reinterpret_cast<const uint4 *>(tt);
  }
#pragma unroll
  for (int o = L / 2; o > 0; o >>= 1) dsum += __shfl_xor(dsum, o);
  if (row < rows && c == 0) D_lm[row] = dsum;
}

// Inverse index of the top-k sets: for each token, the slots e * k + j with
// idx[e][j] = token, listed by start [BH, N + 1] and slot [BH, M * k] (a
// counting sort). One workgroup per (head, range of T tokens), its counters
// in LDS: it reads all of its head's sets, counting the slots of its own
// tokens and those of the tokens below its range (the range's base), scans
// its counts from that base, and places its slots on a second read. The
// order of a token's slots is that of the LDS atomics. Entries outside
// [0, N) are left out of the index.
constexpr int INV_THREADS = 1024, INV_WAVES = INV_THREADS / 64;
constexpr int INV_TMAX = 15360;  // tokens per workgroup: 60 KiB of counters (+ 384 B)

// f(e, tok) for the head's per_head entries, strided over the workgroup, 16
// per thread and call (e[i] the entry, tok[i] its token; -1 pads a short
// batch): up to sixteen 16-byte loads in flight where the rows allow them,
// and the callee's LDS atomics of a batch issued before their results are
// used.
template <class F>
__device__ __forceinline__ void inv_entries(const int32_t *__restrict__ ih, int per_head, F &&f) {
  int e[16], t[16];
  int i = threadIdx.x;
  if ((per_head & 3) == 0 && ((uintptr_t)ih & 15) == 0) {
    const int4 *v = reinterpret_cast<const int4 *>(ih);
    const int n4 = per_head >> 2;
    // sixteen loads in flight (a whole head of 64Ki entries in one round trip)
    for (; i + 15 * INV_THREADS < n4; i += 16 * INV_THREADS) {
      int4 x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = v[i + u * INV_THREADS];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e0 = 4 * (i + (4 * b + u) * INV_THREADS);
          const int4 y = x[4 * b + u];
          e[4 * u] = e0, e[4 * u + 1] = e0 + 1, e[4 * u + 2] = e0 + 2, e[4 * u + 3] = e0 + 3;
          t[4 * u] = y.x, t[4 * u + 1] = y.y, t[4 * u + 2] = y.z, t[4 * u + 3] = y.w;
        }
        f(e, t);
      }
    }
    for (; i + 3 * INV_THREADS < n4; i += 4 * INV_THREADS) {
      int4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = v[i + u * INV_THREADS];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e0 = 4 * (i + u * INV_THREADS);
        e[4 * u] = e0, e[4 * u + 1] = e0 + 1, e[4 * u + 2] = e0 + 2, e[4 * u + 3] = e0 + 3;
        t[4 * u] = x[u].x, t[4 * u + 1] = x[u].y, t[4 * u + 2] = x[u].z, t[4 * u + 3] = x[u].w;
      }
      f(e, t);
    }
#pragma unroll
    for (int q = 4; q < 16; ++q) e[q] = 0, t[q] = -1;
    for (; i < n4; i += INV_THREADS) {
      const int4 x = v[i];
      e[0] = 4 * i, e[1] = 4 * i + 1, e[2] = 4 * i + 2, e[3] = 4 * i + 3;
      t[0] = x.x, t[1] = x.y, t[2] = x.z, t[3] = x.w;
      f(e, t);
    }
    return;
  }
#pragma unroll
  for (int q = 1; q < 16; ++q) e[q] = 0, t[q] = -1;
  for (; i < per_head; i += INV_THREADS) {
    e[0] = i, t[0] = ih[i];
    f(e, t);
  }
}

// Grid: NXCD * ceil(nwork / NXCD) workgroups of INV_THREADS, nwork = BH *
// parts, parts = ceil(N / T); dynamic LDS (T + 2 * INV_WAVES + 64) * 4 bytes.
__global__ __launch_bounds__(INV_THREADS) void inv_index_kernel(const int32_t *__restrict__ idx,
                                                                int32_t *__restrict__ start,
                                                                int32_t *__restrict__ slot, int per_head, int N,
                                                                int T, int parts, int64_t nwork) {
  extern __shared__ uint32_t inv_lds[];  // counters, wave sums, a spare word per lane
  uint32_t *cnt = inv_lds, *wsum = inv_lds + T;
  // a head's ranges on consecutive slots of one XCD, which share its sets in L2
  const int64_t w = xcd_slot((int)blockIdx.x, (int)(gridDim.x / NXCD));
  if (w >= nwork) return;
  const int64_t bh = w / parts;
  const int t0 = (int)(w % parts) * T;
  const uint32_t nt = (uint32_t)min(N - t0, T);
  const int32_t *ih = idx + bh * per_head;
  for (uint32_t i = threadIdx.x; i < nt; i += INV_THREADS) cnt[i] = 0;
  __syncthreads();
  uint32_t below = 0;
  // (entries of other tokens count into a word of their lane past the
  // counters: atomics without branches, whose results wait only once)
  uint32_t *const spare = inv_lds + T + 2 * INV_WAVES + (threadIdx.x & 63);
  inv_entries(ih, per_head, [&](const int(&)[16], const int(&t)[16]) {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const uint32_t r = (uint32_t)t[q] - (uint32_t)t0;
      below += (uint32_t)t[q] < (uint32_t)t0 ? 1u : 0u;
      atomicAdd(r < nt ? &cnt[r] : spare, 1u);
    }
  });
  __syncthreads();
  // exclusive scan of the counts from the base (consecutive runs per thread)
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint32_t per = (nt + INV_THREADS - 1) / INV_THREADS;
  const uint32_t b0 = min(nt, threadIdx.x * per), b1 = min(nt, b0 + per);
  uint32_t sum = 0;
  for (uint32_t i = b0; i < b1; ++i) sum += cnt[i];
  const uint32_t incl = wave_inclusive_scan(sum), bw = wave_sum_u32(below);
  if (lane == 63) {
    wsum[wv] = incl;
    wsum[INV_WAVES + wv] = bw;
  }
  __syncthreads();
  uint32_t before = incl - sum, base = 0, all = 0;
#pragma unroll
  for (int i = 0; i < INV_WAVES; ++i) {
    before += i < wv ? wsum[i] : 0u;
    all += wsum[i];
    base += wsum[INV_WAVES + i];
  }
  before += base;
  for (uint32_t i = b0; i < b1; ++i) {
    const uint32_t c = cnt[i];
    cnt[i] = before;
    before += c;
  }
  __syncthreads();
  int32_t *sh = start + bh * (N + 1) + t0;
  for (uint32_t i = threadIdx.x; i < nt; i += INV_THREADS) sh[i] = (int32_t)cnt[i];
  if (threadIdx.x == 0 && t0 + (int)nt == N) sh[nt] = (int32_t)(base + all);
  __syncthreads();  // (the copy above reads the starts before the atomics move them)
  // place: cnt holds each token's next free position (< base + all <= per_head)
  int32_t *sl = slot + bh * per_head;
  inv_entries(ih, per_head, [&](const int(&e)[16], const int(&t)[16]) {
    uint32_t r[16], pos[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      r[q] = (uint32_t)t[q] - (uint32_t)t0;
      pos[q] = atomicAdd(r[q] < nt ? &cnt[r[q]] : spare, 1u);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q)
      if (r[q] < nt) sl[pos[q]] = e[q];
  });
}

// Exclusive scan of cnt over each head's N tokens into start [BH, N + 1]
// (1024 threads per head, consecutive runs per thread; the merge rounds'
// positions of the surviving tokens).
__global__ __launch_bounds__(1024) void inv_scan_kernel(const int32_t *__restrict__ cnt, int32_t *__restrict__ start,
                                                        int N) {
  __shared__ uint32_t wsum[16];
  const int64_t bh = blockIdx.x;
  const int per = (N + 1023) / 1024;
  const int b0 = threadIdx.x * per, b1 = min(N, b0 + per);
  uint32_t sum = 0;
  for (int i = b0; i < b1; ++i) sum += (uint32_t)cnt[bh * N + i];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t incl = wave_inclusive_scan(sum);
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  uint32_t before = incl - sum, all = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    before += i < w ? wsum[i] : 0u;
    all += wsum[i];
  }
  for (int i = b0; i < b1; ++i) {
    start[bh * (N + 1) + i] = (int32_t)before;
    before += (uint32_t)cnt[bh * N + i];
  }
  if (threadIdx.x == 0) start[bh * (N + 1) + N] = (int32_t)all;
}

// dk_acc, dv_acc of every token = the sum of its staged per-expert rows
// (written, not added: the first contribution). One thread per 4 dims.
template <int D>
__global__ __launch_bounds__(256) void inv_gather_kernel(const float *__restrict__ stage_k,
                                                         const float *__restrict__ stage_v,
                                                         const int32_t *__restrict__ start,
                                                         const int32_t *__restrict__ slot, float *__restrict__ dk,
                                                         float *__restrict__ dv, int64_t rows, int N, int per_head) {
  constexpr int C = D / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = t / C;
  const int c = (int)(t % C);
  if (row >= rows) return;
  const int64_t bh = row / N;
  const int tok = (int)(row % N);
  const int s0 = start[bh * (N + 1) + tok], s1 = start[bh * (N + 1) + tok + 1];
  float4 xk = make_float4(0.f, 0.f, 0.f, 0.f), xv = xk;
  for (int i = s0; i < s1; ++i) {
    const int64_t src = (bh * (int64_t)per_head + slot[bh * (int64_t)per_head + i]) * D + 4 * c;
    const float4 yk = *reinterpret_cast<const float4 *>(stage_k + src);
    const float4 yv = *reinterpret_cast<const float4 *>(stage_v + src);
    xk.x += yk.x; xk.y += yk.y; xk.z += yk.z; xk.w += yk.w;
    xv.x += yv.x; xv.y += yv.y; xv.z += yv.z; xv.w += yv.w;
  }
  *reinterpret_cast<float4 *>(dk + row * D + 4 * c) = xk;
  *reinterpret_cast<float4 *>(dv + row * D + 4 * c) = xv;
}

// Log-sum-exp (log2 units) of every landmark row's scores, from the score
// pass's per-chunk (max, sum) partials: LSE_S waves per 64 consecutive rows
// (a lane per row), wave w combining chunks w, w + LSE_S, ..., then the
// LSE_S partial pairs of each row combined through LDS.
constexpr int LSE_S = 16;
__device__ __forceinline__ void lse_combine(float &m, float &l, float2 x) {
  const float mn = fmaxf(m, x.x);
  if (mn == -INFINITY) return;  // (nothing but empty partials so far)
  l = l * __builtin_amdgcn_exp2f(m - mn) + x.y * __builtin_amdgcn_exp2f(x.x - mn);
  m = mn;
}
__global__ __launch_bounds__(64 * LSE_S) void lse_rows_kernel(const float2 *__restrict__ part_ml,
                                                              float *__restrict__ lse, int64_t rows, int M,
                                                              int nch) {
  __shared__ float2 part[LSE_S][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * 64 + lane;
  float m = -INFINITY, l = 0.f;
  if (t < rows) {
    const int64_t bh = t / M;
    const float2 *src = part_ml + bh * nch * M + (t - bh * M);
    int c = w;
    for (; c + 3 * LSE_S < nch; c += 4 * LSE_S) {
      float2 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = src[(int64_t)(c + u * LSE_S) * M];
#pragma unroll
      for (int u = 0; u < 4; ++u) lse_combine(m, l, x[u]);
    }
    for (; c < nch; c += LSE_S) lse_combine(m, l, src[(int64_t)c * M]);
  }
  part[w][lane] = make_float2(m, l);
  __syncthreads();
  if (w == 0 && t < rows) {
    m = -INFINITY, l = 0.f;
#pragma unroll
    for (int i = 0; i < LSE_S; ++i) lse_combine(m, l, part[i][lane]);
    lse[t] = m + __log2f(l);
  }
}

// The gradients in the io type: dq = the direct part + the pooling backward
// of the landmark queries' gradient (each token of window W_i receives
// dq_lm_i / |W_i|), dk, dv from their accumulators. One thread per 16 dims
// (four 4-dim chunks, FIN_TPR threads per row side by side on each chunk),
// so a token's windows are found once per 16 dims. Along each axis a
// position lies in at most two adaptive windows, among floor(pos * g / G) -
// 1 .. + 1.
template <int D> constexpr int FIN_TPR = D / 16;  // threads per row
template <typename T, int D, bool POOL, bool KV = true>
__global__ __launch_bounds__(256) void bwd_finish_kernel(const float *__restrict__ dq_direct,
                                                         const float *__restrict__ dq_lm,
                                                         const float *__restrict__ dk_acc,
                                                         const float *__restrict__ dv_acc, T *__restrict__ dq,
                                                         T *__restrict__ dk, T *__restrict__ dv, int64_t rows, int N,
                                                         int M, int gh, int gw, int lh, int lw) {
  constexpr int C = FIN_TPR<D>;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = t / C;
  const int c = (int)(t % C);
  if (row >= rows) return;
  int64_t bh;
  int tok;
  if (rows <= (int64_t)UINT32_MAX) {  // (32-bit division where the rows allow it)
    bh = (int64_t)((uint32_t)row / (uint32_t)N);
    tok = (int)((uint32_t)row - (uint32_t)bh * (uint32_t)N);
  } else {
    bh = row / N;
    tok = (int)(row % N);
  }
  const int64_t at = row * D + 4 * c;  // chunk j at at + 4 C j
  float4 x[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) x[j] = *reinterpret_cast<const float4 *>(dq_direct + at + 4 * C * j);
  if (POOL) {
    // 32-bit index arithmetic: positions stay below 2^16 (N <= 65536) and
    // window counts at most 1024 (M <= 1024), so every product below is
    // under 2^27
    const uint32_t pr = (uint32_t)tok / (uint32_t)gw, pc = (uint32_t)tok - pr * (uint32_t)gw;
    const int ar = (int)(pr * (uint32_t)lh / (uint32_t)gh), ac = (int)(pc * (uint32_t)lw / (uint32_t)gw);
    for (int a = max(0, ar - 1); a <= min(lh - 1, ar + 1); ++a) {
      const int r0 = (int)((uint32_t)a * (uint32_t)gh / (uint32_t)lh);
      const int r1 = (int)(((uint32_t)(a + 1) * (uint32_t)gh + (uint32_t)lh - 1u) / (uint32_t)lh);
      if ((int)pr < r0 || (int)pr >= r1) continue;
      for (int b = max(0, ac - 1); b <= min(lw - 1, ac + 1); ++b) {
        const int s0 = (int)((uint32_t)b * (uint32_t)gw / (uint32_t)lw);
        const int s1 = (int)(((uint32_t)(b + 1) * (uint32_t)gw + (uint32_t)lw - 1u) / (uint32_t)lw);
        if ((int)pc < s0 || (int)pc >= s1) continue;
        const float inv = 1.f / (float)((r1 - r0) * (s1 - s0));
        const float *src = dq_lm + (bh * M + a * lw + b) * D + 4 * c;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float4 y = *reinterpret_cast<const float4 *>(src + 4 * C * j);
          x[j].x += y.x * inv;
          x[j].y += y.y * inv;
          x[j].z += y.z * inv;
          x[j].w += y.w * inv;
        }
      }
    }
  }
  auto put = [&](T *dst, int j, float4 f) {
    T vals[4] = {from_f32<T>(f.x), from_f32<T>(f.y), from_f32<T>(f.z), from_f32<T>(f.w)};
    if (sizeof(T) == 2)
      *reinterpret_cast<uint2 *>(dst + at + 4 * C * j) = *reinterpret_cast<const uint2 *>(vals);
    else
      *reinterpret_cast<uint4 *>(dst + at + 4 * C * j) = *reinterpret_cast<const uint4 *>(vals);
  };
#pragma unroll
  for (int j = 0; j < 4; ++j) put(dq, j, x[j]);
  if (KV) {  // (else the landmark-value key pass wrote dk and dv)
    float4 yk[4], yv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      yk[j] = *reinterpret_cast<const float4 *>(dk_acc + at + 4 * C * j);
      yv[j] = *reinterpret_cast<const float4 *>(dv_acc + at + 4 * C * j);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      put(dk, j, yk[j]);
      put(dv, j, yv[j]);
    }
  }
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
  a.q_lse = b.q_lse;
  a.q_D = b.q_D;
  a.N = c.N;
  a.M = c.M;
  a.topk = c.k;
  a.chunk = BWD_CHUNK;
  a.scale = eff_scale(c);
  const unsigned bh = (unsigned)BH(c);
  hipError_t err;
  if (c.use_shared) {
    const int64_t rows = BH(c) * c.M;
    hipLaunchKernelGGL(lse_rows_kernel, dim3((unsigned)((rows + 63) / 64)), dim3(64 * LSE_S), 0, st,
                       (const float2 *)b.part_ml, b.lse_lm, rows, c.M, score_chunks(c));
    if ((err = launched("lse_rows_kernel", st)) != hipSuccess) return err;
  }
  // dQ of the MiTA attention, and each query's log-sum-exp and D
  int tiles = (c.N + ATT_TQ - 1) / ATT_TQ;
  if (c.use_routed) tiles = (tiles + c.M + NXCD - 1) / NXCD * NXCD;
  const dim3 grid((unsigned)tiles, bh);
  const int nlist = (c.use_shared ? c.M : 0) + (c.use_routed ? c.k : 0);
  bool done = false;
  if constexpr (sizeof(T) == 2) {
    // bf16 with the key row list in LDS: the DMA-tiled kernel
    if (list_in_lds(nlist, bwd16_tiles_lds<D>())) {
      constexpr int NG = BWD16_GROUPS<D>;
      const dim3 blk(256 / NG);
      const size_t dyn = (size_t)nlist * sizeof(uint32_t);
      if (c.use_shared && c.use_routed)
        hipLaunchKernelGGL((bwd_att16_kernel<D, true, true, NG>), grid, blk, dyn, st, a);
      else if (c.use_routed)
        hipLaunchKernelGGL((bwd_att16_kernel<D, false, true, NG>), grid, blk, dyn, st, a);
      else
        hipLaunchKernelGGL((bwd_att16_kernel<D, true, false, NG>), grid, blk, dyn, st, a);
      done = true;
    }
  }
  if (!done) {
    if (c.use_shared && c.use_routed)
      hipLaunchKernelGGL((bwd_kernel<T, D, BWD_ATT, true, true>), grid, dim3(256), 0, st, a);
    else if (c.use_routed)
      hipLaunchKernelGGL((bwd_kernel<T, D, BWD_ATT, false, true>), grid, dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((bwd_kernel<T, D, BWD_ATT, true, false>), grid, dim3(256), 0, st, a);
  }
  if ((err = launched("bwd_attend_kernel", st)) != hipSuccess) return err;
  KvArgs kv{};
  kv.q = b.q;
  kv.k = b.k;
  kv.v = b.v;
  kv.dO = b.dO;
  kv.q_lm = b.q_lm;
  kv.v_lm = b.v_lm;
  kv.idx = b.idx;
  kv.perm = b.perm;
  kv.offsets = b.offsets;
  kv.q_lse = b.q_lse;
  kv.q_D = b.q_D;
  kv.stage_k = b.stage_k;
  kv.stage_v = b.stage_v;
  kv.dq_lm = b.dq_lm_acc;
  kv.dv_lm = b.dv_lm_acc;
  kv.N = c.N;
  kv.M = c.M;
  kv.topk = c.k;
  kv.scale = eff_scale(c);
  // bf16 with the landmark values: their key pass owns every token row, so it
  // also sums the routed keys' staged rows and writes dk, dv (no gather pass,
  // no fp32 accumulators of the keys)
  const bool fused_finish = sizeof(T) == 2 && c.use_shared;
  if (c.use_routed) {
    // routed keys: per-expert sums staged, then summed per token
    kv.nblk = (c.k + BWD_KB - 1) / BWD_KB;
    kv.ntotal = c.M * kv.nblk;
    const unsigned nx = (unsigned)((kv.ntotal + NXCD - 1) / NXCD * NXCD);
    if constexpr (sizeof(T) == 2)
      hipLaunchKernelGGL((bwd_kv16_kernel<D, KV_ROUTED, BWD16_GROUPS<D>>), dim3(nx, bh), dim3(256 / BWD16_GROUPS<D>), 0, st,
                         kv);
    else
      hipLaunchKernelGGL((bwd_kv_kernel<T, D, true>), dim3(nx, bh), dim3(256), 0, st, kv);
    if ((err = launched("bwd_kv_kernel", st)) != hipSuccess) return err;
    const int per_head = c.M * c.k;
    // token ranges per head: about one workgroup per CU over all heads (a
    // head's ranges on one XCD), at least 256 tokens each, at most INV_TMAX
    const int64_t heads = BH(c), per_xcd = (heads + NXCD - 1) / NXCD;
    int parts = (int)std::max<int64_t>(1, 256 / (NXCD * per_xcd));
    parts = std::min(parts, std::max(1, c.N / 256));
    parts = std::max(parts, (c.N + INV_TMAX - 1) / INV_TMAX);
    const int span = (c.N + parts - 1) / parts;
    parts = (c.N + span - 1) / span;
    const int64_t nwork = heads * parts;
    hipLaunchKernelGGL(inv_index_kernel, dim3((unsigned)((nwork + NXCD - 1) / NXCD * NXCD)), dim3(INV_THREADS),
                       (size_t)(span + 2 * INV_WAVES + 64) * 4, st, b.idx, b.inv_start, b.inv_slot, per_head, c.N, span, parts,
                       nwork);
    if ((err = launched("inv_index_kernel", st)) != hipSuccess) return err;
    if (!fused_finish) {  // (else the landmark-value key pass sums the staged rows)
      const int64_t rows = BH(c) * c.N;
      hipLaunchKernelGGL((inv_gather_kernel<D>), dim3((unsigned)((rows * (D / 4) + 255) / 256)), dim3(256), 0, st,
                         b.stage_k, b.stage_v, b.inv_start, b.inv_slot, b.dk_acc, b.dv_acc, rows, c.N, per_head);
      if ((err = launched("inv_gather_kernel", st)) != hipSuccess) return err;
    }
  }
  if (c.use_shared) {
    // shared keys (the landmarks): atomic adds per landmark block and query chunk
    kv.nblk = (c.M + BWD_KB - 1) / BWD_KB;
    kv.ntotal = kv.nblk * ((c.N + BWD_QCHUNK - 1) / BWD_QCHUNK);
    const unsigned nx = (unsigned)((kv.ntotal + NXCD - 1) / NXCD * NXCD);
    if constexpr (sizeof(T) == 2)
      hipLaunchKernelGGL((bwd_kv16_kernel<D, KV_SHARED, BWD16_GROUPS<D>>), dim3(nx, bh), dim3(256 / BWD16_GROUPS<D>), 0,
                         st, kv);
    else
      hipLaunchKernelGGL((bwd_kv_kernel<T, D, false>), dim3(nx, bh), dim3(256), 0, st, kv);
    if ((err = launched("bwd_kv_shared_kernel", st)) != hipSuccess) return err;
    // the landmark values (Eq. landmark-value), once their gradient is complete
    const int nlb = (c.M + BWD_TQ - 1) / BWD_TQ, nch = (c.N + BWD_CHUNK - 1) / BWD_CHUNK;
    if constexpr (sizeof(T) == 2) {
      // bf16: the landmark queries' gradient by landmark blocks and key
      // chunks (atomic adds per chunk), then the keys' gradient by token
      // blocks with all landmark rows streamed (each row added once)
      const int64_t mrows = BH(c) * c.M;
      hipLaunchKernelGGL((lmv_prep_kernel<D>), dim3((unsigned)((mrows * (D / 8) + 255) / 256)), dim3(256), 0, st,
                         b.dv_lm_acc, (const bf16_t *)b.v_lm, (bf16_t *)b.dv_lm16, b.D_lm, mrows);
      if ((err = launched("lmv_prep_kernel", st)) != hipSuccess) return err;
      a.dv_lm16 = b.dv_lm16;
      a.D_lm = b.D_lm;
      constexpr int NG = BWD16_GROUPS<D>;
      // longer key chunks than the fp32 kernel's: fewer atomic adds of the
      // partial sums, which all chunks of a landmark block add to the same rows
      a.chunk = BWD16_LMV_CHUNK;
      const int nch16 = (c.N + BWD16_LMV_CHUNK - 1) / BWD16_LMV_CHUNK;
      hipLaunchKernelGGL((bwd_att16_kernel<D, false, false, NG, true>), dim3((unsigned)(nlb * nch16), bh),
                         dim3(256 / NG), (size_t)BWD16_LMV_CHUNK * sizeof(uint32_t), st, a);
      if ((err = launched("bwd_landmark_kernel", st)) != hipSuccess) return err;
      kv.dv_lm16 = b.dv_lm16;
      kv.lse_lm = b.lse_lm;
      kv.D_lm = b.D_lm;
      kv.dk_acc = b.dk_acc;
      kv.dv_acc = b.dv_acc;
      kv.inv_start = c.use_routed ? b.inv_start : nullptr;
      kv.inv_slot = c.use_routed ? b.inv_slot : nullptr;
      kv.dk_out = b.dk;
      kv.dv_out = b.dv;
      kv.ntotal = (c.N + BWD_KB - 1) / BWD_KB;
      const unsigned nxl = (unsigned)((kv.ntotal + NXCD - 1) / NXCD * NXCD);
      if constexpr (D == 64)
        hipLaunchKernelGGL((bwd_kv16_lmv64_kernel<NG>), dim3(nxl, bh), dim3(256 / NG), 0, st, kv);
      else
        hipLaunchKernelGGL((bwd_kv16_kernel<D, KV_LMV, NG>), dim3(nxl, bh), dim3(256 / NG), 0, st, kv);
      if ((err = launched("bwd_kv_landmark_kernel", st)) != hipSuccess) return err;
    } else {
      hipLaunchKernelGGL((bwd_kernel<T, D, BWD_LMV, true, false>), dim3((unsigned)(nlb * nch), bh), dim3(256), 0,
                         st, a);
      if ((err = launched("bwd_landmark_kernel", st)) != hipSuccess) return err;
    }
  }
  const int64_t rows = BH(c) * c.N;
  const int64_t threads = rows * FIN_TPR<D>;
  const dim3 fg((unsigned)((threads + 255) / 256));
  if (fused_finish)
    hipLaunchKernelGGL((bwd_finish_kernel<T, D, true, false>), fg, dim3(256), 0, st, b.dq_direct, b.dq_lm_acc,
                       b.dk_acc, b.dv_acc, (T *)b.dq, (T *)b.dk, (T *)b.dv, rows, c.N, c.M, c.grid_h, c.grid_w,
                       c.lm_h, c.lm_w);
  else if (c.use_shared)
    hipLaunchKernelGGL((bwd_finish_kernel<T, D, true>), fg, dim3(256), 0, st, b.dq_direct, b.dq_lm_acc, b.dk_acc,
                       b.dv_acc, (T *)b.dq, (T *)b.dk, (T *)b.dv, rows, c.N, c.M, c.grid_h, c.grid_w, c.lm_h, c.lm_w);
  else
    hipLaunchKernelGGL((bwd_finish_kernel<T, D, false>), fg, dim3(256), 0, st, b.dq_direct, b.dq_lm_acc, b.dk_acc,
                       b.dv_acc, (T *)b.dq, (T *)b.dk, (T *)b.dv, rows, c.N, c.M, c.grid_h, c.grid_w, c.lm_h, c.lm_w);
  return launched("bwd_finish_kernel", st);
}

hipError_t launch_scan_counts(const int32_t *cnt, int32_t *start, int n, int64_t bh, hipStream_t st) {
  hipLaunchKernelGGL(inv_scan_kernel, dim3((unsigned)bh), dim3(1024), 0, st, cnt, start, n);
  return launched("scan_counts_kernel", st);
}

hipError_t launch_backward(const mita_cfg_t &c, const BwdBufs &b, hipStream_t st) {
  if (c.dtype == MITA_F32) return c.d == 64 ? bwd_t<float, 64>(c, b, st) : bwd_t<float, 128>(c, b, st);
  return c.d == 64 ? bwd_t<bf16_t, 64>(c, b, st) : bwd_t<bf16_t, 128>(c, b, st);
}

}  // namespace mita
