// flash.hpp - one wave's online-softmax attention step over a 64-key tile
// staged in LDS, on MFMA. Used for the landmark values (Eq. landmark-value:
// landmark queries attending over all keys) and for the MiTA output
// (Eq. mita: queries attending over shared plus routed keys).
//
// Layout per wave: 16 queries (the columns of the MFMA tiles). Scores are
// formed transposed, S^T = K Q^T (keys are rows), so every lane owns one query
// column: its running max, running sum and output rescale stay lane-local and
// only the tile max needs a reduction over the four lane groups. P^T leaves
// the score accumulators already in the B-operand layout of O^T += V^T P^T,
// which needs V transposed in LDS (keys contiguous per dimension).
#pragma once
#include "cdna4.hpp"

namespace mita {

constexpr int TK = 64;        // keys per tile
constexpr int BLOCK = 256;    // 4 waves per workgroup
constexpr float LOG2E = 1.4426950408889634f;

template <typename T, int D> struct TileDims {
  static constexpr int VE = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int KSTR = D + VE;             // padded K row (elements)
  static constexpr int VSTR = TK + VE;            // padded V^T row (elements)
  static constexpr int K_ELEMS = TK * KSTR;
  static constexpr int V_ELEMS = D * VSTR;
};

// Cooperative load of up to 64 key/value rows into LDS: Ks row-major [64][D],
// Vt transposed [D][64]. Rows >= nrows are zero-filled (masked keys must
// contribute exact zeros to P V). Row r comes from row (rowidx ? rowidx[r] : r)
// of kbase / vbase. LOAD_V = false stages keys only.
template <typename T, int D, bool LOAD_V = true>
__device__ __forceinline__ void load_kv_tile(T *__restrict__ Ks, T *__restrict__ Vt, const T *__restrict__ kbase,
                                             const T *__restrict__ vbase, const int32_t *__restrict__ rowidx,
                                             int nrows) {
  using TD = TileDims<T, D>;
  constexpr int VE = TD::VE;
  constexpr int CPR = D / VE;
#pragma unroll
  for (int c = threadIdx.x; c < TK * CPR; c += BLOCK) {
    const int r = c / CPR, ch = c % CPR;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (r < nrows) {
      const int64_t src = rowidx ? (int64_t)rowidx[r] : (int64_t)r;
      kv = *reinterpret_cast<const uint4 *>(kbase + src * D + ch * VE);
      if (LOAD_V) vv = *reinterpret_cast<const uint4 *>(vbase + src * D + ch * VE);
    }
    *reinterpret_cast<uint4 *>(Ks + r * TD::KSTR + ch * VE) = kv;
    if (LOAD_V) {
      const T *ve = reinterpret_cast<const T *>(&vv);
#pragma unroll
      for (int e = 0; e < VE; ++e) Vt[(ch * VE + e) * TD::VSTR + r] = ve[e];
    }
  }
}

// S^T for the tile: acc[kb][r] = K[kb*16 + 4g + r] . q[p]  (g = lane / 16, p = lane % 16).
template <typename T, int D>
__device__ __forceinline__ void tile_scores(f32x4 (&acc)[4], const T *__restrict__ Ks, const Frag<T> (&qf)[D / 32]) {
  using TD = TileDims<T, D>;
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    acc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      Frag<T> a;
      a.load(Ks + (kb * 16 + p) * TD::KSTR + ks * 32 + g * 8);
      acc[kb] = mma(a, qf[ks], acc[kb]);
    }
  }
}

// Running state of one wave (16 query columns). m is in the log2 domain.
template <int D> struct Online {
  f32x4 o[D / 16];
  float m, l;
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    m = -INFINITY;
    l = 0.f;
  }
};

// Online-softmax update with the tile's scores (acc, unscaled dot products) and
// O^T += V^T P^T. Keys kb*16 + 4g + r >= nvalid are masked out. sl2 = scale * log2(e).
// The tile must hold at least one valid key.
template <typename T, int D>
__device__ __forceinline__ void tile_softmax_pv(Online<D> &st, const f32x4 (&acc)[4], const T *__restrict__ Vt, int nvalid,
                                                float sl2) {
  using TD = TileDims<T, D>;
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  float t[4][4];
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = kb * 16 + 4 * g + r;
      t[kb][r] = key < nvalid ? acc[kb][r] * sl2 : -INFINITY;
      mx = fmaxf(mx, t[kb][r]);
    }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(st.m, mx);
  const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
  st.m = m_new;
  float ls = 0.f;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      t[kb][r] = __builtin_amdgcn_exp2f(t[kb][r] - m_new);
      ls += t[kb][r];
    }
  st.l = st.l * alpha + ls;
#pragma unroll
  for (int i = 0; i < D / 16; ++i) st.o[i] *= alpha;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    // reduction slice of group g: keys 32j + 4g + (0..3) and 32j + 16 + 4g + (0..3)
    const float pv[8] = {t[2 * j][0],     t[2 * j][1],     t[2 * j][2],     t[2 * j][3],
                         t[2 * j + 1][0], t[2 * j + 1][1], t[2 * j + 1][2], t[2 * j + 1][3]};
    Frag<T> b;
    b.from_f32(pv);
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const T *row = Vt + (db * 16 + p) * TD::VSTR + 32 * j + 4 * g;
      Frag<T> a;
      a.load2x4(row, row + 16);
      st.o[db] = mma(a, b, st.o[db]);
    }
  }
}

// Sum of the per-lane running sums over the four lane groups of a column.
__device__ __forceinline__ float column_sum(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

}  // namespace mita
