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
// The running max of the online softmax is a reference value only: it is
// raised when some query's tile max exceeds it by more than this (log2
// units), so weights stay below 2^8 and the accumulators are rescaled only
// a few times per query instead of on most tiles. Any reference gives the
// same softmax; the weights and sums just carry a common factor.
constexpr float RESCALE_LOG2 = 8.f;

template <typename T, int D> struct TileDims {
  static constexpr int VE = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int KSTR = D + VE;             // padded K row (elements)
  // padded V^T row: 136 bytes (bf16) / 272 bytes (fp32) keep the 8 / 16-byte
  // fragment reads aligned and spread the transposing writes over the banks
  static constexpr int VSTR = TK + 4;
  // bf16, d = 64: V^T row R starts at R * VSTR + 8 * ((R >> 4) & 3). With that
  // shift per 16-row group the transposing stores of a tile (8 chunks of 8
  // rows, 2-key words) fall in 32 distinct banks instead of 8, while the P V
  // fragment reads (16 consecutive rows, one shift) stay conflict-free and in
  // ascending address order.
  static constexpr bool VSHIFT = sizeof(T) == 2 && D == 64;
  static constexpr int K_ELEMS = TK * KSTR;
  static constexpr int V_ELEMS = D * VSTR + (VSHIFT ? 24 : 0);
  __device__ __forceinline__ static int vrow(int row) { return row * VSTR + (VSHIFT ? 8 * ((row >> 4) & 3) : 0); }
};

// Cooperative load of up to 64 key rows into LDS, Ks row-major [64][D]. Rows
// >= nrows are zero-filled. Row r comes from row (rowidx ? rowidx[r] : r) of
// kbase.
template <typename T, int D>
__device__ __forceinline__ void load_k_tile(T *__restrict__ Ks, const T *__restrict__ kbase,
                                            const int32_t *__restrict__ rowidx, int nrows) {
  using TD = TileDims<T, D>;
  constexpr int VE = TD::VE;
  constexpr int CPR = D / VE;
#pragma unroll
  for (int c = threadIdx.x; c < TK * CPR; c += BLOCK) {
    const int r = c / CPR, ch = c % CPR;
    uint4 kv = make_uint4(0, 0, 0, 0);
    if (r < nrows) {
      const int64_t src = rowidx ? (int64_t)rowidx[r] : (int64_t)r;
      kv = *reinterpret_cast<const uint4 *>(kbase + src * D + ch * VE);
    }
    *reinterpret_cast<uint4 *>(Ks + r * TD::KSTR + ch * VE) = kv;
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

// Running state of one wave (16 query columns). m is in the log2 domain and
// at most RESCALE_LOG2 below the largest scaled score seen so far; thr is
// (m + RESCALE_LOG2) / (scale * log2 e), the raw dot product above which m
// has to be raised. The
// running sum of the weights is an MFMA accumulator (an all-ones A operand
// against the same P^T as the values), so every element of lsum holds the
// full sum for its lane's query column, of the very weights (as rounded for
// the MFMA) that multiply V.
template <int D> struct Online {
  f32x4 o[D / 16];
  f32x4 lsum;
  float m, thr;
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    lsum = f32x4{0.f, 0.f, 0.f, 0.f};
    m = -INFINITY;
    thr = -INFINITY;
  }
  __device__ __forceinline__ float l() const { return lsum[0]; }
};

template <typename T> __device__ __forceinline__ Frag<T> ones_frag();
template <> __device__ __forceinline__ Frag<bf16_t> ones_frag<bf16_t>() {
  Frag<bf16_t> f;
  f.v = make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u);  // bf16 1.0 x 8
  return f;
}
template <> __device__ __forceinline__ Frag<float> ones_frag<float>() {
  Frag<float> f;
  f.a = make_float4(1.f, 1.f, 1.f, 1.f);
  f.b = f.a;
  return f;
}

// Online-softmax update with the tile's scores (acc, unscaled dot products) and
// O^T += V^T P^T. sl2 = scale * log2(e) > 0; the reference max is kept in
// scaled log2 units and p = exp2(dot * sl2 - m) is one FMA. Whether the
// reference has to move is decided on each lane's own 16 raw dots against
// thr (a positive scale keeps the order); only then is the column max over
// the four lane groups formed. With MASKED, keys
// kb*16 + 4g + r >= nvalid are excluded (only the last tile of a key range is
// partial). The tile must hold at least one valid key.
template <typename T, int D, bool MASKED = true>
__device__ __forceinline__ void tile_softmax_pv(Online<D> &st, const f32x4 (&acc)[4], const T *__restrict__ Vt, int nvalid,
                                                float sl2) {
  using TD = TileDims<T, D>;
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool ok = !MASKED || kb * 16 + 4 * g + r < nvalid;
      mx = fmaxf(mx, ok ? acc[kb][r] : -INFINITY);
    }
  // a new reference max only when some column's tile max is more than
  // RESCALE_LOG2 above it (always on the first tile: m = -inf)
  if (__ballot(mx > st.thr)) {
    const float m_new = fmaxf(st.m, max_lane_groups(mx) * sl2);
    const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
    st.m = m_new;
    st.thr = (m_new + RESCALE_LOG2) * __builtin_amdgcn_rcpf(sl2);
#pragma unroll
    for (int i = 0; i < D / 16; ++i) st.o[i] *= alpha;
    st.lsum *= alpha;
  }
  const float m_ref = st.m;
  float t[4][4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[kb][r], sl2, -m_ref));
      if (MASKED && kb * 16 + 4 * g + r >= nvalid) e = 0.f;
      t[kb][r] = e;
    }
  const Frag<T> ones = ones_frag<T>();
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    // reduction slice of group g: keys 32j + 4g + (0..3) and 32j + 16 + 4g + (0..3)
    const float pv[8] = {t[2 * j][0],     t[2 * j][1],     t[2 * j][2],     t[2 * j][3],
                         t[2 * j + 1][0], t[2 * j + 1][1], t[2 * j + 1][2], t[2 * j + 1][3]};
    Frag<T> b;
    b.from_f32(pv);
    st.lsum = mma(ones, b, st.lsum);
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const T *row = Vt + TD::vrow(db * 16 + p) + 32 * j + 4 * g;
      Frag<T> a;
      a.load2x4(row, row + 16);
      st.o[db] = mma(a, b, st.o[db]);
    }
  }
}

// Running state of a wave that owns 32 queries: two 16-column groups, each
// kept as in Online (reference max m, its raw-dot threshold thr, weight sums
// as an MFMA accumulator).
template <int D> struct Online2 {
  f32x4 o[2][D / 16];
  f32x4 lsum[2];
  float m[2], thr[2];
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int i = 0; i < D / 16; ++i) o[c][i] = f32x4{0.f, 0.f, 0.f, 0.f};
      lsum[c] = f32x4{0.f, 0.f, 0.f, 0.f};
      m[c] = -INFINITY;
      thr[c] = -INFINITY;
    }
  }
  __device__ __forceinline__ float l(int c) const { return lsum[c][0]; }
  __device__ __forceinline__ float mval(int c) const { return m[c]; }
};

// One wave's online-softmax step over one 32-key half of an LDS tile (keys
// 32h .. 32h + 31) for its 32 queries (fragments qf[c], c = column group):
// S^T = K Q^T for both groups from the same key fragments, then the same
// update as tile_softmax_pv on 8 dots per lane and group, and O^T += V^T P^T
// with every V^T fragment serving both groups. Splitting a tile's keys
// between two waves halves the LDS bytes each wave reads per score. With
// MASKED only keys 32h + i, i < nvalid (>= 1) count.
template <typename T, int D, bool MASKED = false>
__device__ __forceinline__ void half_tile_attend(Online2<D> &st, const T *__restrict__ Ks, const T *__restrict__ Vt,
                                                 int h, const Frag<T> (&qf)[2][D / 32], int nvalid, float sl2) {
  using TD = TileDims<T, D>;
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  f32x4 acc[2][2];  // [group][16-key block]
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    acc[0][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc[1][kb] = acc[0][kb];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      Frag<T> a;
      a.load(Ks + (32 * h + kb * 16 + p) * TD::KSTR + ks * 32 + g * 8);
      acc[0][kb] = mma(a, qf[0][ks], acc[0][kb]);
      acc[1][kb] = mma(a, qf[1][ks], acc[1][kb]);
    }
  }
  float mx[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    mx[c] = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool ok = !MASKED || kb * 16 + 4 * g + r < nvalid;
        mx[c] = fmaxf(mx[c], ok ? acc[c][kb][r] : -INFINITY);
      }
  }
  if (__ballot(mx[0] > st.thr[0] || mx[1] > st.thr[1])) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      // only a column past its own threshold moves its reference, so a
      // query's arithmetic does not depend on the other queries of the tile
      const float cmx = max_lane_groups(mx[c]);
      const float m_new = cmx > st.thr[c] ? fmaxf(st.m[c], cmx * sl2) : st.m[c];
      const float alpha = __builtin_amdgcn_exp2f(st.m[c] - m_new);
      st.m[c] = m_new;
      st.thr[c] = (m_new + RESCALE_LOG2) * __builtin_amdgcn_rcpf(sl2);
#pragma unroll
      for (int i = 0; i < D / 16; ++i) st.o[c][i] *= alpha;
      st.lsum[c] *= alpha;
    }
  }
  const Frag<T> ones = ones_frag<T>();
  Frag<T> b[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    // reduction slice of group g: keys 32h + 4g + (0..3) and 32h + 16 + 4g + (0..3)
    float pv[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float e = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[c][kb][r], sl2, -st.m[c]));
        if (MASKED && kb * 16 + 4 * g + r >= nvalid) e = 0.f;
        pv[4 * kb + r] = e;
      }
    b[c].from_f32(pv);
    st.lsum[c] = mma(ones, b[c], st.lsum[c]);
  }
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    const T *row = Vt + TD::vrow(db * 16 + p) + 32 * h + 4 * g;
    Frag<T> a;
    a.load2x4(row, row + 16);
    st.o[0][db] = mma(a, b[0], st.o[0][db]);
    st.o[1][db] = mma(a, b[1], st.o[1][db]);
  }
}

// ---------------------------------------------------------------------------
// bf16 tiles staged by LDS DMA (global_load_lds_dwordx4: each lane's 16
// bytes land at consecutive LDS addresses, 1 KB per wave instruction, with no
// registers involved). K and V are both kept row-major, rows of D elements
// without padding; 16-byte slot s of row r holds chunk s ^ swz(r). The LDS
// serves 256 bytes per cycle from 64 banks: 16 lanes of a 16-byte read, 32
// lanes of an 8-byte one. The swizzle makes both the K fragment reads (16
// consecutive rows at one chunk) and the V transpose reads (8 rows, 4 pieces
// each, per 32 lanes) touch every bank once per cycle (d = 64). The
// A operand of O^T += V^T P^T comes from ds_read_b64_tr_b16: in each 16-lane
// group, lane 4e + c addresses piece c (4 elements) of row e of a 4 x 16
// block and lane i receives column i, i.e. 4 consecutive keys of one
// dimension.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int swz(int r) { return (r & 6) | ((r >> 3) & 1); }

constexpr int TK32 = 32;  // rows of a DMA-staged tile

template <int D, int ROWS = TK, int NW = 4> struct DmaTile {
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;       // rows per wave instruction
  static constexpr int NI = ROWS / RPI;      // instructions per ROWS-row matrix
  static constexpr int PW = NI / NW;         // per wave of an NW-wave workgroup
  static constexpr int BYTES = ROWS * D * 2; // one ROWS-row matrix
  static_assert(PW >= 1 && NI % NW == 0, "whole instructions per wave");
};

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

// Keep x in a register as computed here: the compiler may not recompute it
// inside a loop (it does so to save registers, at a few VALU instructions per
// use).
template <typename T> __device__ __forceinline__ void pin(T &x) { asm volatile("" : "+v"(x)); }

// Per-lane part of the DMA of one tile, fixed for every tile: the tile row r
// this lane loads (rows start at multiples of 32, so the swizzle of r is the
// same in every tile) and its 16-byte source chunk (sl ^ swz(r)) << 4.
template <int D, int ROWS, int NW = 4> struct DmaLane {
  static constexpr int PW = DmaTile<D, ROWS, NW>::PW;
  uint32_t row[PW];    // r, per instruction of the wave
  uint32_t chunk[PW];  // byte offset of the swizzled chunk within the row
  __device__ __forceinline__ void init(int w, int lane) {
    using DT = DmaTile<D, ROWS, NW>;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int r = (w * PW + j) * DT::RPI + lane / DT::CPR;
      row[j] = (uint32_t)r;
      chunk[j] = (uint32_t)(((lane % DT::CPR) ^ swz(r)) << 4);
      pin(chunk[j]);
    }
  }
};

// Issue the DMA of one tile: rows r < ROWS of K (and, WITH_V, of V) from
// byte offsets offs[r] past kb and vb (without FULL, rows >= nrows take
// offset offs[0]: real data, masked later).
template <int D, bool FULL = false, int ROWS = TK, int NW = 4, bool WITH_V = true>
__device__ __forceinline__ void dma_tile(bf16_t *Kl, bf16_t *Vl, const bf16_t *kb, const bf16_t *vb,
                                         const uint32_t *offs, int nrows) {
  using DT = DmaTile<D, ROWS, NW>;
  // the wave index as a scalar: the LDS destinations (M0) need no readfirstlane
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < DT::PW; ++j) {
    const int ins = w * DT::PW + j;
    const int r = ins * DT::RPI + lane / DT::CPR;
    const int sl = lane % DT::CPR;
    const uint32_t go = offs[FULL || r < nrows ? r : 0] + (uint32_t)((sl ^ swz(r)) << 4);
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(kb) + go,
                                     (lds_void_t *)(reinterpret_cast<char *>(Kl) + ins * 1024), 16, 0, 0);
    if (WITH_V)
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(vb) + go,
                                       (lds_void_t *)(reinterpret_cast<char *>(Vl) + ins * 1024), 16, 0, 0);
  }
}

// The same for a whole tile (every row valid) with the lane's precomputed
// rows and chunks.
template <int D, int ROWS, int NW = 4, bool WITH_V = true>
__device__ __forceinline__ void dma_tile_lane(bf16_t *Kl, bf16_t *Vl, const bf16_t *kb, const bf16_t *vb,
                                              const uint32_t *offs, const DmaLane<D, ROWS, NW> &dl) {
  using DT = DmaTile<D, ROWS, NW>;
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
#pragma unroll
  for (int j = 0; j < DT::PW; ++j) {
    const int ins = w * DT::PW + j;
    const uint32_t go = offs[dl.row[j]] + dl.chunk[j];
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(kb) + go,
                                     (lds_void_t *)(reinterpret_cast<char *>(Kl) + ins * 1024), 16, 0, 0);
    if (WITH_V)
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(vb) + go,
                                       (lds_void_t *)(reinterpret_cast<char *>(Vl) + ins * 1024), 16, 0, 0);
  }
}

// ---------------------------------------------------------------------------
// A wave's online softmax over DMA-staged 32-key tiles for its 16-query
// groups (one MFMA column group each; lane (g, p) holds column p). The score MFMAs start
// from the splat -m of the column's reference max (log2 units; the query
// fragments are pre-scaled by scale * log2 e), so they yield the exp2
// argument directly. The reference is the first tile's column max and moves
// only when a column's shifted scores exceed RESCALE_LOG2. The weight sum is
// kept per lane over the lane's own 8 keys of each tile, from the very bf16
// weights that multiply V (v_dot2c_f32_bf16 against a pair of ones); the
// query's sum is the sum over the four lane groups of its column, formed
// once at the end in a fixed order.
// ---------------------------------------------------------------------------
template <int D> struct Att16 {
  f32x4 o[D / 16];  // O^T: dims 16 db + 4 g + r of query p
  f32x4 nm;         // -m, splat
  f32x4 l;          // the weight sum of query p (an all-ones MFMA row block; every element)
};

// Per-lane LDS byte offsets within one tile buffer, fixed for every tile:
// K fragment of reduction step ks (row p of the first 16-key block; the
// second block is 16 rows on, same swizzle) and the V^T transpose reads of
// dimension block db (row 4 g + e of the first 16-key half; the second half
// is 16 rows on).
template <int D> struct Att16Addr {
  uint32_t k[D / 32];
  uint32_t v[D / 16];
  __device__ __forceinline__ void init() {
    constexpr int RB = 2 * D;  // bytes per row
    const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      k[ks] = (uint32_t)(p * RB + (((4 * ks + g) ^ swz(p)) << 4));
      pin(k[ks]);
    }
    const int e = p >> 2, c4 = p & 3, R = 4 * g + e;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      v[db] = (uint32_t)(R * RB + (((2 * db + (c4 >> 1)) ^ swz(R)) << 4) + ((c4 & 1) << 3));
      pin(v[db]);
    }
  }
};

// The tile functions below run NGB (<= NG) query groups of one wave over the
// same K and V fragments: each fragment read from LDS feeds one MFMA per
// group.

// Shifted scores of the tile's 32 keys (acc[c][kb][r]: key 16 kb + 4 g + r of
// query p of group c).
template <int D, int NGB, int NG>
__device__ __forceinline__ void att16_scores(f32x4 (&acc)[NG][2], const Att16<D> (&st)[NG],
                                             const bf16_t *__restrict__ Kl, const Att16Addr<D> &ad,
                                             const Frag<bf16_t> (&qf)[NG][D / 32]) {
  constexpr int RB = 2 * D;
  const char *kbase = reinterpret_cast<const char *>(Kl);
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int c = 0; c < NGB; ++c) acc[c][kb] = st[c].nm;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      Frag<bf16_t> a;
      a.v = *reinterpret_cast<const uint4 *>(kbase + ad.k[ks] + kb * 16 * RB);
#pragma unroll
      for (int c = 0; c < NGB; ++c) acc[c][kb] = mma(a, qf[c][ks], acc[c][kb]);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// Weights of the tile (exp2 of the shifted scores; with MASKED keys i >=
// nvalid weigh 0), each lane's weight sum, and O^T += V^T P^T per group.
template <int D, bool MASKED, int NGB, int NG>
__device__ __forceinline__ void att16_pv(Att16<D> (&st)[NG], const f32x4 (&acc)[NG][2],
                                         const bf16_t *__restrict__ Vl, const Att16Addr<D> &ad, int nvalid) {
  constexpr int RB = 2 * D;
  const int g = (threadIdx.x & 63) >> 4;
  Frag<bf16_t> b[NG];
#pragma unroll
  for (int c = 0; c < NGB; ++c) {
    float pv[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = __builtin_amdgcn_exp2f(acc[c][kb][r]);
        if (MASKED && kb * 16 + 4 * g + r >= nvalid) x = 0.f;
        pv[4 * kb + r] = x;
      }
    b[c].from_f32(pv);
    // the sum of the rounded weights: an all-ones A operand against the same
    // P^T (every row of the result holds the column sum)
    st[c].l = mma(ones_frag<bf16_t>(), b[c], st[c].l);
  }
  const char *vbase = reinterpret_cast<const char *>(Vl);
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    uint2 half[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
      half[h2] = __builtin_bit_cast(
          uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(vbase + ad.v[db] + h2 * 16 * RB)));
    Frag<bf16_t> a;
    a.v = make_uint4(half[0].x, half[0].y, half[1].x, half[1].y);
    if (db == 0) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int c = 0; c < NGB; ++c) st[c].o[db] = mma(a, b[c], st[c].o[db]);
  }
  __builtin_amdgcn_s_setprio(0);
}

// Maximum of the lane's 8 shifted scores (with MASKED only keys < nvalid).
template <bool MASKED> __device__ __forceinline__ float att16_lane_max(const f32x4 (&acc)[2], int nvalid) {
  const int g = (threadIdx.x & 63) >> 4;
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) mx = fmaxf(mx, (!MASKED || kb * 16 + 4 * g + r < nvalid) ? acc[kb][r] : -INFINITY);
  return mx;
}

// The first tile of a wave: its column maxima become the references.
template <int D, bool MASKED, int NGB, int NG>
__device__ __forceinline__ void att16_first(Att16<D> (&st)[NG], const bf16_t *__restrict__ Kl,
                                            const bf16_t *__restrict__ Vl, const Att16Addr<D> &ad,
                                            const Frag<bf16_t> (&qf)[NG][D / 32], int nvalid) {
#pragma unroll
  for (int c = 0; c < NGB; ++c) {
#pragma unroll
    for (int i = 0; i < D / 16; ++i) st[c].o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    st[c].nm = f32x4{0.f, 0.f, 0.f, 0.f};
    st[c].l = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  f32x4 acc[NG][2];
  att16_scores<D, NGB>(acc, st, Kl, ad, qf);
#pragma unroll
  for (int c = 0; c < NGB; ++c) {
    const float cm = max_lane_groups(att16_lane_max<MASKED>(acc[c], nvalid));
    st[c].nm -= cm;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) acc[c][kb] -= cm;
  }
  att16_pv<D, MASKED, NGB>(st, acc, Vl, ad, nvalid);
}

// A later tile, with the reference check: after the scores, a group some of
// whose columns need it (att16_needs_rescale) is rescaled (att16_rescale),
// then the weights multiply V. The reference of a column moves (by its
// excess) only when the column's shifted scores exceed RESCALE_LOG2, so a
// query's arithmetic does not depend on the other queries of the wave.
__device__ __forceinline__ bool att16_needs_rescale(float mx) { return __ballot(mx > RESCALE_LOG2) != 0; }

template <int D> __device__ __forceinline__ void att16_rescale(Att16<D> &st, f32x4 (&acc)[2], float mx) {
  const float cm = max_lane_groups(mx);
  const float d = cm > RESCALE_LOG2 ? cm : 0.f;
  const float alpha = __builtin_amdgcn_exp2f(-d);
  st.nm -= d;
#pragma unroll
  for (int i = 0; i < D / 16; ++i) st.o[i] *= alpha;
  st.l *= alpha;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) acc[kb] -= d;
}

template <int D, bool MASKED, int NGB, int NG>
__device__ __forceinline__ void att16_next(Att16<D> (&st)[NG], const bf16_t *__restrict__ Kl,
                                           const bf16_t *__restrict__ Vl, const Att16Addr<D> &ad,
                                           const Frag<bf16_t> (&qf)[NG][D / 32], int nvalid) {
  f32x4 acc[NG][2];
  att16_scores<D, NGB>(acc, st, Kl, ad, qf);
#pragma unroll
  for (int c = 0; c < NGB; ++c) {
    const float mx = att16_lane_max<MASKED>(acc[c], nvalid);
    if (att16_needs_rescale(mx)) att16_rescale<D>(st[c], acc[c], mx);
  }
  att16_pv<D, MASKED, NGB>(st, acc, Vl, ad, nvalid);
}

// A later tile without the reference check: the weights exp2(s - m) may
// exceed 2^8 when a score overshoots the first tile's column max; they stay
// finite while the overshoot is below about 2^7 (log2 units), and
// att16_finite tells afterwards whether they did.
template <int D, bool MASKED, int NGB, int NG>
__device__ __forceinline__ void att16_plain(Att16<D> (&st)[NG], const bf16_t *__restrict__ Kl,
                                            const bf16_t *__restrict__ Vl, const Att16Addr<D> &ad,
                                            const Frag<bf16_t> (&qf)[NG][D / 32], int nvalid) {
  f32x4 acc[NG][2];
  att16_scores<D, NGB>(acc, st, Kl, ad, qf);
  att16_pv<D, MASKED, NGB>(st, acc, Vl, ad, nvalid);
}

// Are the query's weight sum and accumulators finite? This lane's parts,
// and'ed over the four lane groups of its column (the same answer in every
// lane of the column).
template <int D> __device__ __forceinline__ bool att16_finite(const Att16<D> &st) {
  bool ok = __builtin_isfinite(st.l[0]);
#pragma unroll
  for (int i = 0; i < D / 16; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) ok = ok && __builtin_isfinite(st.o[i][j]);
  const uint32_t x = ok ? 1u : 0u;
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  const uint32_t pair = a[0] & a[1];
  const auto b = __builtin_amdgcn_permlane32_swap(pair, pair, false, false);
  return (b[0] & b[1]) != 0u;
}

// The query's weight sum: the four lane groups of its column added in a
// fixed order (pairs (0, 1) and (2, 3), then both pairs), the same in every
// lane of the column.
template <int D> __device__ __forceinline__ float att16_sum(const Att16<D> &st) { return st.l[0]; }

// Register-staged copy of one 64-row K/V tile (software pipelining: the
// global loads of the next tile are issued before the current tile is
// processed, the LDS stores after). Thread t owns rows CH*(t / CPR) + j,
// j < CH, at 16-byte chunk t % CPR, so the transposing V store can write the
// CH consecutive keys of one dimension as one packed word. WITH_V = false
// stages keys only.
template <typename T, int D, bool WITH_V = true> struct TileRegs {
  static constexpr int VE = 16 / (int)sizeof(T);
  static constexpr int CPR = D / VE;           // 16-byte chunks per row
  static constexpr int CH = TK * CPR / BLOCK;  // rows per thread
  // the CH 16-byte chunks of K (and V) as one vector value each, so the
  // compiler keeps them in registers (arrays of them could end up in scratch)
  typedef uint32_t vec_t __attribute__((ext_vector_type(4 * CH)));
  vec_t kq, vq;
  __device__ __forceinline__ uint4 kget(int j) const {
    return make_uint4(kq[4 * j], kq[4 * j + 1], kq[4 * j + 2], kq[4 * j + 3]);
  }
  __device__ __forceinline__ uint4 vget(int j) const {
    return make_uint4(vq[4 * j], vq[4 * j + 1], vq[4 * j + 2], vq[4 * j + 3]);
  }
  __device__ __forceinline__ void kset(int j, uint4 x) {
    kq[4 * j] = x.x;
    kq[4 * j + 1] = x.y;
    kq[4 * j + 2] = x.z;
    kq[4 * j + 3] = x.w;
  }
  __device__ __forceinline__ void vset(int j, uint4 x) {
    vq[4 * j] = x.x;
    vq[4 * j + 1] = x.y;
    vq[4 * j + 2] = x.z;
    vq[4 * j + 3] = x.w;
  }
  __device__ __forceinline__ int row0() const { return CH * ((int)threadIdx.x / CPR); }
  __device__ __forceinline__ int chunk() const { return (int)threadIdx.x % CPR; }
  // row r of the tile is source row (rowidx ? rowidx[r] : r); rows >= nrows load zeros
  __device__ __forceinline__ void load(const T *__restrict__ kb, const T *__restrict__ vb, const int32_t *rowidx,
                                       int nrows) {
    const int r0 = row0(), ch = chunk();
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int r = r0 + j;
      uint4 a = make_uint4(0, 0, 0, 0), b = make_uint4(0, 0, 0, 0);
      if (r < nrows) {
        const int64_t src = rowidx ? (int64_t)rowidx[r] : (int64_t)r;
        a = *reinterpret_cast<const uint4 *>(kb + src * D + ch * VE);
        if (WITH_V) b = *reinterpret_cast<const uint4 *>(vb + src * D + ch * VE);
      }
      kset(j, a);
      if (WITH_V) vset(j, b);
    }
  }
  // a full tile: rows 0..63 all valid
  __device__ __forceinline__ void load_full(const T *__restrict__ kb, const T *__restrict__ vb,
                                            const int32_t *rowidx) {
    const int r0 = row0(), ch = chunk();
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int64_t src = rowidx ? (int64_t)rowidx[r0 + j] : (int64_t)(r0 + j);
      kset(j, *reinterpret_cast<const uint4 *>(kb + src * D + ch * VE));
      if (WITH_V) vset(j, *reinterpret_cast<const uint4 *>(vb + src * D + ch * VE));
    }
  }
  // the same from byte offsets: row r of the tile starts offs[r] bytes past
  // kb (and vb); kb and vb are the same for every lane, so the loads take a
  // scalar base and a 32-bit lane offset
  __device__ __forceinline__ void load_off(const T *__restrict__ kb, const T *__restrict__ vb,
                                           const uint32_t *offs, int nrows) {
    const int r0 = row0();
    const uint32_t cb = (uint32_t)chunk() * 16u;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      uint4 a = make_uint4(0, 0, 0, 0), b = make_uint4(0, 0, 0, 0);
      if (r0 + j < nrows) {
        const uint32_t o = offs[r0 + j] + cb;
        a = *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(kb) + o);
        if (WITH_V) b = *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(vb) + o);
      }
      kset(j, a);
      if (WITH_V) vset(j, b);
    }
  }
  __device__ __forceinline__ void load_full_off(const T *__restrict__ kb, const T *__restrict__ vb,
                                                const uint32_t *offs) {
    const int r0 = row0();
    const uint32_t cb = (uint32_t)chunk() * 16u;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const uint32_t o = offs[r0 + j] + cb;
      kset(j, *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(kb) + o));
      if (WITH_V) vset(j, *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(vb) + o));
    }
  }
  __device__ __forceinline__ void store(T *__restrict__ Ks, T *__restrict__ Vt) const {
    using TD = TileDims<T, D>;
    const int r0 = row0(), ch = chunk();
#pragma unroll
    for (int j = 0; j < CH; ++j) *reinterpret_cast<uint4 *>(Ks + (r0 + j) * TD::KSTR + ch * VE) = kget(j);
    if constexpr (WITH_V) store_vt(Vt, ch * VE, r0);
  }
  // V^T rows row .. row+VE-1 (one 8-aligned group, so one swizzle), keys r0 .. r0+CH-1
  __device__ __forceinline__ void store_vt(T *__restrict__ Vt, int row, int r0) const;
};

template <> __device__ __forceinline__ void TileRegs<bf16_t, 64, true>::store_vt(bf16_t *__restrict__ Vt, int row,
                                                                               int r0) const {
  // CH = 2: keys r0, r0+1 of dims 2m, 2m+1 from the two rows' words m
  using TD = TileDims<bf16_t, 64>;
  bf16_t *dst = Vt + TD::vrow(row) + r0;
  const uint4 v0 = vget(0), v1 = vget(1);
  const uint32_t r0w[4] = {v0.x, v0.y, v0.z, v0.w}, r1w[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    *reinterpret_cast<uint32_t *>(dst + (2 * m) * TD::VSTR) = __builtin_amdgcn_perm(r1w[m], r0w[m], 0x05040100u);
    *reinterpret_cast<uint32_t *>(dst + (2 * m + 1) * TD::VSTR) = __builtin_amdgcn_perm(r1w[m], r0w[m], 0x07060302u);
  }
}
template <> __device__ __forceinline__ void TileRegs<bf16_t, 128, true>::store_vt(bf16_t *__restrict__ Vt, int row,
                                                                               int r0) const {
  bf16_t *dst = Vt + row * TileDims<bf16_t, 128>::VSTR + r0;
  // CH = 4: keys r0 .. r0+3 of dims 2m, 2m+1 as one 8-byte word each
  using TD = TileDims<bf16_t, 128>;
  const uint4 v0 = vget(0), v1 = vget(1), v2 = vget(2), v3 = vget(3);
  const uint32_t w0[4] = {v0.x, v0.y, v0.z, v0.w}, w1[4] = {v1.x, v1.y, v1.z, v1.w};
  const uint32_t w2[4] = {v2.x, v2.y, v2.z, v2.w}, w3[4] = {v3.x, v3.y, v3.z, v3.w};
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    *reinterpret_cast<uint2 *>(dst + (2 * m) * TD::VSTR) =
        make_uint2(__builtin_amdgcn_perm(w1[m], w0[m], 0x05040100u), __builtin_amdgcn_perm(w3[m], w2[m], 0x05040100u));
    *reinterpret_cast<uint2 *>(dst + (2 * m + 1) * TD::VSTR) =
        make_uint2(__builtin_amdgcn_perm(w1[m], w0[m], 0x07060302u), __builtin_amdgcn_perm(w3[m], w2[m], 0x07060302u));
  }
}
template <> __device__ __forceinline__ void TileRegs<float, 64, true>::store_vt(float *__restrict__ Vt, int row,
                                                                               int r0) const {
  float *dst = Vt + row * TileDims<float, 64>::VSTR + r0;
  // CH = 4: keys r0 .. r0+3 of each of the 4 dims as one 16-byte word
  using TD = TileDims<float, 64>;
  // vq[4 j + e] = dim e of key r0 + j
#pragma unroll
  for (int e = 0; e < 4; ++e)
    *reinterpret_cast<float4 *>(dst + e * TD::VSTR) =
        make_float4(__uint_as_float(vq[e]), __uint_as_float(vq[4 + e]), __uint_as_float(vq[8 + e]),
                    __uint_as_float(vq[12 + e]));
}
template <> __device__ __forceinline__ void TileRegs<float, 128, true>::store_vt(float *__restrict__ Vt, int row,
                                                                               int r0) const {
  float *dst = Vt + row * TileDims<float, 128>::VSTR + r0;
  // CH = 8: keys r0 .. r0+7 of each of the 4 dims as two 16-byte words
  using TD = TileDims<float, 128>;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = __uint_as_float(vq[4 * j + e]);
    *reinterpret_cast<float4 *>(dst + e * TD::VSTR) = make_float4(x[0], x[1], x[2], x[3]);
    *reinterpret_cast<float4 *>(dst + e * TD::VSTR + 4) = make_float4(x[4], x[5], x[6], x[7]);
  }
}


// Landmark value of one row (Eq. landmark-value) from the score pass's
// per-chunk partials (running max in log2 units, running sum, unnormalised
// accumulator): a log-sum-exp merge over the chunks, by the whole workgroup:
// thread t takes dimension t % D and every (256 / D)-th chunk from t / D on,
// in increasing chunk order; the groups' partial merges are combined through
// LDS. prefetch() issues the loads of a thread's first PF chunks, so that a
// caller can overlap them with other work before finish().
template <typename T, int D, int PF = 8> struct LandmarkMerge {
  static constexpr int NG = 256 / D;
  float2 ml[PF];
  float ov[PF];
  __device__ __forceinline__ void prefetch(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                           int64_t bh, int lm, int M, int nch) {
    const int dim = threadIdx.x % D, grp = threadIdx.x / D;
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      const int c = grp + NG * j;
      if (c < nch) {
        const int64_t prow = (bh * nch + c) * M + lm;
        ml[j] = part_ml[prow];
        ov[j] = part_o[prow * D + dim];
      }
    }
  }
  __device__ __forceinline__ static void step(float &mx, float &L, float &acc, float2 m, float o) {
    const float m_new = fmaxf(mx, m.x);
    const float a = __builtin_amdgcn_exp2f(mx - m_new), b = __builtin_amdgcn_exp2f(m.x - m_new);
    L = L * a + m.y * b;
    acc = acc * a + o * b;
    mx = m_new;
  }
  __device__ __forceinline__ void finish(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                         T *__restrict__ v_lm, int64_t bh, int lm, int M, int nch,
                                         float (*red)[3][D]) const {
    const int dim = threadIdx.x % D, grp = threadIdx.x / D;
    float mx = -INFINITY, L = 0.f, acc = 0.f;
#pragma unroll
    for (int j = 0; j < PF; ++j)
      if (grp + NG * j < nch) step(mx, L, acc, ml[j], ov[j]);
#pragma unroll 4
    for (int c = grp + NG * PF; c < nch; c += NG) {
      const int64_t prow = (bh * nch + c) * M + lm;
      step(mx, L, acc, part_ml[prow], part_o[prow * D + dim]);
    }
    red[grp][0][dim] = mx;
    red[grp][1][dim] = L;
    red[grp][2][dim] = acc;
    __syncthreads();
    if (grp == 0) {
      float m2 = -INFINITY;
#pragma unroll
      for (int g2 = 0; g2 < NG; ++g2) m2 = fmaxf(m2, red[g2][0][dim]);
      float L2 = 0.f, a2 = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < NG; ++g2) {
        const float f = __builtin_amdgcn_exp2f(red[g2][0][dim] - m2);  // a group with no chunk: exp2(-inf) = 0
        L2 += red[g2][1][dim] * f;
        a2 += red[g2][2][dim] * f;
      }
      v_lm[(bh * M + lm) * D + dim] = from_f32<T>(a2 / L2);
    }
  }
};

// The same merge for one (row, dimension) by one thread: the 256 / D
// groups' chunk sequences run one after the other (each in increasing chunk
// order, from the empty state), then the groups are combined in group order,
// with the arithmetic of LandmarkMerge, so the result is the same bit for bit.
// prefetch() loads the first PF chunks' values (PF a multiple of 256 / D),
// so that a caller can overlap them with other work before finish().
template <int D, int PF = 8> struct LandmarkMerge1 {
  static constexpr int NG = 256 / D;
  static_assert(PF % NG == 0, "whole rounds of the groups prefetched");
  float2 ml[PF];
  float ov[PF];
  __device__ __forceinline__ void prefetch(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                           int64_t bh, int lm, int M, int nch, int dim) {
#pragma unroll
    for (int c = 0; c < PF; ++c)
      if (c < nch) {
        const int64_t prow = (bh * nch + c) * M + lm;
        ml[c] = part_ml[prow];
        ov[c] = part_o[prow * D + dim];
      }
  }
  __device__ __forceinline__ float finish(const float2 *__restrict__ part_ml, const float *__restrict__ part_o,
                                          int64_t bh, int lm, int M, int nch, int dim) const {
    float gm[NG], gl[NG], ga[NG];
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      float mx = -INFINITY, L = 0.f, acc = 0.f;
#pragma unroll
      for (int j = 0; j < PF / NG; ++j)
        if (grp + NG * j < nch) LandmarkMerge<float, D>::step(mx, L, acc, ml[grp + NG * j], ov[grp + NG * j]);
      for (int c = grp + PF; c < nch; c += NG) {
        const int64_t prow = (bh * nch + c) * M + lm;
        LandmarkMerge<float, D>::step(mx, L, acc, part_ml[prow], part_o[prow * D + dim]);
      }
      gm[grp] = mx;
      gl[grp] = L;
      ga[grp] = acc;
    }
    return combine(gm, gl, ga);
  }
  __device__ __forceinline__ static float combine(const float (&gm)[NG], const float (&gl)[NG], const float (&ga)[NG]) {
    float m2 = -INFINITY;
#pragma unroll
    for (int g2 = 0; g2 < NG; ++g2) m2 = fmaxf(m2, gm[g2]);
    float L2 = 0.f, a2 = 0.f;
#pragma unroll
    for (int g2 = 0; g2 < NG; ++g2) {
      const float f = __builtin_amdgcn_exp2f(gm[g2] - m2);
      L2 += gl[g2] * f;
      a2 += ga[g2] * f;
    }
    return a2 / L2;
  }
};

template <int D>
__device__ __forceinline__ float merge_landmark_value_1(const float2 *__restrict__ part_ml,
                                                        const float *__restrict__ part_o, int64_t bh, int lm, int M,
                                                        int nch, int dim) {
  constexpr int NG = 256 / D;
  float gm[NG], gl[NG], ga[NG];
#pragma unroll
  for (int grp = 0; grp < NG; ++grp) {
    float mx = -INFINITY, L = 0.f, acc = 0.f;
    for (int c = grp; c < nch; c += NG) {
      const int64_t prow = (bh * nch + c) * M + lm;
      LandmarkMerge<float, D>::step(mx, L, acc, part_ml[prow], part_o[prow * D + dim]);
    }
    gm[grp] = mx;
    gl[grp] = L;
    ga[grp] = acc;
  }
  return LandmarkMerge1<D>::combine(gm, gl, ga);
}


template <typename T, int D>
__device__ __forceinline__ void merge_landmark_value(const float2 *__restrict__ part_ml,
                                                     const float *__restrict__ part_o, T *__restrict__ v_lm,
                                                     int64_t bh, int lm, int M, int nch, float (*red)[3][D]) {
  LandmarkMerge<T, D> m;
  m.prefetch(part_ml, part_o, bh, lm, M, nch);
  m.finish(part_ml, part_o, v_lm, bh, lm, M, nch, red);
}

}  // namespace mita
