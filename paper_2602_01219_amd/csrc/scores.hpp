// scores.hpp - the landmark-key score pass over one key chunk (the tile code
// shared by the score kernel, the fallback rows of the fused selection and
// the launches that combine those rows with routing work).
#pragma once
#include "cdna4.hpp"
#include "flash.hpp"
#include "check.hpp"

namespace mita {

// Neighbouring floats (a zero of either sign steps to the smallest subnormal).
__device__ __forceinline__ float f32_next_down(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) == 0u) return __uint_as_float(0x80000001u);
  return __uint_as_float((u & 0x80000000u) ? u + 1u : u - 1u);
}
__device__ __forceinline__ float f32_next_up(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) == 0u) return __uint_as_float(1u);
  return __uint_as_float((u & 0x80000000u) ? u - 1u : u + 1u);
}

// Bound of a pivot on the unscaled dot: the smallest float t with
// fl(t * scale) >= piv. A rounded product is monotonic in its operand, so for
// scale > 0 and every non-NaN dot a, fl(a * scale) >= piv iff a >= t, and the
// selection test can compare the MFMA dots without scaling them. piv / scale
// lies within a few ulps of t for a normal piv; the walk is capped at 4 steps
// and returns false if it has not settled (a subnormal piv), and then the
// scaled test is used. A NaN piv (no row) gives t = NaN, which lists nothing.
__device__ __forceinline__ bool dot_bound(float piv, float scale, float &t) {
  t = piv / scale;
  if (piv != piv) return true;
  if (t * scale >= piv) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float d = f32_next_down(t);
      if (!(d * scale >= piv)) return true;
      t = d;
    }
    return false;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    t = f32_next_up(t);
    if (t * scale >= piv) return true;
  }
  return false;
}

// ---------------------------------------------------------------------------
// Scores and landmark values. Workgroup = 4 waves x 16 landmarks over one
// chunk of SCORE_NC keys, key tiles of 64 staged in LDS (K row-major, V
// transposed). Each wave forms S^T for its landmarks on MFMA and, per mode:
//  - WRITE_S: writes S = fl(dot) * scale (fp32, landmark-major);
//  - SELECT: lists the keys whose score is >= the row's pivot, in ascending
//    token order, in the (row, chunk) region of the candidate lists (bits of
//    the unscaled dot fl(q . k), token index; the reader scales the dot with
//    the same rounded product fl(dot * scale) as every score) and writes the
//    region's count. In a tile a
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
  uint2 *cand;          // [rows, chunks, SCORE_NC] (unscaled dot bits, token index)
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
  // dotpiv: piv as a bound on the unscaled dots (dot_bound); `scaled` marks
  // the lanes that must test the scaled score instead.
  float piv = 0.f, dotpiv = 0.f;
  bool nan_in = false, scaled = false;
  if (SELECT) {
    const uint32_t plo = lm < M ? sel.plo[row] : 0xffffffffu;
    piv = key_to_float(plo);
    nan_in = plo == ordered_key(-INFINITY);
    scaled = nan_in || !(scale > 0.f && scale < INFINITY) || !dot_bound(piv, scale, dotpiv);
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
    uint32_t m[4] = {0u, 0u, 0u, 0u}, pos = 0u, tot = 0u, ntot = 0u;
    if (active) {
      tile_scores<T, D>(acc, Kc, qf);
      if (SELECT) {
        // per-kb candidate bits m[kb] (bit r); per-kb counts in bytes
        if (nvalid == TK && !__ballot(scaled)) {  // full tile, every lane has a dot bound
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) m[kb] |= (acc[kb][r] >= dotpiv) ? 1u << r : 0u;
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
        uint32_t incl;
        scan_lane_groups(packed, incl, tot);  // tot: per-kb totals of the landmark
        // byte kb of pos: candidates of the landmark before this lane's block kb
        pos = (incl - packed) + (tot << 8) + (tot << 16) + (tot << 24);
        ntot = (tot * 0x01010101u) >> 24;  // candidates of the landmark in the tile
      }
      if (DO_V) {
        if (nvalid == TK)
          tile_softmax_pv<T, D, false>(st, acc, Vc, nvalid, sl2);
        else
          tile_softmax_pv<T, D, true>(st, acc, Vc, nvalid, sl2);
      }
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
            *reinterpret_cast<uint2 *>(cand_w + at) = make_uint2(__float_as_uint(acc[kb][r]), ib + r);
            at += 8u;
          }
      }
      listed += ntot;
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

// Score rows of listed landmark rows (fallback of the fused selection): work
// item = (listed row, key chunk), taken by workgroup b of nb; each item
// recomputes the row's 64-landmark block exactly as the score pass does and
// writes that row only. Ks: two K tile buffers.
template <typename T, int D>
__device__ __forceinline__ void scores_rows_body(T *Ks, int b, int nb, const T *__restrict__ q_lm,
                                                 const T *__restrict__ k, float *__restrict__ S,
                                                 const uint32_t *__restrict__ nrows, const int32_t *__restrict__ rows,
                                                 int N, int M, float scale, int nchunks) {
  const int64_t items = (int64_t)*nrows * nchunks;
  const SelectArgs none{nullptr, nullptr, nullptr};
  for (int64_t it = b; it < items; it += nb) {
    const int row = rows[it / nchunks];
    const int chunk = (int)(it % nchunks);
    const int lm = row % M;
    __syncthreads();  // the previous item's last reads of Ks are done
    score_chunk<T, D, true, false, false>(Ks, nullptr, q_lm, k, nullptr, S, nullptr, nullptr, none, N, M, scale, chunk,
                                          nchunks, lm / 64, row / M, lm);
  }
}

}  // namespace mita

namespace mita {

// ---------------------------------------------------------------------------
// The bf16 score pass with landmark values on the DMA tile machinery of the
// attention (flash.hpp), taken at d = 128, where the products per tile
// outweigh the listing's fixed steps per tile (at d = 64 the 64-key tiles of
// score_chunk are faster). Workgroup = NW waves over one chunk of SCORE_NC
// keys; wave w owns NG groups of 16 landmarks (MFMA column groups), so a
// workgroup covers 16 NG NW landmarks and reads each key chunk once for all
// of them. The keys come in 32-row K and V tiles by LDS DMA, double
// buffered, one barrier per tile. Per tile and group:
//  - the raw dots S^T = K Q^T, accumulated from zero over the same fragments
//    in the same order as score_chunk, so every score has the same value;
//  - SELECT: the candidate bits and their slots as in score_chunk (two
//    16-key blocks per tile), and WRITE_S: the scaled scores; both are stored
//    at the start of the next tile, before its DMA is issued, so that the
//    wait for that DMA (one counter tracks loads and stores) finds the stores
//    long done instead of waiting for fresh ones;
//  - the online softmax of score_chunk (a column's reference max is raised
//    only when its tile max exceeds it by more than RESCALE_LOG2, so the
//    weights stay below 2^8), the exponent one FMA per score, the weights
//    multiplying V through att16_pv (V^T fragments by transposing LDS reads,
//    each serving the NG groups; weight sums by the all-ones MFMA row).
// Partials, counts and candidate regions are laid out as score_chunk writes
// them.
// ---------------------------------------------------------------------------

// DMA of rows [0, 32) of a tile whose rows are contiguous from kb / vb
// (without FULL, rows >= nrows load row 0: real data, masked later).
template <int D, int NW, bool FULL>
__device__ __forceinline__ void dma_rows(bf16_t *Kl, bf16_t *Vl, const bf16_t *kb, const bf16_t *vb,
                                         const DmaLane<D, TK32, NW> &dl, int nrows) {
  using DT = DmaTile<D, TK32, NW>;
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
#pragma unroll
  for (int j = 0; j < DT::PW; ++j) {
    const int ins = w * DT::PW + j;
    const uint32_t r = FULL || dl.row[j] < (uint32_t)nrows ? dl.row[j] : 0u;
    const uint32_t go = r * (uint32_t)(2 * D) + dl.chunk[j];
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(kb) + go,
                                     (lds_void_t *)(reinterpret_cast<char *>(Kl) + ins * 1024), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const char *>(vb) + go,
                                     (lds_void_t *)(reinterpret_cast<char *>(Vl) + ins * 1024), 16, 0, 0);
  }
}

template <int D, int NG, int NW, bool WRITE_S, bool SELECT>
__device__ __forceinline__ void score16_chunk(char *tiles0, char *tiles1, const bf16_t *__restrict__ q_lm,
                                              const bf16_t *__restrict__ k, const bf16_t *__restrict__ v,
                                              float *__restrict__ S, float2 *__restrict__ part_ml,
                                              float *__restrict__ part_o, const SelectArgs &sel, int N, int M,
                                              float scale, int chunk, int nch, int lmblock, int64_t bh) {
  using DT = DmaTile<D, TK32, NW>;
  constexpr bool DEFER = WRITE_S || SELECT;
  auto Ks = [&](auto b) { return reinterpret_cast<bf16_t *>(decltype(b)::value ? tiles1 : tiles0); };
  auto Vs = [&](auto b) { return reinterpret_cast<bf16_t *>((decltype(b)::value ? tiles1 : tiles0) + DT::BYTES); };
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, g = lane >> 4, p = lane & 15;
  const int lmw = (lmblock * NW + w) * NG * 16;  // the wave's first landmark
  int nbusy = 0;                                 // groups with landmarks (the first ones)
#pragma unroll
  for (int c = 0; c < NG; ++c) nbusy += lmw + 16 * c < M ? 1 : 0;

  Frag<bf16_t> qf[NG][D / 32];
  float piv[NG], dotpiv[NG];
  bool nan_in[NG], scaled = false;
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    const int lm = lmw + 16 * c + p;
    const int64_t row = bh * M + lm;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if (lm < M)
        qf[c][ks].load(q_lm + row * D + ks * 32 + g * 8);
      else
        qf[c][ks].zero();
    }
    piv[c] = dotpiv[c] = 0.f;
    nan_in[c] = false;
    if (SELECT) {  // as in score_chunk
      const uint32_t plo = lm < M ? sel.plo[row] : 0xffffffffu;
      piv[c] = key_to_float(plo);
      nan_in[c] = plo == ordered_key(-INFINITY);
      scaled = scaled || nan_in[c] || !(scale > 0.f && scale < INFINITY) || !dot_bound(piv[c], scale, dotpiv[c]);
    }
  }
  // every lane of the wave tests the unscaled dots against its bound
  const bool fast = !__ballot(scaled);
  // SELECT: the candidate regions of group c of this wave start at
  // cand_w + c * gbytes; landmark p's lies lane_off bytes further
  char *cand_w = nullptr;
  const uint32_t gbytes = 16u * (uint32_t)nch * SCORE_NC * 8u;
  const uint32_t lane_off = (uint32_t)p * (uint32_t)nch * SCORE_NC * 8u;
  if (SELECT) cand_w = reinterpret_cast<char *>(sel.cand + ((bh * M + lmw) * nch + chunk) * (int64_t)SCORE_NC);

  const int key_begin = chunk * SCORE_NC, nk = min(N, key_begin + SCORE_NC) - key_begin;
  const int nfull = nk / TK32, rest = nk % TK32;
  const bf16_t *kb_ = k + (bh * N + key_begin) * (int64_t)D, *vb_ = v + (bh * N + key_begin) * (int64_t)D;
  DmaLane<D, TK32, NW> dl;
  dl.init(w, lane);
  Att16Addr<D> ad;
  ad.init();
  Att16<D> st[NG];  // nm stays 0: att16_scores then yields the raw dots
  float m[NG], thr[NG];
  uint32_t listed[NG];
#pragma unroll
  for (int c = 0; c < NG; ++c) {
#pragma unroll
    for (int i = 0; i < D / 16; ++i) st[c].o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    st[c].nm = f32x4{0.f, 0.f, 0.f, 0.f};
    st[c].l = f32x4{0.f, 0.f, 0.f, 0.f};
    m[c] = -INFINITY;
    thr[c] = -INFINITY;
    listed[c] = 0u;
  }
  // the previous tile's dots, candidate flags, slots and list length before it
  f32x4 pacc[NG][2];
  uint32_t ppos[NG], plist[NG];
  int pk0 = 0, pnv = 0;
  const float sl2 = scale * LOG2E;
  wait_loads();

  // NGB: busy groups; FAST: every lane tests the unscaled dots (a masked
  // tile takes the scaled test with its key bound)
  auto run = [&](auto ngb_c, auto fast_c) {
    constexpr int NGB = decltype(ngb_c)::value;
    constexpr bool FAST = decltype(fast_c)::value;
    // is key 16 kb + 4 g + r of group c listed? (the test of the listing,
    // repeated on the kept dots rather than kept as 16 lane masks)
    auto listed_key = [&](int c, float dot, int key, int nv, auto masked_c) {
      constexpr bool MK = decltype(masked_c)::value;
      if (FAST && !MK) return dot >= dotpiv[c];
      const float x = dot * scale;
      return (x >= piv[c] || (nan_in[c] && x != x)) && key < nv;
    };
    // (MK: the kept tile is the partial last one)
    auto store_prev = [&](auto masked_c) {
      constexpr bool MK = decltype(masked_c)::value;
      if (NGB == 0) return;
      if (SELECT) {
        // the slots' token indices (the same for every group)
        uint32_t iv[8];
#pragma unroll
        for (int sl = 0; sl < 8; ++sl) iv[sl] = (uint32_t)(pk0 + 4 * g) + (uint32_t)(16 * (sl >> 2) + (sl & 3));
#pragma unroll
        for (int c = 0; c < NGB; ++c) {
          char *cw = cand_w + c * gbytes;
          const uint32_t base = lane_off + plist[c] * 8u;
#pragma unroll
          for (int kb = 0; kb < 2; ++kb) {
            uint32_t at = base + ((ppos[c] >> (8 * kb)) & 255u) * 8u;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              if (listed_key(c, pacc[c][kb][r], kb * 16 + 4 * g + r, pnv, masked_c)) {
                *reinterpret_cast<uint2 *>(cw + at) = make_uint2(__float_as_uint(pacc[c][kb][r]), iv[4 * kb + r]);
                at += 8u;
              }
            }
          }
        }
      }
      if (WRITE_S) {
#pragma unroll
        for (int c = 0; c < NGB; ++c) {
          const int lm = lmw + 16 * c + p;
          if (lm < M) {
            float *srow = S + (bh * M + lm) * (int64_t)N + pk0;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
              const int key = kb * 16 + 4 * g;
              if (!MK || key + 3 < pnv) {
                *reinterpret_cast<float4 *>(srow + key) =
                    make_float4(pacc[c][kb][0] * scale, pacc[c][kb][1] * scale, pacc[c][kb][2] * scale,
                                pacc[c][kb][3] * scale);
              } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  if (key + r < pnv) srow[key + r] = pacc[c][kb][r] * scale;
              }
            }
          }
        }
      }
    };
    auto tile = [&](const bf16_t *__restrict__ Kc, const bf16_t *__restrict__ Vc, int k0, int nv, auto masked_c) {
      constexpr bool MK = decltype(masked_c)::value;
      if (NGB == 0) return;
      f32x4 acc[NG][2];
      att16_scores<D, NGB>(acc, st, Kc, ad, qf);
      if (SELECT) {
#pragma unroll
        for (int c = 0; c < NGB; ++c) {
          // per-block counts in bytes, scanned over the column's lane groups
          uint32_t n[2] = {0u, 0u};
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) n[kb] += listed_key(c, acc[c][kb][r], kb * 16 + 4 * g + r, nv, masked_c);
          const uint32_t packed = n[0] | (n[1] << 8);
          uint32_t incl, tot;
          scan_lane_groups(packed, incl, tot);
          ppos[c] = (incl - packed) + (tot << 8);
          plist[c] = listed[c];
          listed[c] += (tot + (tot >> 8)) & 255u;
        }
      }
      if (DEFER) {
#pragma unroll
        for (int c = 0; c < NGB; ++c) {
          pacc[c][0] = acc[c][0];
          pacc[c][1] = acc[c][1];
        }
        pk0 = k0;
        pnv = nv;
      }
      // online softmax: reference check on the raw dots, then the exponents
#pragma unroll
      for (int c = 0; c < NGB; ++c) {
        const float mx = att16_lane_max<MK>(acc[c], nv);
        if (__ballot(mx > thr[c])) {
          const float m_new = fmaxf(m[c], max_lane_groups(mx) * sl2);
          const float alpha = __builtin_amdgcn_exp2f(m[c] - m_new);
          m[c] = m_new;
          thr[c] = (m_new + RESCALE_LOG2) * __builtin_amdgcn_rcpf(sl2);
#pragma unroll
          for (int i = 0; i < D / 16; ++i) st[c].o[i] *= alpha;
          st[c].l *= alpha;
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[c][kb][r] = __builtin_fmaf(acc[c][kb][r], sl2, -m[c]);
      }
      att16_pv<D, MK, NGB>(st, acc, Vc, ad, nv);
    };
    // step t: the previous tile's stores, the DMA of tile t + 1 into the
    // other buffer, tile t's arithmetic, then the wait for the DMA and the
    // workgroup barrier (tile t lives in buffer t & 1)
    auto step = [&](int t, auto bc) {
      constexpr int B = decltype(bc)::value;
      if (DEFER && t > 0) store_prev(std::false_type{});  // tile t - 1 < nfull is whole
      const int tn = t + 1;
      if (tn < nfull)
        dma_rows<D, NW, true>(Ks(std::integral_constant<int, B ^ 1>{}), Vs(std::integral_constant<int, B ^ 1>{}),
                              kb_ + (int64_t)tn * TK32 * D, vb_ + (int64_t)tn * TK32 * D, dl, TK32);
      else if (tn == nfull && rest > 0)
        dma_rows<D, NW, false>(Ks(std::integral_constant<int, B ^ 1>{}), Vs(std::integral_constant<int, B ^ 1>{}),
                               kb_ + (int64_t)tn * TK32 * D, vb_ + (int64_t)tn * TK32 * D, dl, rest);
      // the DMA is issued before the tile's arithmetic (the scheduler would
      // otherwise sink it towards its wait)
      __builtin_amdgcn_sched_barrier(0);
      if (t < nfull)
        tile(Ks(bc), Vs(bc), key_begin + t * TK32, TK32, std::false_type{});
      else
        tile(Ks(bc), Vs(bc), key_begin + t * TK32, rest, std::true_type{});
      wait_loads();
      __syncthreads();
    };
    const std::integral_constant<int, 0> b0{};
    const std::integral_constant<int, 1> b1{};
    if (nfull > 0)
      dma_rows<D, NW, true>(Ks(b0), Vs(b0), kb_, vb_, dl, TK32);
    else
      dma_rows<D, NW, false>(Ks(b0), Vs(b0), kb_, vb_, dl, rest);
    wait_loads();
    __syncthreads();
    const int ntile = nfull + (rest > 0 ? 1 : 0);
    int t = 0;
    for (; t + 1 < ntile; t += 2) {
      step(t, b0);
      step(t + 1, b1);
    }
    if (t < ntile) step(t, b0);
    if (DEFER) {
      if (rest > 0)
        store_prev(std::true_type{});
      else
        store_prev(std::false_type{});
    }
  };
  auto run_busy = [&](auto fast_c) {
    if (nbusy == NG)
      run(std::integral_constant<int, NG>{}, fast_c);
    else if (NG > 1 && nbusy == 1)
      run(std::integral_constant<int, 1>{}, fast_c);
    else
      run(std::integral_constant<int, 0>{}, fast_c);
  };
  if (!SELECT || fast)
    run_busy(std::true_type{});
  else
    run_busy(std::false_type{});

  // partials and counts of the chunk, as score_chunk writes them
#pragma unroll
  for (int c = 0; c < NG; ++c) {
    const int lm = lmw + 16 * c + p;
    if (lm >= M) continue;
    const int64_t row = bh * M + lm;
    if (SELECT && g == 0) sel.ccnt[row * nch + chunk] = listed[c];
    const int64_t prow = (bh * nch + chunk) * M + lm;
    if (g == 0) part_ml[prow] = make_float2(m[c], st[c].l[0]);
#pragma unroll
    for (int db = 0; db < D / 16; ++db)
      *reinterpret_cast<float4 *>(part_o + prow * D + db * 16 + 4 * g) =
          make_float4(st[c].o[db][0], st[c].o[db][1], st[c].o[db][2], st[c].o[db][3]);
  }
}

}  // namespace mita
