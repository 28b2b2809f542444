// topk_row.hpp - exact top-k of one score row by one 256-thread workgroup
// (Eq. top-k), used by the top-k kernel and by the launch that combines the
// fallback rows of the fused selection with the routing scan.
//
// Order: larger score first, equal scores by lower token index (-0 == +0;
// NaN inputs are treated as -inf). The k first tokens of that order are
// written in ascending index order.
//
// One 256-thread workgroup per row. Rows of up to 16384 scores are copied
// into LDS by one coalesced pass and every later pass reads LDS; longer rows
// are streamed from memory in every pass (re-reads served by L2 / MALL). A
// pass walks 16 consecutive tokens per thread per step (16-byte loads, the
// next step's loads in flight while one is processed); passes are small
// loops, so the kernel stays compact.
//
// The k-th token of the order, (T, n_cut), is found by narrowing a candidate
// value range that always holds it:
//   0. pivots (long rows, k <= N/4): a histogram of an evenly spaced sample of
//      the row (runs of 4 tokens) gives p_lo < p_hi with (by 4-standard-deviation binomial
//      margins) fewer than k tokens >= p_hi and more than k tokens >= p_lo.
//      One pass counts the tokens >= p_hi and appends those in [p_lo, p_hi)
//      to an LDS list. If the counts confirm that the k-th token lies in
//      [p_lo, p_hi) and the list fits, step 2 follows; otherwise step 1
//      starts from the one of [p_hi, inf), [p_lo, p_hi), (-inf, p_lo) that
//      the counts show holds the k-th token.
//   1. rounds over the stream: block min / max / count of the candidates; a
//      256-bin histogram (bins linear in the value for the first two rounds
//      when the range is finite, which spreads clustered scores; bins over the
//      order-preserving integer key otherwise, which shrink the key span by 2^8
//      per round and so bound the number of rounds) selects the bin holding the
//      target rank. Once at most CAP candidates remain they go to LDS.
//   2. the same rounds over the LDS candidates, until at most 64 remain; one
//      wave then ranks them exactly.
//   If all candidates are equal, the cut among the tied tokens comes from an
//   index-ordered scan of the stream.
// A token is selected iff x > T or (x == T and n <= n_cut); the output is
// written by an index-ordered scan (one block scan per step), so it is ascending.
#pragma once
#include "cdna4.hpp"
#include "check.hpp"

namespace mita {

namespace {

constexpr int NT = 256;  // threads per row
constexpr int NW = NT / 64;
constexpr int NB = 256;  // histogram bins
constexpr int RANKCAP = 64;
constexpr int ITEMS = 16;         // consecutive tokens per thread per stream step
constexpr int CHUNK = ITEMS * NT;  // tokens per stream step

template <int CAP> struct TopkSmem {
  uint32_t hist[NW][NB];
  uint32_t ckey[2][CAP];
  int32_t cidx[2][CAP];
  uint32_t wsum[2][NW];
  float redf[2][NW];
  uint32_t redu[3][NW];
  uint32_t bcast[4];
  uint32_t ccount;
};

__device__ __forceinline__ float canon(float v) {
  if (v != v) v = -INFINITY;  // NaN ranks as -inf
  return v + 0.0f;            // -0 -> +0
}
// Largest float below p in the order where -0 == +0 (p finite or +inf).
__device__ __forceinline__ float float_below(float p) {
  uint32_t kk = ordered_key(p) - 1u;
  if (kk == 0x7fffffffu) kk = 0x7ffffffeu;  // skip -0, which ties with +0
  return key_to_float(kk);
}
__device__ __forceinline__ float fmin_nan(float a, float b) { return b < a ? b : a; }  // NaN b ignored
__device__ __forceinline__ float fmax_nan(float a, float b) { return b > a ? b : a; }

// Where passes read the row from: global memory (streamed, re-reads served by
// L2 / MALL) or a copy in LDS made by one coalesced pass.
template <bool IN_LDS> struct RowSrc;
template <> struct RowSrc<false> {
  const float *__restrict__ s;
  __device__ __forceinline__ float at(int n) const { return s[n]; }
  __device__ __forceinline__ float4 at4(int n) const { return *reinterpret_cast<const float4 *>(s + n); }
};
template <> struct RowSrc<true> {
  const float *s;  // LDS
  __device__ __forceinline__ float at(int n) const { return s[n]; }
  __device__ __forceinline__ float4 at4(int n) const { return *reinterpret_cast<const float4 *>(s + n); }
};

// Load the ITEMS tokens n0 .. n0+ITEMS-1 (zeros past N; callers mask them).
template <bool VEC, typename Src>
__device__ __forceinline__ void load_items(const Src &s, int N, int n0, float (&v)[ITEMS]) {
  if (VEC && n0 + ITEMS <= N) {
#pragma unroll
    for (int e = 0; e < ITEMS; e += 4) {
      const float4 q = s.at4(n0 + e);
      v[e] = q.x;
      v[e + 1] = q.y;
      v[e + 2] = q.z;
      v[e + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < ITEMS; ++e) v[e] = n0 + e < N ? s.at(n0 + e) : 0.f;
  }
}

// Load 4 consecutive tokens starting at a multiple of 4 below N - 3.
template <bool VEC, typename Src>
__device__ __forceinline__ void load_items4(const Src &s, int N, int n0, float (&v)[4]) {
  if (VEC) {
    const float4 q = s.at4(n0);
    v[0] = q.x;
    v[1] = q.y;
    v[2] = q.z;
    v[3] = q.w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = s.at(n0 + e);
  }
}

// Stream the row: f(n, x) for every token n < N (x canonical). Thread t takes
// tokens [base + ITEMS*t, base + ITEMS*(t+1)) of each step; the next step's
// loads are issued before the current step is processed.
template <bool VEC, typename Src, typename F> __device__ __forceinline__ void stream_row(const Src &s, int N, F f) {
  float cur[ITEMS], nxt[ITEMS];
  const int t0 = ITEMS * (int)threadIdx.x;
  load_items<VEC>(s, N, t0, cur);
  for (int base = 0; base < N; base += CHUNK) {
    const int n0 = base + t0;
    if (base + CHUNK < N) load_items<VEC>(s, N, n0 + CHUNK, nxt);
#pragma unroll
    for (int e = 0; e < ITEMS; ++e)
      if (n0 + e < N) f(n0 + e, canon(cur[e]));
#pragma unroll
    for (int e = 0; e < ITEMS; ++e) cur[e] = nxt[e];
  }
}

template <int CAP>
__device__ __forceinline__ void block_min_max_cnt(TopkSmem<CAP> &sh, float &mn, float &mx, uint32_t &cnt) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mn = fmin_nan(mn, __shfl_xor(mn, o));
    mx = fmax_nan(mx, __shfl_xor(mx, o));
    cnt += (uint32_t)__shfl_xor((int)cnt, o);
  }
  if (lane == 0) {
    sh.redf[0][w] = mn;
    sh.redf[1][w] = mx;
    sh.redu[0][w] = cnt;
  }
  __syncthreads();
  mn = INFINITY;
  mx = -INFINITY;
  cnt = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    mn = fmin_nan(mn, sh.redf[0][i]);
    mx = fmax_nan(mx, sh.redf[1][i]);
    cnt += sh.redu[0][i];
  }
  __syncthreads();
}

template <int CAP> __device__ __forceinline__ void block_umin_umax(TopkSmem<CAP> &sh, uint32_t &mn, uint32_t &mx) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  mn = wave_min_u32(mn);
  mx = wave_max_u32(mx);
  if (lane == 0) {
    sh.redu[1][w] = mn;
    sh.redu[2][w] = mx;
  }
  __syncthreads();
  mn = 0xffffffffu;
  mx = 0u;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    mn = min(mn, sh.redu[1][i]);
    mx = max(mx, sh.redu[2][i]);
  }
  __syncthreads();
}

template <int CAP> __device__ __forceinline__ void clear_hist(TopkSmem<CAP> &sh) {
  for (int i = threadIdx.x; i < NW * NB; i += NT) (&sh.hist[0][0])[i] = 0u;
  __syncthreads();
}

// Bin (counted from the top) holding the need-th counted item: returns b*,
// *above = count in higher bins, *in_bin = count in b*.
template <int CAP>
__device__ __forceinline__ int find_bin(TopkSmem<CAP> &sh, int need, uint32_t *above, uint32_t *in_bin) {
  const int tid = threadIdx.x;
  const int b = NB - 1 - tid;  // NT == NB
  uint32_t tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) tot += sh.hist[i][b];
  uint32_t incl = wave_inclusive_scan(tot);
  if ((tid & 63) == 63) sh.wsum[0][tid >> 6] = incl;
  __syncthreads();
  for (int i = 0; i < (tid >> 6); ++i) incl += sh.wsum[0][i];
  const uint32_t ab = incl - tot;
  if (ab < (uint32_t)need && (uint32_t)need <= incl) {
    sh.bcast[0] = (uint32_t)b;
    sh.bcast[1] = ab;
    sh.bcast[2] = tot;
  }
  __syncthreads();
  const int r = (int)sh.bcast[0];
  *above = sh.bcast[1];
  *in_bin = sh.bcast[2];
  __syncthreads();
  return r;
}

// Index-ordered scan of the stream: emit(n, position among flagged tokens)
// for every flagged token. One block scan per stream step.
template <bool VEC, int CAP, typename Src, typename Pred, typename Emit>
__device__ __forceinline__ void ordered_stream(TopkSmem<CAP> &sh, const Src &s, int N, Pred pred, Emit emit) {
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int t0 = ITEMS * tid;
  uint32_t run = 0;
  int par = 0;
  float cur[ITEMS], nxt[ITEMS];
  load_items<VEC>(s, N, t0, cur);
  for (int base = 0; base < N; base += CHUNK) {
    const int n0 = base + t0;
    if (base + CHUNK < N) load_items<VEC>(s, N, n0 + CHUNK, nxt);
    uint32_t fl = 0;
    if (base + CHUNK <= N) {
#pragma unroll
      for (int e = 0; e < ITEMS; ++e) fl |= pred(n0 + e, canon(cur[e])) ? (1u << e) : 0u;
    } else {
#pragma unroll
      for (int e = 0; e < ITEMS; ++e) fl |= (n0 + e < N && pred(n0 + e, canon(cur[e]))) ? (1u << e) : 0u;
    }
    const uint32_t c = (uint32_t)__popc(fl);
    const uint32_t incl = wave_inclusive_scan(c);
    if (lane == 63) sh.wsum[par][w] = incl;
    __syncthreads();
    uint32_t before = run + incl - c, tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint32_t x = sh.wsum[par][i];
      before += i < w ? x : 0u;
      tot += x;
    }
    run += tot;
    par ^= 1;  // double-buffered totals: the next step's write cannot race this read
    while (fl) {
      const int e = __builtin_ctz(fl);
      fl &= fl - 1u;
      emit(n0 + e, before++);
    }
#pragma unroll
    for (int e = 0; e < ITEMS; ++e) cur[e] = nxt[e];
  }
  __syncthreads();
}

}  // namespace

template <int CAP, bool VEC, int ROWCAP>
__device__ __forceinline__ void topk_row(TopkSmem<CAP> &sh, float *lrow, const float *__restrict__ grow,
                                         int32_t *__restrict__ out, int N, int k) {
  constexpr bool IN_LDS = ROWCAP > 0;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  if (IN_LDS) {
    // one coalesced pass copies the row into LDS
    if (VEC) {
      for (int c = tid; c < N / 4; c += NT)
        *reinterpret_cast<float4 *>(lrow + 4 * c) = *reinterpret_cast<const float4 *>(grow + 4 * c);
    } else {
      for (int n = tid; n < N; n += NT) lrow[n] = grow[n];
    }
    __syncthreads();
  }
  RowSrc<IN_LDS> s{IN_LDS ? lrow : grow};

  int need = k;
  float T = 0.f;
  int n_cut = -1;
  bool done = false;
  int in_lds = -1;  // candidates in LDS buffer 0 once >= 0
  // initial candidate range of the stream rounds (inclusive), narrowed by the
  // pivot pass when its verification fails
  float lo0 = -INFINITY, hi0 = INFINITY;

  // ---------------- 0. pivots
  if (N >= 4096 && 4 * (int64_t)k <= N) {
    // sample: from LDS, 4 single tokens per thread at an even stride; from
    // global memory, runs of 4 consecutive tokens (a 16-byte load touches a
    // quarter of the row's 64-byte sectors instead of all of them)
    const int nsamp = IN_LDS ? 4 : min(4, max(1, N / (NT * 64)));
    const int runs = nsamp * NT;
    auto run_start = [&](int q) { return (int)(((int64_t)(q * NT + tid) * (N / 4)) / runs) * 4; };
    auto sample4 = [&](int q, float (&v)[4]) {
      if (IN_LDS) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = s.at((int)(((int64_t)((q * 4 + e) * NT + tid) * N) / (16 * NT)));
      } else {
        load_items4<VEC>(s, N, run_start(q), v);
      }
    };
    float mn = INFINITY, mx = -INFINITY;
    uint32_t ns = 0;
    for (int q = 0; q < nsamp; ++q) {
      float v[4];
      sample4(q, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        mn = fminf(mn, canon(v[e]));
        mx = fmaxf(mx, canon(v[e]));
      }
      ns += 4;
    }
    block_min_max_cnt<CAP>(sh, mn, mx, ns);
    const float span = mx - mn;
    const float inv = (float)NB / span;
    if (__builtin_isfinite(span) && span > 0.f && __builtin_isfinite(inv)) {
      auto vb = [&](float v) {
        const int b = (int)((v - mn) * inv);
        return b < 0 ? 0 : (b > NB - 1 ? NB - 1 : b);
      };
      clear_hist<CAP>(sh);
      for (int q = 0; q < nsamp; ++q) {
        float v[4];
        sample4(q, v);
#pragma unroll
        for (int e = 0; e < 4; ++e) atomicAdd(&sh.hist[w][vb(canon(v[e]))], 1u);
      }
      __syncthreads();
      const float f = (float)k / (float)N * (float)ns;
      const float sd = 4.0f * sqrtf(f);
      const int r_hi = (int)floorf(f - sd);
      const int r_lo = min((int)ceilf(f + sd) + 1, (int)ns);
      float p_hi = INFINITY;
      uint32_t ab, inb;
      if (r_hi >= 1) {
        const int b = find_bin<CAP>(sh, r_hi, &ab, &inb);
        p_hi = b >= NB - 1 ? INFINITY : mn + (float)(b + 1) * (span / (float)NB);
      }
      const int bl = find_bin<CAP>(sh, r_lo, &ab, &inb);
      const float p_lo = mn + (float)max(bl, 1) * (span / (float)NB);
      // One pass: count x >= p_hi; append the token indices with
      // p_lo <= x < p_hi to the LDS list (per step: each thread's candidates
      // as a bit mask, a wave scan for the offsets, one LDS atomic per wave to
      // reserve space, a loop over the set bits). p_lo is finite, so NaN
      // inputs (ranked as -inf) compare below both pivots.
      if (tid == 0) sh.ccount = 0;
      __syncthreads();
      uint32_t c_hi = 0;
      {
        const int t0 = ITEMS * tid;
        float cur[ITEMS], nxt[ITEMS];
        load_items<VEC>(s, N, t0, cur);
        for (int base = 0; base < N; base += CHUNK) {
          const int n0 = base + t0;
          if (base + CHUNK < N) load_items<VEC>(s, N, n0 + CHUNK, nxt);
          uint32_t mm = 0;
          if (base + CHUNK <= N) {
#pragma unroll
            for (int e = 0; e < ITEMS; ++e) {
              const bool hi = cur[e] >= p_hi;
              c_hi += hi;
              mm |= (cur[e] >= p_lo && !hi) ? (1u << e) : 0u;
            }
          } else {
#pragma unroll
            for (int e = 0; e < ITEMS; ++e) {
              const bool ok = n0 + e < N;
              const bool hi = ok && cur[e] >= p_hi;
              c_hi += hi;
              mm |= (ok && cur[e] >= p_lo && !hi) ? (1u << e) : 0u;
            }
          }
          const uint32_t cnt = (uint32_t)__popc(mm);
          const uint32_t incl = wave_inclusive_scan(cnt);
          const uint32_t wtot = (uint32_t)__shfl((int)incl, 63);
          if (wtot) {
            uint32_t slot0 = 0;
            if (lane == 0) slot0 = atomicAdd(&sh.ccount, wtot);
            uint32_t slot = (uint32_t)__shfl((int)slot0, 0) + incl - cnt;
            while (mm) {
              const int e = __builtin_ctz(mm);
              mm &= mm - 1u;
              if (slot < (uint32_t)CAP) sh.cidx[0][slot] = n0 + e;
              ++slot;
            }
          }
#pragma unroll
          for (int e = 0; e < ITEMS; ++e) cur[e] = nxt[e];
        }
      }
      float d0 = 0.f, d1 = 0.f;
      block_min_max_cnt<CAP>(sh, d0, d1, c_hi);  // sums c_hi over the block (and orders the appends)
      const uint32_t c_mid = sh.ccount;
      if (c_mid <= (uint32_t)CAP && c_hi < (uint32_t)k && (uint32_t)k <= c_hi + c_mid) {
        // keys of the candidates, re-read from the (cache-resident) row
        for (int i = tid; i < (int)c_mid; i += NT) sh.ckey[0][i] = ordered_key(canon(s.at(sh.cidx[0][i])));
        __syncthreads();
        need = k - (int)c_hi;
        in_lds = (int)c_mid;
      } else if (c_hi >= (uint32_t)k) {  // the k-th token is >= p_hi
        lo0 = p_hi;
      } else if ((uint32_t)k <= c_hi + c_mid) {  // in [p_lo, p_hi), too many to list
        lo0 = p_lo;
        hi0 = float_below(p_hi);
        need = k - (int)c_hi;
      } else {  // below p_lo
        hi0 = float_below(p_lo);
        need = k - (int)(c_hi + c_mid);
      }
    }
  }

  // ---------------- 1. rounds over the stream
  if (in_lds < 0) {
    float lo = lo0, hi = hi0;
    bool vsel = false, ksel = false;
    float vlo = 0.f, vinv = 0.f;
    uint32_t klo = 0u;
    int kshift = 0, sbin = 0;
    auto vbin_of = [](float v, float base, float inv) {
      const int b = (int)((v - base) * inv);
      return b < 0 ? 0 : (b > NB - 1 ? NB - 1 : b);
    };
    auto is_cand = [&](float v) {
      if (!(v >= lo && v <= hi)) return false;
      if (vsel) return vbin_of(v, vlo, vinv) == sbin;
      if (ksel) return (int)((ordered_key(v) - klo) >> kshift) == sbin;
      return true;
    };
    bool stalled = false;
    // at most two value-binned rounds, then radix rounds that cut the key
    // span by 2^8 each: resolved within 2 + 4 + 1 rounds
    for (int it = 0; it < 10; ++it) {
      float mn = INFINITY, mx = -INFINITY;
      uint32_t cnt = 0;
      stream_row<VEC>(s, N, [&](int, float x) {
        if (is_cand(x)) {
          mn = fminf(mn, x);
          mx = fmaxf(mx, x);
          ++cnt;
        }
      });
      block_min_max_cnt<CAP>(sh, mn, mx, cnt);
      lo = mn;
      hi = mx;
      vsel = ksel = false;
      if (mn == mx) {
        T = mn;
        const int nd = need;
        ordered_stream<VEC, CAP>(sh, s, N, [&](int, float x) { return x == T; },
                                 [&](int n, uint32_t pos) {
                                   if (pos == (uint32_t)(nd - 1)) sh.bcast[3] = (uint32_t)n;
                                 });
        n_cut = (int)sh.bcast[3];
        done = true;
        break;
      }
      if (cnt <= (uint32_t)CAP) {
        if (tid == 0) sh.ccount = 0;
        __syncthreads();
        stream_row<VEC>(s, N, [&](int n, float x) {
          if (x >= lo && x <= hi) {
            const uint32_t slot = atomicAdd(&sh.ccount, 1u);
            if (slot < (uint32_t)CAP) {
              sh.ckey[0][slot] = ordered_key(x);
              sh.cidx[0][slot] = n;
            }
          }
        });
        __syncthreads();
        in_lds = (int)cnt;
        break;
      }
      const float span = mx - mn;
      const bool vmode = it < 2 && !stalled && __builtin_isfinite(mn) && __builtin_isfinite(mx) &&
                         __builtin_isfinite(span) && span > 0.f && __builtin_isfinite((float)NB / span);
      const float inv = vmode ? (float)NB / span : 0.f;
      const uint32_t kmn = ordered_key(mn), kspan = ordered_key(mx) - kmn;
      const int bits = 32 - __clz((int)kspan);
      const int shift = bits > 8 ? bits - 8 : 0;
      clear_hist<CAP>(sh);
      stream_row<VEC>(s, N, [&](int, float x) {
        if (x >= lo && x <= hi) {
          const int b = vmode ? vbin_of(x, mn, inv) : (int)((ordered_key(x) - kmn) >> shift);
          atomicAdd(&sh.hist[w][b], 1u);
        }
      });
      __syncthreads();
      uint32_t above, inb;
      const int bstar = find_bin<CAP>(sh, need, &above, &inb);
      need -= (int)above;
      stalled = vmode && inb == cnt;
      sbin = bstar;
      if (vmode) {
        vsel = true;
        vlo = mn;
        vinv = inv;
      } else {
        ksel = true;
        klo = kmn;
        kshift = shift;
      }
    }
  }

  // ---------------- 2. rounds over the LDS candidates (order-preserving keys)
  if (!done && in_lds >= 0) {
    int cur = 0;
    int c = in_lds;
    for (int it = 0; it < 8; ++it) {
      uint32_t kmn = 0xffffffffu, kmx = 0u;
      for (int i = tid; i < c; i += NT) {
        kmn = min(kmn, sh.ckey[cur][i]);
        kmx = max(kmx, sh.ckey[cur][i]);
      }
      block_umin_umax<CAP>(sh, kmn, kmx);
      if (kmn == kmx) {
        T = key_to_float(kmn);
        const int nd = need;
        ordered_stream<VEC, CAP>(sh, s, N, [&](int, float x) { return x == T; },
                                 [&](int n, uint32_t pos) {
                                   if (pos == (uint32_t)(nd - 1)) sh.bcast[3] = (uint32_t)n;
                                 });
        n_cut = (int)sh.bcast[3];
        done = true;
        break;
      }
      if (c <= RANKCAP) {
        if (w == 0) {
          uint32_t kc = 0u;
          int nc = 0;
          if (lane < c) {
            kc = sh.ckey[cur][lane];
            nc = sh.cidx[cur][lane];
          }
          int rank = 0;
          for (int o = 0; o < c; ++o) {
            const uint32_t ko = sh.ckey[cur][o];
            const int no = sh.cidx[cur][o];
            rank += (ko > kc) || (ko == kc && no < nc);
          }
          if (lane < c && rank == need - 1) {
            sh.bcast[2] = kc;
            sh.bcast[3] = (uint32_t)nc;
          }
        }
        __syncthreads();
        T = key_to_float(sh.bcast[2]);
        n_cut = (int)sh.bcast[3];
        done = true;
        break;
      }
      const uint32_t kspan = kmx - kmn;
      const int bits = 32 - __clz((int)kspan);
      const int shift = bits > 8 ? bits - 8 : 0;
      clear_hist<CAP>(sh);
      for (int i = tid; i < c; i += NT) atomicAdd(&sh.hist[w][(sh.ckey[cur][i] - kmn) >> shift], 1u);
      __syncthreads();
      uint32_t above, inb;
      const int bstar = find_bin<CAP>(sh, need, &above, &inb);
      need -= (int)above;
      if (tid == 0) sh.ccount = 0;
      __syncthreads();
      for (int i0 = 0; i0 < c; i0 += NT) {
        const int i = i0 + tid;
        const bool keep = i < c && (int)((sh.ckey[cur][i] - kmn) >> shift) == bstar;
        const uint64_t b = __ballot(keep);
        uint32_t base = 0;
        if (lane == 0 && b) base = atomicAdd(&sh.ccount, (uint32_t)__popcll(b));
        base = __shfl(base, 0);
        if (keep) {
          const uint32_t slot = base + lanes_below(b);
          sh.ckey[cur ^ 1][slot] = sh.ckey[cur][i];
          sh.cidx[cur ^ 1][slot] = sh.cidx[cur][i];
        }
      }
      __syncthreads();
      cur ^= 1;
      c = (int)inb;
    }
  }

  // ---------------- output: ascending token order
  const float Tf = T;
  const int nc = n_cut;
  ordered_stream<VEC, CAP>(sh, s, N, [&](int n, float x) { return x > Tf || (x == Tf && n <= nc); },
                           [&](int n, uint32_t pos) {
                             if (pos < (uint32_t)k) out[pos] = n;
                           });
}

// Workgroup b of nb walks the *nrows rows listed in rows (every workgroup
// exits at once when there are none). lrow: LDS row copy of ROWCAP floats.
template <int CAP, bool VEC, int ROWCAP>
__device__ __forceinline__ void topk_listed_body(TopkSmem<CAP> &sh, float *lrow, int b, int nb,
                                                 const float *__restrict__ S, int32_t *__restrict__ idx, int N, int k,
                                                 const uint32_t *__restrict__ nrows,
                                                 const int32_t *__restrict__ rows) {
  const uint32_t n = *nrows;
  for (uint32_t f = (uint32_t)b; f < n; f += (uint32_t)nb) {
    const int64_t row = rows[f];
    __syncthreads();  // the previous row's last reads of LDS are done
    topk_row<CAP, VEC, ROWCAP>(sh, lrow, S + row * (int64_t)N, idx + row * (int64_t)k, N, k);
  }
}

}  // namespace mita
