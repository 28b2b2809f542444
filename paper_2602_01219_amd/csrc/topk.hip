// topk.hip - exact top-k per landmark row (Eq. top-k).
//
// Order: larger score first, equal scores by lower token index (-0 == +0).
// The k first tokens of that order are written in ascending index order.
//
// One workgroup per row. The row lives in registers as order-preserving
// uint32 keys (item j of thread t is token j*NT + t, so loads are coalesced).
// The workgroup narrows a candidate set that is always a contiguous run of
// the sorted order:
//   * count / min / max of the candidates (block reduction);
//   * all candidates equal -> the threshold key is known, the cut among the
//     tied tokens is found by an index-ordered scan;
//   * few candidates -> they are ranked exactly in LDS;
//   * otherwise a 256-bin histogram of the candidates (linear bins over the
//     float value range for the first two rounds, which spreads clustered
//     scores; then radix bins over the key range, which shrink the range by
//     at least 128x per round and so guarantee termination) selects the bin
//     holding the target rank.
// The threshold is the pair (T, n_cut) of the k-th token in the order; a
// token is selected iff key > T or (key == T and n <= n_cut). The final
// compaction is an index-ordered scan with ballot / mbcnt, so the output is
// ascending without a sort.
#include "cdna4.hpp"
#include "kernels.hpp"
#include "check.hpp"

namespace mita {

namespace {

constexpr int NB = 256;   // histogram bins
constexpr int CAP = 256;  // exact-ranking capacity

template <int NT> struct TopkShared {
  static constexpr int NW = NT / 64;
  uint32_t hist[NW][NB];
  uint32_t cand_key[CAP];
  int32_t cand_n[CAP];
  uint32_t red[3][NW];
  uint32_t wtot[NW];
  uint32_t bcast[4];
  uint32_t ccount;
};

// Block-wide (sum, min, max); every thread receives the results.
template <int NT>
__device__ __forceinline__ void block_cnt_min_max(TopkShared<NT> &sh, uint32_t &cnt, uint32_t &mn, uint32_t &mx) {
  constexpr int NW = NT / 64;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  cnt = wave_sum_u32(cnt);
  mn = wave_min_u32(mn);
  mx = wave_max_u32(mx);
  if (lane == 0) {
    sh.red[0][w] = cnt;
    sh.red[1][w] = mn;
    sh.red[2][w] = mx;
  }
  __syncthreads();
  cnt = 0;
  mn = 0xffffffffu;
  mx = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    cnt += sh.red[0][i];
    mn = min(mn, sh.red[1][i]);
    mx = max(mx, sh.red[2][i]);
  }
  __syncthreads();
}

// Index-ordered exclusive scan of per-item flags: for every flagged item j,
// emit(j, number of flagged items with a lower token index). The predicate is
// evaluated twice instead of being stored, to keep registers for the keys.
// scan_buf holds IPT*NW counters.
template <int NT, int IPT, typename Pred, typename Emit>
__device__ __forceinline__ void ordered_scan(Pred pred, Emit emit, uint32_t *scan_buf) {
  constexpr int NW = NT / 64;
  constexpr int NE = IPT * NW;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const uint64_t b = __ballot(pred(j));
    if (lane == 0) scan_buf[j * NW + w] = (uint32_t)__popcll(b);
  }
  __syncthreads();
  if (w == 0) {
    constexpr int E = (NE + 63) / 64;
    uint32_t v[E];
    uint32_t sum = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      v[e] = i < NE ? scan_buf[i] : 0u;
      sum += v[e];
    }
    uint32_t run = wave_inclusive_scan(sum) - sum;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      if (i < NE) scan_buf[i] = run;
      run += v[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const bool f = pred(j);
    const uint64_t b = __ballot(f);
    if (f) emit(j, scan_buf[j * NW + w] + lanes_below(b));
  }
  __syncthreads();
}

}  // namespace

template <int NT, int IPT>
__global__ __launch_bounds__(NT) void topk_kernel(const float *__restrict__ S, int32_t *__restrict__ idx, int N,
                                                  int k) {
  constexpr int NW = NT / 64;
  __shared__ TopkShared<NT> sh;
  __shared__ uint32_t scan_buf[IPT * NW];
  const int64_t row = blockIdx.x;
  const float *s = S + row * (int64_t)N;
  int32_t *out = idx + row * (int64_t)k;
  const int tid = threadIdx.x, w = tid >> 6;

  uint32_t key[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int n = j * NT + tid;
    // valid keys are >= 1 (only a NaN pattern moves), so key 0 marks the
    // padding items and is never a candidate or selected
    key[j] = n < N ? max(ordered_key(s[n]), 1u) : 0u;
  }

  // Candidate predicate: valid, lo <= key <= hi, and (after a value-binned
  // round) in the chosen value bin.
  uint32_t lo = 1u, hi = 0xffffffffu;
  bool vsel = false;
  float vlo = 0.f, vinv = 0.f;
  int vbin = 0;
  int need = k;  // rank (1-based) of the target inside the candidate set
  uint32_t T = 0u;
  int n_cut = -1;

  auto value_bin = [](uint32_t kk, float xlo, float inv) {
    asm volatile("" : "+v"(kk));  // keep the decode inside the round loop (registers)
    const float f = (key_to_float(kk) - xlo) * inv;
    const int b = (int)f;
    return b < 0 ? 0 : (b > NB - 1 ? NB - 1 : b);
  };
  auto is_cand = [&](int j) {
    if (key[j] < lo || key[j] > hi) return false;
    return !vsel || value_bin(key[j], vlo, vinv) == vbin;
  };

  // At most 2 value rounds + 5 radix rounds + the resolving round.
  for (int it = 0; it < 16; ++it) {
    uint32_t cnt = 0, kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
    for (int j = 0; j < IPT; ++j)
      if (is_cand(j)) {
        ++cnt;
        kmin = min(kmin, key[j]);
        kmax = max(kmax, key[j]);
      }
    block_cnt_min_max<NT>(sh, cnt, kmin, kmax);
    lo = kmin;
    hi = kmax;
    vsel = false;

    if (kmin == kmax) {
      // Every candidate has key T: take the need-th of them in index order.
      T = kmin;
      ordered_scan<NT, IPT>([&](int j) { return key[j] == T; },
                            [&](int j, uint32_t pos) {
                              if (pos == (uint32_t)(need - 1)) sh.bcast[0] = (uint32_t)(j * NT + tid);
                            },
                            scan_buf);
      n_cut = (int)sh.bcast[0];
      break;
    }

    if (cnt <= (uint32_t)CAP) {
      // Rank the few candidates exactly: (key desc, index asc).
      if (tid == 0) sh.ccount = 0;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < IPT; ++j)
        if (is_cand(j)) {
          const uint32_t slot = atomicAdd(&sh.ccount, 1u);
          if (slot < (uint32_t)CAP) {
            sh.cand_key[slot] = key[j];
            sh.cand_n[slot] = j * NT + tid;
          }
        }
      __syncthreads();
      for (int c = tid; c < (int)cnt; c += NT) {
        const uint32_t kc = sh.cand_key[c];
        const int nc = sh.cand_n[c];
        int rank = 0;
        for (int o = 0; o < (int)cnt; ++o) {
          const uint32_t ko = sh.cand_key[o];
          rank += (ko > kc) || (ko == kc && sh.cand_n[o] < nc);
        }
        if (rank == need - 1) {
          sh.bcast[0] = kc;
          sh.bcast[1] = (uint32_t)nc;
        }
      }
      __syncthreads();
      T = sh.bcast[0];
      n_cut = (int)sh.bcast[1];
      break;
    }

    // Histogram round.
    bool vmode = false;
    float xlo = 0.f, inv = 0.f;
    int shift = 0;
    if (it < 2) {
      xlo = key_to_float(kmin);
      const float xhi = key_to_float(kmax);
      const float span = xhi - xlo;
      if (__builtin_isfinite(xlo) && __builtin_isfinite(xhi) && __builtin_isfinite(span) && span > 0.f) {
        inv = (float)NB / span;
        vmode = __builtin_isfinite(inv) && inv > 0.f;
      }
    }
    if (!vmode) {
      const uint32_t span = kmax - kmin;  // > 0
      const int bits = 32 - __clz((int)span);
      shift = bits > 8 ? bits - 8 : 0;
    }
    for (int i = tid; i < NW * NB; i += NT) (&sh.hist[0][0])[i] = 0u;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      if (key[j] >= kmin && key[j] <= kmax) {
        const int b = vmode ? value_bin(key[j], xlo, inv) : (int)((key[j] - kmin) >> shift);
        atomicAdd(&sh.hist[w][b], 1u);
      }
    }
    __syncthreads();
    // Scan bins from the top: thread t < NB looks at bin NB-1-t.
    uint32_t tot = 0, incl = 0;
    if (tid < NB) {
      const int b = NB - 1 - tid;
#pragma unroll
      for (int i = 0; i < NW; ++i) tot += sh.hist[i][b];
      incl = wave_inclusive_scan(tot);
      if ((tid & 63) == 63) sh.wtot[tid >> 6] = incl;
    }
    __syncthreads();
    if (tid < NB) {
      for (int i = 0; i < (tid >> 6); ++i) incl += sh.wtot[i];
      const uint32_t above = incl - tot;
      if (above < (uint32_t)need && (uint32_t)need <= incl) {
        sh.bcast[0] = (uint32_t)(NB - 1 - tid);
        sh.bcast[1] = above;
      }
    }
    __syncthreads();
    const int bstar = (int)sh.bcast[0];
    need -= (int)sh.bcast[1];
    __syncthreads();
    if (vmode) {
      vsel = true;
      vlo = xlo;
      vinv = inv;
      vbin = bstar;
    } else {
      lo = kmin + ((uint32_t)bstar << shift);
      const uint64_t h = (uint64_t)lo + ((1ull << shift) - 1ull);
      hi = (uint32_t)min<uint64_t>(h, (uint64_t)kmax);
    }
  }

  // Final compaction in ascending token order.
  ordered_scan<NT, IPT>(
      [&](int j) { return key[j] > T || (key[j] == T && j * NT + tid <= n_cut); },
      [&](int j, uint32_t pos) {
        if (pos < (uint32_t)k) out[pos] = j * NT + tid;
      },
      scan_buf);
}

template <int NT, int IPT> static hipError_t topk_t(const mita_cfg_t &c, const float *S, int32_t *idx, hipStream_t st) {
  const int64_t rows = BH(c) * c.M;
  hipLaunchKernelGGL((topk_kernel<NT, IPT>), dim3((unsigned)rows), dim3(NT), 0, st, S, idx, c.N, c.k);
  return hipGetLastError();
}

hipError_t launch_topk(const mita_cfg_t &c, const float *S, int32_t *idx, hipStream_t st) {
  const int N = c.N;
  if (N <= 256) return topk_t<256, 1>(c, S, idx, st);
  if (N <= 512) return topk_t<256, 2>(c, S, idx, st);
  if (N <= 1024) return topk_t<256, 4>(c, S, idx, st);
  if (N <= 2048) return topk_t<256, 8>(c, S, idx, st);
  if (N <= 4096) return topk_t<256, 16>(c, S, idx, st);
  if (N <= 8192) return topk_t<512, 16>(c, S, idx, st);
  if (N <= 16384) return topk_t<1024, 16>(c, S, idx, st);
  if (N <= 32768) return topk_t<1024, 32>(c, S, idx, st);
  return topk_t<1024, 64>(c, S, idx, st);
}

}  // namespace mita
