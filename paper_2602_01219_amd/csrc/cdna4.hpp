// cdna4.hpp - gfx950 (CDNA4) building blocks shared by the MiTA kernels:
// element types, 16x16 MFMA tiles over a 32-wide reduction step, wave64
// reductions and ordered-key helpers.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mita {

typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

constexpr int WAVE = 64;

// bfloat16 storage: raw 16-bit patterns.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }
// Round to nearest even (gfx950 v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
// Two values rounded to bf16 in one instruction: lo = a, hi = b.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

// ---------------------------------------------------------------------------
// Operand fragments.  A 16x16 MFMA tile with a 32-long reduction step: lane l
// (group g = l / 16, position p = l % 16) holds, for the A operand, row p and
// 8 reduction indices of group g; for the B operand, column p and the same 8
// reduction indices. Which 8 indices a group owns is a convention the loader
// chooses; A and B only need to agree. The accumulator holds C[4g + r][p],
// r = 0..3.
// For bf16 the 8 values are one v_mfma_f32_16x16x32_bf16 operand; for fp32
// the step is eight v_mfma_f32_16x16x4_f32, element e of every lane forming
// reduction slice e.
// ---------------------------------------------------------------------------
template <typename T> struct Frag;

template <> struct Frag<bf16_t> {
  uint4 v;  // 8 bf16
  __device__ __forceinline__ void zero() { v = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void load(const bf16_t *p) { v = *reinterpret_cast<const uint4 *>(p); }
  // 4 + 4 values from two places (used for transposed LDS tiles)
  __device__ __forceinline__ void load2x4(const bf16_t *p0, const bf16_t *p1) {
    uint2 a = *reinterpret_cast<const uint2 *>(p0);
    uint2 b = *reinterpret_cast<const uint2 *>(p1);
    v = make_uint4(a.x, a.y, b.x, b.y);
  }
  // from 8 fp32 values (rounded to bf16, two per v_cvt_pk_bf16_f32)
  __device__ __forceinline__ void from_f32(const float *x) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
    v = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

template <> struct Frag<float> {
  float4 a, b;  // 8 fp32
  __device__ __forceinline__ void zero() {
    a = make_float4(0.f, 0.f, 0.f, 0.f);
    b = a;
  }
  __device__ __forceinline__ void load(const float *p) {
    a = *reinterpret_cast<const float4 *>(p);
    b = *reinterpret_cast<const float4 *>(p + 4);
  }
  __device__ __forceinline__ void load2x4(const float *p0, const float *p1) {
    a = *reinterpret_cast<const float4 *>(p0);
    b = *reinterpret_cast<const float4 *>(p1);
  }
  __device__ __forceinline__ void from_f32(const float *x) {
    a = make_float4(x[0], x[1], x[2], x[3]);
    b = make_float4(x[4], x[5], x[6], x[7]);
  }
};

__device__ __forceinline__ f32x4 mma(const Frag<bf16_t> &A, const Frag<bf16_t> &B, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A.v), __builtin_bit_cast(bf16x8, B.v), c,
                                                 0, 0, 0);
}

__device__ __forceinline__ f32x4 mma(const Frag<float> &A, const Frag<float> &B, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.x, B.a.x, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.y, B.a.y, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.z, B.a.z, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.w, B.a.w, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.x, B.b.x, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.y, B.b.y, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.z, B.b.z, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.w, B.b.w, c, 0, 0, 0);
  return c;
}

// 16-byte vector of an element type (8 bf16 or 4 fp32).
template <typename T> struct Vec16 {
  static constexpr int n = 16 / sizeof(T);
};

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t x) { return bf16_to_f32(x.bits); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return bf16_t{f32_to_bf16(x)}; }

// Unpack a 16-byte chunk into fp32 values.
__device__ __forceinline__ void unpack16(const uint4 &u, float *x, const bf16_t *) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack16(const uint4 &u, float *x, const float *) {
  x[0] = __uint_as_float(u.x);
  x[1] = __uint_as_float(u.y);
  x[2] = __uint_as_float(u.z);
  x[3] = __uint_as_float(u.w);
}

// ---------------------------------------------------------------------------
// Wave64 reductions (ds_bpermute based shuffles).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = min(x, (uint32_t)__shfl_xor((int)x, o));
  return x;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = max(x, (uint32_t)__shfl_xor((int)x, o));
  return x;
}
// Maximum over the four 16-lane groups at the same position (lanes p, p+16,
// p+32, p+48), without LDS: v_permlane16_swap(x, x) yields groups (0,0,2,2)
// and (1,1,3,3), v_permlane32_swap the low and high halves. The pairwise
// max is med3(a, b, +inf), which needs no quieting of its inputs.
__device__ __forceinline__ float max_lane_groups(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __builtin_amdgcn_fmed3f(__uint_as_float(a[0]), __uint_as_float(a[1]), INFINITY);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_amdgcn_fmed3f(__uint_as_float(b[0]), __uint_as_float(b[1]), INFINITY);
}

// Inclusive prefix sum `incl` over the four 16-lane groups at the same
// position (lanes p, p+16, p+32, p+48; group g gets the sum over groups 0..g)
// and their total `tot`, without LDS: v_permlane16_swap(x, x) hands each lane
// the values of both groups of its pair (0,1) or (2,3), v_permlane32_swap
// the sums of both pairs. Only sums of the pairs are used, so the order of
// the two swap results does not matter.
__device__ __forceinline__ void scan_lane_groups(uint32_t x, uint32_t &incl, uint32_t &tot) {
  const int g = (threadIdx.x & 63) >> 4;
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  const uint32_t pair = a[0] + a[1];
  const auto b = __builtin_amdgcn_permlane32_swap(pair, pair, false, false);
  tot = b[0] + b[1];
  incl = ((g & 1) ? pair : x) + ((g & 2) ? tot - pair : 0u);
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t y = (uint32_t)__shfl_up((int)x, o);
    if (lane >= o) x += y;
  }
  return x;
}
// Wait until every global load this wave issued so far has landed. Placed
// after the loads that precede a software-pipelined loop (fragments kept in
// registers for the whole loop), it lets the compiler's wait placement inside
// the loop count only the loop's own in-flight loads instead of draining them
// before the first use of those fragments.
// (s_waitcnt fields on gfx9: vmcnt bits 3:0 and 15:14 = 0, expcnt 6:4 = 7 and
// lgkmcnt 11:8 = 15, i.e. no wait on those.)
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Order-preserving map of fp32 to uint32 (larger float -> larger key), with
// -0 mapped like +0 so that signed zeros tie.
__device__ __forceinline__ uint32_t ordered_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_to_float(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}
// Key of a score for the top-k order: NaN ranks as -inf, -0 as +0. Every
// key of a canonical score is >= ordered_key(-inf) = 0x007fffff, so 0 never
// occurs and can mark an empty slot.
__device__ __forceinline__ uint32_t score_key(float x) { return ordered_key(x != x ? -INFINITY : x); }

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t y = ((uint64_t)(uint32_t)__shfl_xor((int)(x >> 32), o) << 32) | (uint32_t)__shfl_xor((int)x, o);
    x = y < x ? y : x;
  }
  return x;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t y = ((uint64_t)(uint32_t)__shfl_xor((int)(x >> 32), o) << 32) | (uint32_t)__shfl_xor((int)x, o);
    x = y > x ? y : x;
  }
  return x;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t x, int src) {
  return ((uint64_t)(uint32_t)__shfl((int)(x >> 32), src) << 32) | (uint32_t)__shfl((int)x, src);
}

}  // namespace mita
