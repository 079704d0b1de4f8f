// Device helpers shared by the gfx950 kernel files of the DMC library
// (bf16 conversion, 16-byte loads, wave reductions, matrix-core operands).
// Internal; included by .hip translation units only.
#pragma once

#include "dmc_internal.h"

namespace dmc {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ float neg_inf() { return -__builtin_huge_valf(); }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (quiet NaN preserved).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return ((u >> 16) | 0x40u) & 0xffffu;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

template <int ES>
__device__ __forceinline__ float load_elem(const void *base, int64_t idx);
template <>
__device__ __forceinline__ float load_elem<2>(const void *base, int64_t idx) {
  return __uint_as_float(uint32_t(static_cast<const uint16_t *>(base)[idx]) << 16);
}
template <>
__device__ __forceinline__ float load_elem<4>(const void *base, int64_t idx) {
  return static_cast<const float *>(base)[idx];
}

// 16-byte vector <-> floats.
template <int ES>
struct V16;
template <>
struct V16<2> {
  static constexpr int N = 8;
  __device__ static __forceinline__ void unpack(const uint4 &r, float *f) {
    f[0] = bf16_lo(r.x); f[1] = bf16_hi(r.x); f[2] = bf16_lo(r.y); f[3] = bf16_hi(r.y);
    f[4] = bf16_lo(r.z); f[5] = bf16_hi(r.z); f[6] = bf16_lo(r.w); f[7] = bf16_hi(r.w);
  }
  // Round to storage; f is replaced by the widened stored values.
  __device__ static __forceinline__ uint4 pack(float *f) {
    uint32_t h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      h[i] = bf16_bits(f[i]);
      f[i] = __uint_as_float(h[i] << 16);
    }
    return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                      h[6] | (h[7] << 16));
  }
};
template <>
struct V16<4> {
  static constexpr int N = 4;
  __device__ static __forceinline__ void unpack(const uint4 &r, float *f) {
    f[0] = __uint_as_float(r.x); f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z); f[3] = __uint_as_float(r.w);
  }
  __device__ static __forceinline__ uint4 pack(float *f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// One lane's slice of a query head (16 bytes of it) with q[0] zeroed, and
// its dot product with the matching 16-byte slice of a key row.  bf16 keeps
// the query packed and uses v_dot2_f32_bf16 (products exact in fp32, fp32
// accumulation); fp32 uses plain FMAs.
template <int ES>
struct QSlice;
template <>
struct QSlice<2> {
  uint4 w;
  __device__ __forceinline__ void load(const char *p, bool first) {
    w = *reinterpret_cast<const uint4 *>(p);
    if (first) w.x &= 0xffff0000u;
  }
  __device__ __forceinline__ float dot(const uint4 &k) const {
    float d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.x),
                                              __builtin_bit_cast(bf16x2_t, k.x), 0.0f, false);
    d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.y),
                                        __builtin_bit_cast(bf16x2_t, k.y), d, false);
    d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.z),
                                        __builtin_bit_cast(bf16x2_t, k.z), d, false);
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.w),
                                           __builtin_bit_cast(bf16x2_t, k.w), d, false);
  }
};
template <>
struct QSlice<4> {
  float f[4];
  __device__ __forceinline__ void load(const char *p, bool first) {
    const uint4 r = *reinterpret_cast<const uint4 *>(p);
    V16<4>::unpack(r, f);
    if (first) f[0] = 0.0f;
  }
  __device__ __forceinline__ float dot(const uint4 &k) const {
    float kf[4];
    V16<4>::unpack(k, kf);
    float d = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) d = fmaf(f[e], kf[e], d);
    return d;
  }
};

__device__ __forceinline__ uint4 ld16(const char *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ void st16(char *p, const uint4 &v) { *reinterpret_cast<uint4 *>(p) = v; }

// E consecutive elements (E = 1 or 2) <-> floats, for the prefill/combine paths.
// (One memory access each; p is aligned to E * ES bytes.)
template <int ES, int E>
__device__ __forceinline__ void load_e(const char *p, float *f) {
  if constexpr (ES == 2 && E == 2) {
    const uint32_t w = *reinterpret_cast<const uint32_t *>(p);
    f[0] = __uint_as_float(w << 16);
    f[1] = __uint_as_float(w & 0xffff0000u);
  } else if constexpr (ES == 4 && E == 2) {
    const float2 w = *reinterpret_cast<const float2 *>(p);
    f[0] = w.x;
    f[1] = w.y;
  } else {
    f[0] = load_elem<ES>(p, 0);
  }
}
// load_e with the nontemporal policy, for data read once (prompt rows).
template <int ES, int E>
__device__ __forceinline__ void load_e_nt(const char *p, float *f) {
  if constexpr (ES == 2 && E == 2) {
    const uint32_t w = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(p));
    f[0] = __uint_as_float(w << 16);
    f[1] = __uint_as_float(w & 0xffff0000u);
  } else if constexpr (ES == 4 && E == 2) {
    typedef float f2_t __attribute__((ext_vector_type(2)));
    const f2_t w = __builtin_nontemporal_load(reinterpret_cast<const f2_t *>(p));
    f[0] = w.x;
    f[1] = w.y;
  } else if constexpr (ES == 2) {
    f[0] = __uint_as_float(uint32_t(__builtin_nontemporal_load(reinterpret_cast<const uint16_t *>(p)))
                           << 16);
  } else {
    f[0] = __builtin_nontemporal_load(reinterpret_cast<const float *>(p));
  }
}
template <int ES, int E>
__device__ __forceinline__ void store_e(char *p, const float *f) {
  if constexpr (ES == 2 && E == 2) {
    *reinterpret_cast<uint32_t *>(p) = bf16_bits(f[0]) | (bf16_bits(f[1]) << 16);
  } else if constexpr (ES == 4 && E == 2) {
    *reinterpret_cast<float2 *>(p) = make_float2(f[0], f[1]);
  } else if constexpr (ES == 2) {
    *reinterpret_cast<uint16_t *>(p) = static_cast<uint16_t>(bf16_bits(f[0]));
  } else {
    *reinterpret_cast<float *>(p) = f[0];
  }
}

// store_e with the nontemporal policy, for rows written once and read much later.
template <int ES, int E>
__device__ __forceinline__ void store_e_nt(char *p, const float *f) {
  if constexpr (ES == 2 && E == 2) {
    __builtin_nontemporal_store(bf16_bits(f[0]) | (bf16_bits(f[1]) << 16),
                                reinterpret_cast<uint32_t *>(p));
  } else {
    store_e<ES, E>(p, f);
  }
}

__device__ __forceinline__ float sigmoid_floor(float x) {
  // omega = sigmoid(x), floored at 2^-100 so a running sum never reaches 0.
  return fmaxf(1.0f / (1.0f + expf(-x)), 0x1p-100f);
}

// Reduction over the LPR lanes of a row group (lanes are grouped in runs of
// LPR); every lane of the group receives the sum.
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
  static_assert(LPR == 8 || LPR == 16 || LPR == 32, "row width");
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x141, 0xF, 0xF, false));  // row_half_mirror
  if (LPR >= 16)
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x140, 0xF, 0xF, false));  // row_mirror
  if (LPR >= 32) x += __shfl_xor(x, 16, 64);
  return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Streaming 16-byte load of cache data that is read once per step.
__device__ __forceinline__ uint4 ld16_stream(const char *p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// v_mfma_f32_16x16x32_bf16 on 16-byte operand slices (8 bf16 per lane).
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma_16x16x32(const uint4 &a, const uint4 &b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
  return bf16_bits(lo) | (bf16_bits(hi) << 16);
}

// Prompt length of batch row b (n when no lengths are given), clamped to [0, n].
__device__ __forceinline__ int clamp_prompt_len(const int32_t *prompt_lens, int n, int b) {
  if (!prompt_lens) return n;
  const int x = prompt_lens[b];
  return x < 0 ? 0 : (x > n ? n : x);
}

}  // namespace
}  // namespace dmc
