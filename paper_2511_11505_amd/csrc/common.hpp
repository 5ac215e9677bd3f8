// Device and host helpers shared by the FarSkip MoE kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define FS_WAVE 64

typedef uint16_t bf16_t;  // bf16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(bf16_t u) { return __uint_as_float(((uint32_t)u) << 16); }

// fp32 -> bf16, round to nearest even.
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(bf16_t, b);
}

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f2bf(v); }

// 16-byte vector of T: 4 floats or 8 bf16.
template <typename T>
struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
  uint4 raw;
  __device__ __forceinline__ float get(int i) const {
    if constexpr (sizeof(T) == 4) {
      return __uint_as_float((&raw.x)[i]);
    } else {
      uint32_t w = (&raw.x)[i >> 1];
      return __uint_as_float((i & 1) ? (w & 0xFFFF0000u) : (w << 16));
    }
  }
  __device__ __forceinline__ void set(int i, float v) {
    if constexpr (sizeof(T) == 4) {
      (&raw.x)[i] = __float_as_uint(v);
    } else {
      uint32_t b = f2bf(v);
      uint32_t& w = (&raw.x)[i >> 1];
      w = (i & 1) ? ((w & 0x0000FFFFu) | (b << 16)) : ((w & 0xFFFF0000u) | b);
    }
  }
};

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

// Wave-wide reductions (64 lanes).
// Wave-wide reductions without LDS traffic: inside each 16-lane row by DPP
// (swap neighbours, swap pairs, mirror each half-row, mirror the row), so
// that every lane of a row holds the row's result, then the four row results
// are read with v_readlane and combined; the result is wave-uniform.  Max
// and arg-max select exactly, so their result does not depend on the tree;
// the sum is one fixed tree.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141; // row_half_mirror
constexpr int kDppMirror = 0x140;     // row_mirror
__device__ __forceinline__ float lane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<kDppXor1>(v);
  v += dpp_f<kDppXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
// Arg-max of (key, idx): larger key wins, equal keys go to the lower idx.
// Bitwise | and & evaluate both comparisons, so this is a compare and two
// selects; a short-circuit || / && compiles to exec-mask branches, a serial
// chain of scalar instructions in every reduction step.
__device__ __forceinline__ void argmax_pick(float& key, int& idx, float k2, int i2) {
  const bool take = (k2 > key) | ((k2 == key) & (i2 < idx));
  key = take ? k2 : key;
  idx = take ? i2 : idx;
}
__device__ __forceinline__ void wave_argmax(float& key, int& idx) {
  argmax_pick(key, idx, dpp_f<kDppXor1>(key), dpp_i<kDppXor1>(idx));
  argmax_pick(key, idx, dpp_f<kDppXor2>(key), dpp_i<kDppXor2>(idx));
  argmax_pick(key, idx, dpp_f<kDppHalfMirror>(key), dpp_i<kDppHalfMirror>(idx));
  argmax_pick(key, idx, dpp_f<kDppMirror>(key), dpp_i<kDppMirror>(idx));
  float k = lane_f(key, 0);
  int i = __builtin_amdgcn_readlane(idx, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16)
    argmax_pick(k, i, lane_f(key, r), __builtin_amdgcn_readlane(idx, r));
  key = k;
  idx = i;
}

static inline int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }
