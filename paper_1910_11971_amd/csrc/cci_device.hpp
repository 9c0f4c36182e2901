// Device-side helpers shared by the CCI kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cci_types.hpp"

namespace cci {

// bf16 is carried as its raw 16-bit pattern; arithmetic happens in fp32.
struct bf16_t {
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bf16, round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T> struct io;
template <> struct io<float> {
  __device__ static __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
  __device__ static __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct io<bf16_t> {
  __device__ static __forceinline__ float load(const bf16_t* p, int64_t i) {
    return bf16_to_f32(p[i].bits);
  }
  __device__ static __forceinline__ void store(bf16_t* p, int64_t i, float v) {
    p[i].bits = f32_to_bf16_rne(v);
  }
};

// Fused epilogue operands (device pointers; null = absent).
template <typename YT>
struct Epilogue {
  const float* scale;
  const float* bias;
  const YT* residual;
  int relu;
};

template <typename YT>
__device__ __forceinline__ float apply_epilogue(float acc, int64_t o, int64_t yoff,
                                                const Epilogue<YT>& ep) {
  float y = acc;
  if (ep.scale) y = y * ep.scale[o];
  if (ep.bias) y = y + ep.bias[o];
  if (ep.residual) y = y + io<YT>::load(ep.residual, yoff);
  if (ep.relu) y = y > 0.0f ? y : (y != y ? y : 0.0f);
  return y;
}

}  // namespace cci
