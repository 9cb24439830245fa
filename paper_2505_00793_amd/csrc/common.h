// Shared device helpers for the MixFlow-MG kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfmg {

typedef uint16_t bf16_t;  // bfloat16 storage
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// float -> bfloat16, round to nearest even (add 0x7fff plus the lsb of the kept
// half, then truncate).  Inputs are finite.
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// Operand element traits: VE elements per 16-byte vector.
template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static constexpr int VE = 8;
  __device__ static __forceinline__ bf16_t from_float(float f) { return f2bf(f); }
  __device__ static __forceinline__ float to_float(bf16_t h) { return bf2f(h); }
};
template <> struct Elem<float> {
  static constexpr int VE = 4;
  __device__ static __forceinline__ float from_float(float f) { return f; }
  __device__ static __forceinline__ float to_float(float f) { return f; }
};

// Four consecutive elements stored with one 8-byte (bf16) or 16-byte (fp32) write.
__device__ __forceinline__ void store4(bf16_t* p, float a, float b, float c, float d) {
  uint2 v;
  v.x = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
  v.y = (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16);
  *reinterpret_cast<uint2*>(p) = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}

enum Act { ACT_TANH = 0, ACT_GELU = 1, ACT_RELU = 2, ACT_NONE = 3 };

__device__ __forceinline__ float act_f(int act, float z) {
  switch (act) {
    case ACT_TANH: return tanhf(z);
    case ACT_GELU: return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
    case ACT_RELU: return z > 0.0f ? z : 0.0f;
    default: return z;
  }
}

// First and second derivative of the activation at z.
__device__ __forceinline__ void act_d12(int act, float z, float& d1, float& d2) {
  switch (act) {
    case ACT_TANH: {
      float t = tanhf(z);
      d1 = 1.0f - t * t;
      d2 = -2.0f * t * d1;
      break;
    }
    case ACT_GELU: {
      float cdf = 0.5f * (1.0f + erff(z * 0.70710678118654752f));
      float pdf = 0.39894228040143268f * expf(-0.5f * z * z);
      d1 = cdf + z * pdf;
      d2 = pdf * (2.0f - z * z);
      break;
    }
    case ACT_RELU:
      d1 = z > 0.0f ? 1.0f : 0.0f;
      d2 = 0.0f;
      break;
    default:
      d1 = 1.0f;
      d2 = 0.0f;
  }
}

// Wavefront (64-lane) sum by butterfly shuffles.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

}  // namespace mfmg
