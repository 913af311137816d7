// Device-side helpers shared by the gfx950 kernels of the chunked MoE layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace memfine {

typedef uint16_t bf16_t;  // bf16 kept as raw bits in memory

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// float -> bf16 bits, round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return ((u >> 16) | 0x40u) & 0xffffu;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Element access for the two storage types of the layer.
template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p) { return bf16_bits_to_f32(*p); }
  __device__ __forceinline__ static void store(bf16_t* p, float v) { *p = (bf16_t)f32_to_bf16_bits(v); }
  static constexpr int kVec = 8;  // elements per 16-byte vector
};
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static void store(float* p, float v) { *p = v; }
  static constexpr int kVec = 4;
};

// Unpack / pack a 16-byte vector of T into floats.
__device__ __forceinline__ void unpack16(const u32x4_t& v, float (&f)[8], bf16_t*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(v[i] << 16);
    f[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack16(const u32x4_t& v, float (&f)[4], float*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(v[i]);
}
__device__ __forceinline__ u32x4_t pack16(const float (&f)[8], bf16_t*) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = f32_to_bf16_bits(f[2 * i]) | (f32_to_bf16_bits(f[2 * i + 1]) << 16);
  return v;
}
__device__ __forceinline__ u32x4_t pack16(const float (&f)[4], float*) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(f[i]);
  return v;
}

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + __expf(-z)); }

}  // namespace memfine
