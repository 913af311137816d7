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

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// Two floats -> two bf16 in one dword (low half = a), round to nearest even;
// one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// Element access for the two storage types of the layer.
template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static constexpr int kVec = 8;  // elements per 16-byte vector
};
template <> struct Elem<float> {
  static constexpr int kVec = 4;
};

// Four consecutive elements of T <-> floats: one 8-byte (bf16) or 16-byte
// (fp32) access; the address must be aligned to it.  Raw is the loaded form,
// so that a batch of loads can be issued before any of them is unpacked.
template <typename T> struct Vec4;
template <> struct Vec4<bf16_t> {
  typedef u32x2_t Raw;
  __device__ __forceinline__ static Raw load_raw(const bf16_t* p) { return *(const u32x2_t*)p; }
  __device__ __forceinline__ static void unpack(const Raw& v, float (&f)[4]) {
    f[0] = __uint_as_float(v[0] << 16);
    f[1] = __uint_as_float(v[0] & 0xffff0000u);
    f[2] = __uint_as_float(v[1] << 16);
    f[3] = __uint_as_float(v[1] & 0xffff0000u);
  }
  __device__ __forceinline__ static void store(bf16_t* p, const float (&f)[4]) {
    u32x2_t v;
    v[0] = pack_bf16x2(f[0], f[1]);
    v[1] = pack_bf16x2(f[2], f[3]);
    *(u32x2_t*)p = v;
  }
};
template <> struct Vec4<float> {
  typedef f32x4_t Raw;
  __device__ __forceinline__ static Raw load_raw(const float* p) { return *(const f32x4_t*)p; }
  __device__ __forceinline__ static void unpack(const Raw& v, float (&f)[4]) {
    f[0] = v[0];
    f[1] = v[1];
    f[2] = v[2];
    f[3] = v[3];
  }
  __device__ __forceinline__ static void store(float* p, const float (&f)[4]) {
    *(f32x4_t*)p = (f32x4_t){f[0], f[1], f[2], f[3]};
  }
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
  for (int i = 0; i < 4; ++i) v[i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
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
