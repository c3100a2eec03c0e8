// 16-byte vector loads/stores of float32 / float16 rows, converted to float.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bevpool {

typedef _Float16 half_t;
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ float to_float(T v) {
  return (float)v;
}

// Load VEC consecutive elements starting at `p` (aligned to VEC*sizeof(T)
// when VEC > 1) into float registers.
template <typename T, int VEC>
struct Vec;

template <>
struct Vec<float, 1> {
  __device__ static __forceinline__ void load(const float* p, float* v) { v[0] = *p; }
  __device__ static __forceinline__ void store(float* p, const float* v) { *p = v[0]; }
};

template <>
struct Vec<half_t, 1> {
  __device__ static __forceinline__ void load(const half_t* p, float* v) { v[0] = (float)*p; }
  __device__ static __forceinline__ void store(half_t* p, const float* v) { *p = (half_t)v[0]; }
};

template <>
struct Vec<float, 4> {
  __device__ static __forceinline__ void load(const float* p, float* v) {
    const float4_t t = *reinterpret_cast<const float4_t*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  }
  __device__ static __forceinline__ void store(float* p, const float* v) {
    float4_t t;
    t.x = v[0]; t.y = v[1]; t.z = v[2]; t.w = v[3];
    *reinterpret_cast<float4_t*>(p) = t;
  }
};

template <>
struct Vec<half_t, 8> {
  __device__ static __forceinline__ void load(const half_t* p, float* v) {
    const half8_t t = *reinterpret_cast<const half8_t*>(p);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (float)t[e];
  }
  __device__ static __forceinline__ void store(half_t* p, const float* v) {
    half8_t t;
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = (half_t)v[e];
    *reinterpret_cast<half8_t*>(p) = t;
  }
};

// float32 output of float16 inputs: 8 floats = two 16-byte stores.
template <>
struct Vec<float, 8> {
  __device__ static __forceinline__ void load(const float* p, float* v) {
    Vec<float, 4>::load(p, v);
    Vec<float, 4>::load(p + 4, v + 4);
  }
  __device__ static __forceinline__ void store(float* p, const float* v) {
    Vec<float, 4>::store(p, v);
    Vec<float, 4>::store(p + 4, v + 4);
  }
};

template <typename T, int VEC>
__device__ __forceinline__ void store_zero(T* p) {
  float z[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) z[e] = 0.f;
  Vec<T, VEC>::store(p, z);
}

}  // namespace bevpool
