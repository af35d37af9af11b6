// Small vector load / store helpers shared by the fixed-size local backward kernels.
#pragma once

#include "tnt_device.h"

namespace tnt {
namespace bwdh {

__device__ __forceinline__ float sum16b(float v) {
  v += __shfl_xor(v, 1, WAVE);
  v += __shfl_xor(v, 2, WAVE);
  v += __shfl_xor(v, 4, WAVE);
  v += __shfl_xor(v, 8, WAVE);
  return v;
}

template <typename IO>
__device__ __forceinline__ void load8(const IO* p, float (&x)[8]);
template <>
__device__ __forceinline__ void load8<__bf16>(const __bf16* p, float (&x)[8]) {
  const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int t = 0; t < 8; ++t) x[t] = (float)v[t];
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float (&x)[8]) {
  const f32x4 u = *reinterpret_cast<const f32x4*>(p), v = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    x[t] = u[t];
    x[t + 4] = v[t];
  }
}
template <typename CT>
__device__ __forceinline__ void store8(CT* p, const float (&x)[8]);
template <>
__device__ __forceinline__ void store8<__bf16>(__bf16* p, const float (&x)[8]) {
  bf16x8 v;
#pragma unroll
  for (int t = 0; t < 8; ++t) v[t] = (__bf16)x[t];
  *reinterpret_cast<bf16x8*>(p) = v;
}
template <>
__device__ __forceinline__ void store8<float>(float* p, const float (&x)[8]) {
  *reinterpret_cast<f32x4*>(p) = f32x4{x[0], x[1], x[2], x[3]};
  *reinterpret_cast<f32x4*>(p + 4) = f32x4{x[4], x[5], x[6], x[7]};
}

template <typename CT>
__device__ __forceinline__ f4 load4(const CT* p);
template <>
__device__ __forceinline__ f4 load4<float>(const float* p) {
  return *reinterpret_cast<const f32x4*>(p);
}
template <>
__device__ __forceinline__ f4 load4<__bf16>(const __bf16* p) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  return f4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}

}  // namespace bwdh
}  // namespace tnt
