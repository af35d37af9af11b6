// Register-resident MFMA tiles as operands (gfx950, bf16 16x16x32).
//
// An accumulator tile holds rows 4(l/16)+r, r = 0..3, of column l%16 in lane
// l.  Two such tiles stacked along the contraction (rows k0..k0+15 and
// k0+16..k0+31) give lane l the contraction indices k0+4(l/16)+r and
// k0+16+4(l/16)+r, one B operand of v_mfma_f32_16x16x32_bf16 whose 32 slots
// are summed in any order: the A operand only has to present the same index in
// the same slot, i.e. two 8-byte reads at k0+4(l/16) and k0+16+4(l/16) of a
// contraction-contiguous row (a_pair) instead of one 16-byte read.  A tile
// used this way contracts over its row index.
#pragma once

#include "tnt_device.h"

namespace tnt {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// The wave's index as a wave-uniform (scalar) value, so that everything
// derived from it stays in scalar registers.
__device__ __forceinline__ int wave_id_uniform() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE));
}

__device__ __forceinline__ bf16x4 cvt4(const f4& a) {
  bf16x4 b;
  b[0] = (__bf16)a[0]; b[1] = (__bf16)a[1]; b[2] = (__bf16)a[2]; b[3] = (__bf16)a[3];
  return b;
}

__device__ __forceinline__ bf16x8 join(const bf16x4& a, const bf16x4& b) {
  bf16x8 f;
  f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
  f[4] = b[0]; f[5] = b[1]; f[6] = b[2]; f[7] = b[3];
  return f;
}

__device__ __forceinline__ bf16x4 zero_bf4() {
  bf16x4 z;
  z[0] = z[1] = z[2] = z[3] = (__bf16)0.0f;
  return z;
}

// A operand row `row` of a contraction-contiguous array (LDS or global),
// contraction indices k0 + 4g + j and k0 + 16 + 4g + j (j = 0..3), matching a
// B operand made of two stacked accumulator tiles; `hi` = false zero-fills the
// second half (a contraction of 16).
__device__ __forceinline__ bf16x8 a_pair(const __bf16* A, int ld, int row, int k0, int g,
                                         bool hi = true) {
  // a 32-bit element offset from the (wave-uniform) base: scalar base + vector
  // offset addressing, one address register per load instead of a pair
  const __bf16* p = A + (uint32_t)(row * ld + k0 + 4 * g);
  const bf16x4 x = *reinterpret_cast<const bf16x4*>(p);
  const bf16x4 y = hi ? *reinterpret_cast<const bf16x4*>(p + 16) : zero_bf4();
  return join(x, y);
}

__device__ __forceinline__ void mma32(f4& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}

}  // namespace tnt
