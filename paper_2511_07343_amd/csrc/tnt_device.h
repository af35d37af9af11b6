// Device-side building blocks of the TNT memory-layer kernels (gfx950).
//
//  * 16x16 MFMA output tiles: bf16 operands (v_mfma_f32_16x16x32_bf16, K step
//    32, K tails of 16 zero-filled) or fp32 operands (v_mfma_f32_16x16x4f32),
//    always accumulating in fp32.  Operands are read through plain pointers
//    (LDS or global), converted to the compute type on load, optionally scaled
//    per contraction index.
//  * Lane layout (checked on gfx950): for a 16x16 output tile, lane l holds
//    rows 4*(l/16)+r, r = 0..3, of column l%16.  The bf16 A operand of lane l
//    is A[l%16][k0 + 8*(l/16) + j], j = 0..7, and B[k0 + 8*(l/16) + j][l%16];
//    the fp32 form takes A[l%16][k0 + l/16] and B[k0 + l/16][l%16].
//  * Activations (exact-erf GELU, SiLU) with first and second derivatives.
//  * Wavefront prefix scans over 64 lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tnt {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int WAVE = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
// The lane index through an opaque move: values derived from it are
// recomputed where they are used instead of being hoisted out of loops and
// kept live (per-lane operand addresses of a long kernel).
__device__ __forceinline__ int lane_id_local() {
  int l = threadIdx.x & (WAVE - 1);
  asm volatile("" : "+v"(l));
  return l;
}
// A global-memory pointer through an opaque move: addresses derived from it
// are not hoisted out of loops, and the move is made on the global address
// space, so the loads through it stay global loads (their completion counter
// can be waited on partially) instead of becoming flat loads.
template <typename T>
__device__ __forceinline__ T* launder_global(T* p) {
  typedef __attribute__((address_space(1))) T gT;
  gT* g = (gT*)p;
  asm volatile("" : "+s"(g));
  return (T*)g;
}
__device__ __forceinline__ int wave_id() { return threadIdx.x / WAVE; }
__device__ __forceinline__ int num_waves() { return blockDim.x / WAVE; }

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(__bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ __bf16 from_f<__bf16>(float x) { return (__bf16)x; }

// ----------------------------------------------------------------------------
// activation sigma and its derivatives (GELU exact erf form, or SiLU)
// ----------------------------------------------------------------------------
enum { ACT_GELU = 0, ACT_SILU = 1 };

struct ActVals { float s, d1, d2; };  // sigma(z), sigma'(z), sigma''(z)

// The logistic function from the hardware exponential and reciprocal
// (v_exp_f32, v_rcp_f32: about 1 ulp each), not the correctly rounded library
// forms: every value it feeds is rounded to bf16 or summed in fp32 next.  For
// z below about -88 the exponential overflows to +inf and the reciprocal
// gives 0, the limit.
__device__ __forceinline__ float sigmoid_fast(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

template <int ACT>
__device__ __forceinline__ float act_f(float z) {
  if (ACT == ACT_GELU) return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
  return z * sigmoid_fast(z);
}

template <int ACT>
__device__ __forceinline__ ActVals act_all(float z) {
  ActVals r;
  if (ACT == ACT_GELU) {
    float cdf = 0.5f * (1.0f + erff(z * 0.70710678118654752f));
    float pdf = 0.39894228040143268f * expf(-0.5f * z * z);
    r.s = z * cdf;
    r.d1 = cdf + z * pdf;
    r.d2 = pdf * (2.0f - z * z);
  } else {
    float sg = sigmoid_fast(z);
    r.s = z * sg;
    r.d1 = sg * (1.0f + z * (1.0f - sg));
    r.d2 = sg * (1.0f - sg) * (2.0f + z * (1.0f - 2.0f * sg));
  }
  return r;
}

// ----------------------------------------------------------------------------
// MFMA tiles
// ----------------------------------------------------------------------------
// Operand layouts.  For A (logical M x K):  KC: A[i*ld + k];  MC: A[k*ld + i].
//                   For B (logical K x N):  KC: B[j*ld + k];  MC: B[k*ld + j].
// "KC" keeps the contraction index contiguous, which is what an MFMA lane
// wants; "MC" is the transposed storage.
enum { KC = 0, MC = 1 };

template <typename CT> struct Mma;

template <> struct Mma<__bf16> {
  static constexpr int KS = 32;
  typedef bf16x8 frag;
  // 8 consecutive-k elements of row/col `idx` starting at k = kb, zero past K.
  template <int LAY, typename E>
  __device__ __forceinline__ static frag load(const E* p, int ld, int idx, int kb, int K,
                                              const float* kscale) {
    frag f;
    if (kb >= K) {
#pragma unroll
      for (int j = 0; j < 8; ++j) f[j] = (__bf16)0.0f;
      return f;
    }
    if (LAY == KC) {
      const E* q = p + (size_t)idx * ld + kb;
      if (sizeof(E) == 2) {
        // 16-byte vector load (callers keep ld and kb multiples of 8)
        f = *reinterpret_cast<const bf16x8*>(q);
        if (kscale) {
#pragma unroll
          for (int j = 0; j < 8; ++j) f[j] = (__bf16)((float)f[j] * kscale[kb + j]);
        }
      } else {
        f32x4 a = *reinterpret_cast<const f32x4*>(q);
        f32x4 b = *reinterpret_cast<const f32x4*>(q + 4);
        float t[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = (__bf16)(kscale ? t[j] * kscale[kb + j] : t[j]);
      }
    } else {
      const E* q = p + (size_t)kb * ld + idx;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float x = to_f(q[(size_t)j * ld]);
        f[j] = (__bf16)(kscale ? x * kscale[kb + j] : x);
      }
    }
    return f;
  }
  __device__ __forceinline__ static void mma(f4& acc, const frag& a, const frag& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
  }
  __device__ __forceinline__ static int kofs(int lane) { return 8 * (lane >> 4); }
};

template <> struct Mma<float> {
  static constexpr int KS = 4;
  typedef float frag;
  template <int LAY, typename E>
  __device__ __forceinline__ static frag load(const E* p, int ld, int idx, int kb, int K,
                                              const float* kscale) {
    if (kb >= K) return 0.0f;
    float x = (LAY == KC) ? to_f(p[(size_t)idx * ld + kb]) : to_f(p[(size_t)kb * ld + idx]);
    return kscale ? x * kscale[kb] : x;
  }
  __device__ __forceinline__ static void mma(f4& acc, const frag& a, const frag& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
  }
  __device__ __forceinline__ static int kofs(int lane) { return lane >> 4; }
};

// acc += A[i0:i0+16, 0:K] * B[0:K, j0:j0+16]; K a multiple of 16 (bf16) or 4 (fp32).
// kscale (optional, length K) multiplies the contraction index.
template <typename CT, int LA, int LB, typename EA, typename EB>
__device__ __forceinline__ void mma_tile(f4& acc, const EA* A, int lda, int i0, const EB* B,
                                         int ldb, int j0, int K, const float* kscale = nullptr) {
  const int l = lane_id();
  const int ko = Mma<CT>::kofs(l);
  const int ia = i0 + (l & 15), jb = j0 + (l & 15);
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += Mma<CT>::KS) {
    auto a = Mma<CT>::template load<LA>(A, lda, ia, k0 + ko, K, kscale);
    auto b = Mma<CT>::template load<LB>(B, ldb, jb, k0 + ko, K, nullptr);
    Mma<CT>::mma(acc, a, b);
  }
}

__device__ __forceinline__ f4 zero4() { return f4{0.f, 0.f, 0.f, 0.f}; }

// A fragment loaded raw from a contraction-contiguous (KC) source and
// converted to the MFMA operand type later, so that many loads can be in
// flight before the first conversion waits for its data.
template <typename CT, typename E> struct RawFrag;
template <> struct RawFrag<__bf16, float> {
  f32x4 a, b;
  __device__ __forceinline__ void load(const float* p, int ld, int idx, int kb) {
    const float* q = p + (size_t)idx * ld + kb;
    a = *reinterpret_cast<const f32x4*>(q);
    b = *reinterpret_cast<const f32x4*>(q + 4);
  }
  __device__ __forceinline__ bf16x8 get() const {
    bf16x8 f;
    f[0] = (__bf16)a[0]; f[1] = (__bf16)a[1]; f[2] = (__bf16)a[2]; f[3] = (__bf16)a[3];
    f[4] = (__bf16)b[0]; f[5] = (__bf16)b[1]; f[6] = (__bf16)b[2]; f[7] = (__bf16)b[3];
    return f;
  }
};
template <> struct RawFrag<__bf16, __bf16> {
  bf16x8 v;
  __device__ __forceinline__ void load(const __bf16* p, int ld, int idx, int kb) {
    v = *reinterpret_cast<const bf16x8*>(p + (size_t)idx * ld + kb);
  }
  __device__ __forceinline__ bf16x8 get() const { return v; }
};
template <> struct RawFrag<float, float> {
  float v;
  __device__ __forceinline__ void load(const float* p, int ld, int idx, int kb) {
    v = p[(size_t)idx * ld + kb];
  }
  __device__ __forceinline__ float get() const { return v; }
};

// visit the 4 elements a lane holds of the 16x16 tile at (i0, j0)
template <typename F>
__device__ __forceinline__ void tile_each(const f4& acc, int i0, int j0, F&& f) {
  const int l = lane_id();
  const int col = j0 + (l & 15);
  const int row = i0 + 4 * (l >> 4);
#pragma unroll
  for (int r = 0; r < 4; ++r) f(row + r, col, acc[r]);
}

// Block-wide GEMM over 16x16 output tiles distributed round-robin to waves:
// out(i, j) = sum_k A(i, k) B(k, j), passed to epi(i, j, value).
template <typename CT, int LA, int LB, typename EA, typename EB, typename Epi>
__device__ __forceinline__ void gemm(int M, int N, int K, const EA* A, int lda, const EB* B,
                                     int ldb, Epi&& epi, const float* kscale = nullptr) {
  const int tn = N >> 4, nt = (M >> 4) * tn;
  for (int t = wave_id(); t < nt; t += num_waves()) {
    const int i0 = (t / tn) << 4, j0 = (t % tn) << 4;
    f4 acc = zero4();
    mma_tile<CT, LA, LB>(acc, A, lda, i0, B, ldb, j0, K, kscale);
    tile_each(acc, i0, j0, epi);
  }
}

// ----------------------------------------------------------------------------
// Register-blocked wave tiles.  An M x N output (multiples of 16, sizes known
// at compile time) is cut into blocks of RB x CB 16x16 tiles: T/8 tiles per
// block (1..8), shaped to need the fewest operand fragments.  Blocks go to the
// waves round-robin.  A wave issues every fragment load of a K step of its
// block before the MFMAs, so a block costs one memory round trip per K step
// rather than one per tile.
// ----------------------------------------------------------------------------
template <int M, int N, int NWAVE = 8> struct Blk {
  static constexpr int TM = M / 16, TN = N / 16, T = TM * TN;
  static constexpr int TPW = T / NWAVE < 1 ? 1 : (T / NWAVE > 8 ? 8 : T / NWAVE);
  static constexpr int pick_rb() {
    int best = 0, cost = 1 << 20;
    for (int rb = 1; rb <= 8; rb <<= 1) {
      const int cb = TPW / rb;
      if (cb < 1 || rb * cb != TPW || rb > TM || cb > TN || TM % rb || TN % cb) continue;
      if (rb + cb <= cost) {  // ties go to the taller block
        cost = rb + cb;
        best = rb;
      }
    }
    return best;
  }
  static constexpr int RB = pick_rb(), CB = RB ? TPW / RB : 0;
  static constexpr int NBM = RB ? TM / RB : 0, NBN = CB ? TN / CB : 0, NB = NBM * NBN;
  static_assert(RB > 0 && CB > 0 && M % 16 == 0 && N % 16 == 0, "unsupported block shape");
};

// visit the wave's blocks of an M x N output: f(i0, j0) at each block corner
template <int M, int N, typename F>
__device__ __forceinline__ void for_blocks(F&& f) {
  using BK = Blk<M, N>;
  for (int b = wave_id(); b < BK::NB; b += num_waves())
    f((b / BK::NBN) * BK::RB * 16, (b % BK::NBN) * BK::CB * 16);
}
// the same over the blocks of Blk<M, N, NWB> (NWB > 8: smaller blocks, several
// per wave, fewer accumulators live at a time)
template <int M, int N, int NWB, typename F>
__device__ __forceinline__ void for_blocks_n(F&& f) {
  using BK = Blk<M, N, NWB>;
  for (int b = wave_id(); b < BK::NB; b += num_waves())
    f((b / BK::NBN) * BK::RB * 16, (b % BK::NBN) * BK::CB * 16);
}

template <int RB, int CB>
__device__ __forceinline__ void zero_blk(f4 (&a)[RB][CB]) {
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < CB; ++c) a[r][c] = zero4();
}

// acc[r][c] += A[i0+16r .., 0:K] B[0:K, j0+16c ..] (K a compile-time constant).
// The K loop stays rolled and double-buffered: the fragments of step k+1 are
// requested before the MFMAs of step k, so one term costs about one memory
// round trip and the live operand registers stay at two steps' worth.
template <typename CT, int LA, int LB, int RB, int CB, int K, typename EA, typename EB>
__device__ __forceinline__ void mma_blk(f4 (&acc)[RB][CB], const EA* A, int lda, int i0,
                                        const EB* B, int ldb, int j0,
                                        const float* kscale = nullptr) {
  typedef Mma<CT> MM;
  const int l = lane_id_local();
  const int ko = MM::kofs(l);
  typename MM::frag fa[RB], fb[CB];
  auto fetch = [&](int k0, typename MM::frag(&xa)[RB], typename MM::frag(&xb)[CB]) {
#pragma unroll
    for (int r = 0; r < RB; ++r)
      xa[r] = MM::template load<LA>(A, lda, i0 + 16 * r + (l & 15), k0 + ko, K, kscale);
#pragma unroll
    for (int c = 0; c < CB; ++c)
      xb[c] = MM::template load<LB>(B, ldb, j0 + 16 * c + (l & 15), k0 + ko, K, nullptr);
  };
  auto apply = [&](const typename MM::frag(&xa)[RB], const typename MM::frag(&xb)[CB]) {
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int c = 0; c < CB; ++c) MM::mma(acc[r][c], xa[r], xb[c]);
  };
  constexpr int NS = (K + MM::KS - 1) / MM::KS;
  constexpr int FRAG_REGS = sizeof(typename MM::frag) / 4;
  constexpr int REGS_A = RB * (sizeof(EA) > sizeof(CT) ? 2 : 1) * FRAG_REGS;
  constexpr int REGS_B = CB * (sizeof(EB) > sizeof(CT) ? 2 : 1) * FRAG_REGS;
  if constexpr (NS > 2 && NS * (REGS_A + REGS_B) <= 128) {
    // small block, long K: every step's loads in flight at once
    typename MM::frag ga[NS][RB], gb[NS][CB];
#pragma unroll
    for (int t = 0; t < NS; ++t) fetch(t * MM::KS, ga[t], gb[t]);
#pragma unroll
    for (int t = 0; t < NS; ++t) apply(ga[t], gb[t]);
    return;
  }
  fetch(0, fa, fb);
#pragma unroll 1
  for (int k0 = MM::KS; k0 < K; k0 += MM::KS) {
    typename MM::frag na[RB], nb[CB];
    fetch(k0, na, nb);
    apply(fa, fb);
#pragma unroll
    for (int r = 0; r < RB; ++r) fa[r] = na[r];
#pragma unroll
    for (int c = 0; c < CB; ++c) fb[c] = nb[c];
  }
  apply(fa, fb);
}

// Two block GEMMs sharing one operand, every K step's fragments in flight before
// the MFMAs (short contractions): x += A B0, y += A B1 (SHARE_A) or
// x += A0 B, y += A1 B (shared B); all operands contraction-contiguous.
template <typename CT, int RB, int CB, int K, bool SHARE_A, typename EA, typename EB>
__device__ __forceinline__ void mma_blk_shared(f4 (&x)[RB][CB], f4 (&y)[RB][CB], const EA* A0,
                                               const EA* A1, int lda, int i0, const EB* B0,
                                               const EB* B1, int ldb, int j0) {
  typedef Mma<CT> MM;
  const int l = lane_id_local();
  const int ko = MM::kofs(l);
  constexpr int NS = (K + MM::KS - 1) / MM::KS;
  static_assert(NS <= 4, "short contractions only: all steps stay in registers");
  typename MM::frag fa[NS][RB], fa1[NS][SHARE_A ? 1 : RB], fb[NS][CB], fb1[NS][SHARE_A ? CB : 1];
#pragma unroll
  for (int t = 0; t < NS; ++t) {
    const int k0 = t * MM::KS + ko;
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      fa[t][r] = MM::template load<KC>(A0, lda, i0 + 16 * r + (l & 15), k0, K, nullptr);
      if constexpr (!SHARE_A) fa1[t][r] = MM::template load<KC>(A1, lda, i0 + 16 * r + (l & 15), k0, K, nullptr);
    }
#pragma unroll
    for (int c = 0; c < CB; ++c) {
      fb[t][c] = MM::template load<KC>(B0, ldb, j0 + 16 * c + (l & 15), k0, K, nullptr);
      if constexpr (SHARE_A) fb1[t][c] = MM::template load<KC>(B1, ldb, j0 + 16 * c + (l & 15), k0, K, nullptr);
    }
  }
#pragma unroll
  for (int t = 0; t < NS; ++t)
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        MM::mma(x[r][c], fa[t][r], fb[t][c]);
        if constexpr (SHARE_A)
          MM::mma(y[r][c], fa[t][r], fb1[t][c]);
        else
          MM::mma(y[r][c], fa1[t][r], fb[t][c]);
      }
}

// f(rb, cb, i, j) once per tile of the block: the lane's rows i .. i+3 of
// column j are acc[rb][cb][0..3]
template <int RB, int CB, typename F>
__device__ __forceinline__ void blk_each4(int i0, int j0, F&& f) {
  const int l = lane_id_local();
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) f(rb, cb, i0 + 16 * rb + 4 * (l >> 4), j0 + 16 * cb + (l & 15));
}

// Block GEMM over the whole output with a per-element epilogue epi(i, j, v).
template <typename CT, int LA, int LB, int M, int N, int K, typename EA, typename EB, typename Epi>
__device__ __forceinline__ void gemm_blk(const EA* A, int lda, const EB* B, int ldb, Epi&& epi,
                                         const float* kscale = nullptr) {
  using BK = Blk<M, N>;
  for_blocks<M, N>([&](int i0, int j0) {
    f4 acc[BK::RB][BK::CB];
    zero_blk(acc);
    mma_blk<CT, LA, LB, BK::RB, BK::CB, K>(acc, A, lda, i0, B, ldb, j0, kscale);
    blk_each4<BK::RB, BK::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) epi(i + r, j, acc[rb][cb][r]);
    });
  });
}

// a lane's value from another lane of its quad (DPP quad_perm pattern CTRL)
template <int CTRL>
__device__ __forceinline__ float quad_perm(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// 4 x 4 transpose within each quad of lanes: before, lane q (= lane & 3) holds
// column q of the quad's block (rows 0..3 in v[0..3]); after, it holds row q
// (columns 0..3).  Two exchanges, with lane q ^ 1 (rows of the lane's parity kept)
// and with lane q ^ 2.
__device__ __forceinline__ f4 quad_transpose(const f4& v) {
  const int q = lane_id() & 3;
  const bool odd = q & 1, hi = q & 2;
  const float x = quad_perm<0xB1>(odd ? v[0] : v[1]);  // from lane q ^ 1
  const float y = quad_perm<0xB1>(odd ? v[2] : v[3]);
  f4 b;
  b[0] = odd ? x : v[0];
  b[1] = odd ? v[1] : x;
  b[2] = odd ? y : v[2];
  b[3] = odd ? v[3] : y;
  const float z = quad_perm<0x4E>(hi ? b[0] : b[2]);  // from lane q ^ 2
  const float w = quad_perm<0x4E>(hi ? b[1] : b[3]);
  f4 u;
  u[0] = hi ? z : b[0];
  u[1] = hi ? w : b[1];
  u[2] = hi ? b[2] : z;
  u[3] = hi ? b[3] : w;
  return u;
}

// four consecutive compute-type elements from one f4 (8- or 16-byte store)
template <typename CT> __device__ __forceinline__ void store4(CT* p, const f4& v);
template <> __device__ __forceinline__ void store4<float>(float* p, const f4& v) {
  *reinterpret_cast<f32x4*>(p) = v;
}
template <> __device__ __forceinline__ void store4<__bf16>(__bf16* p, const f4& v) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 b;
  b[0] = (__bf16)v[0]; b[1] = (__bf16)v[1]; b[2] = (__bf16)v[2]; b[3] = (__bf16)v[3];
  *reinterpret_cast<bf16x4*>(p) = b;
}

// ----------------------------------------------------------------------------
// wavefront scans (64 lanes)
// ----------------------------------------------------------------------------
__device__ __forceinline__ float wave_incl_sum(float x) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    float y = __shfl_up(x, o, WAVE);
    if (l >= o) x += y;
  }
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, WAVE);
  return x;
}

// Block-wide sum; `red` is LDS scratch of at least num_waves() floats.
__device__ __forceinline__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  __syncthreads();
  if (lane_id() == 0) red[wave_id()] = x;
  __syncthreads();
  float t = 0.f;
  for (int w = 0; w < num_waves(); ++w) t += red[w];
  __syncthreads();
  return t;
}

constexpr float LOG_CLAMP = -80.0f;
__device__ __forceinline__ float log_mom(float beta) { return fmaxf(logf(beta), LOG_CLAMP); }
__device__ __forceinline__ float log_keep(float alpha) { return log1pf(-alpha); }

}  // namespace tnt
