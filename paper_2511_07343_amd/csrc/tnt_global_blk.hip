// Global memory, fixed sizes: the chunk phases of the runtime-sized global
// kernels (same quantities and formulas, written out there), restructured
// around register-blocked wave tiles and contraction-contiguous operands:
//
//  forward chunk n   transpose  V1^T, V2^T of the chunk-entry state (bf16)
//                    tile       token tiles: O_G, R, Hk, D1 with every
//                               intermediate in LDS; writes the carry operands
//                               D1^T, Hk^T (hid x C) and (cC K)^T, (b K)^T,
//                               (cC R)^T, (b R)^T (d x C) in bf16
//                    carry      split-K GEMMs over the chunk's tokens into the
//                               split partials that global_carry_reduce sums
//  backward chunk n  transpose  V1^T, V2^T and the exit adjoint's four
//                               transposes
//                    tile       token tiles: the per-token adjoints (d q, d k,
//                               d v, coefficient adjoints) with intermediates in
//                               LDS; writes the operands of the entry adjoint
//                               Zkbar^T, Zqbar^T, Gbar^T, Hk^T, Hq^T (hid x C)
//                               and K^T, Q^T, R^T, Ykbar^T, dO^T (d x C)
//                    state      split-K GEMMs into the partials that
//                               gbwd_state_reduce sums
#include "tnt_device.h"
#include "tnt_kernels.h"

#include <algorithm>

namespace tnt {

namespace {

// tokens per split of the carry / state GEMMs: GTK_LONG where the chunk length
// allows (fewer fp32 partials written and read back)
constexpr int GTK = 256, GTK_LONG = 1024;
// K slab of the LDS-staged carry GEMMs (tokens per round trip)
constexpr int GCARRY_KT = 128;
inline int gtk_of(int C) { return C % GTK_LONG == 0 ? GTK_LONG : GTK; }

template <int H>
constexpr int gtile_rows() {
  return H <= 256 ? 64 : 32;
}

template <typename IO>
__device__ __forceinline__ void gload8(const IO* p, float (&x)[8]);
template <>
__device__ __forceinline__ void gload8<__bf16>(const __bf16* p, float (&x)[8]) {
  const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int t = 0; t < 8; ++t) x[t] = (float)v[t];
}
template <>
__device__ __forceinline__ void gload8<float>(const float* p, float (&x)[8]) {
  const f32x4 u = *reinterpret_cast<const f32x4*>(p), v = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    x[t] = u[t];
    x[t + 4] = v[t];
  }
}
template <typename CT>
__device__ __forceinline__ void gstore8(CT* p, const float (&x)[8]);
template <>
__device__ __forceinline__ void gstore8<__bf16>(__bf16* p, const float (&x)[8]) {
  bf16x8 v;
#pragma unroll
  for (int t = 0; t < 8; ++t) v[t] = (__bf16)x[t];
  *reinterpret_cast<bf16x8*>(p) = v;
}

__device__ __forceinline__ float gsum16(float v) {
  v += __shfl_xor(v, 1, WAVE);
  v += __shfl_xor(v, 2, WAVE);
  v += __shfl_xor(v, 4, WAVE);
  v += __shfl_xor(v, 8, WAVE);
  return v;
}

}  // namespace

// ---------------------------------------------------------------------------
// bf16 copies of a chain's four state matrices: transposed into dst (W1 (hid x
// d) -> [d][hid], W2 (d x hid) -> [hid][d], S1, S2 alike, chain stride
// dst_stride) and as they are into dstn (chain stride dstn_stride); `mask` bit
// m selects matrix m.  One 32 x 32 tile per workgroup.
// ---------------------------------------------------------------------------
template <typename CT>
__global__ void __launch_bounds__(256) gtranspose_kernel(const float* src, size_t src_stride,
                                                         CT* dst, size_t dst_stride, CT* dstn,
                                                         size_t dstn_stride, int d, int h,
                                                         int mask) {
  __shared__ float t[32][33];
  const int m = blockIdx.z;
  if (!((mask >> m) & 1)) return;
  const int chain = blockIdx.y;
  const size_t hd = (size_t)h * d;
  const int R = (m & 1) ? d : h, Cc = (m & 1) ? h : d;
  const int tc = Cc / 32;
  const int r0 = (blockIdx.x / tc) * 32, c0 = (blockIdx.x % tc) * 32;
  const float* s = src + chain * src_stride + m * hd;
  CT* o = dst + (size_t)chain * dst_stride + m * hd;
  CT* on = dstn + (size_t)chain * dstn_stride + m * hd;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8) {
    const size_t e = (size_t)(r0 + k) * Cc + c0 + tx;
    const float x = s[e];
    t[k][tx] = x;
    on[e] = from_f<CT>(x);
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) o[(size_t)(c0 + k) * R + r0 + tx] = from_f<CT>(t[tx][k]);
}

// The carry's reduction fused with the next chunk's state copies: per 32 x 32
// tile of the pair (W_m, S_m) (m = 0: W1, S1 [hid][d]; m = 1: W2, S2 [d][hid]),
//   W' = A_C W + E_C S - sum_splits dW,  S' = B_C S - sum_splits dS
// (fixed split order, four consecutive elements a thread as the unfused
// reduction forms them) into fp32 slot n + 1, and W' in bf16 transposed into
// packT (W1^T, W2^T) and as it is (W1, W2 after 2 hd), the layout the next
// chunk's tile reads.
template <typename CT>
__global__ void __launch_bounds__(256) gcarry_reduce_pack_kernel(GlobalArgs a, int n, int nsplit) {
  __shared__ float t[32][33];
  const Dims D = a.D;
  const int m = blockIdx.z, chain = blockIdx.y;
  const int d = D.d, h = D.hid;
  const size_t hd = (size_t)h * d;
  const int R = m ? d : h, Cc = m ? h : d;  // rows and columns of W_m
  const int tc = Cc / 32;
  const int r0 = (blockIdx.x / tc) * 32, c0 = (blockIdx.x % tc) * 32;
  const float* V = a.states + ((size_t)chain * a.nslots + (n % a.nslots)) * 4 * hd;
  float* Vn = a.states + ((size_t)chain * a.nslots + ((n + 1) % a.nslots)) * 4 * hd;
  const float* P = a.part + (size_t)chain * nsplit * 4 * hd;
  const float* cc = a.chunkc + ((size_t)chain * (D.L / D.C) + n) * 4;
  const float AC = cc[0], BC = cc[1], EC = cc[2];
  CT* pk = (CT*)a.packT + (size_t)chain * 4 * hd;
  {
    const int k = threadIdx.x >> 3, c4 = (threadIdx.x & 7) * 4;
    const size_t e = (size_t)(r0 + k) * Cc + c0 + c4;
    const size_t ew = (size_t)m * hd + e, es = (size_t)(2 + m) * hd + e;
    f32x4 dw = {0.f, 0.f, 0.f, 0.f}, ds = dw;
    for (int sp = 0; sp < nsplit; ++sp) {
      dw += *reinterpret_cast<const f32x4*>(P + (size_t)sp * 4 * hd + ew);
      ds += *reinterpret_cast<const f32x4*>(P + (size_t)sp * 4 * hd + es);
    }
    const f32x4 w = *reinterpret_cast<const f32x4*>(V + ew);
    const f32x4 sv = *reinterpret_cast<const f32x4*>(V + es);
    const f32x4 nw = AC * w + EC * sv - dw;
    *reinterpret_cast<f32x4*>(Vn + ew) = nw;
    *reinterpret_cast<f32x4*>(Vn + es) = BC * sv - ds;
    store4<CT>(pk + 2 * hd + ew, nw);
#pragma unroll
    for (int q = 0; q < 4; ++q) t[k][c4 + q] = nw[q];
  }
  __syncthreads();
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  CT* o = pk + (size_t)m * hd;
  for (int k = ty; k < 32; k += 8) o[(size_t)(c0 + k) * R + r0 + tx] = from_f<CT>(t[tx][k]);
}

template <typename CT>
static void launch_gtranspose(const float* src, size_t src_stride, CT* dst, size_t dst_stride,
                              CT* dstn, size_t dstn_stride, int chains, int d, int h, int mask,
                              hipStream_t st) {
  const dim3 grid((h / 32) * (d / 32), chains, 4);
  hipLaunchKernelGGL(gtranspose_kernel<CT>, grid, dim3(256), 0, st, src, src_stride, dst,
                     dst_stride, dstn, dstn_stride, d, h, mask);
}

// ---------------------------------------------------------------------------
// forward, token tiles of TT rows of chunk n.  KS = false: the retrieval alone
// (Zq -> Hq -> O), for a chunk whose carry nobody reads
// ---------------------------------------------------------------------------
template <int D, int H, bool KS>
constexpr size_t gfwd_tile_lds() {  // padded rows, compute type (2 bytes)
  return (KS ? 2 * (size_t)gtile_rows<H>() * (D + 8) + 3 * (size_t)gtile_rows<H>() * (H + 8)
             : (size_t)gtile_rows<H>() * (D + 8) + (size_t)gtile_rows<H>() * (H + 8)) * 2;
}

template <typename IO, typename CT, int ACT, int D, int H, bool KS>
__global__ void __launch_bounds__(512) gfwd_tile_kernel(GlobalArgs a, int n) {
  constexpr int TT = gtile_rows<H>();
  // rows padded by 16 bytes: the 16-byte operand reads of consecutive rows do
  // not start on the same LDS banks
  constexpr int LD = D + 8, LH = H + 8;
  extern __shared__ __align__(16) unsigned char smem[];
  CT* sQ = reinterpret_cast<CT*>(smem);  // [TT][LD], later R
  CT* sK = sQ + TT * LD;                 // [TT][LD]   (KS only)
  CT* sHq = KS ? sK + TT * LD : sK;      // [TT][LH]
  CT* sHk = sHq + TT * LH;               // [TT][LH]   (KS only)
  CT* sSp = sHk + TT * LH;               // [TT][LH]  s'(Zk)   (KS only)
  __shared__ float cC[TT], bb[TT];
  const Dims Dm = a.D;
  const int C = Dm.C;
  const int chain = blockIdx.y, r0 = blockIdx.x * TT;
  constexpr size_t hd = (size_t)H * D;
  // the chunk-entry state in bf16: V1^T [D][H], V2^T [H][D], V1 [H][D], V2 [D][H]
  const CT* pS = (const CT*)a.packT + (size_t)chain * 4 * hd;
  const CT *V2T = pS + hd, *V1 = pS + 2 * hd, *V2 = pS + 3 * hd;
  CT* op = (CT*)a.opT + (size_t)chain * (2 * (size_t)H + 4 * (size_t)D) * C;
  CT *D1T = op, *HkT = D1T + (size_t)H * C, *KcT = HkT + (size_t)H * C, *KbT = KcT + (size_t)D * C,
     *RcT = KbT + (size_t)D * C, *RbT = RcT + (size_t)D * C;
  const size_t tok0 = (size_t)n * C + r0;
  const size_t cb = (size_t)chain * Dm.L + tok0;
  const IO* q = (const IO*)a.q + cb * D;
  const IO* k = (const IO*)a.k + cb * D;
  const IO* v = (const IO*)a.v + cb * D;
  float* o = a.o_part + cb * D;
  const float* tk = a.tokc + cb * TKS;
  const float rscale = 2.0f / (float)D;

  if (threadIdx.x < TT) {
    cC[threadIdx.x] = tk[(size_t)threadIdx.x * TKS + 0];
    bb[threadIdx.x] = tk[(size_t)threadIdx.x * TKS + 1];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < TT * (D / 8); e += blockDim.x) {
    const int i = e % TT, j0 = (e / TT) * 8;
    float qx[8];
    gload8(q + (size_t)i * D + j0, qx);
    gstore8<CT>(sQ + (size_t)i * LD + j0, qx);
    if constexpr (KS) {
      float kx[8];
      gload8(k + (size_t)i * D + j0, kx);
      gstore8<CT>(sK + (size_t)i * LD + j0, kx);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const size_t et = (size_t)(j0 + t) * C + r0 + i;
        KcT[et] = from_f<CT>(cC[i] * kx[t]);
        KbT[et] = from_f<CT>(bb[i] * kx[t]);
      }
    }
  }
  __syncthreads();
  using BH = Blk<TT, H>;
  using BD = Blk<TT, D>;
  // Zq = Q V1^T -> Hq ; Zk = K V1^T -> Hk, s'(Zk)
  for_blocks<TT, H>([&](int i0, int j0) {
    f4 aq[BH::RB][BH::CB], ak[BH::RB][BH::CB];
    zero_blk(aq);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(aq, sQ, LD, i0, V1, D, j0);
    if constexpr (KS) {
      zero_blk(ak);
      mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ak, sK, LD, i0, V1, D, j0);
    }
    blk_each4<BH::RB, BH::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 hv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t e = (size_t)(i + r) * LH + j;
        sHq[e] = from_f<CT>(act_f<ACT>(aq[rb][cb_][r]));
        if constexpr (KS) {
          const ActVals z = act_all<ACT>(ak[rb][cb_][r]);
          sHk[e] = from_f<CT>(z.s);
          sSp[e] = from_f<CT>(z.d1);
          hv[r] = z.s;
        }
      }
      if constexpr (KS) store4<CT>(HkT + (size_t)j * C + r0 + i, hv);
    });
  });
  __syncthreads();
  // O_G = Hq V2^T ; R = (2/d)(Hk V2^T - V)
  CT* sR = sQ;
  for_blocks<TT, D>([&](int i0, int j0) {
    f4 ao[BD::RB][BD::CB], ay[BD::RB][BD::CB];
    zero_blk(ao);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(ao, sHq, LH, i0, V2, H, j0);
    if constexpr (KS) {
      zero_blk(ay);
      mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(ay, sHk, LH, i0, V2, H, j0);
    }
    blk_each4<BD::RB, BD::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 rc, rbv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ii = i + r;
        const size_t e = (size_t)ii * D + j;
        if (KS || !a.o_final) {
          o[e] = ao[rb][cb_][r];
        } else {  // the layer output: every memory's part in the fixed order
          float sv = ao[rb][cb_][r];
          for (int p = 1; p < a.o_nparts; ++p) sv += o[p * a.o_stride + e];
          reinterpret_cast<IO*>(a.o_final)[cb * D + e] = from_f<IO>(sv);
        }
        if constexpr (KS) {
          const float rv = rscale * (ay[rb][cb_][r] - to_f(v[e]));
          sR[(size_t)ii * LD + j] = from_f<CT>(rv);
          rc[r] = cC[ii] * rv;
          rbv[r] = bb[ii] * rv;
        }
      }
      if constexpr (KS) {
        store4<CT>(RcT + (size_t)j * C + r0 + i, rc);
        store4<CT>(RbT + (size_t)j * C + r0 + i, rbv);
      }
    });
  });
  if constexpr (!KS) return;
  __syncthreads();
  // G = R V2, D1 = G * s'(Zk)
  for_blocks<TT, H>([&](int i0, int j0) {
    f4 ag[BH::RB][BH::CB];
    zero_blk(ag);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ag, sR, LD, i0, V2T, D, j0);
    blk_each4<BH::RB, BH::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 dv;
#pragma unroll
      for (int r = 0; r < 4; ++r) dv[r] = ag[rb][cb_][r] * to_f(sSp[(size_t)(i + r) * LH + j]);
      store4<CT>(D1T + (size_t)j * C + r0 + i, dv);
    });
  });
}

// ---------------------------------------------------------------------------
// acc (the wave's block of an MB x NB output) += sum over the NT terms of
// A_t B_t^T, A_t: MB rows, B_t: NB rows, both K long and contraction-contiguous
// (row stride ld), compute type.  The K range goes through LDS in slabs of KT:
// every thread requests its 16-byte share of the next slab before the MFMAs of
// the current one, so a slab costs one memory round trip for the whole
// workgroup instead of one per K step and wave, and each operand row is read
// from memory once, not once per wave that uses it.  The K order of the
// accumulation is that of the plain block product.  `lds`: (MB + NB) (KT + 8)
// compute-type elements (rows padded by 16 bytes).
// ---------------------------------------------------------------------------
template <typename CT, int MB, int NB, int KT, int NT>
constexpr size_t lds_gemm_bytes() {
  return (size_t)(MB + NB) * (KT + 8) * sizeof(CT);
}

template <typename CT, int MB, int NB, int KT, int NT, int RB, int CB>
__device__ __forceinline__ void lds_gemm_nt(f4 (&acc)[RB][CB], int i0, int j0,
                                            const CT* const (&A)[NT], const CT* const (&B)[NT],
                                            int ld, int K, CT* lds) {
  static_assert(sizeof(CT) == 2 && KT % 32 == 0, "bf16 slabs of whole K steps");
  typedef Mma<CT> MM;
  constexpr int LK = KT + 8, CPR = KT / 8, ITEMS = (MB + NB) * CPR;
  constexpr int PER = (ITEMS + 511) / 512;
  CT* const sA = lds;
  CT* const sB = lds + MB * LK;
  const int spt = K / KT, S = NT * spt;
  bf16x8 pre[PER];
  auto gload = [&](int st) {
    const int t = st / spt, kk = (st - t * spt) * KT;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = threadIdx.x + p * 512;
      if (e < ITEMS) {
        const int row = e / CPR, c = e - row * CPR;
        const CT* src = row < MB ? A[t] + (size_t)row * ld : B[t] + (size_t)(row - MB) * ld;
        pre[p] = *reinterpret_cast<const bf16x8*>(src + kk + 8 * c);
      }
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = threadIdx.x + p * 512;
      if (e < ITEMS) {
        const int row = e / CPR, c = e - row * CPR;
        *reinterpret_cast<bf16x8*>(lds + (size_t)row * LK + 8 * c) = pre[p];
      }
    }
  };
  const int l = lane_id_local();
  const int ko = MM::kofs(l);
  gload(0);
  lstore();
  __syncthreads();
#pragma unroll 1
  for (int st = 0; st < S; ++st) {
    if (st + 1 < S) gload(st + 1);
#pragma unroll
    for (int kk = 0; kk < KT; kk += MM::KS) {
      typename MM::frag fa[RB], fb[CB];
#pragma unroll
      for (int r = 0; r < RB; ++r)
        fa[r] = *reinterpret_cast<const bf16x8*>(sA + (size_t)(i0 + 16 * r + (l & 15)) * LK + kk + ko);
#pragma unroll
      for (int c = 0; c < CB; ++c)
        fb[c] = *reinterpret_cast<const bf16x8*>(sB + (size_t)(j0 + 16 * c + (l & 15)) * LK + kk + ko);
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int c = 0; c < CB; ++c) MM::mma(acc[r][c], fa[r], fb[c]);
    }
    if (st + 1 < S) {
      __syncthreads();  // every wave is done with this slab
      lstore();
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// forward carry partials of token split `blockIdx.x`:
//   m = 0: D1^T (cC K) -> V1 slot,  m = 1: D1^T (b K) -> S1 slot   (hid x d)
//   m = 2: (cC R)^T Hk -> V2 slot,  m = 3: (b R)^T Hk -> S2 slot   (d x hid)
// ---------------------------------------------------------------------------
template <typename CT, int D, int H, int TK>
__global__ void __launch_bounds__(512) gfwd_carry_kernel(GlobalArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int split = blockIdx.x, m = blockIdx.y, chain = blockIdx.z, ns = gridDim.x;
  const int C = a.D.C;
  constexpr size_t hd = (size_t)H * D;
  const CT* op = (const CT*)a.opT + (size_t)chain * (2 * (size_t)H + 4 * (size_t)D) * C;
  const CT *D1T = op, *HkT = D1T + (size_t)H * C, *KcT = HkT + (size_t)H * C,
           *KbT = KcT + (size_t)D * C, *RcT = KbT + (size_t)D * C, *RbT = RcT + (size_t)D * C;
  const size_t k0 = (size_t)split * TK;
  float* P = a.part + ((size_t)chain * ns + split) * 4 * hd;
  CT* lds = reinterpret_cast<CT*>(smem);
  if (m < 2) {
    using BK = Blk<H, D>;
    static_assert(BK::NB == 8, "one block per wave");
    const CT* const As[1] = {D1T + k0};
    const CT* const Bs[1] = {(m == 0 ? KcT : KbT) + k0};
    float* out = P + (m == 0 ? 0 : 2 * hd);
    const int i0 = (wave_id() / BK::NBN) * BK::RB * 16, j0 = (wave_id() % BK::NBN) * BK::CB * 16;
    f4 acc[BK::RB][BK::CB];
    zero_blk(acc);
    lds_gemm_nt<CT, H, D, GCARRY_KT, 1>(acc, i0, j0, As, Bs, C, TK, lds);
    blk_each4<BK::RB, BK::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) out[(size_t)(i + r) * D + j] = acc[rb][cb_][r];
    });
  } else {
    using BK = Blk<D, H>;
    static_assert(BK::NB == 8, "one block per wave");
    const CT* const As[1] = {(m == 2 ? RcT : RbT) + k0};
    const CT* const Bs[1] = {HkT + k0};
    float* out = P + (m == 2 ? hd : 3 * hd);
    const int i0 = (wave_id() / BK::NBN) * BK::RB * 16, j0 = (wave_id() % BK::NBN) * BK::CB * 16;
    f4 acc[BK::RB][BK::CB];
    zero_blk(acc);
    lds_gemm_nt<CT, D, H, GCARRY_KT, 1>(acc, i0, j0, As, Bs, C, TK, lds);
    blk_each4<BK::RB, BK::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) out[(size_t)(i + r) * H + j] = acc[rb][cb_][r];
    });
  }
}

// ---------------------------------------------------------------------------
// backward, token tiles of TT rows of chunk n (exit adjoint in slot (n+1)&1)
// ---------------------------------------------------------------------------
template <typename IO, typename CT, int ACT, int D, int H>
__global__ void __launch_bounds__(512) gbwd_tile_kernel(GlobalArgs a, int n) {
  constexpr int TT = gtile_rows<H>();
  constexpr int TN = D / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  CT* rA = reinterpret_cast<CT*>(smem);  // [TT][D] K
  CT* rB = rA + TT * D;                  // [TT][D] Q, then R
  CT* rC = rB + TT * D;                  // [TT][D] dO, then Ykbar
  CT* rD = rC + TT * D;                  // [TT][H] Zk
  CT* rE = rD + TT * H;                  // [TT][H] Hk, then D1, then Zkbar
  CT* rF = rE + TT * H;                  // [TT][H] Zqbar, then Gbar
  CT* rG = rF + TT * H;                  // [TT][H] D1bar G s''(Zk)
  CT *sK = rA, *sQ = rB, *sR = rB, *sdO = rC, *sYkb = rC, *sZk = rD, *sHk = rE, *sD1 = rE,
     *sZkb = rE, *sZqb = rF, *sGb = rF, *sZkp = rG;
  __shared__ float cC[TT], bb[TT];
  __shared__ float gp[2][TN][TT];
  const Dims Dm = a.D;
  const int C = Dm.C;
  const int chain = blockIdx.y, r0 = blockIdx.x * TT;
  constexpr size_t hd = (size_t)H * D;
  // bf16 copies of the chunk-entry state and the exit adjoint, transposed and as they are
  const CT* pS = (const CT*)a.packT + (size_t)chain * 4 * hd;
  const CT *V1T = pS, *V2T = pS + hd, *V1 = pS + 2 * hd, *V2 = pS + 3 * hd;
  const CT* pA = (const CT*)a.packA + (size_t)chain * 8 * hd;
  const CT *Vb1T = pA, *Vb2T = pA + hd, *Sb1T = pA + 2 * hd, *Sb2T = pA + 3 * hd;
  const CT *Vb1 = pA + 4 * hd, *Vb2 = pA + 5 * hd, *Sb1 = pA + 6 * hd, *Sb2 = pA + 7 * hd;
  CT* op = (CT*)a.opT + (size_t)chain * 5 * ((size_t)H + D) * C;
  CT *ZkbT = op, *ZqbT = ZkbT + (size_t)H * C, *GbT = ZqbT + (size_t)H * C,
     *HkT = GbT + (size_t)H * C, *HqT = HkT + (size_t)H * C, *KT = HqT + (size_t)H * C,
     *QT = KT + (size_t)D * C, *RT = QT + (size_t)D * C, *YkbT = RT + (size_t)D * C,
     *dOT = YkbT + (size_t)D * C;
  const size_t tok0 = (size_t)n * C + r0;
  const size_t cb = (size_t)chain * Dm.L + tok0;
  const IO* q = (const IO*)a.q + cb * D;
  const IO* k = (const IO*)a.k + cb * D;
  const IO* v = (const IO*)a.v + cb * D;
  const IO* dO = (const IO*)a.dO + cb * D;
  const float* tk = a.tokc + cb * TKS;
  float* dtk = a.dtok + cb * 4;
  float* dqp = a.dq_part + cb * D;
  float* dkp = a.dk_part + cb * D;
  float* dvp = a.dv_part + cb * D;
  const float rscale = 2.0f / (float)D;
  const int l = lane_id();

  if (threadIdx.x < TT) {
    cC[threadIdx.x] = tk[(size_t)threadIdx.x * TKS + 0];
    bb[threadIdx.x] = tk[(size_t)threadIdx.x * TKS + 1];
  }
  for (int e = threadIdx.x; e < TT * (D / 8); e += blockDim.x) {
    const int i = e % TT, j0 = (e / TT) * 8;
    float qx[8], kx[8], ox[8];
    gload8(q + (size_t)i * D + j0, qx);
    gload8(k + (size_t)i * D + j0, kx);
    gload8(dO + (size_t)i * D + j0, ox);
    gstore8<CT>(sQ + (size_t)i * D + j0, qx);
    gstore8<CT>(sK + (size_t)i * D + j0, kx);
    gstore8<CT>(sdO + (size_t)i * D + j0, ox);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const size_t et = (size_t)(j0 + t) * C + r0 + i;
      KT[et] = from_f<CT>(kx[t]);
      QT[et] = from_f<CT>(qx[t]);
      dOT[et] = from_f<CT>(ox[t]);
    }
  }
  __syncthreads();
  using BH = Blk<TT, H>;
  using BD = Blk<TT, D>;
  // Zk -> Hk ; Zq -> Hq ; Zqbar = (dO V2) * s'(Zq)
  for_blocks<TT, H>([&](int i0, int j0) {
    f4 ak[BH::RB][BH::CB], aq[BH::RB][BH::CB], ap[BH::RB][BH::CB];
    zero_blk(ak);
    zero_blk(aq);
    zero_blk(ap);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ak, sK, D, i0, V1, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(aq, sQ, D, i0, V1, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ap, sdO, D, i0, V2T, D, j0);
    blk_each4<BH::RB, BH::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 hk, hq, zq;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t e = (size_t)(i + r) * H + j;
        const float zk = ak[rb][cb_][r];
        const ActVals z = act_all<ACT>(aq[rb][cb_][r]);
        hk[r] = act_f<ACT>(zk);
        hq[r] = z.s;
        zq[r] = ap[rb][cb_][r] * z.d1;
        sZk[e] = from_f<CT>(zk);
        sHk[e] = from_f<CT>(hk[r]);
        sZqb[e] = from_f<CT>(zq[r]);
      }
      const size_t et = (size_t)j * C + r0 + i;
      store4<CT>(HkT + et, hk);
      store4<CT>(HqT + et, hq);
      store4<CT>(ZqbT + et, zq);
    });
  });
  __syncthreads();
  // R = (2/d)(Hk V2^T - V) ; T5 = Hk V2bar'^T ; T6 = Hk S2bar'^T ; dq = Zqbar V1
  f4 t3[BD::RB][BD::CB], t4[BD::RB][BD::CB], t5[BD::RB][BD::CB], t6[BD::RB][BD::CB];
  static_assert(BD::NB <= 8, "one (TT x D) block per wave");
  const bool own = wave_id() < BD::NB;
  const int di0 = (wave_id() / BD::NBN) * BD::RB * 16, dj0 = (wave_id() % BD::NBN) * BD::CB * 16;
  zero_blk(t5);
  zero_blk(t6);
  if (own) {
    f4 ay[BD::RB][BD::CB], aq[BD::RB][BD::CB];
    zero_blk(ay);
    zero_blk(aq);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(ay, sHk, H, di0, V2, H, dj0);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(t5, sHk, H, di0, Vb2, H, dj0);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(t6, sHk, H, di0, Sb2, H, dj0);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(aq, sZqb, H, di0, V1T, H, dj0);
    blk_each4<BD::RB, BD::CB>(di0, dj0, [&](int rb, int cb_, int i, int j) {
      f4 rv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t e = (size_t)(i + r) * D + j;
        rv[r] = rscale * (ay[rb][cb_][r] - to_f(v[e]));
        dqp[e] = aq[rb][cb_][r];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sR[(size_t)(i + r) * D + j] = from_f<CT>(rv[r]);  // Q is dead
      store4<CT>(RT + (size_t)j * C + r0 + i, rv);
    });
  }
  __syncthreads();
  // G = R V2 ; D1 = G s'(Zk) ; D1bar = -cC K V1bar'^T - b K S1bar'^T ; Gbar ; Zkp
  for_blocks<TT, H>([&](int i0, int j0) {
    f4 ag[BH::RB][BH::CB], a1[BH::RB][BH::CB], a2[BH::RB][BH::CB];
    zero_blk(ag);
    zero_blk(a1);
    zero_blk(a2);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ag, sR, D, i0, V2T, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(a1, sK, D, i0, Vb1, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(a2, sK, D, i0, Sb1, D, j0);
    blk_each4<BH::RB, BH::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 gv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ii = i + r;
        const size_t e = (size_t)ii * H + j;
        const ActVals z = act_all<ACT>(to_f(sZk[e]));
        const float g = ag[rb][cb_][r];
        const float d1b = -cC[ii] * a1[rb][cb_][r] - bb[ii] * a2[rb][cb_][r];
        sD1[e] = from_f<CT>(g * z.d1);
        gv[r] = d1b * z.d1;
        sGb[e] = from_f<CT>(gv[r]);
        sZkp[e] = from_f<CT>(d1b * g * z.d2);
      }
      store4<CT>(GbT + (size_t)j * C + r0 + i, gv);
    });
  });
  __syncthreads();
  // T3 = D1 V1bar', T4 = D1 S1bar' ; Rbar = -cC T5 - b T6 + Gbar V2^T ; Ykbar ; Vbar ;
  // adjoints of cC_t, b_t: -(K . T3 + R . T5), -(K . T4 + R . T6)
  if (own) {
    f4 ag[BD::RB][BD::CB];
    zero_blk(t3);
    zero_blk(t4);
    zero_blk(ag);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(t3, sD1, H, di0, Vb1T, H, dj0);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(t4, sD1, H, di0, Sb1T, H, dj0);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(ag, sGb, H, di0, V2, H, dj0);
    blk_each4<BD::RB, BD::CB>(di0, dj0, [&](int rb, int cb_, int i, int j) {
      f4 yv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ii = i + r;
        const size_t e = (size_t)ii * D + j;
        const float rbv = -cC[ii] * t5[rb][cb_][r] - bb[ii] * t6[rb][cb_][r] + ag[rb][cb_][r];
        yv[r] = rscale * rbv;
        sYkb[e] = from_f<CT>(yv[r]);
        dvp[e] = -yv[r];
        const float kx = to_f(sK[e]), rx = to_f(sR[e]);
        const float s1 = gsum16(kx * t3[rb][cb_][r] + rx * t5[rb][cb_][r]);
        const float s2 = gsum16(kx * t4[rb][cb_][r] + rx * t6[rb][cb_][r]);
        if ((l & 15) == 0) {
          gp[0][j >> 4][ii] = s1;
          gp[1][j >> 4][ii] = s2;
        }
      }
      store4<CT>(YkbT + (size_t)j * C + r0 + i, yv);
    });
  }
  __syncthreads();
  if (threadIdx.x < TT) {
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int t = 0; t < TN; ++t) {
      s1 += gp[0][t][threadIdx.x];
      s2 += gp[1][t][threadIdx.x];
    }
    dtk[(size_t)threadIdx.x * 4 + 0] = -s1;
    dtk[(size_t)threadIdx.x * 4 + 1] = -s2;
  }
  // Hkbar = -cC R V2bar' - b R S2bar' + Ykbar V2 ; Zkbar = Hkbar s'(Zk) + Zkp
  for_blocks<TT, H>([&](int i0, int j0) {
    f4 a7[BH::RB][BH::CB], a8[BH::RB][BH::CB], ay[BH::RB][BH::CB];
    zero_blk(a7);
    zero_blk(a8);
    zero_blk(ay);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(a7, sR, D, i0, Vb2T, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(a8, sR, D, i0, Sb2T, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ay, sYkb, D, i0, V2T, D, j0);
    blk_each4<BH::RB, BH::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 zv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ii = i + r;
        const size_t e = (size_t)ii * H + j;
        const ActVals z = act_all<ACT>(to_f(sZk[e]));
        const float hkb = -cC[ii] * a7[rb][cb_][r] - bb[ii] * a8[rb][cb_][r] + ay[rb][cb_][r];
        zv[r] = hkb * z.d1 + to_f(sZkp[e]);
        sZkb[e] = from_f<CT>(zv[r]);
      }
      store4<CT>(ZkbT + (size_t)j * C + r0 + i, zv);
    });
  });
  __syncthreads();
  // dk = -cC T3 - b T4 + Zkbar V1
  if (own) {
    f4 ak[BD::RB][BD::CB];
    zero_blk(ak);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(ak, sZkb, H, di0, V1T, H, dj0);
    blk_each4<BD::RB, BD::CB>(di0, dj0, [&](int rb, int cb_, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ii = i + r;
        dkp[(size_t)ii * D + j] =
            -cC[ii] * t3[rb][cb_][r] - bb[ii] * t4[rb][cb_][r] + ak[rb][cb_][r];
      }
    });
  }
}

// ---------------------------------------------------------------------------
// backward tile of the last chunk, whose exit adjoint is zero: every term of
// the key side (T3..T6, D1bar, Gbar, Rbar, Ykbar, Hkbar, Zkbar) vanishes, so dk
// and dv of its tokens are zero and only the query side remains, Zq -> Hq,
// Zqbar = (dO V2) * s'(Zq), dq = Zqbar V1, with the operands of the entry-adjoint
// products that do not vanish (Zqbar^T Q, dO^T Hq)
// ---------------------------------------------------------------------------
template <typename IO, typename CT, int ACT, int D, int H>
__global__ void __launch_bounds__(512) gbwd_tile_last_kernel(GlobalArgs a, int n) {
  constexpr int TT = gtile_rows<H>();
  extern __shared__ __align__(16) unsigned char smem[];
  CT* sQ = reinterpret_cast<CT*>(smem);  // [TT][D]
  CT* sdO = sQ + TT * D;                 // [TT][D]
  CT* sZqb = sdO + TT * D;               // [TT][H]
  const Dims Dm = a.D;
  const int C = Dm.C;
  const int chain = blockIdx.y, r0 = blockIdx.x * TT;
  constexpr size_t hd = (size_t)H * D;
  const CT* pS = (const CT*)a.packT + (size_t)chain * 4 * hd;
  const CT *V1T = pS, *V2T = pS + hd, *V1 = pS + 2 * hd;
  CT* op = (CT*)a.opT + (size_t)chain * 5 * ((size_t)H + D) * C;
  CT *ZqbT = op + (size_t)H * C, *HqT = op + 4 * (size_t)H * C, *QT = op + 5 * (size_t)H * C + (size_t)D * C,
     *dOT = op + 5 * (size_t)H * C + 4 * (size_t)D * C;
  const size_t tok0 = (size_t)n * C + r0;
  const size_t cb = (size_t)chain * Dm.L + tok0;
  const IO* q = (const IO*)a.q + cb * D;
  const IO* dO = (const IO*)a.dO + cb * D;
  float* dtk = a.dtok + cb * 4;
  float* dqp = a.dq_part + cb * D;
  float* dkp = a.dk_part + cb * D;
  float* dvp = a.dv_part + cb * D;

  for (int e = threadIdx.x; e < TT * (D / 8); e += blockDim.x) {
    const int i = e % TT, j0 = (e / TT) * 8;
    float qx[8], ox[8];
    gload8(q + (size_t)i * D + j0, qx);
    gload8(dO + (size_t)i * D + j0, ox);
    gstore8<CT>(sQ + (size_t)i * D + j0, qx);
    gstore8<CT>(sdO + (size_t)i * D + j0, ox);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const size_t et = (size_t)(j0 + t) * C + r0 + i;
      QT[et] = from_f<CT>(qx[t]);
      dOT[et] = from_f<CT>(ox[t]);
    }
  }
  for (int e = threadIdx.x * 4; e < TT * D; e += blockDim.x * 4) {
    *reinterpret_cast<f32x4*>(dkp + e) = f32x4{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4*>(dvp + e) = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (threadIdx.x < TT) {
    dtk[(size_t)threadIdx.x * 4 + 0] = 0.f;
    dtk[(size_t)threadIdx.x * 4 + 1] = 0.f;
  }
  __syncthreads();
  using BH = Blk<TT, H>;
  using BD = Blk<TT, D>;
  // Zq -> Hq ; Zqbar = (dO V2) * s'(Zq)
  for_blocks<TT, H>([&](int i0, int j0) {
    f4 aq[BH::RB][BH::CB], ap[BH::RB][BH::CB];
    zero_blk(aq);
    zero_blk(ap);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(aq, sQ, D, i0, V1, D, j0);
    mma_blk<CT, KC, KC, BH::RB, BH::CB, D>(ap, sdO, D, i0, V2T, D, j0);
    blk_each4<BH::RB, BH::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
      f4 hq, zq;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const ActVals z = act_all<ACT>(aq[rb][cb_][r]);
        hq[r] = z.s;
        zq[r] = ap[rb][cb_][r] * z.d1;
        sZqb[(size_t)(i + r) * H + j] = from_f<CT>(zq[r]);
      }
      const size_t et = (size_t)j * C + r0 + i;
      store4<CT>(HqT + et, hq);
      store4<CT>(ZqbT + et, zq);
    });
  });
  __syncthreads();
  // dq = Zqbar V1
  for_blocks<TT, D>([&](int i0, int j0) {
    f4 aq[BD::RB][BD::CB];
    zero_blk(aq);
    mma_blk<CT, KC, KC, BD::RB, BD::CB, H>(aq, sZqb, H, i0, V1T, H, j0);
    blk_each4<BD::RB, BD::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) dqp[(size_t)(i + r) * D + j] = aq[rb][cb_][r];
    });
  });
}

// ---------------------------------------------------------------------------
// backward entry-adjoint partials of token split `blockIdx.x`:
//   m = 0: Zkbar^T K + Zqbar^T Q            -> V1 slot (hid x d)
//   m = 1: R^T Gbar + Ykbar^T Hk + dO^T Hq  -> V2 slot (d x hid)
// ---------------------------------------------------------------------------
// ZA: the chunk's exit adjoint is zero (its key-side operands vanish): only
// Zqbar^T Q and dO^T Hq remain
template <typename CT, int D, int H, int TK, bool ZA = false>
__global__ void __launch_bounds__(512) gbwd_state_kernel(GlobalArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int split = blockIdx.x, m = blockIdx.y, chain = blockIdx.z, ns = gridDim.x;
  const int C = a.D.C;
  constexpr size_t hd = (size_t)H * D;
  const CT* op = (const CT*)a.opT + (size_t)chain * 5 * ((size_t)H + D) * C;
  const CT *ZkbT = op, *ZqbT = ZkbT + (size_t)H * C, *GbT = ZqbT + (size_t)H * C,
           *HkT = GbT + (size_t)H * C, *HqT = HkT + (size_t)H * C, *KT = HqT + (size_t)H * C,
           *QT = KT + (size_t)D * C, *RT = QT + (size_t)D * C, *YkbT = RT + (size_t)D * C,
           *dOT = YkbT + (size_t)D * C;
  const size_t k0 = (size_t)split * TK;
  float* P = a.part + ((size_t)chain * ns + split) * 4 * hd;
  CT* lds = reinterpret_cast<CT*>(smem);
  if (m == 0) {
    using BK = Blk<H, D>;
    static_assert(BK::NB == 8, "one block per wave");
    const int i0 = (wave_id() / BK::NBN) * BK::RB * 16, j0 = (wave_id() % BK::NBN) * BK::CB * 16;
    f4 acc[BK::RB][BK::CB];
    zero_blk(acc);
    if constexpr (ZA) {
      const CT* const As[1] = {ZqbT + k0};
      const CT* const Bs[1] = {QT + k0};
      lds_gemm_nt<CT, H, D, GCARRY_KT, 1>(acc, i0, j0, As, Bs, C, TK, lds);
    } else {
      const CT* const As[2] = {ZkbT + k0, ZqbT + k0};
      const CT* const Bs[2] = {KT + k0, QT + k0};
      lds_gemm_nt<CT, H, D, GCARRY_KT, 2>(acc, i0, j0, As, Bs, C, TK, lds);
    }
    blk_each4<BK::RB, BK::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) P[(size_t)(i + r) * D + j] = acc[rb][cb_][r];
    });
  } else {
    using BK = Blk<D, H>;
    static_assert(BK::NB == 8, "one block per wave");
    const int i0 = (wave_id() / BK::NBN) * BK::RB * 16, j0 = (wave_id() % BK::NBN) * BK::CB * 16;
    f4 acc[BK::RB][BK::CB];
    zero_blk(acc);
    if constexpr (ZA) {
      const CT* const As[1] = {dOT + k0};
      const CT* const Bs[1] = {HqT + k0};
      lds_gemm_nt<CT, D, H, GCARRY_KT, 1>(acc, i0, j0, As, Bs, C, TK, lds);
    } else {
      const CT* const As[3] = {RT + k0, YkbT + k0, dOT + k0};
      const CT* const Bs[3] = {GbT + k0, HkT + k0, HqT + k0};
      lds_gemm_nt<CT, D, H, GCARRY_KT, 3>(acc, i0, j0, As, Bs, C, TK, lds);
    }
    blk_each4<BK::RB, BK::CB>(i0, j0, [&](int rb, int cb_, int i, int j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) P[hd + (size_t)(i + r) * H + j] = acc[rb][cb_][r];
    });
  }
}

// ---------------------------------------------------------------------------
// launchers: true when the fixed-size path handles the shape
// ---------------------------------------------------------------------------
template <int D, int H>
static bool gblk_shape(const GlobalArgs& a) {
  return a.D.bf16 && a.D.d == D && a.D.hid == H && a.D.C % GTK == 0 &&
         a.D.C % gtile_rows<H>() == 0 && a.packT && a.opT;
}

template <typename IO, typename ACT_T, int ACT, int D, int H>
static hipError_t gfwd_blk_chunk(const GlobalArgs& a, int n, hipStream_t st) {
  typedef __bf16 CT;
  constexpr int TT = gtile_rows<H>();
  const int chains = a.D.B * a.D.H, C = a.D.C;
  constexpr size_t hd = (size_t)H * D;
  // chunk 0's state copies; every later chunk's are written by the reduction
  // that forms its state
  if (n == 0)
    launch_gtranspose<CT>(a.states, (size_t)a.nslots * 4 * hd, (CT*)a.packT, 4 * hd,
                          (CT*)a.packT + 2 * hd, 4 * hd, chains, D, H, 0x3, st);
  static_assert(sizeof(CT) == 2, "gfwd_tile_lds counts 2-byte elements");
  // the backward reads the chunk-entry states only: the carry out of the last
  // chunk (and the tile's key side that feeds it) runs when the caller asks for
  // the final state
  if (a.skip_final_carry && n + 1 == a.D.L / C) {
    GlobalArgs b = a;
    if (b.o_final) {
      hipError_t e = b.parts_ready ? hipStreamWaitEvent(st, b.parts_ready, 0) : hipErrorInvalidValue;
      if (e != hipSuccess) b.o_final = nullptr;  // no fused sum (the caller sums)
    }
    auto kq = gfwd_tile_kernel<IO, CT, ACT, D, H, false>;
    set_lds_limit((const void*)kq);
    hipLaunchKernelGGL(kq, dim3(C / TT, chains), dim3(512), (gfwd_tile_lds<D, H, false>()), st, b, n);
    if (b.o_final && b.o_fused) *b.o_fused = 1;
    return hipGetLastError();
  }
  auto k1 = gfwd_tile_kernel<IO, CT, ACT, D, H, true>;
  set_lds_limit((const void*)k1);
  hipLaunchKernelGGL(k1, dim3(C / TT, chains), dim3(512), (gfwd_tile_lds<D, H, true>()), st, a, n);
  if (a.tile_done && n == a.tile_done_n) {
    const hipError_t e = hipEventRecord(a.tile_done, st);
    if (e != hipSuccess) return e;
    if (a.tile_recorded) *a.tile_recorded = 1;
  }
  const int tk = gtk_of(C), ns = C / tk;
  const int sec = section_begin("global_carry", st);
  constexpr size_t lc = lds_gemm_bytes<CT, H, D, GCARRY_KT, 1>();
  set_lds_limit((const void*)gfwd_carry_kernel<CT, D, H, GTK_LONG>);
  set_lds_limit((const void*)gfwd_carry_kernel<CT, D, H, GTK>);
  if (tk == GTK_LONG)
    hipLaunchKernelGGL((gfwd_carry_kernel<CT, D, H, GTK_LONG>), dim3(ns, 4, chains), dim3(512), lc, st, a);
  else
    hipLaunchKernelGGL((gfwd_carry_kernel<CT, D, H, GTK>), dim3(ns, 4, chains), dim3(512), lc, st, a);
  hipLaunchKernelGGL(gcarry_reduce_pack_kernel<CT>, dim3((unsigned)(hd / 1024), chains, 2), dim3(256), 0,
                     st, a, n, ns);
  section_end(sec, st);
  return hipGetLastError();
}

template <typename IO, typename ACT_T, int ACT, int D, int H>
static hipError_t gbwd_blk_chunk(const GlobalArgs& a, int n, hipStream_t st) {
  typedef __bf16 CT;
  constexpr int TT = gtile_rows<H>();
  const int chains = a.D.B * a.D.H, C = a.D.C;
  constexpr size_t hd = (size_t)H * D;
  // the last chunk (walked first) leaves with a zero adjoint: its tile and
  // state products keep only the terms that do not vanish
  const bool za = n + 1 == a.D.L / C;
  launch_gtranspose<CT>(a.states + (size_t)n * 4 * hd, (size_t)a.nslots * 4 * hd, (CT*)a.packT,
                        4 * hd, (CT*)a.packT + 2 * hd, 4 * hd, chains, D, H, 0x3, st);
  if (za) {
    const size_t lz = (2 * (size_t)TT * D + (size_t)TT * H) * sizeof(CT);
    hipLaunchKernelGGL((gbwd_tile_last_kernel<IO, CT, ACT, D, H>), dim3(C / TT, chains), dim3(512), lz,
                       st, a, n);
  } else {
    launch_gtranspose<CT>(a.adj + (size_t)((n + 1) & 1) * 4 * hd, 2 * 4 * hd, (CT*)a.packA, 8 * hd,
                          (CT*)a.packA + 4 * hd, 8 * hd, chains, D, H, 0xf, st);
    const size_t l1 = (3 * (size_t)TT * D + 4 * (size_t)TT * H) * sizeof(CT);
    auto k1 = gbwd_tile_kernel<IO, CT, ACT, D, H>;
    set_lds_limit((const void*)k1);
    hipLaunchKernelGGL(k1, dim3(C / TT, chains), dim3(512), l1, st, a, n);
  }
  const int tk = gtk_of(C), ns = C / tk;
  const int sec = section_begin("global_bwd_carry", st);
  constexpr size_t ls = lds_gemm_bytes<CT, H, D, GCARRY_KT, 1>();
  set_lds_limit((const void*)gbwd_state_kernel<CT, D, H, GTK>);
  set_lds_limit((const void*)gbwd_state_kernel<CT, D, H, GTK_LONG>);
  set_lds_limit((const void*)gbwd_state_kernel<CT, D, H, GTK, true>);
  set_lds_limit((const void*)gbwd_state_kernel<CT, D, H, GTK_LONG, true>);
  const dim3 gs(ns, 2, chains);
  if (tk == GTK_LONG && za)
    hipLaunchKernelGGL((gbwd_state_kernel<CT, D, H, GTK_LONG, true>), gs, dim3(512), ls, st, a);
  else if (tk == GTK_LONG)
    hipLaunchKernelGGL((gbwd_state_kernel<CT, D, H, GTK_LONG>), gs, dim3(512), ls, st, a);
  else if (za)
    hipLaunchKernelGGL((gbwd_state_kernel<CT, D, H, GTK, true>), gs, dim3(512), ls, st, a);
  else
    hipLaunchKernelGGL((gbwd_state_kernel<CT, D, H, GTK>), gs, dim3(512), ls, st, a);
  const hipError_t e = launch_gbwd_state_reduce(a, n, ns, st);
  section_end(sec, st);
  return e;
}

bool launch_global_fwd_blk(const GlobalArgs& a, int n, hipStream_t st, hipError_t* err) {
  if (a.force_generic) return false;
  if (gblk_shape<64, 256>(a)) {
    *err = a.D.act == ACT_SILU ? gfwd_blk_chunk<__bf16, void, ACT_SILU, 64, 256>(a, n, st)
                               : gfwd_blk_chunk<__bf16, void, ACT_GELU, 64, 256>(a, n, st);
    return true;
  }
  return false;
}

bool launch_global_bwd_blk(const GlobalArgs& a, int n, hipStream_t st, hipError_t* err) {
  if (a.force_generic || !a.packA) return false;
  if (gblk_shape<64, 256>(a)) {
    *err = a.D.act == ACT_SILU ? gbwd_blk_chunk<__bf16, void, ACT_SILU, 64, 256>(a, n, st)
                               : gbwd_blk_chunk<__bf16, void, ACT_GELU, 64, 256>(a, n, st);
    return true;
  }
  return false;
}

// splits used by the fixed-size path (the partial buffer must hold them)
int global_blk_splits(const Dims& D) { return D.C / GTK; }  // the larger count of the two

}  // namespace tnt
