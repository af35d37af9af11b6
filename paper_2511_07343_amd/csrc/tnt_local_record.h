// Per-(unit, chunk) records shared by the chunk-parallel passes of the local
// memories (fixed-size kernels).
//
//  * forward record (in the saved buffer): written by the forward walk and the
//    forward's chunk-parallel retrieval, read by the backward passes — every
//    forward quantity of the chunk that the backward contracts or differentiates
//    through, so the backward does not recompute the forward;
//  * backward record (in the backward workspace): written by the backward's
//    chunk-parallel pass from dO, read by the walk of the carried adjoint and
//    by the gate pass.
//
// C x h elementwise factors (s'(Zk), s''(Zk), G = R W2, s'(Z)) are stored
// fragment-major over the Blk<Cp, hid> decomposition (see frag_ofs): each
// lane's four values of a 16 x 16 tile are contiguous, at a position that
// depends only on the tile and the lane, so any kernel that produces a tile can
// write it where the block-GEMM epilogues of the backward read it.
#pragma once

#include "tnt_device.h"

namespace tnt {
namespace rec {

// forward record, compute type
enum FwdCT {
  Hk, HkT, D1, HT, Sp, Spp, G, Sz,              // C x h (Sp, Spp, G, Sz fragment-major)
  PzT, PoT, StrT,                               // C x C
  K, KT, KcC, Kb, R, RT, RcC, Rb,               // C x d
  XT, XAT, XET, N, NT, QT,                      // C x d
  FWD_CT
};
// forward record, fp32
enum FwdF {
  XK, HH,        // C x C  X K^T, H Hk^T (unmasked; fragment-major over Blk<Cp, Cp>)
  HW2, HS2,      // d x C  (H W2^T)^T, (H S2^T)^T
  kn, cC, bb,    // C      key norms, cC, b
  sc,            // 4      A_C, B_C, E_C
  Cc,            // C(C+1)/2  the chunk coefficients c_{i,tau} (tau <= i), row after row
  cA, cE,        // C      A_i, E_i (pass A of the backward reads these and Cc instead of
                 //        recomputing them; empty unless rec_coefs(C))
  FWD_F
};
// backward record, compute type
enum BwdCT { ZbT, Q1T, dOT, dOAT, dOET, BWD_CT };
// backward record, fp32
enum BwdF {
  Cb,            // C x C  the retrieval's part of cbar
  gA, gE,        // C      the retrieval's dA, dE
  XbQ,           // d x d  Xbar^T Q, then the suffix sum over later chunks
  gCC, gB,       // C      the walk's cC-bar, b-bar
  dots,          // 4      dA_C, dE_C, dB_C (the walk's adjoint . state products)
  BWD_F
};

template <int NB>
struct Lay {
  size_t o[NB];
  size_t n;
};

// offsets rounded to 8 elements: 16-byte alignment for bf16 and fp32 vectors
template <int NB>
__host__ __device__ constexpr Lay<NB> make_lay(const size_t (&sz)[NB]) {
  Lay<NB> y{};
  size_t off = 0;
  for (int i = 0; i < NB; ++i) {
    y.o[i] = off;
    off += (sz[i] + 7) & ~size_t(7);
  }
  y.n = off;
  return y;
}

struct RecLayout {
  Lay<FWD_CT> fc;
  Lay<FWD_F> ff;
  Lay<BWD_CT> bc;
  Lay<BWD_F> bf;
};

// Whether the forward record keeps the chunk coefficients for the backward.  At
// chunks of up to 32 positions, recomputing them (one wave's scan) costs pass A
// more than reading them back; at 64 the 8 KB per chunk they take costs more.
__host__ __device__ constexpr bool rec_coefs(int Cp) { return Cp <= 32; }

__host__ __device__ constexpr RecLayout make_rec_layout(int Cp, int d, int h) {
  const size_t C = Cp, Cd = C * d, Ch = C * h, CC = C * C, dd = (size_t)d * d;
  const size_t sfc[FWD_CT] = {Ch, Ch, Ch, Ch, Ch, Ch, Ch, Ch, CC, CC, CC, Cd, Cd, Cd, Cd,
                              Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd};
  const size_t cr = rec_coefs(Cp) ? C : 0;
  const size_t sff[FWD_F] = {CC, CC, Cd, Cd, C, C, C, 4, cr * (cr + 1) / 2, cr, cr};
  const size_t sbc[BWD_CT] = {Ch, CC, Cd, Cd, Cd};
  const size_t sbf[BWD_F] = {CC, C, C, dd, C, C, 4};
  return RecLayout{make_lay(sfc), make_lay(sff), make_lay(sbc), make_lay(sbf)};
}

}  // namespace rec

// Fragment-major element offset of lane l's four values of the 16 x 16 tile at
// (ti, tj) (multiples of 16) of a CP x N matrix, over the Blk<CP, N>
// decomposition used by the backward's block GEMMs.
template <int CP, int N>
__device__ __forceinline__ size_t frag_ofs(int ti, int tj, int l) {
  using BK = Blk<CP, N>;
  const int blk = (ti / (BK::RB * 16)) * BK::NBN + tj / (BK::CB * 16);
  const int rb = (ti / 16) % BK::RB, cb = (tj / 16) % BK::CB;
  return ((size_t)((blk * BK::RB + rb) * BK::CB + cb) * WAVE + l) * 4;
}

}  // namespace tnt
