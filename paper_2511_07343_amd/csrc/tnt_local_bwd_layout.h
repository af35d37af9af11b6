// Per-unit scratch layout of the local-memory backward kernel (host + device).
#pragma once

#include "tnt_kernels.h"

namespace tnt {

// CT (compute-type) buffers; "T" suffix = transposed copy.
enum BwdCT {
  bQ, bQT, bK, bKT, bN, bNT, bX, bXT, bXAT, bXET, bStr, bStrT,
  bHk, bHkT, bSp, bSpp, bR, bRT, bG, bD1, bD1T, bH, bHT, bSz,
  bPz, bPzT, bPo, bPoT, bdO, bdOT, bdOAT, bdOET, bQ1, bQ1T,
  bZb, bZbT, bQ2, bQ2T, bGb, bGbT, bYkb, bYkbT, bZkb, bZkbT,
  bXb, bXbT, bdXN, bdXNT,
  // row-scaled copies: diag(A) X, diag(E) X, diag(A) dO, diag(E) dO, diag(cC) K,
  // diag(b) K, diag(cC) R, diag(b) R
  bXA, bXE, bdOA, bdOE, bKcC, bKb, bRcC, bRb,
  // transposed copies of the carried adjoint (W1bar^T, S1bar^T: d x h; W2bar^T, S2bar^T: h x d)
  bWb1T, bSb1T, bWb2T, bSb2T, BWD_CT_COUNT
};
// fp32 buffers
enum BwdF32 {
  E_XK, E_HH, E_dOR, E_dZD1, E_Cbar, E_U, E_Kbar, E_Rbar, E_Xbar, E_T3, E_T4, E_T5, E_T6, E_Zkp,
  E_Msym, E_PartA, E_PartE, BWD_F32_COUNT
};

struct BwdLayout {
  size_t ct[BWD_CT_COUNT];
  size_t f32[BWD_F32_COUNT];
  size_t ct_elems, f32_elems;
};

__host__ __device__ constexpr BwdLayout make_bwd_layout(int Cp, int d, int h) {
  BwdLayout yy{};
  BwdLayout* y = &yy;
  const size_t C = Cp;
  size_t sizes[BWD_CT_COUNT] = {};
  const size_t Cd = C * d, Ch = C * h, CC = C * C, HD = (size_t)h * d;
  const size_t s_ct[BWD_CT_COUNT] = {
      Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd, CC, CC,   // Q .. StrT
      Ch, Ch, Ch, Ch, Cd, Cd, Ch, Ch, Ch, Ch, Ch, Ch,   // Hk .. Sz
      CC, CC, CC, CC, Cd, Cd, Cd, Cd, CC, CC,           // Pz .. Q1T
      Ch, Ch, CC, CC, Ch, Ch, Cd, Cd, Ch, Ch,           // Zb .. ZkbT
      Cd, Cd, CC, CC,                                   // Xb .. dXNT
      Cd, Cd, Cd, Cd, Cd, Cd, Cd, Cd,                   // XA .. Rb
      HD, HD, HD, HD};                                  // Wb1T .. Sb2T
  size_t off = 0;
  for (int i = 0; i < BWD_CT_COUNT; ++i) {
    sizes[i] = s_ct[i];
    y->ct[i] = off;
    off += (sizes[i] + 7) & ~size_t(7);
  }
  y->ct_elems = off;
  const size_t hp = (size_t)(h / 16 > d / 16 ? h / 16 : d / 16);
  const size_t s_f[BWD_F32_COUNT] = {CC, CC, CC, CC, CC, CC, Cd, Cd, Cd, Cd, Cd, Cd, Cd, Ch,
                                     (size_t)d * d, hp * C, hp * C};
  off = 0;
  for (int i = 0; i < BWD_F32_COUNT; ++i) {
    y->f32[i] = off;
    off += (s_f[i] + 3) & ~size_t(3);
  }
  y->f32_elems = off;
  return yy;
}

__host__ __device__ inline void bwd_layout(int Cp, int d, int h, BwdLayout* y) {
  *y = make_bwd_layout(Cp, d, h);
}

}  // namespace tnt
