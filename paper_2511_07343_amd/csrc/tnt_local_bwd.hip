// Local memories, backward: one workgroup per unit (batch row, head, shard)
// walks the shard's chunks in reverse, carrying the adjoint of the state
// (W1, W2, S1, S2 and the Q-K sum M).  Each chunk recomputes its forward
// quantities from the saved chunk-entry state and applies the exact adjoint
// of the forward chunk step (see the forward kernel for the step):
//
//   retrieval   O = diag(A) H W2^T + diag(E) H S2^T - (c o H Hk^T) R,  H = s(Z)
//               Z = diag(A) X W1^T + diag(E) X S1^T - (c o X K^T) D1
//   carry       W1' = A_C W1 + E_C S1 - D1^T diag(cC) K,  S1' = B_C S1 - D1^T diag(b) K
//               W2' = A_C W2 + E_C S2 - R^T diag(cC) Hk,  S2' = B_C S2 - R^T diag(b) Hk
//   gradients   D1 = (R W2) * s'(Zk), R = (2/d)(s(Zk) W2^T - V), Zk = K W1^T
//               (second-order terms: s''(Zk), and R, D1 depend on W)
//   projection  X = Q M0^T + tril(Q N^T) N,  M' = M0 + N^T N,  N = K / ||K||
//   gates       A, E, c, cC, b from prefix sums of log(1 - alpha), log beta
//
// The gate adjoints go back through the prefix sums: for la (log-decay) and
// lb (log-momentum) of position j,
//   la_bar_j = Abar_j A_j + Ebar_j E_j + sum_tau cbar_{j tau} c_{j tau} - T_j - Y_j e^{lb_j}
//   lb_bar_j = T_j - sum_i cbar_{i j} c_{i j} + Y_j e^{lb_j} - bbar_j b_j
//              (+ Bbar_C B_C + sum_tau bbar_tau b_tau at j = C-1)
//   T_j = sum_{i>=j} e^{la_i - la_j} U_{i j},  U_{i j} = beta_j U_{i,j-1} + cbar_{i j} eta_j
//   Y_j = sum_{i>=j} Ebar_i e^{la_i - la_j}
// then alpha_bar_j = -(sum_{i>=j} la_bar_i) / (1 - alpha_j) and
// beta_bar_j = (sum_{i>=j} lb_bar_i) / beta_j.
#include "tnt_local_bwd_layout.h"
#include "tnt_local_common.h"

namespace tnt {

__device__ __forceinline__ float sum16(float v) {
  v += __shfl_xor(v, 1, WAVE);
  v += __shfl_xor(v, 2, WAVE);
  v += __shfl_xor(v, 4, WAVE);
  v += __shfl_xor(v, 8, WAVE);
  return v;
}

// iterate the 16x16 output tiles of an M x N result over the waves
template <typename F>
__device__ __forceinline__ void tiles(int M, int N, F&& f) {
  const int tn = N >> 4, nt = (M >> 4) * tn;
  for (int t = wave_id(); t < nt; t += num_waves()) f((t / tn) << 4, (t % tn) << 4);
}

// D_, H_, CP_ > 0 fix the head dim, hidden width and padded chunk at compile
// time (all loops unrolled, buffer offsets constant); 0 reads them from `a`.
template <typename IO, typename CT, int ACT, int D_, int H_, int CP_>
__global__ void __launch_bounds__(512) local_bwd_kernel(LocalBwdArgs a) {
  __shared__ Coef cf;
  __shared__ float gA[MAXC], gE[MAXC], gCC[MAXC], gB[MAXC], gEta[MAXC], gLa[MAXC], gLb[MAXC];
  __shared__ float red[32];
  const Dims D = a.D;
  const int d = D_ ? D_ : D.d, h = H_ ? H_ : D.hid, Cp = CP_ ? CP_ : D.Cp;
  const int C = D.C;
  const int nshard = D.L / D.S;
  const int u = blockIdx.x;
  const int b = u / (D.H * nshard), hh = (u / nshard) % D.H, s = u % nshard;
  const size_t hd = (size_t)h * d;
  const int l = lane_id();
  BwdLayout Y;
  bwd_layout(Cp, d, h, &Y);
  CT* sc = (CT*)a.scratch + (size_t)u * Y.ct_elems;
  float* sf = a.scratch_f32 + (size_t)u * Y.f32_elems;
#define B_(x) (sc + Y.ct[x])
#define F_(x) (sf + Y.f32[x])
  CT *Q = B_(bQ), *QT = B_(bQT), *K = B_(bK), *KT = B_(bKT), *N = B_(bN), *NT = B_(bNT);
  CT *X = B_(bX), *XT = B_(bXT), *XAT = B_(bXAT), *XET = B_(bXET), *Str = B_(bStr),
     *StrT = B_(bStrT);
  CT *Hk = B_(bHk), *HkT = B_(bHkT), *Sp = B_(bSp), *Spp = B_(bSpp), *R = B_(bR), *RT = B_(bRT);
  CT *G = B_(bG), *D1 = B_(bD1), *D1T = B_(bD1T), *H = B_(bH), *HT = B_(bHT), *Sz = B_(bSz);
  CT *Pz = B_(bPz), *PzT = B_(bPzT), *Po = B_(bPo), *PoT = B_(bPoT);
  CT *dO = B_(bdO), *dOT = B_(bdOT), *dOAT = B_(bdOAT), *dOET = B_(bdOET), *Q1 = B_(bQ1),
     *Q1T = B_(bQ1T);
  CT *Zb = B_(bZb), *ZbT = B_(bZbT), *Q2 = B_(bQ2), *Q2T = B_(bQ2T), *Gb = B_(bGb),
     *GbT = B_(bGbT);
  CT *Ykb = B_(bYkb), *YkbT = B_(bYkbT), *Zkb = B_(bZkb), *ZkbT = B_(bZkbT), *Xb = B_(bXb),
     *XbT = B_(bXbT), *dXN = B_(bdXN), *dXNT = B_(bdXNT);
  CT *Wb1T = B_(bWb1T), *Sb1T = B_(bSb1T), *Wb2T = B_(bWb2T), *Sb2T = B_(bSb2T);
  float *fXK = F_(E_XK), *fHH = F_(E_HH), *fdOR = F_(E_dOR), *fdZD1 = F_(E_dZD1), *fCb = F_(E_Cbar),
        *fU = F_(E_U), *fKb = F_(E_Kbar), *fRb = F_(E_Rbar), *fXb = F_(E_Xbar), *fT3 = F_(E_T3),
        *fT4 = F_(E_T4), *fT5 = F_(E_T5), *fT6 = F_(E_T6), *fZkp = F_(E_Zkp), *fMs = F_(E_Msym),
        *pA = F_(E_PartA), *pE = F_(E_PartE);
#undef B_
#undef F_

  const size_t chain = (size_t)b * D.H + hh;
  const size_t cbase = chain * D.L;
  const IO* qg = (const IO*)a.q + cbase * d;
  const IO* kg = (const IO*)a.k + cbase * d;
  const IO* vg = (const IO*)a.v + cbase * d;
  const IO* dOg = (const IO*)a.dO + cbase * d;
  float* dqp = a.dq_part + cbase * d;
  float* dkp = a.dk_part + cbase * d;
  float* dvp = a.dv_part + cbase * d;
  const float* lr = a.lr + cbase;
  const float* mom = a.mom + cbase;
  const float* dec = a.decay + cbase;
  float* dlr = a.dlr + cbase;
  float* dmom = a.dmom + cbase;
  float* ddec = a.ddecay + cbase;
  float* adj = a.adj + (size_t)u * 4 * hd;
  float *Wb1 = adj, *Wb2 = adj + hd, *Sb1 = adj + 2 * hd, *Sb2 = adj + 3 * hd;
  float* madj = a.madj + (size_t)u * d * d;
  const bool shard_qk = D.qk_proj && D.qk_scope == 0;
  const float rscale = 2.0f / (float)d;

  for (size_t e = threadIdx.x; e < 4 * hd; e += blockDim.x) {
    adj[e] = 0.f;
    Wb1T[e] = from_f<CT>(0.f);  // the four transposed copies are contiguous
  }
  for (int e = threadIdx.x; e < d * d; e += blockDim.x) madj[e] = 0.f;
  // gsub > 1: the gradients of a group of gsub chunks are taken at the state
  // entering the group, so the adjoint of that gradient point (Zkbar^T K into
  // W1, R^T Gbar + Ykbar^T Hk into W2) is gathered over the group in `hadj`
  // and joins the carried adjoint at the group's first chunk
  const int gsub = D.gsub > 1 ? D.gsub : 1;
  float* hadj = gsub > 1 ? a.hadj + (size_t)u * 2 * hd : nullptr;
  if (hadj)
    for (size_t e = threadIdx.x; e < 2 * hd; e += blockDim.x) hadj[e] = 0.f;
  __syncthreads();

  const int nch = D.S / C;
  for (int n = nch - 1; n >= 0; --n) {
    const int tok0 = s * D.S + n * C;
    const int ng = n - n % gsub;  // the chunk whose entry state is the gradient point
    const float* st = a.states + ((size_t)u * a.nslots + n) * 4 * hd;
    const float *W1 = st, *W2 = st + hd, *S1 = st + 2 * hd, *S2 = st + 3 * hd;
    const float* stg = a.states + ((size_t)u * a.nslots + ng) * 4 * hd;
    const float *W1g = stg, *W2g = stg + hd;
    const float* Mc = a.mstates + ((size_t)u * a.nslots + n) * d * d;
    // transposed CT copies of the same state (contraction-contiguous operands)
    const CT* pk = (const CT*)a.statesT + ((size_t)u * a.nslots + n) * (4 * hd + (size_t)d * d);
    const CT *W1T = pk, *W2T = pk + hd, *S1T = pk + 2 * hd, *S2T = pk + 3 * hd, *McT = pk + 4 * hd;
    const CT* pkg = (const CT*)a.statesT + ((size_t)u * a.nslots + ng) * (4 * hd + (size_t)d * d);
    const CT *W1gT = pkg, *W2gT = pkg + hd;
    const bool g_first = (n % gsub) == 0;

    // ================= recompute the chunk's forward quantities
    stage_rows<IO, CT>(Q, QT, qg + (size_t)tok0 * d, C, Cp, d);
    stage_rows<IO, CT>(K, KT, kg + (size_t)tok0 * d, C, Cp, d);
    stage_rows<IO, CT>(dO, dOT, dOg + (size_t)tok0 * d, C, Cp, d);
    if (D.qk_proj) unit_keys<IO, CT>(cf, N, NT, kg + (size_t)tok0 * d, C, Cp, d);
    chunk_coefs(cf, lr, mom, dec, tok0, C, Cp);
    for (int e = threadIdx.x; e < Cp * d; e += blockDim.x) {
      const int i = e / d, j = e - i * d;
      const float x = to_f(dO[e]);
      dOAT[(size_t)j * Cp + i] = from_f<CT>(cf.A[i] * x);
      dOET[(size_t)j * Cp + i] = from_f<CT>(cf.E[i] * x);
    }
    if (threadIdx.x < MAXC) {
      gA[threadIdx.x] = gE[threadIdx.x] = gCC[threadIdx.x] = gB[threadIdx.x] = 0.f;
    }
    auto put_x = [&](int i, int j, float x) {
      X[(size_t)i * d + j] = from_f<CT>(x);
      XT[(size_t)j * Cp + i] = from_f<CT>(x);
      XAT[(size_t)j * Cp + i] = from_f<CT>(cf.A[i] * x);
      XET[(size_t)j * Cp + i] = from_f<CT>(cf.E[i] * x);
    };
    if (D.qk_proj) {
      gemm<CT, KC, KC>(Cp, Cp, d, Q, d, N, d, [&](int i, int j, float x) {
        const float y = j <= i ? x : 0.f;
        Str[(size_t)i * Cp + j] = from_f<CT>(y);
        StrT[(size_t)j * Cp + i] = from_f<CT>(y);
      });
      __syncthreads();
      tiles(Cp, d, [&](int i0, int j0) {
        f4 acc = zero4();
        if (shard_qk) mma_tile<CT, KC, KC>(acc, Q, d, i0, Mc, d, j0, d);
        mma_tile<CT, KC, KC>(acc, Str, Cp, i0, NT, Cp, j0, Cp);
        tile_each(acc, i0, j0, put_x);
      });
    } else {
      for (int e = threadIdx.x; e < Cp * d; e += blockDim.x) {
        const int i = e / d, j = e - i * d;
        put_x(i, j, to_f(Q[e]));
      }
    }
    gemm<CT, KC, KC>(Cp, h, d, K, d, W1g, d, [&](int i, int j, float z) {
      const ActVals av = act_all<ACT>(z);
      Hk[(size_t)i * h + j] = from_f<CT>(av.s);
      HkT[(size_t)j * Cp + i] = from_f<CT>(av.s);
      Sp[(size_t)i * h + j] = from_f<CT>(av.d1);
      Spp[(size_t)i * h + j] = from_f<CT>(av.d2);
    });
    __syncthreads();
    gemm<CT, KC, KC>(Cp, d, h, Hk, h, W2g, h, [&](int i, int j, float y) {
      const float r = (i < C) ? rscale * (y - to_f(vg[(size_t)(tok0 + i) * d + j])) : 0.f;
      R[(size_t)i * d + j] = from_f<CT>(r);
      RT[(size_t)j * Cp + i] = from_f<CT>(r);
    });
    __syncthreads();
    gemm<CT, KC, KC>(Cp, h, d, R, d, W2gT, d, [&](int i, int j, float g) {
      const float d1 = g * to_f(Sp[(size_t)i * h + j]);
      G[(size_t)i * h + j] = from_f<CT>(g);
      D1[(size_t)i * h + j] = from_f<CT>(d1);
      D1T[(size_t)j * Cp + i] = from_f<CT>(d1);
    });
    gemm<CT, KC, KC>(Cp, Cp, d, X, d, K, d, [&](int i, int j, float x) {
      fXK[(size_t)i * Cp + j] = x;
      const float p = j <= i ? cf.c[i][j] * x : 0.f;
      Pz[(size_t)i * Cp + j] = from_f<CT>(p);
      PzT[(size_t)j * Cp + i] = from_f<CT>(p);
    });
    __syncthreads();
    tiles(Cp, h, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
      mma_tile<CT, KC, KC>(a1, X, d, i0, W1, d, j0, d);
      mma_tile<CT, KC, KC>(a2, X, d, i0, S1, d, j0, d);
      mma_tile<CT, KC, KC>(a3, Pz, Cp, i0, D1T, Cp, j0, Cp);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const ActVals av = act_all<ACT>(cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r]);
        H[(size_t)i * h + j] = from_f<CT>(av.s);
        HT[(size_t)j * Cp + i] = from_f<CT>(av.s);
        Sz[(size_t)i * h + j] = from_f<CT>(av.d1);
      }
    });
    __syncthreads();
    gemm<CT, KC, KC>(Cp, Cp, h, H, h, Hk, h, [&](int i, int j, float x) {
      fHH[(size_t)i * Cp + j] = x;
      const float p = j <= i ? cf.c[i][j] * x : 0.f;
      Po[(size_t)i * Cp + j] = from_f<CT>(p);
      PoT[(size_t)j * Cp + i] = from_f<CT>(p);
    });
    __syncthreads();

    // ================= backward through the retrieval
    // dOR = dO R^T ; Q1 = c o dOR ; cbar = -HH o dOR
    gemm<CT, KC, KC>(Cp, Cp, d, dO, d, R, d, [&](int i, int j, float x) {
      fdOR[(size_t)i * Cp + j] = x;
      const bool lo = j <= i;
      const float q1 = lo ? cf.c[i][j] * x : 0.f;
      Q1[(size_t)i * Cp + j] = from_f<CT>(q1);
      Q1T[(size_t)j * Cp + i] = from_f<CT>(q1);
      fCb[(size_t)i * Cp + j] = lo ? -fHH[(size_t)i * Cp + j] * x : 0.f;
    });
    __syncthreads();
    // Hbar = diag(A) dO W2 + diag(E) dO S2 - Q1 Hk ; Zbar = Hbar * s'(Z)
    tiles(Cp, h, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
      mma_tile<CT, KC, KC>(a1, dO, d, i0, W2T, d, j0, d);
      mma_tile<CT, KC, KC>(a2, dO, d, i0, S2T, d, j0, d);
      mma_tile<CT, KC, KC>(a3, Q1, Cp, i0, HkT, Cp, j0, Cp);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const float hv = to_f(H[(size_t)i * h + j]);
        const float hb = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
        const float zb = hb * to_f(Sz[(size_t)i * h + j]);
        Zb[(size_t)i * h + j] = from_f<CT>(zb);
        ZbT[(size_t)j * Cp + i] = from_f<CT>(zb);
        const float sa = sum16(a1[r] * hv), se = sum16(a2[r] * hv);
        if ((l & 15) == 0) {
          pA[(size_t)(j0 >> 4) * Cp + i] = sa;
          pE[(size_t)(j0 >> 4) * Cp + i] = se;
        }
      }
    });
    __syncthreads();
    for (int i = threadIdx.x; i < Cp; i += blockDim.x) {
      float sa = 0.f, se = 0.f;
      for (int t = 0; t < (h >> 4); ++t) {
        sa += pA[(size_t)t * Cp + i];
        se += pE[(size_t)t * Cp + i];
      }
      gA[i] += sa;
      gE[i] += se;
    }
    // dZD1 = Zbar D1^T ; Q2 = c o dZD1 ; cbar -= XK o dZD1
    gemm<CT, KC, KC>(Cp, Cp, h, Zb, h, D1, h, [&](int i, int j, float x) {
      fdZD1[(size_t)i * Cp + j] = x;
      const bool lo = j <= i;
      const float q2 = lo ? cf.c[i][j] * x : 0.f;
      Q2[(size_t)i * Cp + j] = from_f<CT>(q2);
      Q2T[(size_t)j * Cp + i] = from_f<CT>(q2);
      if (lo) fCb[(size_t)i * Cp + j] -= fXK[(size_t)i * Cp + j] * x;
    });
    __syncthreads();
    // Xbar = diag(A) Zbar W1 + diag(E) Zbar S1 - Q2 K
    tiles(Cp, d, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
      mma_tile<CT, KC, KC>(a1, Zb, h, i0, W1T, h, j0, h);
      mma_tile<CT, KC, KC>(a2, Zb, h, i0, S1T, h, j0, h);
      mma_tile<CT, KC, KC>(a3, Q2, Cp, i0, KT, Cp, j0, Cp);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const float xv = to_f(X[(size_t)i * d + j]);
        const float xb = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
        fXb[(size_t)i * d + j] = xb;
        Xb[(size_t)i * d + j] = from_f<CT>(xb);
        XbT[(size_t)j * Cp + i] = from_f<CT>(xb);
        const float sa = sum16(a1[r] * xv), se = sum16(a2[r] * xv);
        if ((l & 15) == 0) {
          pA[(size_t)(j0 >> 4) * Cp + i] = sa;
          pE[(size_t)(j0 >> 4) * Cp + i] = se;
        }
      }
    });
    __syncthreads();
    for (int i = threadIdx.x; i < Cp; i += blockDim.x) {
      float sa = 0.f, se = 0.f;
      for (int t = 0; t < (d >> 4); ++t) {
        sa += pA[(size_t)t * Cp + i];
        se += pE[(size_t)t * Cp + i];
      }
      gA[i] += sa;
      gE[i] += se;
    }

    // ================= D1bar, Gbar, second-order part of Zkbar
    // D1bar = -Pz^T Zbar - diag(cC) K W1bar'^T - diag(b) K S1bar'^T
    tiles(Cp, h, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
      mma_tile<CT, KC, KC>(a1, PzT, Cp, i0, ZbT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a2, K, d, i0, Wb1, d, j0, d);
      mma_tile<CT, KC, KC>(a3, K, d, i0, Sb1, d, j0, d);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const size_t e = (size_t)i * h + j;
        const float d1b = -a1[r] - cf.cC[i] * a2[r] - cf.bb[i] * a3[r];
        const float gb = d1b * to_f(Sp[e]);
        Gb[e] = from_f<CT>(gb);
        GbT[(size_t)j * Cp + i] = from_f<CT>(gb);
        fZkp[e] = d1b * to_f(G[e]) * to_f(Spp[e]);
      }
    });
    // T3 = D1 W1bar', T4 = D1 S1bar', T5 = Hk W2bar'^T, T6 = Hk S2bar'^T  (C x d)
    tiles(Cp, d, [&](int i0, int j0) {
      f4 a3 = zero4(), a4 = zero4(), a5 = zero4(), a6 = zero4();
      mma_tile<CT, KC, KC>(a3, D1, h, i0, Wb1T, h, j0, h);
      mma_tile<CT, KC, KC>(a4, D1, h, i0, Sb1T, h, j0, h);
      mma_tile<CT, KC, KC>(a5, Hk, h, i0, Wb2, h, j0, h);
      mma_tile<CT, KC, KC>(a6, Hk, h, i0, Sb2, h, j0, h);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * d + j0 + (l & 15);
        fT3[e] = a3[r];
        fT4[e] = a4[r];
        fT5[e] = a5[r];
        fT6[e] = a6[r];
      }
    });
    __syncthreads();
    // cC_bar = -K.T3 - R.T5 ; b_bar = -K.T4 - R.T6 (row dots)
    for (int i = wave_id(); i < Cp; i += num_waves()) {
      float sc_ = 0.f, sb_ = 0.f;
      for (int j = l; j < d; j += WAVE) {
        const size_t e = (size_t)i * d + j;
        const float kx = to_f(K[e]), rx = to_f(R[e]);
        sc_ += kx * fT3[e] + rx * fT5[e];
        sb_ += kx * fT4[e] + rx * fT6[e];
      }
      sc_ = wave_sum(sc_);
      sb_ = wave_sum(sb_);
      if (l == 0) {
        gCC[i] = -sc_;
        gB[i] = -sb_;
      }
    }
    // Rbar = -Po^T dO - diag(cC) T5 - diag(b) T6 + Gbar W2^T ; Ykbar = (2/d) Rbar ; Vbar = -Ykbar
    tiles(Cp, d, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4();
      mma_tile<CT, KC, KC>(a1, PoT, Cp, i0, dOT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a2, Gb, h, i0, W2g, h, j0, h);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const size_t e = (size_t)i * d + j;
        const float rb = -a1[r] - cf.cC[i] * fT5[e] - cf.bb[i] * fT6[e] + a2[r];
        const float ykb = (i < C) ? rscale * rb : 0.f;
        fRb[e] = rb;
        Ykb[e] = from_f<CT>(ykb);
        YkbT[(size_t)j * Cp + i] = from_f<CT>(ykb);
        if (i < C) dvp[(size_t)(tok0 + i) * d + j] = -ykb;
      }
    });
    __syncthreads();
    // Hkbar = -Q1^T H - diag(cC) R W2bar' - diag(b) R S2bar' + Ykbar W2 ;
    // Zkbar = Hkbar * s'(Zk) + D1bar * G * s''(Zk)
    tiles(Cp, h, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4(), a4 = zero4();
      mma_tile<CT, KC, KC>(a1, Q1T, Cp, i0, HT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a2, R, d, i0, Wb2T, d, j0, d);
      mma_tile<CT, KC, KC>(a3, R, d, i0, Sb2T, d, j0, d);
      mma_tile<CT, KC, KC>(a4, Ykb, d, i0, W2gT, d, j0, d);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const size_t e = (size_t)i * h + j;
        const float hkb = -a1[r] - cf.cC[i] * a2[r] - cf.bb[i] * a3[r] + a4[r];
        const float zkb = hkb * to_f(Sp[e]) + fZkp[e];
        Zkb[e] = from_f<CT>(zkb);
        ZkbT[(size_t)j * Cp + i] = from_f<CT>(zkb);
      }
    });
    __syncthreads();
    // Kbar = -Q2^T X - diag(cC) T3 - diag(b) T4 + Zkbar W1
    tiles(Cp, d, [&](int i0, int j0) {
      f4 a1 = zero4(), a2 = zero4();
      mma_tile<CT, KC, KC>(a1, Q2T, Cp, i0, XT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a2, Zkb, h, i0, W1gT, h, j0, h);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        const size_t e = (size_t)i * d + j;
        fKb[e] = -a1[r] - cf.cC[i] * fT3[e] - cf.bb[i] * fT4[e] + a2[r];
      }
    });
    // ================= Q-K projection backward
    if (D.qk_proj) {
      if (shard_qk)
        for (int e = threadIdx.x; e < d * d; e += blockDim.x) {
          const int i = e / d, j = e - i * d;
          fMs[e] = madj[e] + madj[(size_t)j * d + i];
        }
      gemm<CT, KC, KC>(Cp, Cp, d, Xb, d, N, d, [&](int i, int j, float x) {
        const float y = j <= i ? x : 0.f;
        dXN[(size_t)i * Cp + j] = from_f<CT>(y);
        dXNT[(size_t)j * Cp + i] = from_f<CT>(y);
      });
      __syncthreads();
      // Qbar = Xbar M0 + tril(Xbar N^T) N ; Nbar = Str^T Xbar + tril(Xbar N^T)^T Q + N (Mb' + Mb'^T)
      tiles(Cp, d, [&](int i0, int j0) {
        f4 q1 = zero4(), n1 = zero4();
        if (shard_qk) mma_tile<CT, KC, KC>(q1, Xb, d, i0, McT, d, j0, d);
        mma_tile<CT, KC, KC>(q1, dXN, Cp, i0, NT, Cp, j0, Cp);
        mma_tile<CT, KC, KC>(n1, StrT, Cp, i0, XbT, Cp, j0, Cp);
        mma_tile<CT, KC, KC>(n1, dXNT, Cp, i0, QT, Cp, j0, Cp);
        if (shard_qk) mma_tile<CT, KC, KC>(n1, N, d, i0, fMs, d, j0, d);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          if (i < C) dqp[(size_t)(tok0 + i) * d + j] = q1[r];
          fT3[(size_t)i * d + j] = n1[r];  // Nbar (T3 is no longer needed)
        }
      });
      __syncthreads();
      // Kbar += (Nbar - N (N . Nbar)) / ||k||
      for (int i = wave_id(); i < C; i += num_waves()) {
        const float nr = cf.knorm[i];
        float dt = 0.f;
        for (int j = l; j < d; j += WAVE) dt += to_f(N[(size_t)i * d + j]) * fT3[(size_t)i * d + j];
        dt = wave_sum(dt);
        if (nr > 0.f)
          for (int j = l; j < d; j += WAVE) {
            const size_t e = (size_t)i * d + j;
            fKb[e] += (fT3[e] - to_f(N[e]) * dt) / nr;
          }
      }
    } else {
      for (int e = threadIdx.x; e < C * d; e += blockDim.x)
        dqp[(size_t)tok0 * d + e] = fXb[e];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < C * d; e += blockDim.x) dkp[(size_t)tok0 * d + e] = fKb[e];

    // ================= adjoints of A_C, E_C, B_C (state dot products)
    float pa = 0.f, pe = 0.f, pb = 0.f;
    for (size_t e = threadIdx.x; e < hd; e += blockDim.x) {
      pa += Wb1[e] * W1[e] + Wb2[e] * W2[e];
      pe += Wb1[e] * S1[e] + Wb2[e] * S2[e];
      pb += Sb1[e] * S1[e] + Sb2[e] * S2[e];
    }
    const float dAC = block_sum(pa, red);
    const float dEC = block_sum(pe, red);
    const float dBC = block_sum(pb, red);

    // ================= gate adjoints (wave 0; lanes are chunk positions)
    if (wave_id() == 0) {
      const int i = l;
      if (i < Cp) fCb[(size_t)(C - 1) * Cp + i] += gCC[i];
      if (i == 0) {
        gA[C - 1] += dAC;
        gE[C - 1] += dEC;
      }
    }
    __syncthreads();
    if (wave_id() == 0) {
      const int i = l;
      float eb = 0.f, rows = 0.f, cols = 0.f, Ui = 0.f;
      if (i < Cp) {
        // eta_bar, column sums, row sums of cbar o c
        for (int r = i; r < Cp; ++r) {
          const float cb = fCb[(size_t)r * Cp + i];
          eb += cb * cf.ct[r][i];
          cols += cb * cf.c[r][i];
        }
        eb += gB[i] * cf.ebt[i];
        for (int t = 0; t <= i; ++t) rows += fCb[(size_t)i * Cp + t] * cf.c[i][t];
        // U_{i, j}, j = 0..i
        float lbp = 0.f;
        for (int j = 0; j <= i; ++j) {
          Ui = expf(cf.lb[j] - lbp) * Ui + fCb[(size_t)i * Cp + j] * cf.eta[j];
          lbp = cf.lb[j];
          fU[(size_t)i * Cp + j] = Ui;
        }
      }
      gEta[i] = eb;
      gLa[i] = rows;
      gLb[i] = -cols;
    }
    __syncthreads();
    if (wave_id() == 0) {
      const int j = l;
      float la_b = 0.f, lb_b = 0.f;
      const float bsum = wave_sum(j < Cp ? gB[j] * cf.bb[j] : 0.f);
      if (j < C) {
        float T = 0.f, Yv = 0.f;
        for (int i = j; i < Cp; ++i) {
          const float w = expf(cf.la[i] - cf.la[j]);
          T += w * fU[(size_t)i * Cp + j];
          Yv += w * gE[i];
        }
        const float yl = Yv * expf(cf.lb[j]);
        la_b = gA[j] * cf.A[j] + gE[j] * cf.E[j] + gLa[j] - T - yl;
        lb_b = T + gLb[j] + yl - gB[j] * cf.bb[j];
        if (j == C - 1) lb_b += dBC * cf.BC + bsum;
      }
      // suffix sums over positions
      const float pla = wave_incl_sum(la_b), plb = wave_incl_sum(lb_b);
      const float tla = __shfl(pla, WAVE - 1, WAVE), tlb = __shfl(plb, WAVE - 1, WAVE);
      const float sla = tla - pla + la_b, slb = tlb - plb + lb_b;
      if (j < C) {
        const size_t t = (size_t)tok0 + j;
        const float al = dec[t], be = mom[t];
        dlr[t] = gEta[j];
        ddec[t] = -sla / (1.0f - al);
        dmom[t] = (logf(be) > LOG_CLAMP) ? slb / be : 0.f;
      }
    }
    __syncthreads();

    // ================= adjoint of the chunk-entry state (in place)
    tiles(h, d, [&](int i0, int j0) {  // W1bar, S1bar : h x d
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
      mma_tile<CT, KC, KC>(a1, ZbT, Cp, i0, XAT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a2, ZkbT, Cp, i0, KT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a3, ZbT, Cp, i0, XET, Cp, j0, Cp);
      f4 nw, ns;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * d + j0 + (l & 15);
        const float w = Wb1[e], sv = Sb1[e];
        float gp = a2[r];  // the gradient point's share
        if (hadj) {
          gp += hadj[e];
          hadj[e] = g_first ? 0.f : gp;
          if (!g_first) gp = 0.f;
        }
        nw[r] = cf.AC * w + a1[r] + gp;
        ns[r] = cf.EC * w + cf.BC * sv + a3[r];
        Wb1[e] = nw[r];
        Sb1[e] = ns[r];
      }
      // the lane's 4 rows are consecutive in the transposed copies
      const size_t et = (size_t)(j0 + (l & 15)) * h + i0 + 4 * (l >> 4);
      store4<CT>(Wb1T + et, nw);
      store4<CT>(Sb1T + et, ns);
    });
    tiles(d, h, [&](int i0, int j0) {  // W2bar, S2bar : d x h
      f4 a1 = zero4(), a2 = zero4(), a3 = zero4(), a4 = zero4();
      mma_tile<CT, KC, KC>(a1, dOAT, Cp, i0, HT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a2, RT, Cp, i0, GbT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a3, YkbT, Cp, i0, HkT, Cp, j0, Cp);
      mma_tile<CT, KC, KC>(a4, dOET, Cp, i0, HT, Cp, j0, Cp);
      f4 nw, ns;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * h + j0 + (l & 15);
        const float w = Wb2[e], sv = Sb2[e];
        float gp = a2[r] + a3[r];  // the gradient point's share
        if (hadj) {
          gp += hadj[hd + e];
          hadj[hd + e] = g_first ? 0.f : gp;
          if (!g_first) gp = 0.f;
        }
        nw[r] = cf.AC * w + a1[r] + gp;
        ns[r] = cf.EC * w + cf.BC * sv + a4[r];
        Wb2[e] = nw[r];
        Sb2[e] = ns[r];
      }
      const size_t et = (size_t)(j0 + (l & 15)) * d + i0 + 4 * (l >> 4);
      store4<CT>(Wb2T + et, nw);
      store4<CT>(Sb2T + et, ns);
    });
    if (shard_qk)
      tiles(d, d, [&](int i0, int j0) {
        f4 a1 = zero4();
        mma_tile<CT, KC, KC>(a1, XbT, Cp, i0, QT, Cp, j0, Cp);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * d + j0 + (l & 15);
          madj[e] += a1[r];
        }
      });
    __syncthreads();
  }
  // adjoint of the learned init for this unit
  float* dst = a.dWinit_part + (size_t)u * 2 * hd;
  for (size_t e = threadIdx.x; e < 2 * hd; e += blockDim.x) dst[e] = adj[e];
}

template <typename IO, typename CT, int ACT, int D_, int H_, int CP_>
static bool try_bwd(const LocalBwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (D_ && (a.D.d != D_ || a.D.hid != H_ || a.D.Cp != CP_)) return false;
  if (a.D.act != ACT) return false;
  hipLaunchKernelGGL((local_bwd_kernel<IO, CT, ACT, D_, H_, CP_>), dim3(units), dim3(512), 0,
                     st, a);
  *err = hipGetLastError();
  return true;
}

static hipError_t launch_local_bwd_rest(const LocalBwdArgs& a, int units, hipStream_t st);

hipError_t launch_local_bwd(const LocalBwdArgs& a, int units, hipStream_t st) {
  hipError_t e = hipSuccess;
  if (!a.force_generic && !a.single_walk && launch_local_bwd_split(a, units, st, &e)) return e;
  e = launch_local_bwd_rest(a, units, st);
  if (e == hipSuccess && a.pass_b_done) e = hipEventRecord(a.pass_b_done, st);
  return e;
}

// the one-walk kernels (fixed-size, then runtime-sized)
static hipError_t launch_local_bwd_rest(const LocalBwdArgs& a, int units, hipStream_t st) {
  hipError_t e = hipSuccess;
  // the other kernels recompute from the fp32 chunk-entry states, which a forward
  // that kept them in a ring did not save
  if (a.fslots) return hipErrorInvalidValue;
  if (a.pass_a_done) {
    e = hipEventRecord(a.pass_a_done, st);
    if (e != hipSuccess) return e;
  }
  if (!a.force_generic && launch_local_bwd_blk(a, units, st, &e)) return e;
  if (a.D.bf16) {
    if (try_bwd<__bf16, __bf16, ACT_GELU, 0, 0, 0>(a, units, st, &e) ||
        try_bwd<__bf16, __bf16, ACT_SILU, 0, 0, 0>(a, units, st, &e))
      return e;
  } else {
    if (try_bwd<float, float, ACT_GELU, 0, 0, 0>(a, units, st, &e) ||
        try_bwd<float, float, ACT_SILU, 0, 0, 0>(a, units, st, &e))
      return e;
  }
  return hipErrorInvalidValue;
}

// dW_init[h] = sum over batch rows and shards of the per-unit adjoints
__global__ void reduce_init_kernel(const float* parts, int B, int H, int nshard, size_t hd,
                                   float* dW1, float* dW2) {
  const int hh = blockIdx.y;
  for (size_t e = blockIdx.x * blockDim.x + threadIdx.x; e < 2 * hd;
       e += gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int b = 0; b < B; ++b)
      for (int sh = 0; sh < nshard; ++sh)
        s += parts[(((size_t)b * H + hh) * nshard + sh) * 2 * hd + e];
    if (e < hd)
      dW1[(size_t)hh * hd + e] = s;
    else
      dW2[(size_t)hh * hd + e - hd] = s;
  }
}

hipError_t launch_reduce_init(const float* parts, int B, int H, int nshard, size_t hd2,
                              float* dW1, float* dW2, int d, int hid, int accumulate,
                              hipStream_t st) {
  (void)accumulate;
  (void)d;
  (void)hid;
  const size_t hd = hd2 / 2;
  hipLaunchKernelGGL(reduce_init_kernel, dim3(32, H), dim3(256), 0, st, parts, B, H, nshard, hd,
                     dW1, dW2);
  return hipGetLastError();
}


// Transposed compute-type copies of the saved chunk-entry states, one
// 32 x 32 tile per workgroup and slot: W1 (hid x d) -> W1^T, W2 (d x hid) ->
// W2^T, S1, S2 likewise, and the Q-K sum M (d x d) -> M^T when `with_m`.
// `slots` = units * nslots; out holds 4*hid*d + d*d elements per slot.
template <typename CT>
__global__ void __launch_bounds__(256) pack_states_kernel(const float* st, const float* mst, CT* out,
                                                          size_t slots, int d, int h, int with_m) {
  __shared__ float t[32][33];
  const int m = blockIdx.z;
  if (m == 4 && !with_m) return;
  const size_t hd = (size_t)h * d, slot = 4 * hd + (size_t)d * d;
  const int R = (m == 4 || (m & 1)) ? d : h, Cc = (m != 4 && (m & 1)) ? h : d;
  const int tc = (Cc + 31) / 32, ntiles = ((R + 31) / 32) * tc;
  if ((int)blockIdx.x >= ntiles) return;
  const int r0 = (blockIdx.x / tc) * 32, c0 = (blockIdx.x % tc) * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (size_t z = blockIdx.y; z < slots; z += gridDim.y) {
    const float* src = m == 4 ? mst + z * d * d : st + z * 4 * hd + m * hd;
    CT* dst = out + z * slot + (m == 4 ? 4 * hd : m * hd);
    for (int k = ty; k < 32; k += 8) {
      const int r = r0 + k, c = c0 + tx;
      t[k][tx] = (r < R && c < Cc) ? src[(size_t)r * Cc + c] : 0.f;
    }
    __syncthreads();
    for (int k = ty; k < 32; k += 8) {
      const int c = c0 + k, r = r0 + tx;
      if (c < Cc && r < R) dst[(size_t)c * R + r] = from_f<CT>(t[tx][k]);
    }
    __syncthreads();
  }
}

hipError_t launch_pack_states(const float* states, const float* mstates, void* out, int units,
                              int nslots, int d, int hid, int with_m, int bf16, hipStream_t st) {
  const int tiles = ((hid + 31) / 32) * ((d + 31) / 32);
  const size_t slots = (size_t)units * nslots;
  const dim3 grid(tiles, (unsigned)std::min<size_t>(slots, 65535), 5);
  if (bf16)
    hipLaunchKernelGGL(pack_states_kernel<__bf16>, grid, dim3(256), 0, st, states, mstates,
                       (__bf16*)out, slots, d, hid, with_m);
  else
    hipLaunchKernelGGL(pack_states_kernel<float>, grid, dim3(256), 0, st, states, mstates,
                       (float*)out, slots, d, hid, with_m);
  return hipGetLastError();
}

}  // namespace tnt
