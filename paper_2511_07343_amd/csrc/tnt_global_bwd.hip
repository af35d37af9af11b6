// Global memory, backward.  The chain of global chunks is walked in reverse;
// each chunk n runs
//   phaseA (token tiles, all hidden units): recompute Zk, Hk, R, G, D1 and the
//     retrieval at the chunk-entry state V, then the per-token adjoints
//       D1bar = -diag(cC) K V1bar'^T - diag(b) K S1bar'^T,  Gbar = D1bar * s'(Zk)
//       Rbar  = -diag(cC) Hk V2bar'^T - diag(b) Hk S2bar'^T + Gbar V2^T
//       Hkbar = -diag(cC) R V2bar' - diag(b) R S2bar' + (2/d) Rbar V2
//       Zkbar = Hkbar * s'(Zk) + D1bar * G * s''(Zk)
//       Kbar  = -diag(cC) D1 V1bar' - diag(b) D1 S1bar' + Zkbar V1
//       Qbar  = ((dO V2) * s'(Q V1^T)) V1,  Vbar = -(2/d) Rbar
//     and the adjoints of the chunk coefficients cC_t, b_t;
//   phaseB (hidden slices, all tokens of the chunk): the adjoint of the
//     chunk-entry state
//       V1bar = A_C V1bar' + Zkbar^T K + Zqbar^T Q,      S1bar = E_C V1bar' + B_C S1bar'
//       V2bar = A_C V2bar' + R^T Gbar + Ykbar^T Hk + dO^T Hq,  S2bar = E_C V2bar' + B_C S2bar'
//     recomputing the slice's hidden activations from per-token vectors, plus
//     the state dot products that give the adjoints of A_C, E_C, B_C;
// and finally one scan per chunk turns the coefficient adjoints into
// gradients of lr, mom and decay.
#include "tnt_device.h"
#include "tnt_kernels.h"

#include <algorithm>

namespace tnt {

template <typename F>
__device__ __forceinline__ void gtiles(int M, int N, F&& f) {
  const int tn = N >> 4, nt = (M >> 4) * tn;
  for (int t = wave_id(); t < nt; t += num_waves()) f((t / tn) << 4, (t % tn) << 4);
}

constexpr int GB_TT = 32;  // tokens per phase-A workgroup

// per-workgroup scratch of phase A (CT elements / fp32 elements)
struct GbaLayout {
  size_t K, Q, dO, R, Hk, Sp, Spp, G, D1, Gb, Ykb, Zkb, Zqb, ct_elems;
  size_t T3, T4, T5, T6, Zkp, f_elems;
};
__host__ __device__ inline void gba_layout(int d, int h, GbaLayout* y) {
  const size_t Td = (size_t)GB_TT * d, Th = (size_t)GB_TT * h;
  size_t o = 0;
  y->K = o; o += Td; y->Q = o; o += Td; y->dO = o; o += Td; y->R = o; o += Td;
  y->Hk = o; o += Th; y->Sp = o; o += Th; y->Spp = o; o += Th; y->G = o; o += Th;
  y->D1 = o; o += Th; y->Gb = o; o += Th; y->Ykb = o; o += Td; y->Zkb = o; o += Th;
  y->Zqb = o; o += Th;
  y->ct_elems = o;
  o = 0;
  y->T3 = o; o += Td; y->T4 = o; o += Td; y->T5 = o; o += Td; y->T6 = o; o += Td;
  y->Zkp = o; o += Th;
  y->f_elems = o;
}

size_t global_bwd_scratch_bytes(const Dims& D, size_t* f32_off) {
  GbaLayout y;
  gba_layout(D.d, D.hid, &y);
  const size_t wgs = (size_t)((D.C + GB_TT - 1) / GB_TT) * D.B * D.H;
  const size_t cts = D.bf16 ? 2 : 4;
  const size_t ct_bytes = (wgs * y.ct_elems * cts + 255) & ~size_t(255);
  *f32_off = ct_bytes;
  return ct_bytes + wgs * y.f_elems * sizeof(float);
}

template <typename IO, typename CT, int ACT, int D_, int H_>
__global__ void __launch_bounds__(256) gbwd_a_kernel(GlobalArgs a, int n, void* scratch,
                                                     size_t f32_off) {
  const Dims D = a.D;
  const int d = D_ ? D_ : D.d, h = H_ ? H_ : D.hid, C = D.C;
  const int chain = blockIdx.y;
  const int r0 = blockIdx.x * GB_TT;
  const int rows = min(GB_TT, C - r0);
  const size_t hd = (size_t)h * d;
  const int l = lane_id();
  constexpr int TT = GB_TT;
  GbaLayout Y;
  gba_layout(d, h, &Y);
  const size_t wg = (size_t)chain * gridDim.x + blockIdx.x;
  CT* sc = (CT*)scratch + wg * Y.ct_elems;
  float* sf = (float*)((char*)scratch + f32_off) + wg * Y.f_elems;
  CT *sK = sc + Y.K, *sQ = sc + Y.Q, *sdO = sc + Y.dO, *sR = sc + Y.R, *sHk = sc + Y.Hk,
     *sSp = sc + Y.Sp, *sSpp = sc + Y.Spp, *sG = sc + Y.G, *sD1 = sc + Y.D1, *sGb = sc + Y.Gb,
     *sYkb = sc + Y.Ykb, *sZkb = sc + Y.Zkb, *sZqb = sc + Y.Zqb;
  float *fT3 = sf + Y.T3, *fT4 = sf + Y.T4, *fT5 = sf + Y.T5, *fT6 = sf + Y.T6,
        *fZkp = sf + Y.Zkp;

  const float* V = a.states + ((size_t)chain * a.nslots + n) * 4 * hd;
  const float *V1 = V, *V2 = V + hd;
  const float* Ab = a.adj + ((size_t)chain * 2 + ((n + 1) & 1)) * 4 * hd;  // adjoint of V_{n+1}
  const float *Vb1 = Ab, *Vb2 = Ab + hd, *Sb1 = Ab + 2 * hd, *Sb2 = Ab + 3 * hd;
  const size_t tok0 = (size_t)n * C + r0;
  const size_t cb = (size_t)chain * D.L + tok0;
  const IO* q = (const IO*)a.q + cb * d;
  const IO* k = (const IO*)a.k + cb * d;
  const IO* v = (const IO*)a.v + cb * d;
  const IO* dO = (const IO*)a.dO + cb * d;
  const float* tk = a.tokc + cb * TKS;
  float* dtk = a.dtok + cb * 4;
  float* Rg = a.Rbuf + ((size_t)chain * C + r0) * d;
  float* dRg = a.dRbuf + ((size_t)chain * C + r0) * d;
  float* dqp = a.dq_part + cb * d;
  float* dkp = a.dk_part + cb * d;
  float* dvp = a.dv_part + cb * d;
  const float rscale = 2.0f / (float)d;
  __shared__ float cC[TT], bb[TT];

  for (int e = threadIdx.x; e < TT * d; e += blockDim.x) {
    const int i = e / d;
    const bool in = i < rows;
    sK[e] = from_f<CT>(in ? to_f(k[e]) : 0.f);
    sQ[e] = from_f<CT>(in ? to_f(q[e]) : 0.f);
    sdO[e] = from_f<CT>(in ? to_f(dO[e]) : 0.f);
  }
  if (threadIdx.x < TT) {
    const int i = threadIdx.x;
    cC[i] = i < rows ? tk[(size_t)i * TKS + 0] : 0.f;
    bb[i] = i < rows ? tk[(size_t)i * TKS + 1] : 0.f;
  }
  __syncthreads();
  // Zk -> Hk, s', s'' ; Zq -> s'(Zq) ; Zqbar = (dO V2) * s'(Zq)
  gtiles(TT, h, [&](int i0, int j0) {
    f4 az = zero4(), aq = zero4(), ap = zero4();
    mma_tile<CT, KC, KC>(az, sK, d, i0, V1, d, j0, d);
    mma_tile<CT, KC, KC>(aq, sQ, d, i0, V1, d, j0, d);
    mma_tile<CT, KC, MC>(ap, sdO, d, i0, V2, h, j0, d);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * h + j0 + (l & 15);
      const ActVals z = act_all<ACT>(az[r]);
      const ActVals zq = act_all<ACT>(aq[r]);
      sHk[e] = from_f<CT>(z.s);
      sSp[e] = from_f<CT>(z.d1);
      sSpp[e] = from_f<CT>(z.d2);
      sZqb[e] = from_f<CT>(ap[r] * zq.d1);
    }
  });
  __syncthreads();
  // R = (2/d)(Hk V2^T - V) ; T5 = Hk V2bar'^T ; T6 = Hk S2bar'^T ; Qbar = Zqbar V1
  gtiles(TT, d, [&](int i0, int j0) {
    f4 ay = zero4(), a5 = zero4(), a6 = zero4(), aq = zero4();
    mma_tile<CT, KC, KC>(ay, sHk, h, i0, V2, h, j0, h);
    mma_tile<CT, KC, KC>(a5, sHk, h, i0, Vb2, h, j0, h);
    mma_tile<CT, KC, KC>(a6, sHk, h, i0, Sb2, h, j0, h);
    mma_tile<CT, KC, MC>(aq, sZqb, h, i0, V1, d, j0, h);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
      const size_t e = (size_t)i * d + j;
      const float rv = i < rows ? rscale * (ay[r] - to_f(v[e])) : 0.f;
      sR[e] = from_f<CT>(rv);
      fT5[e] = a5[r];
      fT6[e] = a6[r];
      if (i < rows) {
        Rg[e] = rv;
        dqp[e] = aq[r];
      }
    }
  });
  __syncthreads();
  // G = R V2 ; D1 = G s' ; D1bar = -cC K V1bar'^T - b K S1bar'^T ; Gbar, Zkbar part
  gtiles(TT, h, [&](int i0, int j0) {
    f4 ag = zero4(), a1 = zero4(), a2 = zero4();
    mma_tile<CT, KC, MC>(ag, sR, d, i0, V2, h, j0, d);
    mma_tile<CT, KC, KC>(a1, sK, d, i0, Vb1, d, j0, d);
    mma_tile<CT, KC, KC>(a2, sK, d, i0, Sb1, d, j0, d);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 4 * (l >> 4) + r;
      const size_t e = (size_t)i * h + j0 + (l & 15);
      const float sp = to_f(sSp[e]);
      const float d1b = -cC[i] * a1[r] - bb[i] * a2[r];
      sG[e] = from_f<CT>(ag[r]);
      sD1[e] = from_f<CT>(ag[r] * sp);
      sGb[e] = from_f<CT>(d1b * sp);
      fZkp[e] = d1b * ag[r] * to_f(sSpp[e]);
    }
  });
  __syncthreads();
  // T3 = D1 V1bar', T4 = D1 S1bar' ; Rbar = -cC T5 - b T6 + Gbar V2^T ; Ykbar ; Vbar
  gtiles(TT, d, [&](int i0, int j0) {
    f4 a3 = zero4(), a4 = zero4(), ag = zero4();
    mma_tile<CT, KC, MC>(a3, sD1, h, i0, Vb1, d, j0, h);
    mma_tile<CT, KC, MC>(a4, sD1, h, i0, Sb1, d, j0, h);
    mma_tile<CT, KC, KC>(ag, sGb, h, i0, V2, h, j0, h);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
      const size_t e = (size_t)i * d + j;
      fT3[e] = a3[r];
      fT4[e] = a4[r];
      const float rb = -cC[i] * fT5[e] - bb[i] * fT6[e] + ag[r];
      const float ykb = i < rows ? rscale * rb : 0.f;
      sYkb[e] = from_f<CT>(ykb);
      if (i < rows) {
        dRg[e] = ykb;
        dvp[e] = -ykb;
      }
    }
  });
  __syncthreads();
  // adjoints of cC_t, b_t (row dots over d)
  for (int i = wave_id(); i < rows; i += num_waves()) {
    float s1 = 0.f, s2 = 0.f;
    for (int j = l; j < d; j += WAVE) {
      const size_t e = (size_t)i * d + j;
      const float kx = to_f(sK[e]), rx = to_f(sR[e]);
      s1 += kx * fT3[e] + rx * fT5[e];
      s2 += kx * fT4[e] + rx * fT6[e];
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    if (l == 0) {
      dtk[(size_t)i * 4 + 0] = -s1;
      dtk[(size_t)i * 4 + 1] = -s2;
    }
  }
  // Hkbar = -cC R V2bar' - b R S2bar' + Ykbar V2 ; Zkbar
  gtiles(TT, h, [&](int i0, int j0) {
    f4 a7 = zero4(), a8 = zero4(), ay = zero4();
    mma_tile<CT, KC, MC>(a7, sR, d, i0, Vb2, h, j0, d);
    mma_tile<CT, KC, MC>(a8, sR, d, i0, Sb2, h, j0, d);
    mma_tile<CT, KC, MC>(ay, sYkb, d, i0, V2, h, j0, d);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 4 * (l >> 4) + r;
      const size_t e = (size_t)i * h + j0 + (l & 15);
      const float hkb = -cC[i] * a7[r] - bb[i] * a8[r] + ay[r];
      sZkb[e] = from_f<CT>(hkb * to_f(sSp[e]) + fZkp[e]);
    }
  });
  __syncthreads();
  // Kbar = -cC T3 - b T4 + Zkbar V1
  gtiles(TT, d, [&](int i0, int j0) {
    f4 ak = zero4();
    mma_tile<CT, KC, MC>(ak, sZkb, h, i0, V1, d, j0, h);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
      const size_t e = (size_t)i * d + j;
      if (i < rows) dkp[e] = -cC[i] * fT3[e] - bb[i] * fT4[e] + ak[r];
    }
  });
}

// ---- phase B: adjoint of the chunk-entry state, one hidden slice per workgroup
constexpr int GBB_HS = 16;
constexpr int GBB_TT = 32;

template <typename IO, typename CT, int ACT, int D_, int H_>
__global__ void __launch_bounds__(256) gbwd_b_kernel(GlobalArgs a, int n) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Dims D = a.D;
  const int d = D_ ? D_ : D.d, h = H_ ? H_ : D.hid, C = D.C;
  const int chain = blockIdx.z;
  const int s0 = blockIdx.x * GBB_HS;
  const int split = blockIdx.y, nsplit = gridDim.y;
  const size_t hd = (size_t)h * d;
  const int l = lane_id();
  constexpr int TT = GBB_TT, HS = GBB_HS;
  const float* V = a.states + ((size_t)chain * a.nslots + n) * 4 * hd;
  const float *V1 = V, *V2 = V + hd;
  const float* Ab = a.adj + ((size_t)chain * 2 + ((n + 1) & 1)) * 4 * hd;
  const float *Vb1 = Ab, *Vb2 = Ab + hd, *Sb1 = Ab + 2 * hd, *Sb2 = Ab + 3 * hd;
  float* P = a.part + ((size_t)chain * nsplit + split) * 4 * hd;
  CT* sK = (CT*)smem;            // [TT][d]
  CT* sQ = sK + TT * d;
  CT* sdO = sQ + TT * d;
  CT* sR = sdO + TT * d;
  CT* sYk = sR + TT * d;
  CT* sKT = sYk + TT * d;        // [d][TT]
  CT* sQT = sKT + TT * d;
  CT* sdOT = sQT + TT * d;
  CT* sRT = sdOT + TT * d;
  CT* sYkT = sRT + TT * d;
  CT* sZkbT = sYkT + TT * d;     // [HS][TT]
  CT* sZqbT = sZkbT + HS * TT;
  CT* sGbT = sZqbT + HS * TT;
  CT* sHkT = sGbT + HS * TT;
  CT* sHqT = sHkT + HS * TT;
  __shared__ float cC[TT], bb[TT];
  const size_t cb0 = (size_t)chain * D.L + (size_t)n * C;
  const IO* qg = (const IO*)a.q + cb0 * d;
  const IO* kg = (const IO*)a.k + cb0 * d;
  const IO* dOg = (const IO*)a.dO + cb0 * d;
  const float* tk = a.tokc + cb0 * TKS;
  const float* Rg = a.Rbuf + (size_t)chain * C * d;
  const float* dRg = a.dRbuf + (size_t)chain * C * d;

  const int nt1 = d >> 4;
  f4 av1[2], av2[2];
  for (int x = 0; x < 2; ++x) av1[x] = av2[x] = zero4();

  const int ntile = (C + TT - 1) / TT;
  const int tb = split * ntile / nsplit, te = (split + 1) * ntile / nsplit;
  for (int r0 = tb * TT; r0 < te * TT; r0 += TT) {
    const int rows = min(TT, C - r0);
    for (int e = threadIdx.x; e < TT * d; e += blockDim.x) {
      const int i = e / d, j = e - i * d;
      const bool in = i < rows;
      const size_t g = (size_t)(r0 + i) * d + j;
      const float kx = in ? to_f(kg[g]) : 0.f, qx = in ? to_f(qg[g]) : 0.f;
      const float ox = in ? to_f(dOg[g]) : 0.f, rx = in ? Rg[g] : 0.f, yx = in ? dRg[g] : 0.f;
      sK[e] = from_f<CT>(kx); sQ[e] = from_f<CT>(qx); sdO[e] = from_f<CT>(ox);
      sR[e] = from_f<CT>(rx); sYk[e] = from_f<CT>(yx);
      const size_t et = (size_t)j * TT + i;
      sKT[et] = from_f<CT>(kx); sQT[et] = from_f<CT>(qx); sdOT[et] = from_f<CT>(ox);
      sRT[et] = from_f<CT>(rx); sYkT[et] = from_f<CT>(yx);
    }
    if (threadIdx.x < TT) {
      const int i = threadIdx.x;
      cC[i] = i < rows ? tk[(size_t)(r0 + i) * TKS + 0] : 0.f;
      bb[i] = i < rows ? tk[(size_t)(r0 + i) * TKS + 1] : 0.f;
    }
    __syncthreads();
    for (int t = wave_id(); t < TT / 16; t += num_waves()) {
      const int i0 = t * 16;
      f4 az = zero4(), ag = zero4(), a1 = zero4(), a2 = zero4(), a7 = zero4(), a8 = zero4(),
         ay = zero4(), aq = zero4(), ap = zero4();
      mma_tile<CT, KC, KC>(az, sK, d, i0, V1 + (size_t)s0 * d, d, 0, d);
      mma_tile<CT, KC, MC>(ag, sR, d, i0, V2 + s0, h, 0, d);
      mma_tile<CT, KC, KC>(a1, sK, d, i0, Vb1 + (size_t)s0 * d, d, 0, d);
      mma_tile<CT, KC, KC>(a2, sK, d, i0, Sb1 + (size_t)s0 * d, d, 0, d);
      mma_tile<CT, KC, MC>(a7, sR, d, i0, Vb2 + s0, h, 0, d);
      mma_tile<CT, KC, MC>(a8, sR, d, i0, Sb2 + s0, h, 0, d);
      mma_tile<CT, KC, MC>(ay, sYk, d, i0, V2 + s0, h, 0, d);
      mma_tile<CT, KC, KC>(aq, sQ, d, i0, V1 + (size_t)s0 * d, d, 0, d);
      mma_tile<CT, KC, MC>(ap, sdO, d, i0, V2 + s0, h, 0, d);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = l & 15;
        const ActVals z = act_all<ACT>(az[r]);
        const ActVals zq = act_all<ACT>(aq[r]);
        const float d1b = -cC[i] * a1[r] - bb[i] * a2[r];
        const float gb = d1b * z.d1;
        const float hkb = -cC[i] * a7[r] - bb[i] * a8[r] + ay[r];
        const float zkb = hkb * z.d1 + d1b * ag[r] * z.d2;
        const size_t et = (size_t)j * TT + i;
        sZkbT[et] = from_f<CT>(zkb);
        sZqbT[et] = from_f<CT>(ap[r] * zq.d1);
        sGbT[et] = from_f<CT>(gb);
        sHkT[et] = from_f<CT>(z.s);
        sHqT[et] = from_f<CT>(zq.s);
      }
    }
    __syncthreads();
    for (int x = 0, t = wave_id(); t < nt1; t += num_waves(), ++x) {
      const int j0 = t * 16;
      mma_tile<CT, KC, KC>(av1[x], sZkbT, TT, 0, sKT, TT, j0, TT);
      mma_tile<CT, KC, KC>(av1[x], sZqbT, TT, 0, sQT, TT, j0, TT);
      mma_tile<CT, KC, KC>(av2[x], sRT, TT, j0, sGbT, TT, 0, TT);
      mma_tile<CT, KC, KC>(av2[x], sYkT, TT, j0, sHkT, TT, 0, TT);
      mma_tile<CT, KC, KC>(av2[x], sdOT, TT, j0, sHqT, TT, 0, TT);
    }
    __syncthreads();
  }
  // partial sums of this token split (combined in fixed order by gbwd_state_reduce)
  for (int x = 0, t = wave_id(); t < nt1; t += num_waves(), ++x) {
    const int j0 = t * 16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      {
        const int i = 4 * (l >> 4) + r, j = j0 + (l & 15);
        P[(size_t)(s0 + i) * d + j] = av1[x][r];
      }
      {
        const int i = j0 + 4 * (l >> 4) + r, j = l & 15;
        P[hd + (size_t)i * h + s0 + j] = av2[x][r];
      }
    }
  }
}

// adjoint of the chunk-entry state from the split partials (fixed order):
//   V1bar = A_C V1bar' + sum dV1,  S1bar = E_C V1bar' + B_C S1bar'   (and V2, S2 alike)
// plus the state dot products that give the adjoints of A_C, E_C, B_C.
__global__ void __launch_bounds__(256) gbwd_state_reduce(GlobalArgs a, int n, int nsplit) {
  const Dims D = a.D;
  const int chain = blockIdx.y;
  const size_t hd = (size_t)D.hid * D.d;
  const float* V = a.states + ((size_t)chain * a.nslots + n) * 4 * hd;
  const float* Ab = a.adj + ((size_t)chain * 2 + ((n + 1) & 1)) * 4 * hd;
  float* An = a.adj + ((size_t)chain * 2 + (n & 1)) * 4 * hd;
  const float* P = a.part + (size_t)chain * nsplit * 4 * hd;
  const float* cc = a.chunkc + ((size_t)chain * (D.L / D.C) + n) * 4;
  const float AC = cc[0], BC = cc[1], EC = cc[2];
  __shared__ float red[16];
  float pa = 0.f, pe = 0.f, pb = 0.f;
  for (size_t e4 = blockIdx.x * blockDim.x + threadIdx.x; e4 < hd / 4;
       e4 += gridDim.x * blockDim.x) {
    const size_t e = e4 * 4;
#pragma unroll
    for (int m = 0; m < 2; ++m) {  // m = 0: (V1, S1), m = 1: (V2, S2)
      const size_t ew = (size_t)m * hd + e, es = (size_t)(2 + m) * hd + e;
      f32x4 dv = {0.f, 0.f, 0.f, 0.f};
      for (int sp = 0; sp < nsplit; ++sp)
        dv += *reinterpret_cast<const f32x4*>(P + (size_t)sp * 4 * hd + ew);
      const f32x4 w = *reinterpret_cast<const f32x4*>(Ab + ew);
      const f32x4 sv = *reinterpret_cast<const f32x4*>(Ab + es);
      const f32x4 vw = *reinterpret_cast<const f32x4*>(V + ew);
      const f32x4 vs = *reinterpret_cast<const f32x4*>(V + es);
      const f32x4 nw = AC * w + dv;
      *reinterpret_cast<f32x4*>(An + ew) = nw;
      *reinterpret_cast<f32x4*>(An + es) = EC * w + BC * sv;
      if (n == 0) *reinterpret_cast<f32x4*>(a.dWinit + (size_t)chain * 2 * hd + ew) = nw;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        pa += w[j] * vw[j];
        pe += w[j] * vs[j];
        pb += sv[j] * vs[j];
      }
    }
  }
  pa = block_sum(pa, red);
  pe = block_sum(pe, red);
  pb = block_sum(pb, red);
  if (threadIdx.x == 0) {
    float* dc = a.dchunk + (((size_t)chain * (D.L / D.C) + n) * gridDim.x + blockIdx.x) * 4;
    dc[0] = pa;
    dc[1] = pe;
    dc[2] = pb;
    dc[3] = 0.f;
  }
}

hipError_t launch_gbwd_state_reduce(const GlobalArgs& a, int n, int nsplit, hipStream_t st) {
  hipLaunchKernelGGL(gbwd_state_reduce, dim3(GRED_BLOCKS, a.D.B * a.D.H), dim3(256), 0, st, a, n,
                     nsplit);
  return hipGetLastError();
}

int global_bwd_splits(const Dims& D) {
  const int tiles = (D.C + GBB_TT - 1) / GBB_TT;
  return std::max(1, std::min(16, tiles / 4));
}

template <typename IO, typename CT, int ACT, int D_, int H_>
static hipError_t launch_gbwd_dims(const GlobalArgs& a, int n, void* scratch, size_t f32_off,
                                   hipStream_t st) {
  const Dims& D = a.D;
  dim3 ga((D.C + GB_TT - 1) / GB_TT, D.B * D.H);
  hipLaunchKernelGGL((gbwd_a_kernel<IO, CT, ACT, D_, H_>), ga, dim3(256), 0, st, a, n, scratch, f32_off);
  const int ns = global_bwd_splits(D);
  dim3 gb(D.hid / GBB_HS, ns, D.B * D.H);
  const size_t lds = (10 * (size_t)GBB_TT * D.d + 5 * GBB_HS * GBB_TT) * sizeof(CT);
  set_lds_limit((const void*)gbwd_b_kernel<IO, CT, ACT, D_, H_>);
  hipLaunchKernelGGL((gbwd_b_kernel<IO, CT, ACT, D_, H_>), gb, dim3(256), lds, st, a, n);
  hipLaunchKernelGGL(gbwd_state_reduce, dim3(GRED_BLOCKS, D.B * D.H), dim3(256), 0, st, a, n, ns);
  return hipGetLastError();
}

template <typename IO, typename CT, int ACT>
static hipError_t launch_gbwd_t(const GlobalArgs& a, int n, void* scratch, size_t f32_off,
                                hipStream_t st) {
  if (!a.force_generic) {
    if constexpr (sizeof(IO) == 2) {
      if (a.D.d == 64 && a.D.hid == 256)
        return launch_gbwd_dims<IO, CT, ACT, 64, 256>(a, n, scratch, f32_off, st);
      if (a.D.d == 128 && a.D.hid == 512)
        return launch_gbwd_dims<IO, CT, ACT, 128, 512>(a, n, scratch, f32_off, st);
    } else {
      if (a.D.d == 16 && a.D.hid == 32)
        return launch_gbwd_dims<IO, CT, ACT, 16, 32>(a, n, scratch, f32_off, st);
    }
  }
  return launch_gbwd_dims<IO, CT, ACT, 0, 0>(a, n, scratch, f32_off, st);
}

hipError_t launch_global_bwd_chunk(const GlobalArgs& a, int n, hipStream_t st) {
  hipError_t err = hipSuccess;
  if (launch_global_bwd_blk(a, n, st, &err)) return err;
  void* sc = a.scratch;
  const size_t fo = a.scratch_f32_off;
  if (a.D.bf16)
    return a.D.act == ACT_GELU ? launch_gbwd_t<__bf16, __bf16, ACT_GELU>(a, n, sc, fo, st)
                               : launch_gbwd_t<__bf16, __bf16, ACT_SILU>(a, n, sc, fo, st);
  return a.D.act == ACT_GELU ? launch_gbwd_t<float, float, ACT_GELU>(a, n, sc, fo, st)
                             : launch_gbwd_t<float, float, ACT_SILU>(a, n, sc, fo, st);
}

// zero the adjoint slot that chunk L/C - 1 reads
__global__ void gbwd_zero_kernel(GlobalArgs a, int slot) {
  const size_t hd = (size_t)a.D.hid * a.D.d;
  float* p = a.adj + ((size_t)blockIdx.y * 2 + slot) * 4 * hd;
  for (size_t e = blockIdx.x * blockDim.x + threadIdx.x; e < 4 * hd; e += gridDim.x * blockDim.x)
    p[e] = 0.f;
}

hipError_t launch_global_bwd_zero(const GlobalArgs& a, int slot, hipStream_t st) {
  hipLaunchKernelGGL(gbwd_zero_kernel, dim3(16, a.D.B * a.D.H), dim3(256), 0, st, a, slot);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// gate adjoints of one global chunk (one wavefront per (chunk, chain)).  With
// F_m = sum_{t<=m} cCbar_t eta_t e^{lb_m - lb_t} (forward affine scan),
//   la_bar_m = -e^{la_C - la_m} (F_m + Ebar_C e^{lb_m})       (+ sum cCbar cC + Abar A_C + Ebar E_C at m = C-1)
//   lb_bar_m =  e^{la_C - la_m} (F_m + Ebar_C e^{lb_m}) - cCbar_m cC_m - bbar_m b_m
//                                                         (+ sum bbar b + Bbar B_C at m = C-1)
//   eta_bar_m = cCbar_m s_m + bbar_m e^{lb_C - lb_m}
// then suffix sums give the decay and momentum gradients.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(64) global_gate_bwd_kernel(GlobalArgs a, int nslices) {
  const int n = blockIdx.x, chain = blockIdx.y;
  const int C = a.D.C, L = a.D.L;
  const size_t base = (size_t)chain * L + (size_t)n * C;
  const float* lr = a.lr + base;
  const float* mom = a.mom + base;
  const float* dec = a.decay + base;
  const float* tk = a.tokc + base * TKS;
  const float* dtk = a.dtok + base * 4;
  float* dlr = a.dlr + base;
  float* dmom = a.dmom + base;
  float* ddec = a.ddecay + base;
  const int l = lane_id();
  const int E = (C + WAVE - 1) / WAVE;
  const int i0 = min(l * E, C), i1 = min(i0 + E, C);
  const float* cc = a.chunkc + ((size_t)chain * (L / C) + n) * 4;
  const float AC = cc[0], BC = cc[1], EC = cc[2];
  float dAC = 0.f, dEC = 0.f, dBC = 0.f;
  {
    const float* dc = a.dchunk + ((size_t)chain * (L / C) + n) * nslices * 4;
    for (int s = 0; s < nslices; ++s) {
      dAC += dc[s * 4 + 0];
      dEC += dc[s * 4 + 1];
      dBC += dc[s * 4 + 2];
    }
  }
  const float laC = tk[(size_t)(C - 1) * TKS + 2];
  // sums over the chunk: sum cCbar cC, sum bbar b
  float scc = 0.f, sbb = 0.f;
  for (int i = i0; i < i1; ++i) {
    scc += dtk[(size_t)i * 4 + 0] * tk[(size_t)i * TKS + 0];
    sbb += dtk[(size_t)i * 4 + 1] * tk[(size_t)i * TKS + 1];
  }
  scc = wave_sum(scc);
  sbb = wave_sum(sbb);
  // forward affine scan F_m = beta_m F_{m-1} + x_m, x_m = cCbar_m eta_m
  float P = 1.f, Q = 0.f;  // segment map F_out = P F_in + Q
  for (int i = i0; i < i1; ++i) {
    const float bm = mom[i];
    Q = bm * Q + dtk[(size_t)i * 4 + 0] * lr[i];
    P = bm * P;
  }
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    const float Pp = __shfl_up(P, o, WAVE), Qp = __shfl_up(Q, o, WAVE);
    if (l >= o) {  // compose: this segment after the earlier ones
      Q = P * Qp + Q;
      P = P * Pp;
    }
  }
  float Fin = __shfl_up(Q, 1, WAVE);
  if (l == 0) Fin = 0.f;
  // per-token la_bar, lb_bar and the segment's sums (pass 1), then suffix sums (pass 2)
  float F = Fin, segA = 0.f, segB = 0.f;
  for (int i = i0; i < i1; ++i) {
    F = mom[i] * F + dtk[(size_t)i * 4 + 0] * lr[i];
    const float la = tk[(size_t)i * TKS + 2], lb = tk[(size_t)i * TKS + 3];
    const float w = expf(laC - la) * F + dEC * expf(laC - la + lb);
    float lab = -w, lbb = w - dtk[(size_t)i * 4 + 0] * tk[(size_t)i * TKS + 0] -
                          dtk[(size_t)i * 4 + 1] * tk[(size_t)i * TKS + 1];
    if (i == C - 1) {
      lab += scc + dAC * AC + dEC * EC;
      lbb += sbb + dBC * BC;
    }
    segA += lab;
    segB += lbb;
  }
  const float ia = wave_incl_sum(segA), ib = wave_incl_sum(segB);
  const float ta = __shfl(ia, WAVE - 1, WAVE), tb = __shfl(ib, WAVE - 1, WAVE);
  float sufA = ta - ia + segA, sufB = tb - ib + segB;  // sum over i >= i0
  F = Fin;
  for (int i = i0; i < i1; ++i) {
    F = mom[i] * F + dtk[(size_t)i * 4 + 0] * lr[i];
    const float la = tk[(size_t)i * TKS + 2], lb = tk[(size_t)i * TKS + 3];
    const float w = expf(laC - la) * F + dEC * expf(laC - la + lb);
    float lab = -w, lbb = w - dtk[(size_t)i * 4 + 0] * tk[(size_t)i * TKS + 0] -
                          dtk[(size_t)i * 4 + 1] * tk[(size_t)i * TKS + 1];
    if (i == C - 1) {
      lab += scc + dAC * AC + dEC * EC;
      lbb += sbb + dBC * BC;
    }
    dlr[i] = dtk[(size_t)i * 4 + 0] * tk[(size_t)i * TKS + 4] +
             dtk[(size_t)i * 4 + 1] * tk[(size_t)i * TKS + 5];
    ddec[i] = -sufA / (1.0f - dec[i]);
    const float be = mom[i];
    dmom[i] = (logf(be) > LOG_CLAMP) ? sufB / be : 0.f;
    sufA -= lab;
    sufB -= lbb;
  }
}

hipError_t launch_global_gate_bwd(const GlobalArgs& a, hipStream_t st) {
  dim3 grid(a.D.L / a.D.C, a.D.B * a.D.H);
  hipLaunchKernelGGL(global_gate_bwd_kernel, grid, dim3(64), 0, st, a, GRED_BLOCKS);
  return hipGetLastError();
}

// dW_init of the global memory: sum over the batch rows of each head
__global__ void reduce_gw_kernel(const float* part, int B, int H, size_t hd, float* dW1,
                                 float* dW2) {
  const int hh = blockIdx.y;
  for (size_t e = blockIdx.x * blockDim.x + threadIdx.x; e < 2 * hd;
       e += gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += part[((size_t)b * H + hh) * 2 * hd + e];
    if (e < hd)
      dW1[(size_t)hh * hd + e] = s;
    else
      dW2[(size_t)hh * hd + e - hd] = s;
  }
}

hipError_t launch_reduce_global_init(const float* part, int B, int H, size_t hd, float* dW1,
                                     float* dW2, hipStream_t st) {
  hipLaunchKernelGGL(reduce_gw_kernel, dim3(32, H), dim3(256), 0, st, part, B, H, hd, dW1, dW2);
  return hipGetLastError();
}

}  // namespace tnt
