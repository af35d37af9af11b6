// Local memories, forward, for fixed sizes (head dim D, hidden HID, padded
// chunk CP) whose chunk working set fits in the 160 KB LDS of a CU.  Same
// chunk step as local_fwd_kernel (see tnt_local_fwd.hip); here every loop has
// a compile-time trip count and every chunk intermediate stays on chip:
//
//   LDS  Hk [CP][HID]   s(K W1^T)                         bf16/fp32 (CT)
//        D1 [CP][HID]   (R W2) * s'(K W1^T)
//        U  [CP][HID]   reused in turn: Q-K temporaries (Q, N, N^T, tril(Q N^T)),
//                       then the chunk-entry W2 (CT copy, [D][HID]), then H = s(Z)
//        X, K, R [CP][D], P [CP][CP], gate coefficients
//   VGPR s'(K W1^T) between the two GEMMs that share its output tiles
//
// The fp32 state (W1, W2, S1, S2 and the Q-K sum) lives in global memory,
// one slot per chunk boundary; contraction-contiguous operands are read from
// it directly, the carry reads the entry slot and writes the next one.
#include "tnt_local_common.h"

namespace tnt {

struct CoefF {  // forward-only gate coefficients (no ct)
  float c[MAXC][MAXC + 1];
  float A[MAXC], E[MAXC], la[MAXC], lb[MAXC], eta[MAXC], cC[MAXC], bb[MAXC];
  float knorm[MAXC];
  float AC, BC, EC;
};

__device__ __forceinline__ void chunk_coefs_f(CoefF& cf, const float* lr, const float* mom,
                                              const float* dec, int tok0, int C, int Cp) {
  if (wave_id() == 0) {
    const int i = lane_id();
    const bool in = i < C;
    const float eta = in ? lr[tok0 + i] : 0.f;
    const float lmb = in ? log_mom(mom[tok0 + i]) : 0.f;
    const float lka = in ? log_keep(dec[tok0 + i]) : 0.f;
    const float la = wave_incl_sum(lka);
    const float lb = wave_incl_sum(lmb);
    cf.la[i] = la;
    cf.lb[i] = lb;
    cf.eta[i] = eta;
    cf.A[i] = expf(la);
  }
  __syncthreads();
  if (wave_id() == 0) {
    const int i = lane_id();
    if (i < Cp) {
      float e = 0.f;
      for (int m = 0; m <= i; ++m) e += expf(cf.la[i] - cf.la[m] + cf.lb[m]);
      cf.E[i] = e;
      const int tau = i;
      const float lbt = cf.lb[tau];
      for (int r = 0; r < tau; ++r) cf.c[r][tau] = 0.f;
      float x = 1.0f;
      cf.c[tau][tau] = cf.eta[tau];
      for (int r = tau + 1; r < Cp; ++r) {
        x = expf(cf.la[r] - cf.la[r - 1]) * x + expf(cf.lb[r] - lbt);
        cf.c[r][tau] = cf.eta[tau] * x;
      }
    }
  }
  __syncthreads();
  if (wave_id() == 0) {
    const int tau = lane_id();
    if (tau < Cp) {
      const float et = (tau < C) ? expf(cf.lb[C - 1] - cf.lb[tau]) : 0.f;
      cf.bb[tau] = cf.eta[tau] * et;
      cf.cC[tau] = cf.c[C - 1][tau];
    }
    if (tau == 0) {
      cf.AC = cf.A[C - 1];
      cf.BC = expf(cf.lb[C - 1]);
      cf.EC = cf.E[C - 1];
    }
  }
  __syncthreads();
}

// LDS carve-up (CT elements)
template <int D, int HID, int CP>
struct FwdLds {
  static constexpr int cmax(int x, int y) { return x > y ? x : y; }
  static constexpr int USZ = cmax(cmax(CP, D) * HID, 3 * CP * D + CP * CP);
  static constexpr int Hk = 0;
  static constexpr int D1 = Hk + CP * HID;
  static constexpr int U = D1 + CP * HID;
  static constexpr int X = U + USZ;
  static constexpr int K = X + CP * D;
  static constexpr int R = K + CP * D;
  static constexpr int P = R + CP * D;
  static constexpr int total = P + CP * CP;
  // inside U during the Q-K phase
  static constexpr int uQ = U, uN = U + CP * D, uNT = U + 2 * CP * D, uS = U + 3 * CP * D;
};

template <typename CT, int D, int HID, int CP>
constexpr size_t fwd_fast_lds_bytes() {
  return (size_t)FwdLds<D, HID, CP>::total * sizeof(CT);
}

template <typename IO, typename CT, int ACT, int D, int HID, int CP>
__global__ void __launch_bounds__(512) local_fwd_fast_kernel(LocalFwdArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ CoefF cf;
  using Ly = FwdLds<D, HID, CP>;
  constexpr int NW = 8;                       // waves
  constexpr int TNH = HID / 16, TMC = CP / 16;
  constexpr int TILES_CH = TMC * TNH;         // tiles of a CP x HID result
  constexpr int PER_WAVE = (TILES_CH + NW - 1) / NW;
  CT* L = (CT*)smem;
  CT *sHk = L + Ly::Hk, *sD1 = L + Ly::D1, *sU = L + Ly::U, *sX = L + Ly::X, *sK = L + Ly::K,
     *sR = L + Ly::R, *sP = L + Ly::P;
  CT *sQ = L + Ly::uQ, *sN = L + Ly::uN, *sNT = L + Ly::uNT, *sS = L + Ly::uS;
  CT* sW2 = sU;  // chunk-entry W2 copy [D][HID]
  CT* sH = sU;

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int u = blockIdx.x;
  const int b = u / (Dm.H * nshard), hh = (u / nshard) % Dm.H, s = u % nshard;
  constexpr size_t hd = (size_t)HID * D;
  const size_t chain = (size_t)b * Dm.H + hh;
  const IO* q = (const IO*)a.q + chain * Dm.L * D;
  const IO* k = (const IO*)a.k + chain * Dm.L * D;
  const IO* v = (const IO*)a.v + chain * Dm.L * D;
  float* o = a.o_part + chain * Dm.L * D;
  const float* lr = a.lr + chain * Dm.L;
  const float* mom = a.mom + chain * Dm.L;
  const float* dec = a.decay + chain * Dm.L;
  float* st = a.states + (size_t)u * a.nslots * 4 * hd;
  float* mst = a.mstates + (size_t)u * a.nslots * D * D;
  const bool qk = Dm.qk_proj;
  const bool shard_qk = Dm.qk_proj && Dm.qk_scope == 0;
  const float rscale = 2.0f / (float)D;
  const int l = lane_id(), w = wave_id();

  {
    const float* W1i = a.W1i + hh * hd;
    const float* W2i = a.W2i + hh * hd;
    for (int e = threadIdx.x * 4; e < (int)hd; e += blockDim.x * 4) {
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(W1i + e);
      const f32x4 x2 = *reinterpret_cast<const f32x4*>(W2i + e);
      *reinterpret_cast<f32x4*>(st + e) = x1;
      *reinterpret_cast<f32x4*>(st + hd + e) = x2;
      *reinterpret_cast<f32x4*>(st + 2 * hd + e) = f32x4{0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4*>(st + 3 * hd + e) = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (shard_qk)
      for (int e = threadIdx.x; e < D * D; e += blockDim.x) mst[e] = 0.f;
  }
  __syncthreads();

  const int nch = Dm.S / C;
  for (int n = 0; n < nch; ++n) {
    const int tok0 = s * Dm.S + n * C;
    const float* cur = st + (size_t)(n % a.nslots) * 4 * hd;
    float* nxt = st + (size_t)((n + 1) % a.nslots) * 4 * hd;
    const float *W1 = cur, *W2 = cur + hd, *S1 = cur + 2 * hd, *S2 = cur + 3 * hd;
    float *W1n = nxt, *W2n = nxt + hd, *S1n = nxt + 2 * hd, *S2n = nxt + 3 * hd;
    const float* Mc = mst + (size_t)(n % a.nslots) * D * D;
    float* Mn = mst + (size_t)((n + 1) % a.nslots) * D * D;

    // ---- stage Q, K (rows >= C zero), unit keys, gate coefficients
    for (int e = threadIdx.x; e < CP * D; e += blockDim.x) {
      const int i = e / D;
      const bool in = i < C;
      sQ[e] = from_f<CT>(in ? to_f(q[(size_t)tok0 * D + e]) : 0.f);
      sK[e] = from_f<CT>(in ? to_f(k[(size_t)tok0 * D + e]) : 0.f);
    }
    if (qk) {
      for (int i = w; i < CP; i += NW) {
        float ss = 0.f;
        if (i < C)
          for (int j = l; j < D; j += WAVE) {
            const float x = to_f(k[(size_t)(tok0 + i) * D + j]);
            ss += x * x;
          }
        ss = wave_sum(ss);
        if (l == 0) cf.knorm[i] = sqrtf(ss);
      }
    }
    chunk_coefs_f(cf, lr, mom, dec, tok0, C, CP);  // barriers inside
    if (qk) {
      for (int e = threadIdx.x; e < CP * D; e += blockDim.x) {
        const int i = e / D, j = e - i * D;
        const float nr = cf.knorm[i];
        const float x = (i < C && nr > 0.f) ? to_f(k[(size_t)(tok0 + i) * D + j]) / nr : 0.f;
        sN[e] = from_f<CT>(x);
        sNT[(size_t)j * CP + i] = from_f<CT>(x);
      }
      __syncthreads();
      gemm<CT, KC, KC>(CP, CP, D, sQ, D, sN, D, [&](int i, int j, float x) {
        sS[(size_t)i * CP + j] = from_f<CT>(j <= i ? x : 0.f);
      });
      __syncthreads();
      {
        constexpr int tn = D / 16, nt = TMC * tn;
        for (int t = w; t < nt; t += NW) {
          const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
          f4 acc = zero4();
          if (shard_qk) mma_tile<CT, KC, KC>(acc, sQ, D, i0, Mc, D, j0, D);
          mma_tile<CT, KC, KC>(acc, sS, CP, i0, sNT, CP, j0, CP);
          tile_each(acc, i0, j0, [&](int i, int j, float x) { sX[(size_t)i * D + j] = from_f<CT>(x); });
        }
      }
      if (shard_qk)
        gemm<CT, KC, KC>(D, D, CP, sNT, CP, sNT, CP, [&](int i, int j, float x) {
          Mn[(size_t)i * D + j] = Mc[(size_t)i * D + j] + x;
        });
    } else {
      for (int e = threadIdx.x; e < CP * D; e += blockDim.x) sX[e] = sQ[e];
    }

    // ---- Zk = K W1^T -> Hk (LDS), s'(Zk) (registers)
    f4 spr[PER_WAVE];
#pragma unroll
    for (int x = 0; x < PER_WAVE; ++x) {
      const int t = w + x * NW;
      if (t < TILES_CH) {
        const int i0 = (t / TNH) * 16, j0 = (t % TNH) * 16;
        f4 acc = zero4();
        mma_tile<CT, KC, KC>(acc, sK, D, i0, W1, D, j0, D);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          const ActVals av = act_all<ACT>(acc[r]);
          sHk[(size_t)i * HID + j] = from_f<CT>(av.s);
          spr[x][r] = av.d1;
        }
      }
    }
    __syncthreads();  // Q-K temporaries in U are dead from here
    // chunk-entry W2 -> U as CT [D][HID]
    for (int e = threadIdx.x * 4; e < (int)hd; e += blockDim.x * 4) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(W2 + e);
#pragma unroll
      for (int j = 0; j < 4; ++j) sW2[e + j] = from_f<CT>(x[j]);
    }
    __syncthreads();

    // ---- R = (2/d) (Hk W2^T - V)
    {
      constexpr int tn = D / 16, nt = TMC * tn;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 acc = zero4();
        mma_tile<CT, KC, KC>(acc, sHk, HID, i0, sW2, HID, j0, HID);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          const float rv = (i < C) ? rscale * (acc[r] - to_f(v[(size_t)(tok0 + i) * D + j])) : 0.f;
          sR[(size_t)i * D + j] = from_f<CT>(rv);
        }
      }
    }
    __syncthreads();

    // ---- D1 = (R W2) * s'(Zk), same tiles as Zk
#pragma unroll
    for (int x = 0; x < PER_WAVE; ++x) {
      const int t = w + x * NW;
      if (t < TILES_CH) {
        const int i0 = (t / TNH) * 16, j0 = (t % TNH) * 16;
        f4 acc = zero4();
        mma_tile<CT, KC, MC>(acc, sR, D, i0, sW2, HID, j0, D);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          sD1[(size_t)i * HID + j] = from_f<CT>(acc[r] * spr[x][r]);
        }
      }
    }
    __syncthreads();

    // ---- carry into the next slot
    {
      constexpr int tn = D / 16, nt = (HID / 16) * tn;  // W1', S1' : HID x D
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 aw = zero4(), as = zero4();
        // A[i][tau] = D1[tau][i] (x cC_tau or b_tau), B[tau][j] = K[tau][j]
        mma_tile<CT, MC, MC>(aw, sD1, HID, i0, sK, D, j0, CP, cf.cC);
        mma_tile<CT, MC, MC>(as, sD1, HID, i0, sK, D, j0, CP, cf.bb);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * D + j0 + (l & 15);
          W1n[e] = cf.AC * W1[e] + cf.EC * S1[e] - aw[r];
          S1n[e] = cf.BC * S1[e] - as[r];
        }
      }
    }
    {
      constexpr int tn = HID / 16, nt = (D / 16) * tn;  // W2', S2' : D x HID
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 aw = zero4(), as = zero4();
        // A[i][tau] = R[tau][i] (x cC_tau or b_tau), B[tau][j] = Hk[tau][j]
        mma_tile<CT, MC, MC>(aw, sR, D, i0, sHk, HID, j0, CP, cf.cC);
        mma_tile<CT, MC, MC>(as, sR, D, i0, sHk, HID, j0, CP, cf.bb);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * HID + j0 + (l & 15);
          W2n[e] = cf.AC * W2[e] + cf.EC * S2[e] - aw[r];
          S2n[e] = cf.BC * S2[e] - as[r];
        }
      }
    }

    // ---- retrieval, dual form
    {
      constexpr int tn = CP / 16, nt = TMC * tn;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 acc = zero4();
        mma_tile<CT, KC, KC>(acc, sX, D, i0, sK, D, j0, D);
        tile_each(acc, i0, j0, [&](int i, int j, float x) {
          sP[(size_t)i * CP + j] = from_f<CT>(j <= i ? cf.c[i][j] * x : 0.f);
        });
      }
    }
    __syncthreads();  // P ready; the W2 copy in U is dead
#pragma unroll
    for (int x = 0; x < PER_WAVE; ++x) {
      const int t = w + x * NW;
      if (t < TILES_CH) {
        const int i0 = (t / TNH) * 16, j0 = (t % TNH) * 16;
        f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
        mma_tile<CT, KC, KC>(a1, sX, D, i0, W1, D, j0, D);
        mma_tile<CT, KC, KC>(a2, sX, D, i0, S1, D, j0, D);
        mma_tile<CT, KC, MC>(a3, sP, CP, i0, sD1, HID, j0, CP);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          const float z = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
          sH[(size_t)i * HID + j] = from_f<CT>(act_f<ACT>(z));
        }
      }
    }
    __syncthreads();
    {
      constexpr int tn = CP / 16, nt = TMC * tn;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 acc = zero4();
        mma_tile<CT, KC, KC>(acc, sH, HID, i0, sHk, HID, j0, HID);
        tile_each(acc, i0, j0, [&](int i, int j, float x) {
          sP[(size_t)i * CP + j] = from_f<CT>(j <= i ? cf.c[i][j] * x : 0.f);
        });
      }
    }
    __syncthreads();
    {
      constexpr int tn = D / 16, nt = TMC * tn;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
        mma_tile<CT, KC, KC>(a1, sH, HID, i0, W2, HID, j0, HID);
        mma_tile<CT, KC, KC>(a2, sH, HID, i0, S2, HID, j0, HID);
        mma_tile<CT, KC, MC>(a3, sP, CP, i0, sR, D, j0, CP);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          if (i < C) o[(size_t)(tok0 + i) * D + j] = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
        }
      }
    }
    __syncthreads();
  }
}

template <typename IO, typename CT, int ACT, int D, int HID, int CP>
static bool try_fast(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (a.D.d != D || a.D.hid != HID || a.D.Cp != CP || a.D.act != ACT) return false;
  constexpr size_t lds = fwd_fast_lds_bytes<CT, D, HID, CP>();
  if (lds + sizeof(CoefF) > 160 * 1024) return false;
  auto kern = local_fwd_fast_kernel<IO, CT, ACT, D, HID, CP>;
  set_lds_limit((const void*)kern);
  hipLaunchKernelGGL(kern, dim3(units), dim3(512), lds, st, a);
  *err = hipGetLastError();
  return true;
}

// Returns true (and the launch status) when a fixed-size kernel handles `a`.
bool launch_local_fwd_fast(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (a.D.bf16) {
    return try_fast<__bf16, __bf16, ACT_SILU, 64, 256, 64>(a, units, st, err) ||
           try_fast<__bf16, __bf16, ACT_SILU, 64, 256, 32>(a, units, st, err) ||
           try_fast<__bf16, __bf16, ACT_SILU, 64, 256, 16>(a, units, st, err) ||
           try_fast<__bf16, __bf16, ACT_GELU, 64, 256, 64>(a, units, st, err) ||
           try_fast<__bf16, __bf16, ACT_GELU, 64, 256, 16>(a, units, st, err);
  }
  return try_fast<float, float, ACT_GELU, 16, 32, 16>(a, units, st, err) ||
         try_fast<float, float, ACT_SILU, 16, 32, 16>(a, units, st, err);
}

}  // namespace tnt
