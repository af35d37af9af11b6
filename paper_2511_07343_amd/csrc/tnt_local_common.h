// Pieces of one local-memory chunk step shared by the forward and backward
// kernels: staging of the chunk's tokens, the gate coefficients of the
// momentum / decay recurrence, the Q-K projection and the chunk-entry
// gradient quantities.  Internal to the library.
#pragma once

#include "tnt_device.h"
#include "tnt_kernels.h"

namespace tnt {

constexpr int MAXC = 64;  // largest padded chunk handled by one workgroup

// Gate coefficients of one chunk (positions i, tau = 0..Cp-1, 0-indexed).
//   la_i = sum_{j<=i} log(1 - alpha_j),  lb_i = sum_{j<=i} log beta_j
//   A_i = e^{la_i},  E_i = sum_{m<=i} e^{la_i - la_m + lb_m}
//   ct_{i,tau} = sum_{m=tau}^{i} e^{la_i - la_m + lb_m - lb_tau}   (tau <= i)
//   c_{i,tau} = eta_tau ct_{i,tau};  W_i = A_i W0 + E_i S0 - sum_tau c_{i,tau} u_tau
//   momentum weights at the chunk end: b_tau = eta_tau e^{lb_{C-1} - lb_tau}
// Padded positions (i >= C) carry eta = 0, alpha = 0, beta = 1.
struct Coef {
  float c[MAXC][MAXC + 1];
  float ct[MAXC][MAXC + 1];
  float A[MAXC], E[MAXC], la[MAXC], lb[MAXC], eta[MAXC], cC[MAXC], bb[MAXC], ebt[MAXC];
  float knorm[MAXC];
  float AC, BC, EC;
  float red[32];
};

// Columns of the coefficient matrix, one prefix affine scan over the rows
// (lanes) per column tau, the columns dealt to the waves:
//   ct_{r,tau} = e^{la_r - la_{r-1}} ct_{r-1,tau} + e^{lb_r - lb_tau}  (r >= tau),
//   ct_{r,tau} = 0 (r < tau), c = eta_tau ct.  Every multiplier and term is at most 1.
// Wave 0 also scans E_i = e^{la_i - la_{i-1}} E_{i-1} + e^{lb_i}.  The prefix
// arrays la, lb, eta must be in LDS.  No barrier.
__device__ __forceinline__ void affine_scan_up(float& a, float& b) {  // inclusive, over lanes
  const int r = lane_id();
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    const float pa = __shfl_up(a, o, WAVE), pb = __shfl_up(b, o, WAVE);
    if (r >= o) {
      b = a * pb + b;
      a = a * pa;
    }
  }
}
// `put(r, tau, ct)` receives ct_{r,tau} for every row r < Cp of every column.
template <typename Put>
__device__ __forceinline__ void coef_scan_columns(const float* la, const float* lb, int Cp,
                                                  const Put& put, float* E) {
  const int r = lane_id();
  const float lar = la[r < Cp ? r : Cp - 1], lbr = lb[r < Cp ? r : Cp - 1];
  const float ar = r > 0 && r < Cp ? expf(lar - la[r - 1]) : 0.f;
  for (int tau = wave_id(); tau < Cp; tau += num_waves()) {
    float a = ar, b = (r >= tau && r < Cp) ? expf(lbr - lb[tau]) : 0.f;
    affine_scan_up(a, b);
    if (r < Cp) put(r, tau, b);
  }
  if (wave_id() == 0) {
    float a = ar, b = r < Cp ? expf(lbr) : 0.f;
    affine_scan_up(a, b);
    if (r < Cp) E[r] = b;
  }
}
template <int STRIDE>
__device__ __forceinline__ void coef_columns(const float* la, const float* lb, const float* eta,
                                             int Cp, float (*ct)[STRIDE], float (*c)[STRIDE],
                                             float* E) {
  coef_scan_columns(la, lb, Cp, [&](int r, int tau, float b) {
    if (ct) ct[r][tau] = b;
    c[r][tau] = eta[tau] * b;
  }, E);
}

// Fill `cf` for the chunk whose first token is `tok0` (gate arrays already
// offset to the chain).  All threads call.  Ends with a barrier.
__device__ __forceinline__ void chunk_coefs(Coef& cf, const float* lr, const float* mom,
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
  coef_columns(cf.la, cf.lb, cf.eta, Cp, cf.ct, cf.c, cf.E);
  __syncthreads();
  if (wave_id() == 0) {
    const int tau = lane_id();
    if (tau < Cp) {
      const float et = (tau < C) ? expf(cf.lb[C - 1] - cf.lb[tau]) : 0.f;
      cf.ebt[tau] = et;
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

// The coefficients without ct / ebt (retrieval and carry only; smaller LDS
// footprint), for chunks of at most N (padded) positions.
template <int N>
struct alignas(16) CoefFN {  // 16-byte aligned: c is copied in 16-byte groups
  static_assert(N <= MAXC, "one wave scans a chunk");
  // the lower triangle of c (c_{i,tau} = 0 for tau > i), row after row:
  // c_{i,tau} at i (i + 1) / 2 + tau
  float c[N * (N + 1) / 2];
  float A[N], E[N], la[N], lb[N], eta[N], cC[N], bb[N];
  float knorm[N];
  float AC, BC, EC;
  // c_{i,j}; for j > i the value read is another entry's, to be masked by the
  // caller (every index stays inside the array)
  __device__ __forceinline__ float cc(int i, int j) const { return c[i * (i + 1) / 2 + j]; }
};
using CoefF = CoefFN<MAXC>;

template <int N>
__device__ __forceinline__ void chunk_coefs_f(CoefFN<N>& cf, const float* lr, const float* mom,
                                              const float* dec, int tok0, int C, int Cp) {
  if (wave_id() == 0) {
    const int i = lane_id();
    const bool in = i < C;
    const float eta = in ? lr[tok0 + i] : 0.f;
    const float lmb = in ? log_mom(mom[tok0 + i]) : 0.f;
    const float lka = in ? log_keep(dec[tok0 + i]) : 0.f;
    const float la = wave_incl_sum(lka);
    const float lb = wave_incl_sum(lmb);
    if (i < N) {
      cf.la[i] = la;
      cf.lb[i] = lb;
      cf.eta[i] = eta;
      cf.A[i] = expf(la);
    }
  }
  __syncthreads();
  coef_scan_columns(cf.la, cf.lb, Cp, [&](int r, int tau, float b) {
    if (tau <= r) cf.c[r * (r + 1) / 2 + tau] = cf.eta[tau] * b;
  }, cf.E);
  __syncthreads();
  if (wave_id() == 0) {
    const int tau = lane_id();
    if (tau < Cp) {
      const float et = (tau < C) ? expf(cf.lb[C - 1] - cf.lb[tau]) : 0.f;
      cf.bb[tau] = cf.eta[tau] * et;
      cf.cC[tau] = tau < C ? cf.cc(C - 1, tau) : 0.f;
    }
    if (tau == 0) {
      cf.AC = cf.A[C - 1];
      cf.BC = expf(cf.lb[C - 1]);
      cf.EC = cf.E[C - 1];
    }
  }
  __syncthreads();
}

// The coefficients of the gate adjoints, for chunks of at most N (padded)
// positions: ct packed like CoefFN's c.  c_{i,tau} = eta_tau ct_{i,tau} is the
// product the scan forms for c, so cc() equals the stored c bit for bit.
template <int N>
struct CoefGN {
  static_assert(N <= MAXC, "one wave scans a chunk");
  float ct[N * (N + 1) / 2];
  float A[N], E[N], la[N], lb[N], eta[N], bb[N], ebt[N];
  float BC;
  // ct_{i,j} and c_{i,j} for j <= i
  __device__ __forceinline__ float ctt(int i, int j) const { return ct[i * (i + 1) / 2 + j]; }
  __device__ __forceinline__ float cc(int i, int j) const { return eta[j] * ct[i * (i + 1) / 2 + j]; }
};

template <int N>
__device__ __forceinline__ void chunk_coefs_g(CoefGN<N>& cf, const float* lr, const float* mom,
                                              const float* dec, int tok0, int C, int Cp) {
  if (wave_id() == 0) {
    const int i = lane_id();
    const bool in = i < C;
    const float eta = in ? lr[tok0 + i] : 0.f;
    const float lmb = in ? log_mom(mom[tok0 + i]) : 0.f;
    const float lka = in ? log_keep(dec[tok0 + i]) : 0.f;
    const float la = wave_incl_sum(lka);
    const float lb = wave_incl_sum(lmb);
    if (i < N) {
      cf.la[i] = la;
      cf.lb[i] = lb;
      cf.eta[i] = eta;
      cf.A[i] = expf(la);
    }
  }
  __syncthreads();
  coef_scan_columns(cf.la, cf.lb, Cp, [&](int r, int tau, float b) {
    if (tau <= r) cf.ct[r * (r + 1) / 2 + tau] = b;
  }, cf.E);
  __syncthreads();
  if (wave_id() == 0) {
    const int tau = lane_id();
    if (tau < Cp) {
      const float et = (tau < C) ? expf(cf.lb[C - 1] - cf.lb[tau]) : 0.f;
      cf.ebt[tau] = et;
      cf.bb[tau] = cf.eta[tau] * et;
    }
    if (tau == 0) cf.BC = expf(cf.lb[C - 1]);
  }
  __syncthreads();
}

// The retrieval's chunk coefficients c (packed), A, E from a forward record: the
// values chunk_coefs_f forms, bit for bit (the retrieval computed them from the
// same gates).  All threads call; ends with a barrier.
template <int N>
__device__ __forceinline__ void coefs_from_record_f(CoefFN<N>& cf, const float* cc, const float* vA,
                                                    const float* vE, int Cp) {
  for (int e = threadIdx.x; e < Cp; e += blockDim.x) {
    cf.A[e] = vA[e];
    cf.E[e] = vE[e];
  }
  const int np = Cp * (Cp + 1) / 2;
  for (int e = threadIdx.x * 4; e < np; e += blockDim.x * 4) {
    if (e + 4 <= np) {
      *reinterpret_cast<f32x4*>(cf.c + e) = *reinterpret_cast<const f32x4*>(cc + e);
    } else {
      for (int q = e; q < np; ++q) cf.c[q] = cc[q];
    }
  }
  __syncthreads();
}

// Stage a [Cp][d] tile of an I/O tensor (rows >= C zero) into CT storage,
// optionally also its transpose [d][Cp].
template <typename IO, typename CT>
__device__ __forceinline__ void stage_rows(CT* dst, CT* dstT, const IO* src, int C, int Cp,
                                           int d) {
  for (int e = threadIdx.x; e < Cp * d; e += blockDim.x) {
    const int i = e / d, j = e - i * d;
    const float x = (i < C) ? to_f(src[(size_t)i * d + j]) : 0.f;
    if (dst) dst[(size_t)i * d + j] = from_f<CT>(x);
    if (dstT) dstT[(size_t)j * Cp + i] = from_f<CT>(x);
  }
}

// Row norms of the staged keys and the unit keys N = K / ||K|| (zero rows
// stay zero), stored as [Cp][d] and [d][Cp].
template <typename IO, typename CT>
__device__ __forceinline__ void unit_keys(Coef& cf, CT* N, CT* NT, const IO* k, int C, int Cp,
                                          int d) {
  for (int i = threadIdx.x; i < Cp; i += blockDim.x) {
    float s = 0.f;
    if (i < C)
      for (int j = 0; j < d; ++j) {
        const float x = to_f(k[(size_t)i * d + j]);
        s += x * x;
      }
    cf.knorm[i] = sqrtf(s);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < Cp * d; e += blockDim.x) {
    const int i = e / d, j = e - i * d;
    const float nr = cf.knorm[i];
    const float x = (i < C && nr > 0.f) ? to_f(k[(size_t)i * d + j]) / nr : 0.f;
    N[(size_t)i * d + j] = from_f<CT>(x);
    NT[(size_t)j * Cp + i] = from_f<CT>(x);
  }
}

// The carry's coefficients only (cC, b, A_C, B_C, E_C), without the C x C
// matrix: cC_t = eta_t y_t with y_t = sum_{m >= t} e^{(la_C - la_m) + (lb_m - lb_t)}
// obeys y_t = e^{la_C - la_t} + e^{lb_{t+1} - lb_t} y_{t+1}, a suffix affine scan
// over the lanes whose terms and multipliers are all at most 1.  One wave;
// ends with a barrier.  Overwrites those fields of `cf` (every walk takes its
// carry from here).
template <typename CF>
__device__ __forceinline__ void carry_coefs(CF& cf, const float* lr, const float* mom,
                                            const float* dec, int tok0, int C, int Cp) {
  if (wave_id() == 0) {
    const int i = lane_id();
    const bool in = i < C;
    const float eta = in ? lr[tok0 + i] : 0.f;
    const float lmb = in ? log_mom(mom[tok0 + i]) : 0.f;
    const float lka = in ? log_keep(dec[tok0 + i]) : 0.f;
    const float la = wave_incl_sum(lka), lb = wave_incl_sum(lmb);
    const float laC = __shfl(la, C - 1, WAVE), lbC = __shfl(lb, C - 1, WAVE);
    const float lbn = __shfl_down(lb, 1, WAVE);
    float ya = in ? expf(laC - la) : 0.f;
    float yb = (i + 1 < C) ? expf(lbn - lb) : 0.f;
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
      const float pa = __shfl_down(ya, o, WAVE), pb = __shfl_down(yb, o, WAVE);
      if (i + o < WAVE) {
        ya = ya + yb * pa;
        yb = yb * pb;
      }
    }
    const float ec = wave_sum(in ? expf(laC - la + lb) : 0.f);
    if (i < Cp) {
      cf.cC[i] = in ? eta * ya : 0.f;
      cf.bb[i] = in ? eta * expf(lbC - lb) : 0.f;
    }
    if (i == 0) {
      cf.AC = expf(laC);
      cf.BC = expf(lbC);
      cf.EC = ec;
    }
  }
  __syncthreads();
}

}  // namespace tnt
