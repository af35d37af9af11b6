// Global memory, forward (global update rule, Sec. 4.1.1 box; App. E) and the
// small helpers of the layer (output sum, init-gradient reduction).
//
// The global memory is one sequential chain per (batch row, head) over L/C_G
// chunks.  Inside a chunk nothing is sequential: retrieval reads the
// chunk-entry state V_{xi(t,C_G)} (Sec. 4.1.2 retrieval box) and every
// gradient is taken at that state, so each chunk runs as
//   scan  : gate coefficients of every chunk at once (inputs only)
//   phase1: token tiles -> O_G = s(Q V1^T) V2^T and R = (2/d) (s(K V1^T) V2^T - V)
//   phase2: hidden slices -> V1' = A_C V1 + E_C S1 - D1^T diag(cC) K,
//           S1' = B_C S1 - D1^T diag(b) K (V2', S2' alike with R^T, Hk), where
//           the slice's Hk and D1 = (R V2) * s'(K V1^T) are recomputed from R.
#include "tnt_device.h"
#include "tnt_kernels.h"

#include <algorithm>

namespace tnt {

// ---------------------------------------------------------------------------
// gate coefficients of a global chunk (one 512-thread workgroup per (chunk,
// chain); each thread owns a contiguous segment of the chunk's tokens).
// tokc[t] = {cC_t, b_t, la_t, lb_t, s_t, e^{lb_C - lb_t}}; chunkc[n] = {A_C, B_C, E_C, 0} with
//   cC_t = eta_t s_t,  s_t = sum_{m>=t} e^{la_C - la_m + lb_m - lb_t}
//        = e^{la_C - la_t} + beta_{t+1} s_{t+1}          (suffix affine scan)
//   b_t  = eta_t e^{lb_C - lb_t},  E_C = beta_0 s_0.
// The prefix sums la, lb and the suffix scan of s run as wavefront scans
// joined across the workgroup's waves through LDS.  When the chunk's records
// fit in LDS (C_G <= GSCAN_STAGE_MAX) they are assembled there and written out
// whole, consecutive threads on consecutive 16-byte pieces, so every 32-byte
// record reaches memory as one full sector (the unused two floats as zeros).
// ---------------------------------------------------------------------------
constexpr int GSCAN_THREADS = 512;
constexpr int GSCAN_WAVES = GSCAN_THREADS / WAVE;
constexpr int GSCAN_STAGE_MAX = 4096;  // tokens of a chunk whose records are staged in LDS

__global__ void __launch_bounds__(GSCAN_THREADS) global_scan_kernel(GlobalArgs a, int stage) {
  extern __shared__ __align__(16) float srec[];           // [C][TKS] when staged
  __shared__ float wa[GSCAN_WAVES], wb[GSCAN_WAVES];      // per-wave gate log sums
  __shared__ float wp[GSCAN_WAVES], wq[GSCAN_WAVES];      // per-wave affine maps
  __shared__ float s_in[GSCAN_WAVES + 1];                 // s at each wave's end
  const int n = blockIdx.x, chain = blockIdx.y;
  const int C = a.D.C, L = a.D.L;
  const size_t base = (size_t)chain * L + (size_t)n * C;
  const float* lr = a.lr + base;
  const float* mom = a.mom + base;
  const float* dec = a.decay + base;
  float* const tkg = a.tokc + base * TKS;
  float* const tk = stage ? srec : tkg;  // where the records are assembled
  const int l = lane_id(), w = wave_id(), t = threadIdx.x;
  const int E = (C + GSCAN_THREADS - 1) / GSCAN_THREADS;
  const int i0 = min(t * E, C), i1 = min(i0 + E, C);
  float sa = 0.f, sb = 0.f;
  for (int i = i0; i < i1; ++i) {
    sa += log_keep(dec[i]);
    sb += log_mom(mom[i]);
  }
  const float ia = wave_incl_sum(sa), ib = wave_incl_sum(sb);
  if (l == WAVE - 1) {
    wa[w] = ia;
    wb[w] = ib;
  }
  __syncthreads();
  float oa = 0.f, ob = 0.f, laC = 0.f, lbC = 0.f;
  for (int v = 0; v < GSCAN_WAVES; ++v) {
    if (v < w) {
      oa += wa[v];
      ob += wb[v];
    }
    laC += wa[v];
    lbC += wb[v];
  }
  float pa = oa + ia - sa, pb = ob + ib - sb;
  for (int i = i0; i < i1; ++i) {
    pa += log_keep(dec[i]);
    pb += log_mom(mom[i]);
    *reinterpret_cast<float2*>(tk + (size_t)i * TKS + 2) = make_float2(pa, pb);
    if (stage) *reinterpret_cast<float2*>(tk + (size_t)i * TKS + 6) = make_float2(0.f, 0.f);
  }
  // segment affine map s_{i0} = P s_{i1} + Q (own writes are visible to the thread)
  float P = 1.f, Q = 0.f;
  for (int i = i1 - 1; i >= i0; --i) {
    const float ai = expf(laC - tk[(size_t)i * TKS + 2]);
    const float mi = (i + 1 < C) ? mom[i + 1] : 0.f;
    Q = ai + mi * Q;
    P = mi * P;
  }
  // suffix composition over the wave's lanes: G_l = F_l o F_{l+1} o ... o F_63
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    const float Po = __shfl_down(P, o, WAVE), Qo = __shfl_down(Q, o, WAVE);
    if (l + o < WAVE) {
      Q = P * Qo + Q;
      P = P * Po;
    }
  }
  if (l == 0) {
    wp[w] = P;
    wq[w] = Q;
  }
  __syncthreads();
  if (t == 0) {  // s at the end of each wave's tokens, from the chunk's end (s = 0) back
    float sv = 0.f;
    s_in[GSCAN_WAVES] = 0.f;
    for (int v = GSCAN_WAVES - 1; v >= 0; --v) {
      s_in[v + 1] = sv;
      sv = wp[v] * sv + wq[v];
    }
  }
  __syncthreads();
  const float send = s_in[w + 1];  // s at the first token after this wave's tokens
  const float Pn = __shfl_down(P, 1, WAVE), Qn = __shfl_down(Q, 1, WAVE);
  float sv = (l == WAVE - 1) ? send : Pn * send + Qn;  // s at this thread's i1
  for (int i = i1 - 1; i >= i0; --i) {
    const float ai = expf(laC - tk[(size_t)i * TKS + 2]);
    const float mi = (i + 1 < C) ? mom[i + 1] : 0.f;
    sv = ai + mi * sv;
    const float ebt = expf(lbC - tk[(size_t)i * TKS + 3]);
    *reinterpret_cast<float2*>(tk + (size_t)i * TKS + 0) = make_float2(lr[i] * sv, lr[i] * ebt);
    *reinterpret_cast<float2*>(tk + (size_t)i * TKS + 4) = make_float2(sv, ebt);
  }
  if (t == 0) {
    float* cc = a.chunkc + ((size_t)chain * (L / C) + n) * 4;
    cc[0] = expf(laC);
    cc[1] = expf(lbC);
    cc[2] = (C > 0 ? mom[0] : 0.f) * sv;  // thread 0 ends at i = 0: sv = s_0
    cc[3] = 0.f;
  }
  if (stage) {
    __syncthreads();
    static_assert(TKS % 4 == 0, "whole 16-byte pieces per record");
    for (int e = t * 4; e < C * TKS; e += GSCAN_THREADS * 4)
      *reinterpret_cast<f32x4*>(tkg + e) = *reinterpret_cast<const f32x4*>(srec + e);
  }
}

hipError_t launch_global_scan(const GlobalArgs& a, hipStream_t st) {
  dim3 grid(a.D.L / a.D.C, a.D.B * a.D.H);
  const int stage = a.D.C <= GSCAN_STAGE_MAX;
  const size_t lds = stage ? (size_t)a.D.C * TKS * sizeof(float) : 0;
  if (stage) set_lds_limit((const void*)global_scan_kernel);
  hipLaunchKernelGGL(global_scan_kernel, grid, dim3(GSCAN_THREADS), lds, st, a, stage);
  return hipGetLastError();
}

// slot 0 of every chain = (W1_init, W2_init, 0, 0)
__global__ void global_init_kernel(GlobalArgs a) {
  const int chain = blockIdx.y;
  const int hh = chain % a.D.H;
  const size_t hd = (size_t)a.D.hid * a.D.d;
  float* st = a.states + (size_t)chain * a.nslots * 4 * hd;
  for (size_t e = blockIdx.x * blockDim.x + threadIdx.x; e < hd; e += gridDim.x * blockDim.x) {
    st[e] = a.W1i[hh * hd + e];
    st[hd + e] = a.W2i[hh * hd + e];
    st[2 * hd + e] = 0.f;
    st[3 * hd + e] = 0.f;
  }
}

hipError_t launch_global_init(const GlobalArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(global_init_kernel, dim3(16, a.D.B * a.D.H), dim3(256), 0, st, a);
  return hipGetLastError();
}

// token-tile rows per phase-1 workgroup, chosen so the tile fits in LDS
static int g1_rows(const Dims& D) {
  const size_t cts = D.bf16 ? 2 : 4;
  for (int tt = 64; tt > 16; tt >>= 1)
    if ((2 * (size_t)tt * D.d + (size_t)tt * D.hid) * cts <= 96 * 1024) return tt;
  return 16;
}

// ---- phase 1: retrieval at the chunk-entry state and R = (2/d) (f(V, k) - v)
template <typename IO, typename CT, int ACT, int D_, int H_>
__global__ void __launch_bounds__(256) global_p1_kernel(GlobalArgs a, int n, int TT) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Dims D = a.D;
  const int d = D_ ? D_ : D.d, h = H_ ? H_ : D.hid, C = D.C;
  const int chain = blockIdx.y;
  const int r0 = blockIdx.x * TT;                 // first row of the tile inside the chunk
  const int rows = min(TT, C - r0);
  const size_t hd = (size_t)h * d;
  const float* V = a.states + ((size_t)chain * a.nslots + (n % a.nslots)) * 4 * hd;
  const float *V1 = V, *V2 = V + hd;
  CT* sQ = (CT*)smem;
  CT* sK = sQ + (size_t)TT * d;
  CT* sH = sK + (size_t)TT * d;
  const size_t tok0 = (size_t)n * C + r0;
  const IO* q = (const IO*)a.q + ((size_t)chain * D.L + tok0) * d;
  const IO* k = (const IO*)a.k + ((size_t)chain * D.L + tok0) * d;
  const IO* v = (const IO*)a.v + ((size_t)chain * D.L + tok0) * d;
  float* o = a.o_part + ((size_t)chain * D.L + tok0) * d;
  float* R = a.Rbuf + ((size_t)chain * C + r0) * d;
  const float rscale = 2.0f / (float)d;  // d(1/d ||y - v||^2)/dy
  for (int e = threadIdx.x; e < TT * d; e += blockDim.x) {
    const int i = e / d;
    sQ[e] = from_f<CT>(i < rows ? to_f(q[e]) : 0.f);
    sK[e] = from_f<CT>(i < rows ? to_f(k[e]) : 0.f);
  }
  __syncthreads();
  gemm<CT, KC, KC>(TT, h, d, sQ, d, V1, d, [&](int i, int j, float z) {
    sH[(size_t)i * h + j] = from_f<CT>(act_f<ACT>(z));
  });
  __syncthreads();
  gemm<CT, KC, KC>(TT, d, h, sH, h, V2, h, [&](int i, int j, float x) {
    if (i < rows) o[(size_t)i * d + j] = x;
  });
  __syncthreads();
  gemm<CT, KC, KC>(TT, h, d, sK, d, V1, d, [&](int i, int j, float z) {
    sH[(size_t)i * h + j] = from_f<CT>(act_f<ACT>(z));
  });
  __syncthreads();
  gemm<CT, KC, KC>(TT, d, h, sH, h, V2, h, [&](int i, int j, float y) {
    if (i < rows) R[(size_t)i * d + j] = rscale * (y - to_f(v[(size_t)i * d + j]));
  });
}

// ---- phase 2: the carry, one hidden slice of 16 rows per workgroup
constexpr int G2_HS = 16;

static int g2_rows(const Dims& D) {
  const size_t cts = D.bf16 ? 2 : 4;
  for (int tt = 64; tt > 16; tt >>= 1)
    if ((6 * (size_t)tt * D.d + 2 * (size_t)G2_HS * tt) * cts <= 112 * 1024) return tt;
  return 16;
}

template <typename IO, typename CT, int ACT, int D_, int H_>
__global__ void __launch_bounds__(256) global_p2_kernel(GlobalArgs a, int n, int TT) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Dims D = a.D;
  const int d = D_ ? D_ : D.d, h = H_ ? H_ : D.hid, C = D.C;
  const int chain = blockIdx.z;
  const int s0 = blockIdx.x * G2_HS;
  const int split = blockIdx.y, nsplit = gridDim.y;
  const size_t hd = (size_t)h * d;
  const float* V = a.states + ((size_t)chain * a.nslots + (n % a.nslots)) * 4 * hd;
  const float *V1 = V, *V2 = V + hd;
  float* P = a.part + ((size_t)chain * nsplit + split) * 4 * hd;  // this split's partial sums
  constexpr int HS = G2_HS;
  CT* sK = (CT*)smem;                 // [TT][d]
  CT* sR = sK + TT * d;               // [TT][d]
  CT* sKcT = sR + TT * d;             // [d][TT]
  CT* sKbT = sKcT + d * TT;
  CT* sRcT = sKbT + d * TT;
  CT* sRbT = sRcT + d * TT;
  CT* sHkT = sRbT + d * TT;           // [HS][TT]
  CT* sD1T = sHkT + HS * TT;          // [HS][TT]
  const size_t tokc0 = (size_t)chain * D.L + (size_t)n * C;
  const float* tk = a.tokc + tokc0 * TKS;
  const IO* kk = (const IO*)a.k + tokc0 * d;
  const float* Rb = a.Rbuf + (size_t)chain * C * d;

  // persistent accumulators: V1/S1 slice (HS x d) and V2/S2 slice (d x HS)
  const int nt1 = d >> 4;  // tiles of the (HS x d) slice; the (d x HS) slice has as many
  f4 aw1[2], as1[2], aw2[2], as2[2];
  for (int x = 0; x < 2; ++x) aw1[x] = as1[x] = aw2[x] = as2[x] = zero4();

  const int ntile = (C + TT - 1) / TT;
  const int tb = split * ntile / nsplit, te = (split + 1) * ntile / nsplit;
  for (int r0 = tb * TT; r0 < te * TT; r0 += TT) {
    const int rows = min(TT, C - r0);
    for (int e = threadIdx.x; e < TT * d; e += blockDim.x) {
      const int i = e / d, j = e - i * d;
      const bool in = i < rows;
      const float kx = in ? to_f(kk[(size_t)(r0 + i) * d + j]) : 0.f;
      const float rx = in ? Rb[(size_t)(r0 + i) * d + j] : 0.f;
      const float cc = in ? tk[(size_t)(r0 + i) * TKS + 0] : 0.f;
      const float bb = in ? tk[(size_t)(r0 + i) * TKS + 1] : 0.f;
      sK[e] = from_f<CT>(kx);
      sR[e] = from_f<CT>(rx);
      sKcT[(size_t)j * TT + i] = from_f<CT>(cc * kx);
      sKbT[(size_t)j * TT + i] = from_f<CT>(bb * kx);
      sRcT[(size_t)j * TT + i] = from_f<CT>(cc * rx);
      sRbT[(size_t)j * TT + i] = from_f<CT>(bb * rx);
    }
    __syncthreads();
    // Zk and G for the slice: TT x HS, two accumulators per tile
    for (int t = wave_id(); t < TT / 16; t += num_waves()) {
      const int i0 = t * 16;
      f4 az = zero4(), ag = zero4();
      mma_tile<CT, KC, KC>(az, sK, d, i0, V1 + (size_t)s0 * d, d, 0, d);
      mma_tile<CT, KC, MC>(ag, sR, d, i0, V2 + s0, h, 0, d);
      const int l = lane_id();
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = l & 15;
        const ActVals av = act_all<ACT>(az[r]);
        sHkT[(size_t)j * TT + i] = from_f<CT>(av.s);
        sD1T[(size_t)j * TT + i] = from_f<CT>(ag[r] * av.d1);
      }
    }
    __syncthreads();
    for (int x = 0, t = wave_id(); t < nt1; t += num_waves(), ++x) {
      const int j0 = t * 16;
      mma_tile<CT, KC, KC>(aw1[x], sD1T, TT, 0, sKcT, TT, j0, TT);
      mma_tile<CT, KC, KC>(as1[x], sD1T, TT, 0, sKbT, TT, j0, TT);
      mma_tile<CT, KC, KC>(aw2[x], sRcT, TT, j0, sHkT, TT, 0, TT);
      mma_tile<CT, KC, KC>(as2[x], sRbT, TT, j0, sHkT, TT, 0, TT);
    }
    __syncthreads();
  }
  // partial sums of this token split (combined in fixed order by global_carry_reduce)
  const int l = lane_id();
  for (int x = 0, t = wave_id(); t < nt1; t += num_waves(), ++x) {
    const int j0 = t * 16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      {  // V1 / S1 slice element (s0 + i, j)
        const int i = 4 * (l >> 4) + r, j = j0 + (l & 15);
        const size_t e = (size_t)(s0 + i) * d + j;
        P[e] = aw1[x][r];
        P[2 * hd + e] = as1[x][r];
      }
      {  // V2 / S2 slice element (j0 + row, s0 + col)
        const int i = j0 + 4 * (l >> 4) + r, j = l & 15;
        const size_t e = (size_t)i * h + s0 + j;
        P[hd + e] = aw2[x][r];
        P[3 * hd + e] = as2[x][r];
      }
    }
  }
}

// V' = A_C V + E_C S - sum_splits dV,  S' = B_C S - sum_splits dS  (fixed split order)
__global__ void __launch_bounds__(256) global_carry_reduce(GlobalArgs a, int n, int nsplit) {
  const Dims D = a.D;
  const int chain = blockIdx.y;
  const size_t hd = (size_t)D.hid * D.d;
  const float* V = a.states + ((size_t)chain * a.nslots + (n % a.nslots)) * 4 * hd;
  float* Vn = a.states + ((size_t)chain * a.nslots + ((n + 1) % a.nslots)) * 4 * hd;
  const float* P = a.part + (size_t)chain * nsplit * 4 * hd;
  const float* cc = a.chunkc + ((size_t)chain * (D.L / D.C) + n) * 4;
  const float AC = cc[0], BC = cc[1], EC = cc[2];
  for (size_t e4 = blockIdx.x * blockDim.x + threadIdx.x; e4 < hd / 4;
       e4 += gridDim.x * blockDim.x) {
    const size_t e = e4 * 4;
#pragma unroll
    for (int m = 0; m < 2; ++m) {  // m = 0: (W1, S1), m = 1: (W2, S2)
      const size_t ew = (size_t)m * hd + e, es = (size_t)(2 + m) * hd + e;
      f32x4 dw = {0.f, 0.f, 0.f, 0.f}, ds = dw;
      for (int sp = 0; sp < nsplit; ++sp) {
        dw += *reinterpret_cast<const f32x4*>(P + (size_t)sp * 4 * hd + ew);
        ds += *reinterpret_cast<const f32x4*>(P + (size_t)sp * 4 * hd + es);
      }
      const f32x4 w = *reinterpret_cast<const f32x4*>(V + ew);
      const f32x4 sv = *reinterpret_cast<const f32x4*>(V + es);
      *reinterpret_cast<f32x4*>(Vn + ew) = AC * w + EC * sv - dw;
      *reinterpret_cast<f32x4*>(Vn + es) = BC * sv - ds;
    }
  }
}

hipError_t launch_global_carry_reduce(const GlobalArgs& a, int n, int nsplit, hipStream_t st) {
  hipLaunchKernelGGL(global_carry_reduce, dim3(GRED_BLOCKS, a.D.B * a.D.H), dim3(256), 0, st, a, n,
                     nsplit);
  return hipGetLastError();
}

int global_fwd_splits(const Dims& D) {
  const int tiles = (D.C + 63) / 64;
  return std::max(1, std::min(16, tiles / 4));
}

template <typename IO, typename CT, int ACT, int D_, int H_>
static hipError_t launch_gfwd_dims(const GlobalArgs& a, int n, hipStream_t st) {
  const Dims& D = a.D;
  const int TT = g1_rows(D);
  const size_t cts = sizeof(CT);
  dim3 g1((D.C + TT - 1) / TT, D.B * D.H);
  const size_t l1 = (2 * (size_t)TT * D.d + (size_t)TT * D.hid) * cts;
  set_lds_limit((const void*)global_p1_kernel<IO, CT, ACT, D_, H_>);
  hipLaunchKernelGGL((global_p1_kernel<IO, CT, ACT, D_, H_>), g1, dim3(256), l1, st, a, n, TT);
  const int T2 = g2_rows(D);
  const int ns = global_fwd_splits(D);
  dim3 g2(D.hid / G2_HS, ns, D.B * D.H);
  const size_t l2 = (6 * (size_t)T2 * D.d + 2 * (size_t)G2_HS * T2) * cts;
  set_lds_limit((const void*)global_p2_kernel<IO, CT, ACT, D_, H_>);
  hipLaunchKernelGGL((global_p2_kernel<IO, CT, ACT, D_, H_>), g2, dim3(256), l2, st, a, n, T2);
  hipLaunchKernelGGL(global_carry_reduce, dim3(GRED_BLOCKS, D.B * D.H), dim3(256), 0, st, a, n,
                     ns);
  return hipGetLastError();
}

template <typename IO, typename CT, int ACT>
static hipError_t launch_gfwd_t(const GlobalArgs& a, int n, hipStream_t st) {
  if (!a.force_generic) {
    if constexpr (sizeof(IO) == 2) {
      if (a.D.d == 64 && a.D.hid == 256) return launch_gfwd_dims<IO, CT, ACT, 64, 256>(a, n, st);
      if (a.D.d == 128 && a.D.hid == 512)
        return launch_gfwd_dims<IO, CT, ACT, 128, 512>(a, n, st);
    } else {
      if (a.D.d == 16 && a.D.hid == 32) return launch_gfwd_dims<IO, CT, ACT, 16, 32>(a, n, st);
    }
  }
  return launch_gfwd_dims<IO, CT, ACT, 0, 0>(a, n, st);
}

hipError_t launch_global_fwd_chunk(const GlobalArgs& a, int n, hipStream_t st) {
  hipError_t err = hipSuccess;
  if (launch_global_fwd_blk(a, n, st, &err)) return err;
  if (a.D.bf16)
    return a.D.act == ACT_GELU ? launch_gfwd_t<__bf16, __bf16, ACT_GELU>(a, n, st)
                               : launch_gfwd_t<__bf16, __bf16, ACT_SILU>(a, n, st);
  return a.D.act == ACT_GELU ? launch_gfwd_t<float, float, ACT_GELU>(a, n, st)
                             : launch_gfwd_t<float, float, ACT_SILU>(a, n, st);
}

// ---------------------------------------------------------------------------
// o = sum of the per-memory fp32 partials, written in the I/O dtype
// ---------------------------------------------------------------------------
template <typename IO, int NP>
__global__ void sum_out_kernel(SumJobs jobs, int njobs, size_t stride, size_t n, size_t per8,
                               size_t seg8) {
  // fixed-order sum of NP fp32 partials, 8 elements per thread (two 16-byte
  // loads per partial, all issued before the sum, one store), jobs along
  // blockIdx.y; the 8-element vectors taken are the first seg8 of every per8
  // (n: the count of elements taken)
  const int y = blockIdx.y;
  if (y >= njobs) return;
  const float* parts = jobs.parts[y];
  IO* out = (IO*)jobs.out[y];
  const size_t n8 = n / 8;
  for (size_t u = (size_t)blockIdx.x * blockDim.x + threadIdx.x; u < n8;
       u += (size_t)gridDim.x * blockDim.x) {
    const size_t v = seg8 == per8 ? u : (u / seg8) * per8 + u % seg8;
    f32x4 x0[NP], x1[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const float* q = parts + p * stride + v * 8;
      x0[p] = *reinterpret_cast<const f32x4*>(q);
      x1[p] = *reinterpret_cast<const f32x4*>(q + 4);
    }
    f32x4 s0 = x0[0], s1 = x1[0];
#pragma unroll
    for (int p = 1; p < NP; ++p) {
      s0 += x0[p];
      s1 += x1[p];
    }
    if constexpr (sizeof(IO) == 2) {
      bf16x8 o;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        o[t] = (__bf16)s0[t];
        o[t + 4] = (__bf16)s1[t];
      }
      *reinterpret_cast<bf16x8*>(out + v * 8) = o;
    } else {
      *reinterpret_cast<f32x4*>(out + v * 8) = s0;
      *reinterpret_cast<f32x4*>(out + v * 8 + 4) = s1;
    }
  }
  // tail (n not a multiple of 8; whole runs only)
  for (size_t e = n8 * 8 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    float sacc = 0.f;
    for (int p = 0; p < NP; ++p) sacc += parts[p * stride + e];
    out[e] = from_f<IO>(sacc);
  }
}

template <typename IO>
static hipError_t sum_outs_io(const SumJobs& jobs, int njobs, int nparts, size_t stride, size_t n,
                              size_t per8, size_t seg8, hipStream_t st) {
  // one 8-element vector per thread where the grid allows it
  const int blocks = (int)std::max<size_t>(1, std::min<size_t>((n / 8 + 255) / 256, 65535));
  const dim3 g(blocks, njobs), b(256);
  switch (nparts) {
    case 1: hipLaunchKernelGGL((sum_out_kernel<IO, 1>), g, b, 0, st, jobs, njobs, stride, n, per8, seg8); break;
    case 2: hipLaunchKernelGGL((sum_out_kernel<IO, 2>), g, b, 0, st, jobs, njobs, stride, n, per8, seg8); break;
    case 3: hipLaunchKernelGGL((sum_out_kernel<IO, 3>), g, b, 0, st, jobs, njobs, stride, n, per8, seg8); break;
    case 4: hipLaunchKernelGGL((sum_out_kernel<IO, 4>), g, b, 0, st, jobs, njobs, stride, n, per8, seg8); break;
    case 5: hipLaunchKernelGGL((sum_out_kernel<IO, 5>), g, b, 0, st, jobs, njobs, stride, n, per8, seg8); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_sum_outs(const SumJobs& jobs, int njobs, int nparts, size_t stride, size_t n,
                           int bf16, hipStream_t st) {
  return bf16 ? sum_outs_io<__bf16>(jobs, njobs, nparts, stride, n, n / 8, n / 8, st)
              : sum_outs_io<float>(jobs, njobs, nparts, stride, n, n / 8, n / 8, st);
}

hipError_t launch_sum_out_runs(const float* parts, int nparts, size_t stride, size_t nseq, size_t per,
                               size_t seg, void* out, int bf16, hipStream_t st) {
  if (per % 8 || seg % 8 || seg > per) return hipErrorInvalidValue;
  if (seg == 0 || nseq == 0) return hipSuccess;
  SumJobs jobs{};
  jobs.parts[0] = parts;
  jobs.out[0] = out;
  const size_t n = nseq * seg;
  return bf16 ? sum_outs_io<__bf16>(jobs, 1, nparts, stride, n, per / 8, seg / 8, st)
              : sum_outs_io<float>(jobs, 1, nparts, stride, n, per / 8, seg / 8, st);
}

hipError_t launch_sum_out(const float* parts, int nparts, size_t stride, size_t n, void* out,
                          int bf16, hipStream_t st) {
  SumJobs jobs{};
  jobs.parts[0] = parts;
  jobs.out[0] = out;
  return launch_sum_outs(jobs, 1, nparts, stride, n, bf16, st);
}

// final global state (slot `last`) -> [B*H][4][hid*d]
__global__ void copy_final_kernel(const float* states, int nslots, size_t slot_elems, int last,
                                  float* out) {
  const int chain = blockIdx.y;
  const float* src = states + ((size_t)chain * nslots + last) * slot_elems;
  float* dst = out + (size_t)chain * slot_elems;
  for (size_t e = blockIdx.x * blockDim.x + threadIdx.x; e < slot_elems;
       e += gridDim.x * blockDim.x)
    dst[e] = src[e];
}

hipError_t launch_copy_final(const float* states, int nslots, int nchains, size_t slot_elems,
                             int last, float* out, hipStream_t st) {
  hipLaunchKernelGGL(copy_final_kernel, dim3(32, nchains), dim3(256), 0, st, states, nslots,
                     slot_elems, last, out);
  return hipGetLastError();
}

// The saved buffer's header, one 4-byte word per thread.
__global__ void write_header_kernel(uint32_t* dst, SavedHeader h) {
  constexpr int W = (int)(sizeof(SavedHeader) / 4);
  static_assert(sizeof(SavedHeader) % 4 == 0, "whole words");
  const int i = threadIdx.x;
  if (i < W) dst[i] = reinterpret_cast<const uint32_t*>(&h)[i];
}

hipError_t launch_write_header(void* dst, const SavedHeader& h, hipStream_t st) {
  hipLaunchKernelGGL(write_header_kernel, dim3(1), dim3(64), 0, st, (uint32_t*)dst, h);
  return hipGetLastError();
}

}  // namespace tnt
