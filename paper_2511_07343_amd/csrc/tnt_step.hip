// Step-wise forward (prefill / decode) of the TNT memory layer from a carried
// state.
//
// Within a chunk every gradient is taken at the chunk-entry weights (Sec. 2.2)
// and folded in with momentum and decay (App. D), so the chunkwise rule has an
// exact token-by-token form once the entry weights are kept beside the
// running ones:
//     u_t = grad_W l(W^; k_t, v_t)           (W^ = weights entering t's chunk)
//     S_t = mom_t S_{t-1} - lr_t u_t,    W_t = (1 - decay_t) W_{t-1} + S_t,
// and W^ <- W at every chunk start.  The global memory reads at its entry
// state, o_G = f(V^, q_t) (Sec. 4.1.2 retrieval box); a local memory resets
// (W^, W, S, M) to (W_init, W_init, 0, 0) at each shard start, adds
// k_t k_t^T / ||k_t||^2 to its Q-K sum M and reads at W_t after the update,
// o_i = f(W_t, M q_t) (Sec. 4.1.1 local update, Sec. 4.1.2; App. C).
//
// The state of every (memory, chain) is split by hidden unit into G slices of
// HS = min(64, hid): slice g owns rows [g HS, (g+1) HS) of W^1, W1, S1 and the
// same columns of W^2, W2, S2, and one workgroup per (slice, chain, memory)
// touches nothing else of the state.  Each token takes three launches:
//   K1: chunk / shard boundary of the slice; z = W^1 k (and the global
//       retrieval's W^1 q) for the slice's rows; s(z), s'(z) to scratch; the
//       slice's share of W^2 s(z) (and W^2 s(W^1 q)); a local memory's query
//       x = M_t q (slice 0);
//   K2: r = (2/d)(sum of the shares - v); the slice's delta = (W^2^T r) s'(z);
//       the gated update of the slice; a local memory's W1_t x on the fresh
//       rows and its share of W2_t s(W1_t x); M += k k^T / ||k||^2 (slice 0);
//   K3: o = sum of the retrieval shares (global memory first, fixed order).
// The work is matrix-vector products and rank-one updates of the fp32 state
// (HBM-bound), with 16-byte loads issued in batches; there is no contraction
// long enough for MFMA tiles.
#include "tnt_device.h"
#include "tnt_kernels.h"

namespace tnt {

namespace {

constexpr int STEP_THREADS = 256;
constexpr int STEP_MAX_D = 128, STEP_MAX_H = 512;
constexpr int SEG4 = 16;                  // 16-byte loads a thread issues before reducing
constexpr int STEP_PART = 4096;           // LDS floats of the partial sums

// One row-dot job: y[r] = A[r] . x (and y2[r] = A[r] . x2 when x2 is set) for r < R.
struct RowJob {
  const float* A;
  int R, N, lda;  // rows, row length, row stride (floats)
  const float *x, *x2;
  float *y, *y2;
};

// Runs up to two jobs in one pass.  Each row is cut into segments of up to
// SEG4 float4; a thread loads a whole segment, then forms its dots with the
// job's vectors; the segment sums meet in `part` (at most STEP_PART floats:
// R * segments * vectors summed over the jobs).
__device__ __forceinline__ void row_dots_2(const RowJob j0, const RowJob j1, float* part) {
  const int s0 = (j0.N / 4) < SEG4 ? 1 : (j0.N / 4) / SEG4;
  const int s1 = (j1.N / 4) < SEG4 ? 1 : (j1.N / 4) / SEG4;
  const int n0 = j0.R * s0, n1 = j1.R * s1;
  const int v0 = j0.x2 ? 2 : 1;
  float* part1 = part + v0 * n0;
  for (int it = threadIdx.x; it < n0 + n1; it += blockDim.x) {
    const bool first = it < n0;
    // the job's fields picked by value (a reference would put the jobs in scratch)
    const float* jA = first ? j0.A : j1.A;
    const float* jx = first ? j0.x : j1.x;
    const float* jx2 = first ? j0.x2 : j1.x2;
    const int jN = first ? j0.N : j1.N, jld = first ? j0.lda : j1.lda;
    const int S = first ? s0 : s1, ii = first ? it : it - n0;
    const int n4 = jN / 4, seg4 = n4 < SEG4 ? n4 : SEG4;
    const int r = ii / S, sg = ii - r * S;
    const f4* row = reinterpret_cast<const f4*>(jA + (size_t)r * jld) + sg * seg4;
    f4 buf[SEG4];
#pragma unroll
    for (int c = 0; c < SEG4; ++c)
      if (c < seg4) buf[c] = row[c];
    const f4* x4 = reinterpret_cast<const f4*>(jx) + sg * seg4;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < SEG4; ++c)
      if (c < seg4) {
        const f4 xv = x4[c];
        acc += buf[c][0] * xv[0] + buf[c][1] * xv[1] + buf[c][2] * xv[2] + buf[c][3] * xv[3];
      }
    (first ? part : part1)[ii] = acc;
    if (jx2) {
      const f4* y4 = reinterpret_cast<const f4*>(jx2) + sg * seg4;
      float acc2 = 0.f;
#pragma unroll
      for (int c = 0; c < SEG4; ++c)
        if (c < seg4) {
          const f4 xv = y4[c];
          acc2 += buf[c][0] * xv[0] + buf[c][1] * xv[1] + buf[c][2] * xv[2] + buf[c][3] * xv[3];
        }
      (first ? part + n0 : part1 + n1)[ii] = acc2;
    }
  }
  __syncthreads();
  for (int r = threadIdx.x; r < j0.R + j1.R; r += blockDim.x) {
    const bool first = r < j0.R;
    float* jy = first ? j0.y : j1.y;
    float* jy2 = first ? j0.y2 : j1.y2;
    const bool two = first ? j0.x2 != nullptr : j1.x2 != nullptr;
    const int S = first ? s0 : s1, rr = first ? r : r - j0.R, n = first ? n0 : n1;
    const float* pp = first ? part : part1;
    float acc = 0.f;
    for (int sg = 0; sg < S; ++sg) acc += pp[rr * S + sg];
    jy[rr] = acc;
    if (two) {
      float acc2 = 0.f;
      for (int sg = 0; sg < S; ++sg) acc2 += pp[n + rr * S + sg];
      jy2[rr] = acc2;
    }
  }
}

__device__ __forceinline__ void row_dots(const float* A, int R, int N, const float* x, float* y,
                                         float* part) {
  const RowJob j0{A, R, N, N, x, nullptr, y, nullptr}, none{A, 0, N, N, x, nullptr, y, nullptr};
  row_dots_2(j0, none, part);
}

// y[c] = sum_r A[r][c] x[r] for c < N.  A thread takes four columns (one
// float4) over a run of up to SEG4 rows, loading the run first; the run sums
// meet in `part` (N/4 * runs * 4 <= STEP_PART here).
__device__ __forceinline__ void col_dots(const float* A, int R, int N, int lda, const float* x,
                                         float* y, float* part) {
  const int n4 = N / 4, ld4 = lda / 4;
  const int run = R < SEG4 ? R : SEG4;
  const int nr = R / run;
  const f4* A4 = reinterpret_cast<const f4*>(A);
  f4* p4 = reinterpret_cast<f4*>(part);
  for (int it = threadIdx.x; it < n4 * nr; it += blockDim.x) {
    const int c4 = it % n4, rr = it / n4;
    const int r0 = rr * run;
    f4 buf[SEG4];
#pragma unroll
    for (int i = 0; i < SEG4; ++i)
      if (i < run) buf[i] = A4[(size_t)(r0 + i) * ld4 + c4];
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < SEG4; ++i)
      if (i < run) acc += buf[i] * x[r0 + i];
    p4[it] = acc;
  }
  __syncthreads();
  for (int c = threadIdx.x; c < N; c += blockDim.x) {
    const int c4 = c >> 2, e = c & 3;
    float acc = 0.f;
    for (int rr = 0; rr < nr; ++rr) acc += part[(size_t)(rr * n4 + c4) * 4 + e];
    y[c] = acc;
  }
}

}  // namespace

// scratch of one (memory, chain), floats: s(z) [hid], s'(z) [hid], x [d],
// then per slice the shares W^2 s(z) [G][d], global W^2 s(W^1 q) [G][d] and
// local W2_t s(W1_t x) [G][d]
struct StepScr {
  float *a, *sp, *x, *yp, *yq, *y2;
};
__device__ __forceinline__ StepScr step_scr(const StepArgs& a, int m, int chain) {
  float* b = a.scratch + ((size_t)m * a.B * a.H + chain) * a.sc_stride;
  StepScr s;
  s.a = b;
  s.sp = b + a.hid;
  s.x = b + 2 * a.hid;
  s.yp = s.x + a.d;
  s.yq = s.yp + (size_t)a.G * a.d;
  s.y2 = s.yq + (size_t)a.G * a.d;
  return s;
}

template <typename IO, int ACT>
__global__ void __launch_bounds__(STEP_THREADS) step_k1(StepArgs a) {
  __shared__ __align__(16) float sq[STEP_MAX_D], sk[STEP_MAX_D], sx[STEP_MAX_D], sy[STEP_MAX_D],
      syq[STEP_MAX_D];
  __shared__ __align__(16) float sz[64], sa[64], szq[64], saq[64];
  __shared__ __align__(16) float part[STEP_PART];
  __shared__ float red[STEP_THREADS / WAVE];
  const int g = blockIdx.x, chain = blockIdx.y, m = blockIdx.z;
  const int H = a.H, d = a.d, hid = a.hid, HS = a.HS, j0 = g * HS;
  const int b = chain / H, h = chain - b * H, t = a.t;
  const long long p = a.pos + t;
  const bool global = a.has_global && m == 0;
  const size_t hd = (size_t)hid * d;
  float* base = a.state + ((size_t)m * a.B * H + chain) * a.mem_stride;
  float *Wh1 = base, *Wh2 = base + hd, *W1 = base + 2 * hd, *W2 = base + 3 * hd,
        *S1 = base + 4 * hd, *S2 = base + 5 * hd, *Mq = base + 6 * hd;
  const StepScr sc = step_scr(a, m, chain);
  const size_t tok = ((size_t)chain * a.T + t) * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    sq[i] = to_f(((const IO*)a.q)[tok + i]);
    sk[i] = to_f(((const IO*)a.k)[tok + i]);
  }

  // chunk / shard boundary, restricted to the slice (and M on slice 0)
  const bool reset = !global && p % a.S[m] == 0;
  if (reset || p % a.C[m] == 0) {
    const float* W1i = a.W1i + ((size_t)m * H + h) * hd;
    const float* W2i = a.W2i + ((size_t)m * H + h) * hd;
    for (int e = threadIdx.x; e < HS * d; e += blockDim.x) {  // rows of W^1, W1, S1
      const size_t i1 = (size_t)j0 * d + e;
      if (reset) {
        Wh1[i1] = W1[i1] = W1i[i1];
        S1[i1] = 0.f;
      } else {
        Wh1[i1] = W1[i1];
      }
    }
    for (int e = threadIdx.x; e < HS * d; e += blockDim.x) {  // columns of W^2, W2, S2
      const int i = e / HS, jj = e - i * HS;
      const size_t i2 = (size_t)i * hid + j0 + jj;
      if (reset) {
        Wh2[i2] = W2[i2] = W2i[i2];
        S2[i2] = 0.f;
      } else {
        Wh2[i2] = W2[i2];
      }
    }
    if (!global && g == 0 && (reset || a.qk_scope == 1))
      for (int e = threadIdx.x; e < d * d; e += blockDim.x) Mq[e] = 0.f;
  }
  __syncthreads();

  // z = W^1 k on the slice's rows (and the global retrieval's W^1 q); a local
  // memory's M_{t-1} q on slice 0
  const bool proj = !global && a.qk_proj && g == 0;
  {
    const RowJob r1{Wh1 + (size_t)j0 * d, HS, d, d, sk, global ? sq : nullptr, sz,
                    global ? szq : nullptr};
    const RowJob r2{Mq, proj ? d : 0, d, d, sq, nullptr, sx, nullptr};
    row_dots_2(r1, r2, part);
  }
  __syncthreads();
  for (int jj = threadIdx.x; jj < HS; jj += blockDim.x) {
    const ActVals av = act_all<ACT>(sz[jj]);
    sa[jj] = av.s;
    sc.a[j0 + jj] = av.s;
    sc.sp[j0 + jj] = av.d1;
    if (global) saq[jj] = act_f<ACT>(szq[jj]);
  }
  __syncthreads();
  // the slice's share of W^2 s(z) (and of W^2 s(W^1 q))
  {
    const RowJob r1{Wh2 + j0, d, HS, hid, sa, global ? saq : nullptr, sy, global ? syq : nullptr};
    const RowJob none{Wh2, 0, HS, hid, sa, nullptr, sy, nullptr};
    row_dots_2(r1, none, part);
  }
  float kk = 0.f, kq = 0.f;
  if (!global && g == 0) {
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
      kk += sk[i] * sk[i];
      kq += sk[i] * sq[i];
    }
  }
  kk = block_sum(kk, red);  // (barrier inside: the shares are complete)
  kq = block_sum(kq, red);
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    sc.yp[(size_t)g * d + i] = sy[i];
    if (global) sc.yq[(size_t)g * d + i] = syq[i];
    // local query x = M_t q = M_{t-1} q + k (k . q) / ||k||^2, or q
    if (!global && g == 0) {
      const float ikk = kk > 0.f ? 1.0f / kk : 0.f;
      sc.x[i] = a.qk_proj ? sx[i] + sk[i] * (kq * ikk) : sq[i];
    }
  }
}

template <typename IO, int ACT>
__global__ void __launch_bounds__(STEP_THREADS) step_k2(StepArgs a) {
  __shared__ __align__(16) float sk[STEP_MAX_D], sr[STEP_MAX_D], sx[STEP_MAX_D], sy[STEP_MAX_D];
  __shared__ __align__(16) float sa[64], sp[64], sg[64], sz[64];
  __shared__ __align__(16) float part[STEP_PART];
  __shared__ float red[STEP_THREADS / WAVE];
  const int g = blockIdx.x, chain = blockIdx.y, m = blockIdx.z;
  const int B = a.B, H = a.H, d = a.d, hid = a.hid, HS = a.HS, G = a.G, j0 = g * HS;
  const int b = chain / H, h = chain - b * H, t = a.t;
  const bool global = a.has_global && m == 0;
  const size_t hd = (size_t)hid * d;
  float* base = a.state + ((size_t)m * B * H + chain) * a.mem_stride;
  float *Wh2 = base + hd, *W1 = base + 2 * hd, *W2 = base + 3 * hd, *S1 = base + 4 * hd,
        *S2 = base + 5 * hd, *Mq = base + 6 * hd;
  const StepScr sc = step_scr(a, m, chain);
  const size_t tok = ((size_t)chain * a.T + t) * d;
  const size_t gi = (((size_t)m * B + b) * H + h) * a.T + t;
  const float eta = a.lr[gi], beta = a.mom[gi], alpha = a.decay[gi];
  const float rs = 2.0f / (float)d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    sk[i] = to_f(((const IO*)a.k)[tok + i]);
    float y = 0.f;
    for (int gg = 0; gg < G; ++gg) y += sc.yp[(size_t)gg * d + i];
    sr[i] = rs * (y - to_f(((const IO*)a.v)[tok + i]));
    if (!global) sx[i] = sc.x[i];
  }
  for (int jj = threadIdx.x; jj < HS; jj += blockDim.x) {
    sa[jj] = sc.a[j0 + jj];
    sp[jj] = sc.sp[j0 + jj];
  }
  __syncthreads();
  // delta = (W^2^T r) * s'(z) on the slice
  col_dots(Wh2 + j0, d, HS, hid, sr, sg, part);
  __syncthreads();
  for (int jj = threadIdx.x; jj < HS; jj += blockDim.x) sg[jj] *= sp[jj];
  __syncthreads();

  // gated update of the slice (16-byte accesses, UNR per array in flight);
  // a local memory also forms z'[j] = W1_t[j] . x from the fresh rows (the
  // d/4 lanes of a row are adjacent in a wave and sum by shuffles)
  const float keep = 1.0f - alpha;
  constexpr int UNR = 4;
  const int g4 = d / 4, h4 = HS / 4, n4 = HS * d / 4;  // n4: a multiple of 64
  const f4* k4 = reinterpret_cast<const f4*>(sk);
  const f4* x4 = reinterpret_cast<const f4*>(sx);
  const f4* a4 = reinterpret_cast<const f4*>(sa);
  {
    f4 *S14 = reinterpret_cast<f4*>(S1 + (size_t)j0 * d), *W14 = reinterpret_cast<f4*>(W1 + (size_t)j0 * d);
    for (int e0 = threadIdx.x; e0 < n4; e0 += UNR * blockDim.x) {
      f4 s1[UNR], w1[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = e0 + u * blockDim.x;
        if (e < n4) {
          s1[u] = S14[e];
          w1[u] = W14[e];
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = e0 + u * blockDim.x;
        if (e < n4) {  // whole waves take this branch
          const int jj = e / g4, l4 = e - jj * g4;
          const f4 n1 = beta * s1[u] - (eta * sg[jj]) * k4[l4];
          const f4 nw = keep * w1[u] + n1;
          S14[e] = n1;
          W14[e] = nw;
          if (!global) {
            const f4 xv = x4[l4];
            float zp = nw[0] * xv[0] + nw[1] * xv[1] + nw[2] * xv[2] + nw[3] * xv[3];
            for (int o_ = 1; o_ < g4; o_ <<= 1) zp += __shfl_xor(zp, o_, WAVE);
            if (l4 == 0) sz[jj] = zp;
          }
        }
      }
    }
  }
  {
    for (int e0 = threadIdx.x; e0 < n4; e0 += UNR * blockDim.x) {
      f4 s2[UNR], w2[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = e0 + u * blockDim.x;
        if (e < n4) {
          const int i = e / h4, c4 = e - i * h4;
          const size_t ofs = (size_t)i * hid + j0 + 4 * c4;
          s2[u] = *reinterpret_cast<const f4*>(S2 + ofs);
          w2[u] = *reinterpret_cast<const f4*>(W2 + ofs);
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = e0 + u * blockDim.x;
        if (e < n4) {
          const int i = e / h4, c4 = e - i * h4;
          const size_t ofs = (size_t)i * hid + j0 + 4 * c4;
          const f4 n2 = beta * s2[u] - (eta * sr[i]) * a4[c4];
          *reinterpret_cast<f4*>(S2 + ofs) = n2;
          *reinterpret_cast<f4*>(W2 + ofs) = keep * w2[u] + n2;
        }
      }
    }
  }
  if (!global && g == 0) {
    float kk = 0.f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) kk += sk[i] * sk[i];
    kk = block_sum(kk, red);
    const float ikk = kk > 0.f ? 1.0f / kk : 0.f;
    for (int e = threadIdx.x; e < d * d; e += blockDim.x) {
      const int i = e / d, j = e - i * d;
      Mq[e] += sk[i] * sk[j] * ikk;
    }
  }
  if (global) return;
  __syncthreads();
  // the slice's share of the local retrieval W2_t s(W1_t x)
  for (int jj = threadIdx.x; jj < HS; jj += blockDim.x) sa[jj] = act_f<ACT>(sz[jj]);
  __syncthreads();
  {
    const RowJob r1{W2 + j0, d, HS, hid, sa, nullptr, sy, nullptr};
    const RowJob none{W2, 0, HS, hid, sa, nullptr, sy, nullptr};
    row_dots_2(r1, none, part);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < d; i += blockDim.x) sc.y2[(size_t)g * d + i] = sy[i];
}

// o = the global retrieval's shares, then each local memory's (fixed order)
template <typename IO>
__global__ void __launch_bounds__(128) step_k3(StepArgs a) {
  const int chain = blockIdx.x, d = a.d, G = a.G;
  IO* o = (IO*)a.o + ((size_t)chain * a.T + a.t) * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    float acc = 0.f;
    for (int m = 0; m < a.M; ++m) {
      const StepScr sc = step_scr(a, m, chain);
      const float* sh = (a.has_global && m == 0) ? sc.yq : sc.y2;
      for (int gg = 0; gg < G; ++gg) acc += sh[(size_t)gg * d + i];
    }
    o[i] = from_f<IO>(acc);
  }
}

// state blocks of every (memory, chain): W^1 = W1 = W1_init[m][h], W^2 = W2 =
// W2_init[m][h], S = 0, M = 0
__global__ void __launch_bounds__(256) step_init_kernel(StepArgs a) {
  const int chain = blockIdx.x, m = blockIdx.y;
  const int h = chain % a.H;
  const size_t hd = (size_t)a.hid * a.d;
  float* base = a.state + ((size_t)m * a.B * a.H + chain) * a.mem_stride;
  const float* W1i = a.W1i + ((size_t)m * a.H + h) * hd;
  const float* W2i = a.W2i + ((size_t)m * a.H + h) * hd;
  for (size_t e = threadIdx.x; e < hd; e += blockDim.x) {
    base[e] = base[2 * hd + e] = W1i[e];
    base[hd + e] = base[3 * hd + e] = W2i[e];
    base[4 * hd + e] = 0.f;
    base[5 * hd + e] = 0.f;
  }
  for (size_t e = 6 * hd + threadIdx.x; e < a.mem_stride; e += blockDim.x) base[e] = 0.f;
}

// the global memory's block from a forward's final state [chain][4][hid*d]
// (V1, V2, S1, S2): W^1 = W1 = V1, W^2 = W2 = V2, S1, S2
__global__ void __launch_bounds__(256) step_from_final_kernel(StepArgs a, const float* fin) {
  const int chain = blockIdx.x;
  const size_t hd = (size_t)a.hid * a.d;
  float* base = a.state + (size_t)chain * a.mem_stride;  // memory 0
  const float* f = fin + (size_t)chain * 4 * hd;
  for (size_t e = threadIdx.x; e < hd; e += blockDim.x) {
    base[e] = base[2 * hd + e] = f[e];
    base[hd + e] = base[3 * hd + e] = f[hd + e];
    base[4 * hd + e] = f[2 * hd + e];
    base[5 * hd + e] = f[3 * hd + e];
  }
}

hipError_t launch_step_from_final(const StepArgs& a, const float* fin, hipStream_t st) {
  hipLaunchKernelGGL(step_init_kernel, dim3(a.B * a.H, a.M), dim3(256), 0, st, a);
  if (a.has_global && fin)
    hipLaunchKernelGGL(step_from_final_kernel, dim3(a.B * a.H), dim3(256), 0, st, a, fin);
  return hipGetLastError();
}

size_t step_state_floats(int d, int hid) { return 6 * (size_t)hid * d + (size_t)d * d; }

size_t step_scratch_floats(int d, int hid) {
  const int HS = hid < 64 ? hid : 64, G = hid / HS;
  const size_t n = 2 * (size_t)hid + d + 3 * (size_t)G * d;
  return (n + 63) / 64 * 64;
}

hipError_t launch_step_init(const StepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(step_init_kernel, dim3(a.B * a.H, a.M), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <typename IO, int ACT>
static hipError_t step_tokens(StepArgs a, hipStream_t st) {
  const dim3 grid(a.G, a.B * a.H, a.M), block(STEP_THREADS);
  for (int t = 0; t < a.T; ++t) {
    a.t = t;
    hipLaunchKernelGGL((step_k1<IO, ACT>), grid, block, 0, st, a);
    hipLaunchKernelGGL((step_k2<IO, ACT>), grid, block, 0, st, a);
    hipLaunchKernelGGL((step_k3<IO>), dim3(a.B * a.H), dim3(128), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_step(const StepArgs& a, hipStream_t st) {
  if (a.d > STEP_MAX_D || a.hid > STEP_MAX_H || a.HS > 64 || a.G * a.HS != a.hid || !a.scratch)
    return hipErrorInvalidValue;
  if (a.bf16)
    return a.act == ACT_SILU ? step_tokens<__bf16, ACT_SILU>(a, st) : step_tokens<__bf16, ACT_GELU>(a, st);
  return a.act == ACT_SILU ? step_tokens<float, ACT_SILU>(a, st) : step_tokens<float, ACT_GELU>(a, st);
}

}  // namespace tnt
