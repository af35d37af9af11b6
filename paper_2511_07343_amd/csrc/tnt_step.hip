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
// One workgroup per (batch row, head) chain walks the step's tokens and the
// layer's memories in order.  The work per token is a handful of matrix-vector
// products and rank-one updates of the fp32 state (HBM-bound), done with
// coalesced wave-per-row dot products, thread-per-column dot products and
// elementwise passes; there is no contraction long enough for MFMA tiles.
#include "tnt_device.h"
#include "tnt_kernels.h"

namespace tnt {

namespace {

constexpr int STEP_THREADS = 512;
constexpr int STEP_MAX_D = 128, STEP_MAX_H = 512;
constexpr int SEG4 = 16;                  // 16-byte loads a thread issues before reducing
constexpr int STEP_PART = 4096;           // LDS floats of the partial sums

// One row-dot job: y[r] = A[r] . x (and y2[r] = A[r] . x2 when x2 is set) for r < R.
struct RowJob {
  const float* A;
  int R, N;
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
    const int jN = first ? j0.N : j1.N;
    const int S = first ? s0 : s1, ii = first ? it : it - n0;
    const int n4 = jN / 4, seg4 = n4 < SEG4 ? n4 : SEG4;
    const int r = ii / S, sg = ii - r * S;
    const f4* row = reinterpret_cast<const f4*>(jA) + (size_t)r * n4 + sg * seg4;
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
  const RowJob j0{A, R, N, x, nullptr, y, nullptr}, none{A, 0, N, x, nullptr, y, nullptr};
  row_dots_2(j0, none, part);
}

// y[c] = sum_r A[r][c] x[r] for c < N.  A thread takes four columns (one
// float4) over a run of up to SEG4 rows, loading the run first; the run sums
// meet in `part` (N/4 * runs * 4 <= STEP_PART here).
__device__ __forceinline__ void col_dots(const float* A, int R, int N, const float* x, float* y,
                                         float* part) {
  const int n4 = N / 4;
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
      if (i < run) buf[i] = A4[(size_t)(r0 + i) * n4 + c4];
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

template <typename IO, int ACT>
__global__ void __launch_bounds__(STEP_THREADS) step_kernel(StepArgs a) {
  __shared__ __align__(16) float sq[STEP_MAX_D], sk[STEP_MAX_D], sv[STEP_MAX_D], sx[STEP_MAX_D],
      sy[STEP_MAX_D], sr[STEP_MAX_D], so[STEP_MAX_D];
  __shared__ __align__(16) float sz[STEP_MAX_H], sa[STEP_MAX_H], sp[STEP_MAX_H], sg[STEP_MAX_H],
      szq[STEP_MAX_H], saq[STEP_MAX_H];
  __shared__ __align__(16) float syq[STEP_MAX_D];
  __shared__ __align__(16) float part[STEP_PART];
  __shared__ float red[STEP_THREADS / WAVE];
  const int chain = blockIdx.x;
  const int B = a.B, H = a.H, T = a.T, d = a.d, hid = a.hid;
  const int b = chain / H, h = chain - b * H;
  const size_t hd = (size_t)hid * d;
  const IO* q = (const IO*)a.q + (size_t)chain * T * d;
  const IO* k = (const IO*)a.k + (size_t)chain * T * d;
  const IO* v = (const IO*)a.v + (size_t)chain * T * d;
  IO* o = (IO*)a.o + (size_t)chain * T * d;
  const float rs = 2.0f / (float)d;

  for (int t = 0; t < T; ++t) {
    const long long p = a.pos + t;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
      sq[i] = to_f(q[(size_t)t * d + i]);
      sk[i] = to_f(k[(size_t)t * d + i]);
      sv[i] = to_f(v[(size_t)t * d + i]);
      so[i] = 0.f;
    }
    __syncthreads();
    float kk = 0.f, kq = 0.f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
      kk += sk[i] * sk[i];
      kq += sk[i] * sq[i];
    }
    kk = block_sum(kk, red);
    kq = block_sum(kq, red);
    const float ikk = kk > 0.f ? 1.0f / kk : 0.f;

    for (int m = 0; m < a.M; ++m) {
      const bool global = a.has_global && m == 0;
      const int C = a.C[m];
      float* base = a.state + ((size_t)m * B * H + chain) * a.mem_stride;
      float *Wh1 = base, *Wh2 = base + hd, *W1 = base + 2 * hd, *W2 = base + 3 * hd,
            *S1 = base + 4 * hd, *S2 = base + 5 * hd, *Mq = base + 6 * hd;
      const size_t gi = (((size_t)m * B + b) * H + h) * T + t;
      const float eta = a.lr[gi], beta = a.mom[gi], alpha = a.decay[gi];

      // chunk / shard boundaries
      if (!global && p % a.S[m] == 0) {
        const float* W1i = a.W1i + ((size_t)m * H + h) * hd;
        const float* W2i = a.W2i + ((size_t)m * H + h) * hd;
        for (size_t e = threadIdx.x; e < hd; e += blockDim.x) {
          Wh1[e] = W1[e] = W1i[e];
          Wh2[e] = W2[e] = W2i[e];
          S1[e] = 0.f;
          S2[e] = 0.f;
        }
        for (int e = threadIdx.x; e < d * d; e += blockDim.x) Mq[e] = 0.f;
      } else if (p % C == 0) {
        for (size_t e = threadIdx.x; e < hd; e += blockDim.x) {
          Wh1[e] = W1[e];
          Wh2[e] = W2[e];
        }
        if (!global && a.qk_scope == 1)
          for (int e = threadIdx.x; e < d * d; e += blockDim.x) Mq[e] = 0.f;
      }
      __syncthreads();

      // phase 1: z = W^1 k, and in the same pass the global retrieval's W^1 q
      // or a local memory's M_{t-1} q
      const bool proj = !global && a.qk_proj;
      {
        const RowJob g1{Wh1, hid, d, sk, global ? sq : nullptr, sz, global ? szq : nullptr};
        const RowJob g2{Mq, proj ? d : 0, d, sq, nullptr, sx, nullptr};
        row_dots_2(g1, g2, part);
      }
      __syncthreads();
      for (int j = threadIdx.x; j < hid; j += blockDim.x) {
        const ActVals av = act_all<ACT>(sz[j]);
        sa[j] = av.s;
        sp[j] = av.d1;
        if (global) saq[j] = act_f<ACT>(szq[j]);
      }
      __syncthreads();
      // phase 2: y = W^2 s(z) (and the global retrieval W^2 s(W^1 q))
      {
        const RowJob g1{Wh2, d, hid, sa, global ? saq : nullptr, sy, global ? syq : nullptr};
        const RowJob none{Wh2, 0, hid, sa, nullptr, sy, nullptr};
        row_dots_2(g1, none, part);
      }
      __syncthreads();
      for (int i = threadIdx.x; i < d; i += blockDim.x) {
        sr[i] = rs * (sy[i] - sv[i]);
        if (global) so[i] += syq[i];
        // local query x = M_t q = M_{t-1} q + k (k . q) / ||k||^2, or q
        if (!global) sx[i] = proj ? sx[i] + sk[i] * (kq * ikk) : sq[i];
      }
      __syncthreads();
      // phase 3: delta = (W^2^T r) * s'(z)
      col_dots(Wh2, d, hid, sr, sg, part);
      __syncthreads();
      for (int j = threadIdx.x; j < hid; j += blockDim.x) sg[j] *= sp[j];
      __syncthreads();

      // phase 4: gated update, u1 = delta k^T (hid x d), u2 = r s(z)^T (d x hid),
      // 16-byte accesses, UNR per array in flight per thread.  A local memory
      // also forms z'[j] = W1_t[j] . x here: the d/4 lanes holding one row of
      // W1 are adjacent within a wave and sum by shuffles (fixed order).
      const float keep = 1.0f - alpha;
      {
        constexpr int UNR = 4;
        const int hd4 = (int)(hd / 4), g4 = d / 4;
        f4 *S14 = reinterpret_cast<f4*>(S1), *W14 = reinterpret_cast<f4*>(W1),
           *S24 = reinterpret_cast<f4*>(S2), *W24 = reinterpret_cast<f4*>(W2);
        const f4* k4 = reinterpret_cast<const f4*>(sk);
        const f4* a4 = reinterpret_cast<const f4*>(sa);
        const f4* x4 = reinterpret_cast<const f4*>(sx);
        for (int e0 = threadIdx.x; e0 < hd4; e0 += UNR * blockDim.x) {
          f4 s1[UNR], w1[UNR], s2[UNR], w2[UNR];
#pragma unroll
          for (int u = 0; u < UNR; ++u) {
            const int e = e0 + u * blockDim.x;
            if (e < hd4) {
              s1[u] = S14[e];
              w1[u] = W14[e];
              s2[u] = S24[e];
              w2[u] = W24[e];
            }
          }
#pragma unroll
          for (int u = 0; u < UNR; ++u) {
            const int e = e0 + u * blockDim.x;
            if (e < hd4) {  // hd4 is a multiple of 64: whole waves take this branch
              const int j1 = e / g4, l4 = e - j1 * g4;                   // W1, S1: [hid][d]
              const int i2 = (4 * e) / hid, j4 = (4 * e - i2 * hid) / 4;  // W2, S2: [d][hid]
              const f4 n1 = beta * s1[u] - (eta * sg[j1]) * k4[l4];
              const f4 n2 = beta * s2[u] - (eta * sr[i2]) * a4[j4];
              const f4 nw1 = keep * w1[u] + n1;
              S14[e] = n1;
              W14[e] = nw1;
              S24[e] = n2;
              W24[e] = keep * w2[u] + n2;
              if (!global) {
                const f4 xv = x4[l4];
                float zp = nw1[0] * xv[0] + nw1[1] * xv[1] + nw1[2] * xv[2] + nw1[3] * xv[3];
                for (int o_ = 1; o_ < g4; o_ <<= 1) zp += __shfl_xor(zp, o_, WAVE);
                if (l4 == 0) sz[j1] = zp;
              }
            }
          }
        }
      }
      if (!global) {
        for (int e = threadIdx.x; e < d * d; e += blockDim.x) {
          const int i = e / d, j = e - i * d;
          Mq[e] += sk[i] * sk[j] * ikk;
        }
      }
      __syncthreads();

      if (!global) {  // local retrieval at W_t: o += W2_t s(z')
        for (int j = threadIdx.x; j < hid; j += blockDim.x) sa[j] = act_f<ACT>(sz[j]);
        __syncthreads();
        row_dots(W2, d, hid, sa, sy, part);
        __syncthreads();
        for (int i = threadIdx.x; i < d; i += blockDim.x) so[i] += sy[i];
        __syncthreads();
      }
    }
    for (int i = threadIdx.x; i < d; i += blockDim.x) o[(size_t)t * d + i] = from_f<IO>(so[i]);
    __syncthreads();
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

size_t step_state_floats(int d, int hid) { return 6 * (size_t)hid * d + (size_t)d * d; }

hipError_t launch_step_init(const StepArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(step_init_kernel, dim3(a.B * a.H, a.M), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_step(const StepArgs& a, hipStream_t st) {
  if (a.d > STEP_MAX_D || a.hid > STEP_MAX_H) return hipErrorInvalidValue;
  const dim3 grid(a.B * a.H), block(STEP_THREADS);
  if (a.bf16) {
    if (a.act == ACT_SILU)
      hipLaunchKernelGGL((step_kernel<__bf16, ACT_SILU>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((step_kernel<__bf16, ACT_GELU>), grid, block, 0, st, a);
  } else {
    if (a.act == ACT_SILU)
      hipLaunchKernelGGL((step_kernel<float, ACT_SILU>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((step_kernel<float, ACT_GELU>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace tnt
