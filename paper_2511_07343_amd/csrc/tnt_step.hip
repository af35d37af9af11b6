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

// y[r] = sum_c A[r][c] x[c] for r < R.  Each row is cut into segments of up
// to SEG4 float4; a thread loads a whole segment, then reduces it; the
// segment sums meet in `part` (R * segments <= STEP_PART / 4 here).
__device__ __forceinline__ void row_dots(const float* A, int R, int N, const float* x, float* y,
                                         float* part) {
  const int n4 = N / 4;
  const int seg4 = n4 < SEG4 ? n4 : SEG4;
  const int S = n4 / seg4;
  const f4* A4 = reinterpret_cast<const f4*>(A);
  const f4* x4 = reinterpret_cast<const f4*>(x);
  for (int it = threadIdx.x; it < R * S; it += blockDim.x) {
    const int r = it / S, sg = it - r * S;
    const f4* row = A4 + (size_t)r * n4 + sg * seg4;
    f4 buf[SEG4];
#pragma unroll
    for (int c = 0; c < SEG4; ++c)
      if (c < seg4) buf[c] = row[c];
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < SEG4; ++c)
      if (c < seg4) {
        const f4 xv = x4[sg * seg4 + c];
        acc += buf[c][0] * xv[0] + buf[c][1] * xv[1] + buf[c][2] * xv[2] + buf[c][3] * xv[3];
      }
    part[it] = acc;
  }
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += blockDim.x) {
    float acc = 0.f;
    for (int sg = 0; sg < S; ++sg) acc += part[r * S + sg];
    y[r] = acc;
  }
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

// f(W, x) = W2 s(W1 x) added into acc[d]; z, a: hid-sized LDS vectors
template <int ACT>
__device__ void retrieve_add(const float* W1, const float* W2, int d, int hid, const float* x,
                             float* z, float* a, float* y, float* acc, float* part) {
  row_dots(W1, hid, d, x, z, part);
  __syncthreads();
  for (int j = threadIdx.x; j < hid; j += blockDim.x) a[j] = act_f<ACT>(z[j]);
  __syncthreads();
  row_dots(W2, d, hid, a, y, part);
  __syncthreads();
  for (int i = threadIdx.x; i < d; i += blockDim.x) acc[i] += y[i];
  __syncthreads();
}

}  // namespace

template <typename IO, int ACT>
__global__ void __launch_bounds__(STEP_THREADS) step_kernel(StepArgs a) {
  __shared__ __align__(16) float sq[STEP_MAX_D], sk[STEP_MAX_D], sv[STEP_MAX_D], sx[STEP_MAX_D],
      sy[STEP_MAX_D], sr[STEP_MAX_D], so[STEP_MAX_D];
  __shared__ __align__(16) float sz[STEP_MAX_H], sa[STEP_MAX_H], sp[STEP_MAX_H], sg[STEP_MAX_H];
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
    float kk = 0.f;
    for (int i = threadIdx.x; i < d; i += blockDim.x) kk += sk[i] * sk[i];
    kk = block_sum(kk, red);
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

      // global retrieval at the chunk-entry state
      if (global) retrieve_add<ACT>(Wh1, Wh2, d, hid, sq, sz, sa, sy, so, part);

      // inner gradient at the chunk-entry weights:
      // z = W^1 k, r = (2/d)(W^2 s(z) - v), delta = (W^2^T r) * s'(z)
      row_dots(Wh1, hid, d, sk, sz, part);
      __syncthreads();
      for (int j = threadIdx.x; j < hid; j += blockDim.x) {
        const ActVals av = act_all<ACT>(sz[j]);
        sa[j] = av.s;
        sp[j] = av.d1;
      }
      __syncthreads();
      row_dots(Wh2, d, hid, sa, sy, part);
      __syncthreads();
      for (int i = threadIdx.x; i < d; i += blockDim.x) sr[i] = rs * (sy[i] - sv[i]);
      __syncthreads();
      col_dots(Wh2, d, hid, sr, sg, part);
      __syncthreads();
      for (int j = threadIdx.x; j < hid; j += blockDim.x) sg[j] *= sp[j];
      __syncthreads();

      // gated update: u1 = delta k^T (hid x d), u2 = r s(z)^T (d x hid)
      // (16-byte accesses, UNR of them per array in flight per thread)
      const float keep = 1.0f - alpha;
      {
        constexpr int UNR = 4;
        const int hd4 = (int)(hd / 4);
        f4 *S14 = reinterpret_cast<f4*>(S1), *W14 = reinterpret_cast<f4*>(W1),
           *S24 = reinterpret_cast<f4*>(S2), *W24 = reinterpret_cast<f4*>(W2);
        const f4* k4 = reinterpret_cast<const f4*>(sk);
        const f4* a4 = reinterpret_cast<const f4*>(sa);
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
            if (e < hd4) {
              const int j1 = (4 * e) / d, l4 = (4 * e - j1 * d) / 4;   // W1, S1: [hid][d]
              const int i2 = (4 * e) / hid, j4 = (4 * e - i2 * hid) / 4;  // W2, S2: [d][hid]
              const f4 n1 = beta * s1[u] - (eta * sg[j1]) * k4[l4];
              const f4 n2 = beta * s2[u] - (eta * sr[i2]) * a4[j4];
              S14[e] = n1;
              W14[e] = keep * w1[u] + n1;
              S24[e] = n2;
              W24[e] = keep * w2[u] + n2;
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

      if (!global) {  // local retrieval at W_t, queried at M_t q_t (or q_t)
        const float* xq = sq;
        if (a.qk_proj) {
          row_dots(Mq, d, d, sq, sx, part);
          __syncthreads();
          xq = sx;
        }
        retrieve_add<ACT>(W1, W2, d, hid, xq, sz, sa, sy, so, part);
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
