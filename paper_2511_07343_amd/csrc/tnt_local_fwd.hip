// Local memories, forward: one workgroup per unit (batch row, head, shard)
// runs the shard's chunk loop.  Units are independent because every shard
// starts from the learned init (local update rule with reset, Sec. 4.1.1;
// App. E), so the grid covers all (b, h, shard) at once.
//
// Chunk step (chunk-entry state W1, W2, S1, S2, M0; 0-indexed positions):
//   X   = Q M0^T + tril(Q N^T) N                 Q-K projection incl. token t (App. C)
//   Zk  = K W1^T,  Hk = s(Zk)                    memory MLP on the keys at the
//   R   = (2/d) (Hk W2^T - V)                    chunk-entry weights (Sec. 2.2)
//   D1  = (R W2) * s'(Zk)                        u_tau = (D1_tau k_tau^T, R_tau Hk_tau^T)
//   W1' = A_C W1 + E_C S1 - D1^T diag(cC) K      state carry with momentum / decay
//   S1' = B_C S1 - D1^T diag(b) K                (W2', S2' alike with R^T, Hk)
//   Z   = diag(A) X W1^T + diag(E) X S1^T - (c o X K^T) D1      retrieval at W_t,
//   O   = diag(A) s(Z) W2^T + diag(E) s(Z) S2^T - (c o s(Z) Hk^T) R   causal in-chunk
// which equals f(W_t, x_t) with W_t after token t's own update, without ever
// forming W_t (dual form of the per-token recurrence).
#include "tnt_local_common.h"

namespace tnt {

size_t local_plan(const Dims& D, LocalPlan* p, bool backward) {
  const size_t Cp = D.Cp, d = D.d, h = D.hid;
  size_t off = 0;
  auto take = [&](size_t n) { size_t o = off; off += (n + 7) & ~size_t(7); return o; };
  *p = LocalPlan{};
  p->Q = take(Cp * d); p->K = take(Cp * d); p->N = take(Cp * d); p->NT = take(d * Cp);
  p->X = take(Cp * d); p->KcT = take(d * Cp); p->KbT = take(d * Cp);
  p->R = take(Cp * d); p->RT = take(d * Cp); p->RcT = take(d * Cp); p->RbT = take(d * Cp);
  p->S = take(Cp * Cp); p->P = take(Cp * Cp);
  p->Hk = take(Cp * h); p->HkT = take(h * Cp); p->Sp = take(Cp * h); p->D1T = take(h * Cp);
  p->H = take(Cp * h);
  if (backward) {
    p->Spp = take(Cp * h); p->G = take(Cp * h); p->D1 = take(Cp * h); p->Sz = take(Cp * h);
    p->HT = take(h * Cp); p->dZ = take(Cp * h); p->dZT = take(h * Cp); p->dGT = take(h * Cp);
    p->dZkT = take(h * Cp); p->dYkT = take(d * Cp); p->dXT = take(d * Cp); p->QT = take(d * Cp);
    p->KT = take(d * Cp); p->XT = take(d * Cp); p->XAT = take(d * Cp); p->XET = take(d * Cp);
    p->dOT = take(d * Cp); p->dOAT = take(d * Cp); p->dOET = take(d * Cp);
    p->PzT = take(Cp * Cp); p->PoT = take(Cp * Cp); p->Q1T = take(Cp * Cp);
    p->Q2T = take(Cp * Cp); p->dXN = take(Cp * Cp); p->dXNT = take(Cp * Cp); p->ST = take(Cp * Cp);
    p->Rb = take(Cp * d);
  }
  p->elems = off;
  return off;
}

template <typename IO, typename CT, int ACT>
__global__ void __launch_bounds__(512) local_fwd_kernel(LocalFwdArgs a) {
  __shared__ Coef cf;
  const Dims D = a.D;
  const int d = D.d, h = D.hid, C = D.C, Cp = D.Cp;
  const int nshard = D.L / D.S;
  const int u = blockIdx.x;
  const int b = u / (D.H * nshard), hh = (u / nshard) % D.H, s = u % nshard;
  const size_t hd = (size_t)h * d;
  const LocalPlan& P = a.plan;
  CT* sc = (CT*)a.scratch + (size_t)u * P.elems;
  CT *sQ = sc + P.Q, *sK = sc + P.K, *sN = sc + P.N, *sNT = sc + P.NT, *sX = sc + P.X;
  CT *sKcT = sc + P.KcT, *sKbT = sc + P.KbT, *sR = sc + P.R, *sRT = sc + P.RT;
  CT *sRcT = sc + P.RcT, *sRbT = sc + P.RbT, *sS = sc + P.S, *sP = sc + P.P;
  CT *sHk = sc + P.Hk, *sHkT = sc + P.HkT, *sSp = sc + P.Sp, *sD1T = sc + P.D1T, *sH = sc + P.H;

  const size_t chain = (size_t)b * D.H + hh;
  const IO* q = (const IO*)a.q + chain * D.L * d;
  const IO* k = (const IO*)a.k + chain * D.L * d;
  const IO* v = (const IO*)a.v + chain * D.L * d;
  float* o = a.o_part + chain * D.L * d;
  const float* lr = a.lr + chain * D.L;
  const float* mom = a.mom + chain * D.L;
  const float* dec = a.decay + chain * D.L;
  float* st = a.states + (size_t)u * a.nslots * 4 * hd;
  float* mst = a.mstates + (size_t)u * a.nslots * d * d;
  const bool shard_qk = D.qk_proj && D.qk_scope == 0;
  const float rscale = 2.0f / (float)d;  // d(1/d ||y - v||^2)/dy

  {  // slot 0 = learned init, zero momentum, zero Q-K sum
    const float* W1i = a.W1i + hh * hd;
    const float* W2i = a.W2i + hh * hd;
    for (size_t e = threadIdx.x; e < hd; e += blockDim.x) {
      st[e] = W1i[e];
      st[hd + e] = W2i[e];
      st[2 * hd + e] = 0.f;
      st[3 * hd + e] = 0.f;
    }
    if (shard_qk)
      for (int e = threadIdx.x; e < d * d; e += blockDim.x) mst[e] = 0.f;
  }
  __syncthreads();

  const int nch = D.S / C;
  const int gsub = D.gsub > 1 ? D.gsub : 1;
  for (int n = 0; n < nch; ++n) {
    const int tok0 = s * D.S + n * C;
    const float* cur = st + (size_t)(n % a.nslots) * 4 * hd;
    // the state the chunk's gradients are taken at: its own entry state, or with
    // gsub > 1 the state entering its group of gsub chunks (every slot is kept then)
    const float* gpt = st + (size_t)((n - n % gsub) % a.nslots) * 4 * hd;
    const float *W1g = gpt, *W2g = gpt + hd;
    float* nxt = st + (size_t)((n + 1) % a.nslots) * 4 * hd;
    const float *W1 = cur, *W2 = cur + hd, *S1 = cur + 2 * hd, *S2 = cur + 3 * hd;
    float *W1n = nxt, *W2n = nxt + hd, *S1n = nxt + 2 * hd, *S2n = nxt + 3 * hd;
    const float* Mc = mst + (size_t)(n % a.nslots) * d * d;
    float* Mn = mst + (size_t)((n + 1) % a.nslots) * d * d;

    // ---- stage tokens, gate coefficients
    stage_rows<IO, CT>(sQ, nullptr, q + (size_t)tok0 * d, C, Cp, d);
    stage_rows<IO, CT>(sK, nullptr, k + (size_t)tok0 * d, C, Cp, d);
    if (D.qk_proj) unit_keys<IO, CT>(cf, sN, sNT, k + (size_t)tok0 * d, C, Cp, d);
    chunk_coefs(cf, lr, mom, dec, tok0, C, Cp);  // ends with a barrier

    // ---- Q-K projection: X = Q M0^T + tril(Q N^T) N ; M' = M0 + N^T N
    if (D.qk_proj) {
      gemm<CT, KC, KC>(Cp, Cp, d, sQ, d, sN, d, [&](int i, int j, float x) {
        sS[(size_t)i * Cp + j] = from_f<CT>(j <= i ? x : 0.f);
      });
      __syncthreads();
      {
        const int tn = d >> 4, nt = (Cp >> 4) * tn;
        for (int t = wave_id(); t < nt; t += num_waves()) {
          const int i0 = (t / tn) << 4, j0 = (t % tn) << 4;
          f4 acc = zero4();
          if (shard_qk) mma_tile<CT, KC, KC>(acc, sQ, d, i0, Mc, d, j0, d);
          mma_tile<CT, KC, KC>(acc, sS, Cp, i0, sNT, Cp, j0, Cp);
          tile_each(acc, i0, j0, [&](int i, int j, float x) { sX[(size_t)i * d + j] = from_f<CT>(x); });
        }
      }
      if (shard_qk)
        gemm<CT, KC, KC>(d, d, Cp, sNT, Cp, sNT, Cp, [&](int i, int j, float x) {
          Mn[(size_t)i * d + j] = Mc[(size_t)i * d + j] + x;
        });
    } else {
      for (int e = threadIdx.x; e < Cp * d; e += blockDim.x) sX[e] = sQ[e];
    }

    // ---- Zk = K W1^T -> Hk, s'(Zk)
    gemm<CT, KC, KC>(Cp, h, d, sK, d, W1g, d, [&](int i, int j, float z) {
      const ActVals av = act_all<ACT>(z);
      sHk[(size_t)i * h + j] = from_f<CT>(av.s);
      sHkT[(size_t)j * Cp + i] = from_f<CT>(av.s);
      sSp[(size_t)i * h + j] = from_f<CT>(av.d1);
    });
    // scaled key copies for the carry
    for (int e = threadIdx.x; e < Cp * d; e += blockDim.x) {
      const int i = e / d, j = e - i * d;
      const float x = to_f(sK[e]);
      sKcT[(size_t)j * Cp + i] = from_f<CT>(cf.cC[i] * x);
      sKbT[(size_t)j * Cp + i] = from_f<CT>(cf.bb[i] * x);
    }
    __syncthreads();

    // ---- R = (2/d) (Hk W2^T - V)
    gemm<CT, KC, KC>(Cp, d, h, sHk, h, W2g, h, [&](int i, int j, float y) {
      const float r = (i < C) ? rscale * (y - to_f(v[(size_t)(tok0 + i) * d + j])) : 0.f;
      sR[(size_t)i * d + j] = from_f<CT>(r);
      sRT[(size_t)j * Cp + i] = from_f<CT>(r);
      sRcT[(size_t)j * Cp + i] = from_f<CT>(cf.cC[i] * r);
      sRbT[(size_t)j * Cp + i] = from_f<CT>(cf.bb[i] * r);
    });
    __syncthreads();

    // ---- D1 = (R W2) * s'(Zk)
    gemm<CT, KC, MC>(Cp, h, d, sR, d, W2g, h, [&](int i, int j, float g) {
      sD1T[(size_t)j * Cp + i] = from_f<CT>(g * to_f(sSp[(size_t)i * h + j]));
    });
    __syncthreads();

    // ---- carry into the next slot
    {
      const int tn = d >> 4, nt = (h >> 4) * tn;  // W1', S1' : h x d
      for (int t = wave_id(); t < nt; t += num_waves()) {
        const int i0 = (t / tn) << 4, j0 = (t % tn) << 4;
        f4 aw = zero4(), as = zero4();
        mma_tile<CT, KC, KC>(aw, sD1T, Cp, i0, sKcT, Cp, j0, Cp);
        mma_tile<CT, KC, KC>(as, sD1T, Cp, i0, sKbT, Cp, j0, Cp);
        const int l = lane_id();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * d + j0 + (l & 15);
          W1n[e] = cf.AC * W1[e] + cf.EC * S1[e] - aw[r];
          S1n[e] = cf.BC * S1[e] - as[r];
        }
      }
    }
    {
      const int tn = h >> 4, nt = (d >> 4) * tn;  // W2', S2' : d x h
      for (int t = wave_id(); t < nt; t += num_waves()) {
        const int i0 = (t / tn) << 4, j0 = (t % tn) << 4;
        f4 aw = zero4(), as = zero4();
        mma_tile<CT, KC, KC>(aw, sRcT, Cp, i0, sHkT, Cp, j0, Cp);
        mma_tile<CT, KC, KC>(as, sRbT, Cp, i0, sHkT, Cp, j0, Cp);
        const int l = lane_id();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * h + j0 + (l & 15);
          W2n[e] = cf.AC * W2[e] + cf.EC * S2[e] - aw[r];
          S2n[e] = cf.BC * S2[e] - as[r];
        }
      }
    }

    // ---- retrieval, dual form
    gemm<CT, KC, KC>(Cp, Cp, d, sX, d, sK, d, [&](int i, int j, float x) {
      sP[(size_t)i * Cp + j] = from_f<CT>(j <= i ? cf.c[i][j] * x : 0.f);
    });
    __syncthreads();
    {
      const int tn = h >> 4, nt = (Cp >> 4) * tn;
      for (int t = wave_id(); t < nt; t += num_waves()) {
        const int i0 = (t / tn) << 4, j0 = (t % tn) << 4;
        f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
        mma_tile<CT, KC, KC>(a1, sX, d, i0, W1, d, j0, d);
        mma_tile<CT, KC, KC>(a2, sX, d, i0, S1, d, j0, d);
        mma_tile<CT, KC, KC>(a3, sP, Cp, i0, sD1T, Cp, j0, Cp);
        const int l = lane_id();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          const float z = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
          sH[(size_t)i * h + j] = from_f<CT>(act_f<ACT>(z));
        }
      }
    }
    __syncthreads();
    gemm<CT, KC, KC>(Cp, Cp, h, sH, h, sHk, h, [&](int i, int j, float x) {
      sP[(size_t)i * Cp + j] = from_f<CT>(j <= i ? cf.c[i][j] * x : 0.f);
    });
    __syncthreads();
    {
      const int tn = d >> 4, nt = (Cp >> 4) * tn;
      for (int t = wave_id(); t < nt; t += num_waves()) {
        const int i0 = (t / tn) << 4, j0 = (t % tn) << 4;
        f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
        mma_tile<CT, KC, KC>(a1, sH, h, i0, W2, h, j0, h);
        mma_tile<CT, KC, KC>(a2, sH, h, i0, S2, h, j0, h);
        mma_tile<CT, KC, KC>(a3, sP, Cp, i0, sRT, Cp, j0, Cp);
        const int l = lane_id();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          if (i < C) o[(size_t)(tok0 + i) * d + j] = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
        }
      }
    }
    __syncthreads();
  }
}

template <typename IO, typename CT>
static hipError_t launch_local_fwd_t(const LocalFwdArgs& a, int units, hipStream_t st) {
  dim3 grid(units), block(512);
  if (a.D.act == ACT_GELU)
    hipLaunchKernelGGL((local_fwd_kernel<IO, CT, ACT_GELU>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((local_fwd_kernel<IO, CT, ACT_SILU>), grid, block, 0, st, a);
  return hipGetLastError();
}

hipError_t launch_local_fwd(const LocalFwdArgs& a, int units, hipStream_t st) {
  hipError_t e = hipSuccess;
  if (!a.force_generic && launch_local_fwd_fast(a, units, st, &e)) return e;
  e = a.D.bf16 ? launch_local_fwd_t<__bf16, __bf16>(a, units, st)
               : launch_local_fwd_t<float, float>(a, units, st);
  if (e != hipSuccess || !a.statesT) return e;
  // the runtime-sized kernel writes fp32 states only: transpose them in one pass
  return launch_pack_states(a.states, a.mstates, a.statesT, units, a.nslots, a.D.d, a.D.hid,
                            a.D.qk_proj && a.D.qk_scope == 0, a.D.bf16, st);
}

}  // namespace tnt
