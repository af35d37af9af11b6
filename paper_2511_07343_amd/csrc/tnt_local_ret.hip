// Retrieval of every (unit, chunk) of a local memory at once, for the
// fixed-size shapes of the register-resident walk (d 64, hid 256, C_L <= 64,
// bf16): one workgroup per (unit, chunk), from the chunk-entry state the walk
// saved (W1^T, W2^T, S1^T, S2^T in the compute type), the walk's D1^T and R of
// the chunk, and its Hk (Sec. 4.1.2 retrieval box, local memories; the dual
// form of the chunk rule of Sec. 2.2 with the gates of App. D):
//
//   x_t = M_t q_t  (Q-K projection, App. C):  X = Q M_0 + tril(Q N^T) N
//   P   = c o (X K^T)                       (c_{i,tau} = 0 for tau > i)
//   Z   = diag(A) X W1^T + diag(E) X S1^T - P D1,   H = s(Z)
//   Po  = c o (H Hk^T)
//   O   = diag(A) H W2^T + diag(E) H S2^T - Po R
//
// It also writes the chunk's forward record fields that the backward passes
// read and that the walk does not write (K, R, X and their scaled and
// transposed forms, Q^T, N, N^T, tril(Q N^T)^T, Pz^T, Po^T, H^T, s'(Z), X K^T,
// H Hk^T, (H W2^T)^T, (H S2^T)^T, key norms and the carry coefficients).
//
// Sized for two workgroups per CU: LDS holds X, K, R (rows padded by 16 bytes
// so that the 16-byte operand reads of consecutive rows do not start on the
// same banks) and one region used in turn by the Q-K temporaries (Q, N, N^T,
// tril(Q N^T)) and by the retrieval's P and H; the contractions with Hk and D1
// take their B operands straight from global memory, the chunk coefficients
// keep only the lower triangle of c, and the kernel is built for at most 128
// VGPRs.
#include "tnt_local_common.h"
#include "tnt_local_record.h"

namespace tnt {

namespace {

template <int D, int HID, int CP>
struct RetLds {
  static constexpr int cmax(int x, int y) { return x > y ? x : y; }
  static constexpr int LDD = D + 8, LDC = CP + 8, LDH = HID + 8;
  static constexpr int X = 0, K = X + CP * LDD, R = K + CP * LDD, U = R + CP * LDD;
  // phase 1 (Q-K projection and the record): Q, N [CP][LDD], N^T [D][LDC], tril(Q N^T) [CP][LDC]
  static constexpr int Q = U, N = Q + CP * LDD, NT = N + CP * LDD, S = NT + D * LDC;
  static constexpr int U1 = 2 * CP * LDD + D * LDC + CP * LDC;
  // phase 2 (the retrieval): P [CP][LDC] (P, then Po), H [CP][LDH]
  static constexpr int P = U, H = P + CP * LDC;
  static constexpr int U2 = CP * LDC + CP * LDH;
  static constexpr int total = U + cmax(U1, U2);
  static_assert(K % 8 == 0 && R % 8 == 0 && U % 8 == 0 && N % 8 == 0 && NT % 8 == 0 &&
                    S % 8 == 0 && H % 8 == 0 && total % 8 == 0,
                "16-byte aligned rows");
};

}  // namespace

template <int D, int HID, int CP>
constexpr size_t ret_lds_bytes() {
  return (size_t)RetLds<D, HID, CP>::total * 2;
}

template <typename IO, int ACT, int D, int HID, int CP>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4, 8)))
local_ret_kernel(LocalFwdArgs a) {
  using CT = __bf16;
  using Ly = RetLds<D, HID, CP>;
  constexpr int LDD = Ly::LDD, LDC = Ly::LDC, LDH = Ly::LDH;
  constexpr int NW = 8;
  constexpr int TNH = HID / 16, TMC = CP / 16;
  constexpr int KS = Mma<CT>::KS;
  constexpr int NKD = D / KS, NKH = HID / KS;
  constexpr int NS = (TNH + NW - 1) / NW;  // 16-column strips of HID per wave
  static_assert(NW % (D / 16) == 0, "one column strip of D per wave");
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ CoefFN<CP> cf;
  CT* L = (CT*)smem;
  CT *sX = L + Ly::X, *sK = L + Ly::K, *sR = L + Ly::R;
  CT *sQ = L + Ly::Q, *sN = L + Ly::N, *sNT = L + Ly::NT, *sS = L + Ly::S;
  CT *sP = L + Ly::P, *sH = L + Ly::H;

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int nch = Dm.S / C;
  const int u = (int)blockIdx.x / nch, n = (int)blockIdx.x % nch;
  const int b = u / (Dm.H * nshard), hh = (u / nshard) % Dm.H, s = u % nshard;
  constexpr size_t hd = (size_t)HID * D;
  const size_t chain = (size_t)b * Dm.H + hh;
  const IO* q = (const IO*)a.q + chain * Dm.L * D;
  const IO* k = (const IO*)a.k + chain * Dm.L * D;
  float* o = a.o_part + chain * Dm.L * D;
  const float* lr = a.lr + chain * Dm.L;
  const float* mom = a.mom + chain * Dm.L;
  const float* dec = a.decay + chain * Dm.L;
  const bool qk = Dm.qk_proj;
  const bool shard_qk = Dm.qk_proj && Dm.qk_scope == 0;
  const int l = lane_id(), w = wave_id();
  const int ko = Mma<CT>::kofs(l);
  constexpr size_t PS = 4 * hd + (size_t)D * D;               // CT elements per transposed slot
  constexpr size_t FS = 2 * (size_t)CP * HID + (size_t)CP * D;  // the walk's buffer per chunk
  constexpr rec::RecLayout RL = rec::make_rec_layout(CP, D, HID);
  const size_t t = (size_t)u * nch + n;
  const CT* const fsn = (const CT*)a.fsplit + t * FS;           // Hk | D1^T | R
  CT* const fr = a.frec ? (CT*)a.frec + t * RL.fc.n : nullptr;
  float* const frf = fr ? a.frec_f + t * RL.ff.n : nullptr;
  const CT* const gHk = fr ? fr + RL.fc.o[rec::Hk] : fsn;       // [CP][HID], where the walk left it
  const CT* const gD1T = fsn + (size_t)CP * HID;                // [HID][CP]
  const CT* const pkc = (const CT*)a.statesT + ((size_t)u * a.nslots + n) * PS;  // entry state
  const float* Mc = a.mstates + ((size_t)u * a.nslots + n) * D * D;
  const int tok0 = s * Dm.S + n * C;

  // R of the chunk, requested first (one 16-byte vector per thread and pass)
  constexpr int RV = CP * D / 8, RPER = (RV + 511) / 512;
  bf16x8 rbuf[RPER];
#pragma unroll
  for (int p = 0; p < RPER; ++p) {
    const int vi = (int)threadIdx.x + 512 * p;
    if (vi < RV) rbuf[p] = *reinterpret_cast<const bf16x8*>(fsn + 2 * (size_t)CP * HID + (size_t)vi * 8);
  }

  // ---- stage Q, K (16-byte loads; rows >= C zero), key norms, gate coefficients
  {
    constexpr int VEC = 16 / sizeof(IO), LPR = D / VEC;  // lanes per row
    static_assert(LPR >= 1 && LPR <= WAVE && (LPR & (LPR - 1)) == 0, "rows within one wave");
    static_assert((CP * D / VEC) % WAVE == 0, "whole waves stage");
    for (int e = threadIdx.x * VEC; e < CP * D; e += 512 * VEC) {
      const int i = e / D;
      const int el = i * LDD + (e - i * D);
      float ss = 0.f;
      if (i < C) {
        const IO* pq = q + (size_t)tok0 * D + e;
        const IO* pk = k + (size_t)tok0 * D + e;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          sQ[el + j] = from_f<CT>(to_f(pq[j]));
          const CT kv = from_f<CT>(to_f(pk[j]));
          sK[el + j] = kv;
          ss += to_f(kv) * to_f(kv);
        }
      } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          sQ[el + j] = from_f<CT>(0.f);
          sK[el + j] = from_f<CT>(0.f);
        }
      }
#pragma unroll
      for (int o2 = 1; o2 < LPR; o2 <<= 1) ss += __shfl_xor(ss, o2, WAVE);
      if ((threadIdx.x & (LPR - 1)) == 0) cf.knorm[i] = sqrtf(ss);  // visible after the coefficients' barrier
    }
  }
  chunk_coefs_f(cf, lr, mom, dec, tok0, C, CP);  // barriers inside (K staged)
#pragma unroll
  for (int p = 0; p < RPER; ++p) {
    const int vi = (int)threadIdx.x + 512 * p;
    if (vi < RV) {
      const int e = vi * 8, i = e / D;
      *reinterpret_cast<bf16x8*>(sR + i * LDD + (e - i * D)) = rbuf[p];
    }
  }

  // ---- Q-K projection: X = Q M_0 + tril(Q N^T) N (shard scope; chunk scope
  // without the M_0 term), X = Q without it
  if (qk) {
    for (int e = threadIdx.x; e < CP * D; e += 512) {
      const int i = e / D, j = e - i * D;
      const float nr = cf.knorm[i];
      const float x = (i < C && nr > 0.f) ? to_f(sK[i * LDD + j]) / nr : 0.f;
      sN[i * LDD + j] = from_f<CT>(x);
      sNT[(size_t)j * LDC + i] = from_f<CT>(x);
    }
    __syncthreads();
    gemm<CT, KC, KC>(CP, CP, D, sQ, LDD, sN, LDD, [&](int i, int j, float x) {
      sS[(size_t)i * LDC + j] = from_f<CT>(j <= i ? x : 0.f);
    });
    __syncthreads();
    constexpr int tn = D / 16, nt = TMC * tn;
    RawFrag<CT, float> bm[NKD];
    const int cs = w % tn;
    if (shard_qk)
#pragma unroll
      for (int ks = 0; ks < NKD; ++ks) bm[ks].load(Mc, D, cs * 16 + (l & 15), ks * KS + ko);
    for (int tt = w; tt < nt; tt += NW) {
      const int i0 = (tt / tn) * 16, j0 = cs * 16;
      f4 acc = zero4();
      if (shard_qk) {
#pragma unroll
        for (int ks = 0; ks < NKD; ++ks) {
          auto av = Mma<CT>::template load<KC>(sQ, LDD, i0 + (l & 15), ks * KS + ko, D, nullptr);
          Mma<CT>::mma(acc, av, bm[ks].get());
        }
      }
      mma_tile<CT, KC, KC>(acc, sS, LDC, i0, sNT, LDC, j0, CP);
      tile_each(acc, i0, j0, [&](int i, int j, float x) { sX[(size_t)i * LDD + j] = from_f<CT>(x); });
    }
  } else {
    for (int e = threadIdx.x; e < CP * D; e += 512) {
      const int el = (e / D) * LDD + e % D;
      sX[el] = sQ[el];
    }
  }
  __syncthreads();

  // ---- the forward record: K, R and their scaled / transposed forms, X^T scaled
  // and as it is, Q^T,
  // N, N^T, tril(Q N^T)^T (eight destination elements per thread, 16-byte
  // stores; transposed destinations gather their eight sources from LDS)
  if (fr) {
    auto st8 = [&](int field, size_t e0, const float (&x)[8]) {
      bf16x8 vv;
#pragma unroll
      for (int qq = 0; qq < 8; ++qq) vv[qq] = (__bf16)x[qq];
      *reinterpret_cast<bf16x8*>(fr + RL.fc.o[field] + e0) = vv;
    };
    auto cp8 = [&](int field, size_t e0, const CT* src) {
      *reinterpret_cast<bf16x8*>(fr + RL.fc.o[field] + e0) = *reinterpret_cast<const bf16x8*>(src);
    };
    for (int v = threadIdx.x; v < CP * D / 8; v += 512) {
      const size_t e0 = (size_t)v * 8;
      const int i = (int)(e0 / D);
      const int jt = (int)(e0 / CP), it = (int)(e0 % CP);  // transposed [D][CP]: rows it..it+7
      const size_t ed = (size_t)i * LDD + e0 % D;          // [CP][D] element e0 in LDS
      const size_t ec = (size_t)jt * LDC + it;             // [D][CP] element e0 in LDS
      cp8(rec::K, e0, sK + ed);
      cp8(rec::R, e0, sR + ed);
      float kc[8], kb[8], rc[8], rb[8], kt[8], rt[8], xt[8], xa[8], xe[8], qt[8];
#pragma unroll
      for (int qq = 0; qq < 8; ++qq) {
        const float kx = to_f(sK[ed + qq]), rx = to_f(sR[ed + qq]);
        kc[qq] = cf.cC[i] * kx;
        kb[qq] = cf.bb[i] * kx;
        rc[qq] = cf.cC[i] * rx;
        rb[qq] = cf.bb[i] * rx;
        const size_t es = (size_t)(it + qq) * LDD + jt;
        kt[qq] = to_f(sK[es]);
        rt[qq] = to_f(sR[es]);
        xt[qq] = to_f(sX[es]);
        xa[qq] = cf.A[it + qq] * xt[qq];
        xe[qq] = cf.E[it + qq] * xt[qq];
        qt[qq] = to_f(sQ[es]);
      }
      st8(rec::KcC, e0, kc);
      st8(rec::Kb, e0, kb);
      st8(rec::RcC, e0, rc);
      st8(rec::Rb, e0, rb);
      st8(rec::KT, e0, kt);
      st8(rec::RT, e0, rt);
      st8(rec::XT, e0, xt);
      st8(rec::XAT, e0, xa);
      st8(rec::XET, e0, xe);
      st8(rec::QT, e0, qt);
      if (qk) {
        cp8(rec::N, e0, sN + ed);
        cp8(rec::NT, e0, sNT + ec);
      }
    }
    if (qk)
      for (int v = threadIdx.x; v < CP * CP / 8; v += 512) {
        const size_t e0 = (size_t)v * 8;
        const int jt = (int)(e0 / CP), it = (int)(e0 % CP);
        float x[8];
#pragma unroll
        for (int qq = 0; qq < 8; ++qq) x[qq] = to_f(sS[(size_t)(it + qq) * LDC + jt]);
        st8(rec::StrT, e0, x);
      }
    if (threadIdx.x < CP) {
      const int i = threadIdx.x;
      frf[RL.ff.o[rec::kn] + i] = cf.knorm[i];
      frf[RL.ff.o[rec::cC] + i] = cf.cC[i];
      frf[RL.ff.o[rec::bb] + i] = cf.bb[i];
      if constexpr (rec::rec_coefs(CP)) {
        frf[RL.ff.o[rec::cA] + i] = cf.A[i];
        frf[RL.ff.o[rec::cE] + i] = cf.E[i];
      }
    }
    if constexpr (rec::rec_coefs(CP)) {  // the packed coefficient matrix, 16-byte stores
      constexpr int NP = CP * (CP + 1) / 2;
      static_assert(NP % 4 == 0, "whole 16-byte groups");
      for (int e = threadIdx.x * 4; e < NP; e += 512 * 4)
        *reinterpret_cast<f32x4*>(frf + RL.ff.o[rec::Cc] + e) = *reinterpret_cast<const f32x4*>(cf.c + e);
    }
    if (threadIdx.x == 0) {
      frf[RL.ff.o[rec::sc] + 0] = cf.AC;
      frf[RL.ff.o[rec::sc] + 1] = cf.BC;
      frf[RL.ff.o[rec::sc] + 2] = cf.EC;
    }
  }
  __syncthreads();  // the Q-K temporaries are dead: their region takes P and H

  // ---- P = c o (X K^T)
  {
    constexpr int tn = CP / 16, nt = TMC * tn;
    for (int tt = w; tt < nt; tt += NW) {
      const int i0 = (tt / tn) * 16, j0 = (tt % tn) * 16;
      f4 acc = zero4();
      mma_tile<CT, KC, KC>(acc, sX, LDD, i0, sK, LDD, j0, D);
      f4 pv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        pv[r] = j <= i ? cf.cc(i, j) * acc[r] : 0.f;
        sP[(size_t)i * LDC + j] = from_f<CT>(pv[r]);
      }
      if (fr) {
        store4<float>(frf + RL.ff.o[rec::XK] + frag_ofs<CP, CP>(i0, j0, l), acc);
        store4<CT>(fr + RL.fc.o[rec::PzT] + (size_t)(j0 + (l & 15)) * CP + i0 + 4 * (l >> 4), pv);
      }
    }
  }
  // ---- Z = diag(A) X W1^T + diag(E) X S1^T - P D1, H = s(Z): the wave's hidden
  // strips; W1, S1 from the walk's W1^T, S1^T [D][HID] and D1 from D1^T [HID][CP]
  // (contraction-major reads), all requested before the barrier
  {
    typename Mma<CT>::frag bw[NS][NKD], bs[NS][NKD];
    typename Mma<CT>::frag bd[NS][(CP + KS - 1) / KS];
    constexpr int NKC = (CP + KS - 1) / KS;
#pragma unroll
    for (int y = 0; y < NS; ++y) {
      const int sidx = w + NW * y;
      if (sidx < TNH) {
#pragma unroll
        for (int ks = 0; ks < NKD; ++ks) {
          bw[y][ks] = Mma<CT>::template load<MC>(pkc, HID, sidx * 16 + (l & 15), ks * KS + ko, D, nullptr);
          bs[y][ks] = Mma<CT>::template load<MC>(pkc + 2 * hd, HID, sidx * 16 + (l & 15), ks * KS + ko,
                                                 D, nullptr);
        }
#pragma unroll
        for (int ks = 0; ks < NKC; ++ks)
          bd[y][ks] = Mma<CT>::template load<KC>(gD1T, CP, sidx * 16 + (l & 15), ks * KS + ko, CP, nullptr);
      }
    }
    __syncthreads();  // P ready
#pragma unroll
    for (int y = 0; y < NS; ++y) {
      const int sidx = w + NW * y;
      if (sidx >= TNH) continue;
#pragma unroll 1
      for (int it = 0; it < TMC; ++it) {
        const int i0 = it * 16, j0 = sidx * 16;
        f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
#pragma unroll
        for (int ks = 0; ks < NKD; ++ks) {
          auto av = Mma<CT>::template load<KC>(sX, LDD, i0 + (l & 15), ks * KS + ko, D, nullptr);
          Mma<CT>::mma(a1, av, bw[y][ks]);
          Mma<CT>::mma(a2, av, bs[y][ks]);
        }
#pragma unroll
        for (int ks = 0; ks < NKC; ++ks) {
          auto av = Mma<CT>::template load<KC>(sP, LDC, i0 + (l & 15), ks * KS + ko, CP, nullptr);
          Mma<CT>::mma(a3, av, bd[y][ks]);
        }
        f4 hv, szv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          const float z = cf.A[i] * a1[r] + cf.E[i] * a2[r] - a3[r];
          if (fr) {
            const ActVals av = act_all<ACT>(z);
            sH[(size_t)i * LDH + j] = from_f<CT>(av.s);
            hv[r] = av.s;
            szv[r] = av.d1;
          } else {
            sH[(size_t)i * LDH + j] = from_f<CT>(act_f<ACT>(z));
          }
        }
        if (fr) {
          store4<CT>(fr + RL.fc.o[rec::HT] + (size_t)(j0 + (l & 15)) * CP + i0 + 4 * (l >> 4), hv);
          store4<CT>(fr + RL.fc.o[rec::Sz] + frag_ofs<CP, HID>(i0, j0, l), szv);
        }
      }
    }
  }
  __syncthreads();  // H ready; P is dead
  // ---- Po = c o (H Hk^T): Hk rows straight from global memory
  {
    constexpr int tn = CP / 16, nt = TMC * tn;
    for (int tt = w; tt < nt; tt += NW) {
      const int i0 = (tt / tn) * 16, j0 = (tt % tn) * 16;
      f4 acc = zero4();
      mma_tile<CT, KC, KC>(acc, sH, LDH, i0, gHk, HID, j0, HID);
      f4 pv;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        pv[r] = j <= i ? cf.cc(i, j) * acc[r] : 0.f;
        sP[(size_t)i * LDC + j] = from_f<CT>(pv[r]);
      }
      if (fr) {
        store4<float>(frf + RL.ff.o[rec::HH] + frag_ofs<CP, CP>(i0, j0, l), acc);
        store4<CT>(fr + RL.fc.o[rec::PoT] + (size_t)(j0 + (l & 15)) * CP + i0 + 4 * (l >> 4), pv);
      }
    }
  }
  // ---- O = diag(A) H W2^T + diag(E) H S2^T - Po R: one column strip of D per
  // wave; the W2^T, S2^T strip in halves of HID
  {
    constexpr int tn = D / 16, nt = TMC * tn;
    constexpr int PT = (nt + NW - 1) / NW;
    constexpr int HALF = NKH < 2 ? NKH : 2;
    const int cs = w % tn;
    f4 a1[PT], a2[PT];
#pragma unroll
    for (int x = 0; x < PT; ++x) a1[x] = a2[x] = zero4();
    bool synced = false;
#pragma unroll
    for (int hb = 0; hb < NKH; hb += HALF) {
      typename Mma<CT>::frag bw[HALF], bs[HALF];
#pragma unroll
      for (int kk = 0; kk < HALF; ++kk)
        if (hb + kk < NKH) {
          bw[kk] = Mma<CT>::template load<MC>(pkc + hd, D, cs * 16 + (l & 15), (hb + kk) * KS + ko, HID,
                                              nullptr);
          bs[kk] = Mma<CT>::template load<MC>(pkc + 3 * hd, D, cs * 16 + (l & 15), (hb + kk) * KS + ko,
                                              HID, nullptr);
        }
      if (!synced) {
        __syncthreads();  // Po ready
        synced = true;
      }
#pragma unroll
      for (int x = 0; x < PT; ++x) {
        const int tt = w + NW * x;
        if (tt >= nt) continue;
        const int i0 = (tt / tn) * 16;
#pragma unroll
        for (int kk = 0; kk < HALF; ++kk)
          if (hb + kk < NKH) {
            auto av = Mma<CT>::template load<KC>(sH, LDH, i0 + (l & 15), (hb + kk) * KS + ko, HID, nullptr);
            Mma<CT>::mma(a1[x], av, bw[kk]);
            Mma<CT>::mma(a2[x], av, bs[kk]);
          }
      }
    }
#pragma unroll
    for (int x = 0; x < PT; ++x) {
      const int tt = w + NW * x;
      if (tt >= nt) continue;
      const int i0 = (tt / tn) * 16, j0 = cs * 16;
      f4 a3 = zero4();
      mma_tile<CT, KC, MC>(a3, sP, LDC, i0, sR, LDD, j0, CP);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
        if (i < C) o[(size_t)(tok0 + i) * D + j] = cf.A[i] * a1[x][r] + cf.E[i] * a2[x][r] - a3[r];
      }
      if (fr) {  // transposed [D][CP]: the lane's four rows are contiguous
        const size_t et = (size_t)(j0 + (l & 15)) * CP + i0 + 4 * (l >> 4);
        store4<float>(frf + RL.ff.o[rec::HW2] + et, a1[x]);
        store4<float>(frf + RL.ff.o[rec::HS2] + et, a2[x]);
      }
    }
  }
}

// Launches the retrieval for the shapes it is built for; false otherwise.
template <typename IO, int ACT, int D, int HID, int CP>
static bool try_ret(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (a.D.d != D || a.D.hid != HID || a.D.Cp != CP || a.D.act != ACT) return false;
  constexpr size_t lds = ret_lds_bytes<D, HID, CP>();
  static_assert(lds + sizeof(CoefFN<CP>) <= 160 * 1024, "LDS of one CU");
  auto kern = local_ret_kernel<IO, ACT, D, HID, CP>;
  if (!lds_fits((const void*)kern, lds)) {  // the compiled static LDS, not the estimate
    *err = hipErrorInvalidConfiguration;
    return true;
  }
  set_lds_limit((const void*)kern);
  const int nch = a.D.S / a.D.C;
  hipLaunchKernelGGL(kern, dim3(units * nch), dim3(512), lds, st, a);
  *err = hipGetLastError();
  return true;
}

bool launch_local_ret(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (!a.D.bf16 || !a.statesT || !a.fsplit || a.nslots <= a.D.S / a.D.C) return false;
  return try_ret<__bf16, ACT_SILU, 64, 256, 64>(a, units, st, err) ||
         try_ret<__bf16, ACT_SILU, 64, 256, 32>(a, units, st, err) ||
         try_ret<__bf16, ACT_SILU, 64, 256, 16>(a, units, st, err) ||
         try_ret<__bf16, ACT_GELU, 64, 256, 64>(a, units, st, err) ||
         try_ret<__bf16, ACT_GELU, 64, 256, 16>(a, units, st, err);
}

}  // namespace tnt
