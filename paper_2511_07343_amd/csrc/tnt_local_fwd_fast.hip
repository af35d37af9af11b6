// Local memories, forward, for fixed sizes (head dim D, hidden HID, padded
// chunk CP) whose chunk working set fits in the 160 KB LDS of a CU.  Same
// chunk step as local_fwd_kernel (see tnt_local_fwd.hip); here every loop has
// a compile-time trip count and every chunk intermediate stays on chip:
//
//   LDS  Hk [CP][HID]   s(K W1^T)                         bf16/fp32 (CT)
//        D1^T [HID][CP] ((R W2) * s'(K W1^T))^T
//        U              reused in turn: Q-K temporaries (Q, N, N^T, tril(Q N^T)),
//                       the chunk-entry W2 (CT copy, [D][HID]), K^T and R^T for the
//                       carry, then H = s(Z) [CP][HID]
//        X, K, R [CP][D], P [CP][CP], gate coefficients
//   VGPR s'(K W1^T) between the two GEMMs that share its output tiles
//
// The fp32 state (W1, W2, S1, S2 and the Q-K sum) lives in global memory,
// one slot per chunk boundary; contraction-contiguous operands are read from
// it directly, the carry reads the entry slot and writes the next one.  When
// the states are saved for the backward pass, the carry also writes the CT
// transposes of the new state (W1^T, W2^T, S1^T, S2^T, M^T) from the same
// registers: four consecutive rows of an MFMA output tile are four contiguous
// elements of the transpose.
#include "tnt_local_common.h"
#include "tnt_local_record.h"

namespace tnt {

// LDS carve-up (CT elements); leading dimensions LDD, LDC, LDH are the
// matrices' own widths plus PD (0 here: the walk modes' LDS also holds W2).
template <int D, int HID, int CP, int PD>
struct FwdLds {
  static constexpr int cmax(int x, int y) { return x > y ? x : y; }
  static constexpr int LDD = D + PD, LDC = CP + PD, LDH = HID + PD;
  // U: H [CP][LDH] and the Q-K temporaries; the walk modes (PD = 0) also hold
  // the chunk-entry W2 ([D][HID] or W2^T [HID][D]) and K^T, R^T [D][CP] there
  static constexpr int USZ = cmax(cmax(CP * LDH, 2 * CP * LDD + D * LDC + CP * LDC),
                                  PD == 0 ? cmax(D * HID, 2 * D * CP) : 0);
  static constexpr int Hk = 0;                 // [CP][LDH]
  static constexpr int D1 = Hk + CP * LDH;     // D1^T [HID][LDC]
  static constexpr int U = D1 + HID * LDC;
  static constexpr int X = U + USZ;            // [CP][LDD]
  static constexpr int K = X + CP * LDD;
  static constexpr int R = K + CP * LDD;
  static constexpr int P = R + CP * LDD;       // [CP][LDC]
  static constexpr int total = P + CP * LDC;
  // inside U during the Q-K phase: Q, N [CP][LDD], N^T [D][LDC], tril(Q N^T) [CP][LDC]
  static constexpr int uQ = U, uN = U + CP * LDD, uNT = U + 2 * CP * LDD, uS = uNT + D * LDC;
  static_assert(USZ % 8 == 0 && D1 % 8 == 0 && U % 8 == 0 && X % 8 == 0 && K % 8 == 0 &&
                    R % 8 == 0 && P % 8 == 0 && uNT % 8 == 0 && uS % 8 == 0,
                "16-byte aligned rows");
};

template <typename CT, int D, int HID, int CP, int PD>
constexpr size_t fwd_fast_lds_bytes() {
  return (size_t)FwdLds<D, HID, CP, PD>::total * sizeof(CT);
}

// Modes of the kernel.  FWD_FULL: one workgroup per unit walks its chunks and
// does everything.  When every chunk-entry state is saved, the walk is split:
// FWD_CHAIN walks the chunks doing only what the next state needs (keys, the
// chunk gradient, the carry, the Q-K sum) and leaves Hk, D1^T and R of every
// chunk in a buffer (for the shapes and kernel families the register-resident
// walk does not take); local_ret_kernel then takes the retrieval of every
// (unit, chunk) at once, one workgroup each, from the saved entry state and
// that buffer.
enum { FWD_FULL = 0, FWD_CHAIN = 1 };

// per-chunk buffer of the split forward: Hk [CP][HID], D1^T [HID][CP], R [CP][D]
template <int D, int HID, int CP>
constexpr size_t fwd_split_elems() {
  return 2 * (size_t)CP * HID + (size_t)CP * D;
}

template <typename IO, typename CT, int ACT, int D, int HID, int CP, int MODE>
__global__ void __launch_bounds__(512) local_fwd_fast_kernel(LocalFwdArgs a) {
  constexpr bool WALK = true, RETR = MODE != FWD_CHAIN;
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ CoefFN<CP> cf;  // the coefficients of a CP-row chunk
  using Ly = FwdLds<D, HID, CP, 0>;
  constexpr int LDD = Ly::LDD, LDC = Ly::LDC, LDH = Ly::LDH;
  constexpr int NW = 8;                       // waves
  constexpr int TNH = HID / 16, TMC = CP / 16;
  constexpr int KS = Mma<CT>::KS;
  constexpr int NKD = D / KS, NKH = HID / KS;
  constexpr int NS = (TNH + NW - 1) / NW;     // 16-column strips of HID per wave
  static_assert(NW % (D / 16) == 0, "one column strip of D per wave");
  static_assert((HID / 16) * (D / 16) % NW == 0, "state tiles spread evenly over waves");
  static_assert((size_t)HID * D % (512 * 4) == 0, "W2 copy in whole float4s per thread");
  static_assert(sizeof(CT) == 2, "the fixed-size forward computes in bf16");
  CT* L = (CT*)smem;
  CT *sHk = L + Ly::Hk, *sD1 = L + Ly::D1, *sU = L + Ly::U, *sX = L + Ly::X, *sK = L + Ly::K,
     *sR = L + Ly::R, *sP = L + Ly::P;
  CT *sQ = L + Ly::uQ, *sN = L + Ly::uN, *sNT = L + Ly::uNT, *sS = L + Ly::uS;
  CT* sW2 = sU;  // chunk-entry W2 copy: [D][HID], or W2^T [HID][D] in the walk
  CT* sH = sU;

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int nch = Dm.S / C;
  const int u = (int)blockIdx.x;
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
  const int fsl = a.fslots ? a.fslots : a.nslots;  // fp32 state slots the walk cycles through
  float* st = a.states + (size_t)u * fsl * 4 * hd;
  float* mst = a.mstates + (size_t)u * a.nslots * D * D;
  constexpr size_t PS = 4 * hd + (size_t)D * D;  // CT elements per transposed slot
  CT* const pku = a.statesT ? (CT*)a.statesT + (size_t)u * a.nslots * PS : nullptr;
  const bool qk = Dm.qk_proj;
  const bool shard_qk = Dm.qk_proj && Dm.qk_scope == 0;
  const float rscale = 2.0f / (float)D;
  const int l = lane_id(), w = wave_id();
  const int ko = Mma<CT>::kofs(l);
  constexpr size_t FS = fwd_split_elems<D, HID, CP>();
  constexpr rec::RecLayout RL = rec::make_rec_layout(CP, D, HID);

  if (WALK) {
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
    if (pku) {  // slot 0 transposes; destination-ordered writes
      for (int e = threadIdx.x; e < (int)hd; e += blockDim.x) {
        const int c1 = e / HID, r1 = e - c1 * HID;  // W1^T [D][HID]
        const int c2 = e / D, r2 = e - c2 * D;      // W2^T [HID][D]
        pku[e] = from_f<CT>(W1i[(size_t)r1 * D + c1]);
        pku[hd + e] = from_f<CT>(W2i[(size_t)r2 * HID + c2]);
        pku[2 * hd + e] = pku[3 * hd + e] = from_f<CT>(0.f);
      }
      if (shard_qk)
        for (int e = threadIdx.x; e < D * D; e += blockDim.x) pku[4 * hd + e] = from_f<CT>(0.f);
    }
  }
  __syncthreads();

  for (int n = 0; n < nch; ++n) {
    CT* const fsn = (MODE == FWD_FULL) ? nullptr : (CT*)a.fsplit + ((size_t)u * nch + n) * FS;
    // the chunk's forward record (walk: s'(Zk), s''(Zk), G; retrieval: the rest)
    CT* const fr = (MODE != FWD_FULL && a.frec) ? (CT*)a.frec + ((size_t)u * nch + n) * RL.fc.n : nullptr;
    float* const frf = fr ? a.frec_f + ((size_t)u * nch + n) * RL.ff.n : nullptr;
    const int tok0 = s * Dm.S + n * C;
    const float* cur = st + (size_t)(n % fsl) * 4 * hd;
    float* nxt = st + (size_t)((n + 1) % fsl) * 4 * hd;
    const float *W1 = cur, *W2 = cur + hd, *S1 = cur + 2 * hd, *S2 = cur + 3 * hd;
    float *W1n = nxt, *W2n = nxt + hd, *S1n = nxt + 2 * hd, *S2n = nxt + 3 * hd;
    const float* Mc = mst + (size_t)(n % a.nslots) * D * D;
    float* Mn = mst + (size_t)((n + 1) % a.nslots) * D * D;
    CT* const pkn = pku ? pku + (size_t)((n + 1) % a.nslots) * PS : nullptr;
    const CT* const pkc = pku ? pku + (size_t)(n % a.nslots) * PS : nullptr;  // entry state, bf16 T

    // ---- stage Q, K (16-byte loads; rows >= C zero), key norms, gate coefficients
    {
      constexpr int VEC = 16 / sizeof(IO), LPR = D / VEC;  // lanes per row
      static_assert(LPR >= 1 && LPR <= WAVE && (LPR & (LPR - 1)) == 0, "rows within one wave");
      static_assert((CP * D / VEC) % WAVE == 0, "whole waves stage");
      for (int e = threadIdx.x * VEC; e < CP * D; e += blockDim.x * VEC) {
        const int i = e / D;
        const int el = i * LDD + (e - i * D);  // LDS position of element e
        float ss = 0.f;
        if (i < C) {
          const IO* pq = q + (size_t)tok0 * D + e;
          const IO* pk = k + (size_t)tok0 * D + e;
#pragma unroll
          for (int j = 0; j < VEC; ++j) {
            if (RETR) sQ[el + j] = from_f<CT>(to_f(pq[j]));
            const CT kv = from_f<CT>(to_f(pk[j]));
            sK[el + j] = kv;
            ss += to_f(kv) * to_f(kv);
          }
        } else {
#pragma unroll
          for (int j = 0; j < VEC; ++j) {
            if (RETR) sQ[el + j] = from_f<CT>(0.f);
            sK[el + j] = from_f<CT>(0.f);
          }
        }
#pragma unroll
        for (int o = 1; o < LPR; o <<= 1) ss += __shfl_xor(ss, o, WAVE);
        if ((threadIdx.x & (LPR - 1)) == 0) cf.knorm[i] = sqrtf(ss);  // visible after the coefficients' barrier
      }
    }
    if (RETR) chunk_coefs_f(cf, lr, mom, dec, tok0, C, CP);  // barriers inside (K staged)
    if (WALK) carry_coefs(cf, lr, mom, dec, tok0, C, CP);
    if (qk) {
      for (int e = threadIdx.x; e < CP * D; e += blockDim.x) {
        const int i = e / D, j = e - i * D;
        const float nr = cf.knorm[i];
        const float x = (i < C && nr > 0.f) ? to_f(sK[i * LDD + j]) / nr : 0.f;
        sN[i * LDD + j] = from_f<CT>(x);
        sNT[(size_t)j * LDC + i] = from_f<CT>(x);
      }
      __syncthreads();
      if (RETR) {
      gemm<CT, KC, KC>(CP, CP, D, sQ, LDD, sN, LDD, [&](int i, int j, float x) {
        sS[(size_t)i * LDC + j] = from_f<CT>(j <= i ? x : 0.f);
      });
      __syncthreads();
      {
        // X tiles: one column strip of D per wave (NW % (D/16) == 0)
        constexpr int tn = D / 16, nt = TMC * tn;
        RawFrag<CT, float> bm[NKD];  // converted at use (small)
        const int cs = w % tn;
        if (shard_qk)
#pragma unroll
          for (int ks = 0; ks < NKD; ++ks) bm[ks].load(Mc, D, cs * 16 + (l & 15), ks * KS + ko);
        for (int t = w; t < nt; t += NW) {
          const int i0 = (t / tn) * 16, j0 = cs * 16;
          f4 acc = zero4();
          if (shard_qk) {
#pragma unroll
            for (int ks = 0; ks < NKD; ++ks) {
              auto a = Mma<CT>::template load<KC>(sQ, LDD, i0 + (l & 15), ks * KS + ko, D, nullptr);
              Mma<CT>::mma(acc, a, bm[ks].get());
            }
          }
          mma_tile<CT, KC, KC>(acc, sS, LDC, i0, sNT, LDC, j0, CP);
          tile_each(acc, i0, j0, [&](int i, int j, float x) { sX[(size_t)i * LDD + j] = from_f<CT>(x); });
        }
      }
      }
      if (WALK && shard_qk) {
        constexpr int tn = D / 16, nt = tn * tn;
        for (int t = w; t < nt; t += NW) {
          const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
          float mo[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) mo[r] = Mc[(size_t)(i0 + 4 * (l >> 4) + r) * D + j0 + (l & 15)];
          f4 acc = zero4();
          mma_tile<CT, KC, KC>(acc, sNT, LDC, i0, sNT, LDC, j0, CP);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            acc[r] += mo[r];
            Mn[(size_t)(i0 + 4 * (l >> 4) + r) * D + j0 + (l & 15)] = acc[r];
          }
          if (pkn) store4<CT>(pkn + 4 * hd + (size_t)(j0 + (l & 15)) * D + i0 + 4 * (l >> 4), acc);
        }
      }
    } else if (RETR) {
      for (int e = threadIdx.x; e < CP * D; e += blockDim.x) {
        const int el = (e / D) * LDD + e % D;
        sX[el] = sQ[el];
      }
    }

    if constexpr (WALK) {
    // ---- Zk = K W1^T -> Hk (LDS), s'(Zk) (registers); each wave owns NS column strips
    CT spr[NS][TMC][4];  // s'(Zk) in the compute type
    {
      typename Mma<CT>::frag bw[NS][NKD];
      if constexpr (MODE == FWD_CHAIN) {
        // W1 from the entry state's compute-type transpose W1^T [D][HID] (written by the
        // previous step's carry; the same rounding as a conversion of the fp32 state)
#pragma unroll
        for (int y = 0; y < NS; ++y) {
          const int sidx = w + NW * y;
          if (sidx < TNH)
#pragma unroll
            for (int ks = 0; ks < NKD; ++ks)
              bw[y][ks] = Mma<CT>::template load<MC>(pkc, HID, sidx * 16 + (l & 15), ks * KS + ko, D,
                                                     nullptr);
        }
      } else {
        RawFrag<CT, float> raw[NS][NKD];
#pragma unroll
        for (int y = 0; y < NS; ++y) {
          const int sidx = w + NW * y;
          if (sidx < TNH)
#pragma unroll
            for (int ks = 0; ks < NKD; ++ks) raw[y][ks].load(W1, D, sidx * 16 + (l & 15), ks * KS + ko);
        }
#pragma unroll
        for (int y = 0; y < NS; ++y)
#pragma unroll
          for (int ks = 0; ks < NKD; ++ks) bw[y][ks] = raw[y][ks].get();
      }
#pragma unroll
      for (int y = 0; y < NS; ++y) {
        const int sidx = w + NW * y;
        if (sidx >= TNH) continue;
#pragma unroll
        for (int it = 0; it < TMC; ++it) {
          const int i0 = it * 16, j0 = sidx * 16;
          f4 acc = zero4();
#pragma unroll
          for (int ks = 0; ks < NKD; ++ks) {
            auto a = Mma<CT>::template load<KC>(sK, LDD, i0 + (l & 15), ks * KS + ko, D, nullptr);
            Mma<CT>::mma(acc, a, bw[y][ks]);
          }
          f4 hv, d1v, d2v;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
            const ActVals av = act_all<ACT>(acc[r]);
            sHk[(size_t)i * LDH + j] = from_f<CT>(av.s);
            spr[y][it][r] = from_f<CT>(av.d1);
            hv[r] = av.s;
            d1v[r] = av.d1;
            d2v[r] = av.d2;
          }
          if (MODE == FWD_CHAIN && fr) {
            const size_t fo = frag_ofs<CP, HID>(i0, j0, l);
            store4<CT>(fr + RL.fc.o[rec::Sp] + fo, d1v);
            store4<CT>(fr + RL.fc.o[rec::Spp] + fo, d2v);
            // Hk^T [HID][CP]: the lane's four rows are contiguous
            store4<CT>(fr + RL.fc.o[rec::HkT] + (size_t)(j0 + (l & 15)) * CP + i0 + 4 * (l >> 4), hv);
          }
        }
      }
    }
    __syncthreads();  // Q-K temporaries in U are dead from here
    // chunk-entry W2 -> U: the walk copies its compute-type transpose W2^T [HID][D];
    // the one-walk kernel converts the fp32 state to CT [D][HID] (all loads first)
    if constexpr (MODE == FWD_CHAIN) {
      constexpr int V8 = 16 / sizeof(CT), PER = (int)(hd / (512 * V8));
      static_assert(hd % (512 * V8) == 0, "W2^T copy in whole 16-byte vectors per thread");
      bf16x8 x[PER];
#pragma unroll
      for (int p = 0; p < PER; ++p)
        x[p] = *reinterpret_cast<const bf16x8*>(pkc + hd + (size_t)(threadIdx.x + 512 * p) * V8);
#pragma unroll
      for (int p = 0; p < PER; ++p)
        *reinterpret_cast<bf16x8*>(sW2 + (size_t)(threadIdx.x + 512 * p) * V8) = x[p];
    } else {
      constexpr int PER = (int)(hd / (512 * 4));
      f32x4 x[PER];
#pragma unroll
      for (int p = 0; p < PER; ++p)
        x[p] = *reinterpret_cast<const f32x4*>(W2 + (size_t)(threadIdx.x + 512 * p) * 4);
#pragma unroll
      for (int p = 0; p < PER; ++p)
#pragma unroll
        for (int j = 0; j < 4; ++j) sW2[(size_t)(threadIdx.x + 512 * p) * 4 + j] = from_f<CT>(x[p][j]);
    }
    __syncthreads();

    // ---- R = (2/d) (Hk W2^T - V)
    {
      constexpr int tn = D / 16, nt = TMC * tn;
      constexpr int PT = (nt + NW - 1) / NW;
      float vv[PT][4];
#pragma unroll
      for (int x = 0; x < PT; ++x) {
        const int t = w + NW * x;
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r;
          vv[x][r] = (t < nt && i < C) ? to_f(v[(size_t)(tok0 + i) * D + j0 + (l & 15)]) : 0.f;
        }
      }
#pragma unroll
      for (int x = 0; x < PT; ++x) {
        const int t = w + NW * x;
        if (t >= nt) continue;
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 acc = zero4();
        if constexpr (MODE == FWD_CHAIN)
          mma_tile<CT, KC, MC>(acc, sHk, LDH, i0, sW2, D, j0, HID);  // sW2 = W2^T
        else
          mma_tile<CT, KC, KC>(acc, sHk, LDH, i0, sW2, HID, j0, HID);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          const float rv = (i < C) ? rscale * (acc[r] - vv[x][r]) : 0.f;
          sR[(size_t)i * LDD + j] = from_f<CT>(rv);
        }
      }
    }
    __syncthreads();

    // ---- D1 = (R W2) * s'(Zk), same strips as Zk
#pragma unroll
    for (int y = 0; y < NS; ++y) {
      const int sidx = w + NW * y;
      if (sidx >= TNH) continue;
#pragma unroll
      for (int it = 0; it < TMC; ++it) {
        const int i0 = it * 16, j0 = sidx * 16;
        f4 acc = zero4();
        if constexpr (MODE == FWD_CHAIN)
          mma_tile<CT, KC, KC>(acc, sR, LDD, i0, sW2, D, j0, D);  // sW2 = W2^T
        else
          mma_tile<CT, KC, MC>(acc, sR, LDD, i0, sW2, HID, j0, D);
        f4 dv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          dv[r] = acc[r] * to_f(spr[y][it][r]);
          sD1[(size_t)j * LDC + i] = from_f<CT>(dv[r]);  // D1^T
        }
        if (MODE == FWD_CHAIN && fr) {
          store4<CT>(fr + RL.fc.o[rec::G] + frag_ofs<CP, HID>(i0, j0, l), acc);
          CT* const d1r = fr + RL.fc.o[rec::D1] + (size_t)(i0 + 4 * (l >> 4)) * HID + j0 + (l & 15);
#pragma unroll
          for (int r = 0; r < 4; ++r) d1r[(size_t)r * HID] = from_f<CT>(dv[r]);  // D1 [CP][HID]
        }
      }
    }
    __syncthreads();

    // ---- K^T, R^T into U (the W2 copy is dead), then the carry
    CT* sKT = sU;              // [D][CP]
    CT* sRT = sU + CP * D;     // [D][CP]
    for (int e = threadIdx.x; e < CP * D; e += blockDim.x) {
      const int i = e / D, j = e - i * D;
      sKT[(size_t)j * CP + i] = sK[i * LDD + j];
      sRT[(size_t)j * CP + i] = sR[i * LDD + j];
    }
    __syncthreads();
    if constexpr (MODE == FWD_CHAIN) {
      // Hk (into the forward record when there is one), D1^T, R for the retrieval
      // pass (LDS reads only; overlaps the carry)
      for (size_t e = threadIdx.x * 8; e < FS; e += blockDim.x * 8) {
        const CT* src = e < (size_t)CP * HID ? sHk + e
                        : e < 2 * (size_t)CP * HID ? sD1 + (e - (size_t)CP * HID)
                                                   : sR + (e - 2 * (size_t)CP * HID);
        CT* dst = (fr && e < (size_t)CP * HID) ? fr + RL.fc.o[rec::Hk] + e : fsn + e;
        *reinterpret_cast<bf16x8*>(dst) = *reinterpret_cast<const bf16x8*>(src);
      }
    }
    {
      constexpr int tn = D / 16, nt = (HID / 16) * tn;  // W1', S1' : HID x D
      constexpr int PT = nt / NW, BT = PT < 4 ? PT : 4;
#pragma unroll 1
      for (int xb = 0; xb < PT; xb += BT) {
      float pw[BT][4], ps[BT][4];
#pragma unroll
      for (int xx = 0; xx < BT; ++xx) {
        const int x = xb + xx;
        const int t = w + NW * x;
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * D + j0 + (l & 15);
          pw[xx][r] = W1[e];
          ps[xx][r] = S1[e];
        }
      }
#pragma unroll
      for (int xx = 0; xx < BT; ++xx) {
        const int x = xb + xx;
        const int t = w + NW * x;
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 aw = zero4(), as = zero4();
        // A[i][tau] = D1^T[i][tau] (x cC_tau or b_tau), B[tau][j] = K^T[j][tau]
        mma_tile<CT, KC, KC>(aw, sD1, LDC, i0, sKT, CP, j0, CP, cf.cC);
        mma_tile<CT, KC, KC>(as, sD1, LDC, i0, sKT, CP, j0, CP, cf.bb);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * D + j0 + (l & 15);
          aw[r] = cf.AC * pw[xx][r] + cf.EC * ps[xx][r] - aw[r];
          as[r] = cf.BC * ps[xx][r] - as[r];
          W1n[e] = aw[r];
          S1n[e] = as[r];
        }
        if (pkn) {
          const size_t et = (size_t)(j0 + (l & 15)) * HID + i0 + 4 * (l >> 4);
          store4<CT>(pkn + et, aw);
          store4<CT>(pkn + 2 * hd + et, as);
        }
      }
      }
    }
    {
      constexpr int tn = HID / 16, nt = (D / 16) * tn;  // W2', S2' : D x HID
      constexpr int PT = nt / NW, BT = PT < 4 ? PT : 4;
#pragma unroll 1
      for (int xb = 0; xb < PT; xb += BT) {
      float pw[BT][4], ps[BT][4];
#pragma unroll
      for (int xx = 0; xx < BT; ++xx) {
        const int x = xb + xx;
        const int t = w + NW * x;
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * HID + j0 + (l & 15);
          pw[xx][r] = W2[e];
          ps[xx][r] = S2[e];
        }
      }
#pragma unroll
      for (int xx = 0; xx < BT; ++xx) {
        const int x = xb + xx;
        const int t = w + NW * x;
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 aw = zero4(), as = zero4();
        // A[i][tau] = R^T[i][tau] (x cC_tau or b_tau), B[tau][j] = Hk[tau][j]
        mma_tile<CT, KC, MC>(aw, sRT, CP, i0, sHk, LDH, j0, CP, cf.cC);
        mma_tile<CT, KC, MC>(as, sRT, CP, i0, sHk, LDH, j0, CP, cf.bb);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i0 + 4 * (l >> 4) + r) * HID + j0 + (l & 15);
          aw[r] = cf.AC * pw[xx][r] + cf.EC * ps[xx][r] - aw[r];
          as[r] = cf.BC * ps[xx][r] - as[r];
          W2n[e] = aw[r];
          S2n[e] = as[r];
        }
        if (pkn) {
          const size_t et = (size_t)(j0 + (l & 15)) * D + i0 + 4 * (l >> 4);
          store4<CT>(pkn + hd + et, aw);
          store4<CT>(pkn + 3 * hd + et, as);
        }
      }
      }
    }

    }  // WALK

    // ---- retrieval, dual form
    if constexpr (RETR) {
    {
      constexpr int tn = CP / 16, nt = TMC * tn;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
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
    {
      __syncthreads();  // P ready; K^T / R^T in U are dead
#pragma unroll
      for (int y = 0; y < NS; ++y) {
        const int sidx = w + NW * y;
        if (sidx >= TNH) continue;
        typename Mma<CT>::frag bw[NKD], bs[NKD];
        {
          RawFrag<CT, float> rw[NKD], rs[NKD];
#pragma unroll
          for (int ks = 0; ks < NKD; ++ks) {
            rw[ks].load(W1, D, sidx * 16 + (l & 15), ks * KS + ko);
            rs[ks].load(S1, D, sidx * 16 + (l & 15), ks * KS + ko);
          }
#pragma unroll
          for (int ks = 0; ks < NKD; ++ks) {
            bw[ks] = rw[ks].get();
            bs[ks] = rs[ks].get();
          }
        }
#pragma unroll 1
        for (int it = 0; it < TMC; ++it) {
          const int i0 = it * 16, j0 = sidx * 16;
          f4 a1 = zero4(), a2 = zero4(), a3 = zero4();
#pragma unroll
          for (int ks = 0; ks < NKD; ++ks) {
            auto a = Mma<CT>::template load<KC>(sX, LDD, i0 + (l & 15), ks * KS + ko, D, nullptr);
            Mma<CT>::mma(a1, a, bw[ks]);
            Mma<CT>::mma(a2, a, bs[ks]);
          }
          mma_tile<CT, KC, KC>(a3, sP, LDC, i0, sD1, LDC, j0, CP);
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
    __syncthreads();
    {
      constexpr int tn = CP / 16, nt = TMC * tn;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / tn) * 16, j0 = (t % tn) * 16;
        f4 acc = zero4();
        mma_tile<CT, KC, KC>(acc, sH, LDH, i0, sHk, LDH, j0, HID);
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
    // O: one column strip of D per wave; the W2 / S2 strip is loaded in halves of HID
    {
      constexpr int tn = D / 16, nt = TMC * tn;
      constexpr int PT = (nt + NW - 1) / NW;
      constexpr int HALF = NKH < 2 ? NKH : 2;  // k-steps per batch of W2 / S2 loads
      const int cs = w % tn;
      f4 a1[PT], a2[PT];
#pragma unroll
      for (int x = 0; x < PT; ++x) a1[x] = a2[x] = zero4();
      bool synced = false;
#pragma unroll
      for (int hb = 0; hb < NKH; hb += HALF) {
        typename Mma<CT>::frag bw[HALF], bs[HALF];
        {
          RawFrag<CT, float> rw[HALF], rs[HALF];
#pragma unroll
          for (int kk = 0; kk < HALF; ++kk)
            if (hb + kk < NKH) {
              rw[kk].load(W2, HID, cs * 16 + (l & 15), (hb + kk) * KS + ko);
              rs[kk].load(S2, HID, cs * 16 + (l & 15), (hb + kk) * KS + ko);
            }
#pragma unroll
          for (int kk = 0; kk < HALF; ++kk) {
            bw[kk] = rw[kk].get();
            bs[kk] = rs[kk].get();
          }
        }
        if (!synced) {
          __syncthreads();  // Po ready
          synced = true;
        }
#pragma unroll
        for (int x = 0; x < PT; ++x) {
          const int t = w + NW * x;
          if (t >= nt) continue;
          const int i0 = (t / tn) * 16;
#pragma unroll
          for (int kk = 0; kk < HALF; ++kk)
            if (hb + kk < NKH) {
              auto a = Mma<CT>::template load<KC>(sH, LDH, i0 + (l & 15), (hb + kk) * KS + ko, HID,
                                                  nullptr);
              Mma<CT>::mma(a1[x], a, bw[kk]);
              Mma<CT>::mma(a2[x], a, bs[kk]);
            }
        }
      }
#pragma unroll
      for (int x = 0; x < PT; ++x) {
        const int t = w + NW * x;
        if (t >= nt) continue;
        const int i0 = (t / tn) * 16, j0 = cs * 16;
        f4 a3 = zero4();
        mma_tile<CT, KC, MC>(a3, sP, LDC, i0, sR, LDD, j0, CP);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * (l >> 4) + r, j = j0 + (l & 15);
          if (i < C)
            o[(size_t)(tok0 + i) * D + j] = cf.A[i] * a1[x][r] + cf.E[i] * a2[x][r] - a3[r];
        }
        if (fr) {  // transposed [D][CP]: the lane's four rows are contiguous
          const size_t et = (size_t)(j0 + (l & 15)) * CP + i0 + 4 * (l >> 4);
          store4<float>(frf + RL.ff.o[rec::HW2] + et, a1[x]);
          store4<float>(frf + RL.ff.o[rec::HS2] + et, a2[x]);
        }
      }
    }
    }  // RETR
    __syncthreads();
  }
}

template <typename IO, typename CT, int ACT, int D, int HID, int CP>
static bool try_fast(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err, size_t* bytes) {
  if (a.D.d != D || a.D.hid != HID || a.D.Cp != CP || a.D.act != ACT) return false;
  constexpr size_t lds = fwd_fast_lds_bytes<CT, D, HID, CP, 0>();
  if (lds + sizeof(CoefFN<CP>) > 160 * 1024) return false;
  const int nch = a.D.S / a.D.C;
  if (bytes) {  // size query: the split forward's per-chunk buffer
    *bytes = (size_t)units * nch * fwd_split_elems<D, HID, CP>() * sizeof(CT);
    return true;
  }
  {  // the compiled static LDS of every mode, not the estimate
    auto k0 = local_fwd_fast_kernel<IO, CT, ACT, D, HID, CP, FWD_FULL>;
    auto k1 = local_fwd_fast_kernel<IO, CT, ACT, D, HID, CP, FWD_CHAIN>;
    if (!lds_fits((const void*)k0, lds) || !lds_fits((const void*)k1, lds)) {
      *err = hipErrorInvalidConfiguration;
      return true;
    }
  }
  if (a.fsplit && a.statesT && a.nslots > nch) {
    // the walk (register-resident state where built, else this kernel's walk
    // mode), then the retrieval of every chunk at once
    hipError_t we = hipSuccess;
    const int sec = section_begin("local_carry", st);  // the state carry alone, for its GB/s
    if (!launch_local_walk(a, units, st, &we)) {
      auto kc = local_fwd_fast_kernel<IO, CT, ACT, D, HID, CP, FWD_CHAIN>;
      set_lds_limit((const void*)kc);
      hipLaunchKernelGGL(kc, dim3(units), dim3(512), lds, st, a);
    }
    section_end(sec, st);
    if (we != hipSuccess) {
      *err = we;
      return true;
    }
    hipError_t re = hipSuccess;
    if (!launch_local_ret(a, units, st, &re)) re = hipErrorInvalidConfiguration;
    if (re != hipSuccess) {
      *err = re;
      return true;
    }
  } else {
    auto kern = local_fwd_fast_kernel<IO, CT, ACT, D, HID, CP, FWD_FULL>;
    set_lds_limit((const void*)kern);
    hipLaunchKernelGGL(kern, dim3(units), dim3(512), lds, st, a);
  }
  *err = hipGetLastError();
  return true;
}

static bool dispatch_fast(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err,
                          size_t* bytes) {
  if (a.D.bf16) {
    return try_fast<__bf16, __bf16, ACT_SILU, 64, 256, 64>(a, units, st, err, bytes) ||
           try_fast<__bf16, __bf16, ACT_SILU, 64, 256, 32>(a, units, st, err, bytes) ||
           try_fast<__bf16, __bf16, ACT_SILU, 64, 256, 16>(a, units, st, err, bytes) ||
           try_fast<__bf16, __bf16, ACT_GELU, 64, 256, 64>(a, units, st, err, bytes) ||
           try_fast<__bf16, __bf16, ACT_GELU, 64, 256, 16>(a, units, st, err, bytes);
  }
  return false;  // fp32 shapes (the tiny smoke workload) take the runtime-sized kernel
}

// Returns true (and the launch status) when a fixed-size kernel handles `a`.
bool launch_local_fwd_fast(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  return dispatch_fast(a, units, st, err, nullptr);
}

// Bytes of the per-chunk buffer of the split forward (0: no fixed-size kernel for D).
size_t local_fwd_split_bytes(const Dims& D, int units) {
  LocalFwdArgs a{};
  a.D = D;
  size_t bytes = 0;
  hipError_t e = hipSuccess;
  return dispatch_fast(a, units, nullptr, &e, &bytes) ? bytes : 0;
}

}  // namespace tnt
