// Local memories, backward, fixed sizes, in three passes.
//
// The backward of one chunk is affine in the carried adjoint of the chunk's
// exit state (W1', S1', W2', S2' bar): the backward of the retrieval (driven by
// dO), the query / key / value adjoints it feeds and the Q-K projection do not
// depend on it.  The forward already wrote every forward quantity of every
// chunk that the backward needs into the chunk's forward record (see
// tnt_local_record.h), so the reverse walk over a shard's chunks is split:
//
//   pass A  (all chunks of all units at once, a persistent grid) takes the
//           backward of the retrieval from dO and the forward record, writes
//           the chunk's dq and its share of dk, and leaves a backward record:
//           the dO operands the walk contracts, the retrieval's gate
//           cotangents (cbar, dA, dE) and Xbar^T Q for the Q-K state adjoint;
//   pass B  (one workgroup per unit, chunks in reverse) walks the carried
//           adjoint back: T3..T6, D1bar / Gbar, Rbar (dv), Zkbar, the carried
//           part of Kbar and the chunk-entry adjoint, four block barriers a chunk;
//   scan    turns the per-chunk Xbar^T Q into the suffix sums the Q-K projection
//           carries back to each chunk (shard-scoped projection only);
//   pass C  (all chunks at once) finishes the gate adjoints (dlr, dmom,
//           ddecay) and adds the carried Q-K term to dk.
//
// Each step's formulas are those of the single-walk kernels (the runtime-sized
// kernel writes them out); only the place where each term is taken differs.
// Wave-block GEMMs (Blk / mma_blk) and fragment-major elementwise factors as in
// the single-walk fixed-size kernel.
#include "tnt_local_common.h"
#include "tnt_local_bwd_helpers.h"
#include "tnt_local_record.h"

namespace tnt {

using namespace bwdh;

namespace {

// ---------------------------------------------------------------------------
// temporaries (element offsets; CT = compute type)
// ---------------------------------------------------------------------------
struct SplitLayout {
  rec::RecLayout r;
};

constexpr SplitLayout make_split_layout(int Cp, int d, int h) {
  return SplitLayout{rec::make_rec_layout(Cp, d, h)};
}

// Dynamic LDS of pass A (CT = compute type, fp32 where named):
//   Zb   [CP][H] CT  Zbar (phases 2-4), then Kbar, Nbar [CP][D] fp32 each
//   pA, pE  [(D/16)][CP] fp32  partial row sums of the Xbar epilogue
//   U    one region used in turn:
//        phases 0-2: dO [CP][D] CT, Q1 [CP][CP] CT, partial dA, dE [D/8][CP] fp32
//        phases 3-:  Q2, Q2T [CP][CP] CT (later dXN, dXNT), Xbar [CP][D], Xbar^T [D][CP] CT
// cbar stays in the registers of the wave that owns its tiles (phases 1 and 3
// walk the same C x C blocks); the retrieval's dA, dE in the registers of the
// thread of their position.  About 66 KB at 64 rows with the chunk
// coefficients' 10 KB: two workgroups per CU.
template <typename CT, int CP, int D, int H>
struct ALds {
  static constexpr size_t cmax(size_t x, size_t y) { return x > y ? x : y; }
  static constexpr size_t zb = 0;
  static constexpr size_t pa = zb + cmax((size_t)CP * H * sizeof(CT), 2 * (size_t)CP * D * sizeof(float));
  static constexpr size_t pe = pa + (size_t)(D / 16) * CP * sizeof(float);
  static constexpr size_t u = pe + (size_t)(D / 16) * CP * sizeof(float);
  // phases 0-2
  static constexpr size_t dO = u;
  static constexpr size_t q1 = dO + (size_t)CP * D * sizeof(CT);
  static constexpr size_t dpa = q1 + (size_t)CP * CP * sizeof(CT);
  static constexpr size_t dpe = dpa + (size_t)(D / 8) * CP * sizeof(float);
  static constexpr size_t ua = dpe + (size_t)(D / 8) * CP * sizeof(float) - u;
  // phases 3-
  static constexpr size_t q2 = u;
  static constexpr size_t q2t = q2 + (size_t)CP * CP * sizeof(CT);
  static constexpr size_t xb = q2t + (size_t)CP * CP * sizeof(CT);
  static constexpr size_t xbt = xb + (size_t)CP * D * sizeof(CT);
  static constexpr size_t ub = xbt + (size_t)D * CP * sizeof(CT) - u;
  static constexpr size_t total = u + cmax(ua, ub);
  static_assert(pa % 16 == 0 && u % 16 == 0 && q1 % 16 == 0 && dpa % 16 == 0 && q2t % 16 == 0 &&
                    xb % 16 == 0 && xbt % 16 == 0,
                "16-byte aligned regions");
};


template <typename CT, int CP, int D, int H>
constexpr size_t split_a_lds() {
  return ALds<CT, CP, D, H>::total;
}
// static LDS of pass A: the chunk coefficients
constexpr size_t SPLIT_A_STATIC = sizeof(CoefF);

// pass B: a CP x H compute-type slot (Gbar, then Zkbar); T3, T4 and T5, T6
// (fragment-major fp32, CP x D each; the T5/T6 space holds Zkbar^T, H x CP
// compute type, from phase 3 on); Ykbar and Ykbar^T (CP x D compute type each);
// per-column-tile partial row sums for cC_bar, b_bar (K . T3, K . T4, R . T5, R . T6:
// (D/16) x CP fp32 each);
// Gbar^T (H x CP compute type)
template <typename CT, int CP, int D, int H>
struct SplitBLds {
  static constexpr size_t cmax(size_t x, size_t y) { return x > y ? x : y; }
  static constexpr size_t slot = (size_t)CP * H * sizeof(CT);
  static constexpr size_t t34 = slot;
  static constexpr size_t t56 = t34 + 2 * (size_t)CP * D * sizeof(float);
  static constexpr size_t ykb = t56 + cmax(2 * (size_t)CP * D * sizeof(float), (size_t)H * CP * sizeof(CT));
  static constexpr size_t ykbt = ykb + (size_t)CP * D * sizeof(CT);
  static constexpr size_t pc = ykbt + (size_t)CP * D * sizeof(CT);
  static constexpr size_t pb = pc + (size_t)(D / 16) * CP * sizeof(float);
  static constexpr size_t pc2 = pb + (size_t)(D / 16) * CP * sizeof(float);
  static constexpr size_t pb2 = pc2 + (size_t)(D / 16) * CP * sizeof(float);
  static constexpr size_t gbt = pb2 + (size_t)(D / 16) * CP * sizeof(float);
  static constexpr size_t total = gbt + (size_t)H * CP * sizeof(CT);
};
template <typename CT, int CP, int D, int H>
constexpr size_t split_b_lds() {
  return SplitBLds<CT, CP, D, H>::total;
}
// pass C: cbar (CP x CP fp32) and the gate partials (5 x 8 x CP fp32); the Q-K
// term uses the same space first (Mbar in padded rows, D x (D + 1) fp32, then
// Nbar, CP x D fp32, in the same place; Msym: D x D compute type after it)
template <typename CT, int CP, int D>
constexpr size_t split_c_lds() {
  static_assert(CP <= D + 1, "Nbar fits where Mbar was");
  const size_t gate = ((size_t)CP * CP + 40 * (size_t)CP) * sizeof(float);
  const size_t qk = (size_t)D * (D + 1) * sizeof(float) + (size_t)D * D * sizeof(CT);
  return gate > qk ? gate : qk;
}

}  // namespace

struct SplitPtrs {
  void* brec;       // CT   [units * nch][r.bc.n]  backward records
  float* brec_f;    // fp32 [units * nch][r.bf.n]
  int units;
  int n0, nc;       // passes A and B: the chunks n0 .. n0 + nc - 1 of every unit
};

// ===========================================================================
// pass A: backward of the retrieval of every chunk, from dO and the forward record
// ===========================================================================
// Built for 128 VGPRs and ALds' LDS, so that two workgroups share a CU and
// overlap each other's waits.  One workgroup per chunk: a grid-stride loop lets
// the compiler hoist every per-lane address out of the loop, and at 128 VGPRs
// those hoisted values spill.
template <typename IO, typename CT, int ACT, int D, int H, int CP>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4, 8)))
local_bwd_ret_kernel(LocalBwdArgs a, SplitPtrs P) {
  __shared__ CoefF cf;
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int d = D, h = H, Cp = CP;
  using AL = ALds<CT, CP, D, H>;
  CT* const Zb = reinterpret_cast<CT*>(smem + AL::zb);  // C x h slot
  float* const pA = reinterpret_cast<float*>(smem + AL::pa);
  float* const pE = reinterpret_cast<float*>(smem + AL::pe);
  CT* const dO = reinterpret_cast<CT*>(smem + AL::dO);
  CT* const Q1 = reinterpret_cast<CT*>(smem + AL::q1);
  float* const dpa = reinterpret_cast<float*>(smem + AL::dpa);  // [D/8][CP] partial dA, dE
  float* const dpe = reinterpret_cast<float*>(smem + AL::dpe);
  CT* const Q2 = reinterpret_cast<CT*>(smem + AL::q2);
  CT* const Q2T = reinterpret_cast<CT*>(smem + AL::q2t);
  CT* const dXN = Q2;    // the Q-K phase, once Q2 and Q2^T are dead
  CT* const dXNT = Q2T;
  CT* const Xb = reinterpret_cast<CT*>(smem + AL::xb);
  CT* const XbT = reinterpret_cast<CT*>(smem + AL::xbt);
  // Kbar and Nbar (fp32 C x d each) take the Zbar slot once Xbar has read it
  float *fKb = reinterpret_cast<float*>(smem + AL::zb), *fNb = fKb + CP * D;

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int nch = Dm.S / C;
  const int total = P.units * P.nc;
  constexpr size_t hd = (size_t)h * d;
  constexpr SplitLayout Y = make_split_layout(CP, D, H);
  const bool shard_qk = Dm.qk_proj && Dm.qk_scope == 0;
  using BCD = Blk<CP, D>;
  using BCC = Blk<CP, CP>;
  using BDD = Blk<D, D>;
  constexpr int NWH = 16;  // C x h products in blocks of half the usual size
  using BCH = Blk<CP, H, NWH>;
  static_assert(BCC::NB <= 8, "each wave owns at most one C x C block (its cbar tiles)");

  if (const int tl = blockIdx.x; tl < total) {  // one chunk per workgroup
    const int u = tl / P.nc, n = P.n0 + (tl - u * P.nc);
    const int t = u * nch + n;
    const int b = u / (Dm.H * nshard), hh = (u / nshard) % Dm.H, s = u % nshard;
    const CT* fr = (const CT*)a.frec + (size_t)t * Y.r.fc.n;
    const float* frf = a.frec_f + (size_t)t * Y.r.ff.n;
    CT* br = (CT*)P.brec + (size_t)t * Y.r.bc.n;
    float* brf = P.brec_f + (size_t)t * Y.r.bf.n;
    fr = launder_global(fr);
    frf = launder_global(frf);
    br = launder_global(br);
    brf = launder_global(brf);
    const size_t cbase = ((size_t)b * Dm.H + hh) * Dm.L;
    const IO* dOg = (const IO*)a.dO + cbase * d;
    float* dqp = a.dq_part + cbase * d;
    float* dkp = a.dk_part + cbase * d;
#define FR_(x) (fr + Y.r.fc.o[rec::x])
#define FRF_(x) (frf + Y.r.ff.o[rec::x])
#define BR_(x) (br + Y.r.bc.o[rec::x])
#define BRF_(x) (brf + Y.r.bf.o[rec::x])
    const CT *HkT = FR_(HkT), *D1 = FR_(D1), *Sz = FR_(Sz), *KT = FR_(KT), *R = FR_(R),
             *XT = FR_(XT), *N = FR_(N), *NT = FR_(NT), *QT = FR_(QT), *StrT = FR_(StrT);
    const float *fXK = FRF_(XK), *fHH = FRF_(HH), *fHW2 = FRF_(HW2), *fHS2 = FRF_(HS2),
                *knorm = FRF_(kn);
    CT *ZbT = BR_(ZbT), *Q1T = BR_(Q1T), *dOT = BR_(dOT), *dOAT = BR_(dOAT), *dOET = BR_(dOET);
    const int tok0 = s * Dm.S + n * C;
    const int l = lane_id_local();
    const CT* pk = (const CT*)a.statesT + ((size_t)u * a.nslots + n) * (4 * hd + (size_t)d * d);
    const CT *W1T = pk, *W2T = pk + hd, *S1T = pk + 2 * hd, *S2T = pk + 3 * hd, *McT = pk + 4 * hd;

    // ---- chunk coefficients; stage dO (one (row, 8-column block) per thread,
    // consecutive threads on consecutive rows) and its scaled and transposed
    // forms for the backward record; partial dA, dE of the retrieval,
    // sum_k dO_ik (H W2^T)_ik (S2 likewise)
    if constexpr (rec::rec_coefs(CP))
      coefs_from_record_f(cf, FRF_(Cc), FRF_(cA), FRF_(cE), Cp);  // ends with a barrier
    else
      chunk_coefs_f(cf, a.lr + cbase, a.mom + cbase, a.decay + cbase, tok0, C, Cp);  // likewise
    constexpr int JB = D / 8, ITEMS = CP * JB, PER = (ITEMS + 511) / 512;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int e = threadIdx.x + p * 512;
      if (e < ITEMS) {
        const int i = e % CP, j0 = (e / CP) * 8;
        const size_t en = (size_t)i * d + j0;
        float ox[8];
        if (i < C) {
          load8(dOg + (size_t)(tok0 + i) * d + j0, ox);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) ox[q] = 0.f;
        }
        float sa = 0.f, se = 0.f;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const size_t et = (size_t)(j0 + q) * Cp + i;  // consecutive lanes: consecutive i
          const float w2 = fHW2[et], s2 = fHS2[et];
          dOT[et] = from_f<CT>(ox[q]);
          dOAT[et] = from_f<CT>(cf.A[i] * ox[q]);
          dOET[et] = from_f<CT>(cf.E[i] * ox[q]);
          const float oq = to_f(from_f<CT>(ox[q]));  // dO as the contractions see it
          sa += oq * w2;
          se += oq * s2;
        }
        store8<CT>(dO + en, ox);
        dpa[(j0 / 8) * CP + i] = sa;
        dpe[(j0 / 8) * CP + i] = se;
      }
    }
    __syncthreads();
    float gAi = 0.f, gEi = 0.f;  // thread i's retrieval dA_i, dE_i
    if (threadIdx.x < Cp) {
      const int i = threadIdx.x;
#pragma unroll
      for (int q = 0; q < JB; ++q) {  // fixed order: deterministic
        gAi += dpa[q * CP + i];
        gEi += dpe[q * CP + i];
      }
    }
    // dOR = dO R^T ; Q1 = c o dOR ; cbar = -HH o dOR (kept in the wave's registers)
    f4 cbr[BCC::RB][BCC::CB];
    zero_blk(cbr);
    for_blocks<CP, CP>([&](int i0, int j0) {
      f4 hhv[BCC::RB][BCC::CB];  // H Hk^T, requested ahead of the product
      blk_each4<BCC::RB, BCC::CB>(i0, j0, [&](int rb, int cb, int, int) {
        hhv[rb][cb] = load4<float>(fHH + frag_ofs<CP, CP>(i0 + 16 * rb, j0 + 16 * cb, l));
      });
      f4 acc[BCC::RB][BCC::CB];
      zero_blk(acc);
      mma_blk<CT, KC, KC, BCC::RB, BCC::CB, D>(acc, dO, d, i0, R, d, j0);
      blk_each4<BCC::RB, BCC::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        const f4 hv = hhv[rb][cb];
        f4 qv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = i + r;
          const float x = acc[rb][cb][r];
          const bool lo = j <= ii;
          qv[r] = lo ? cf.cc(ii, j) * x : 0.f;
          Q1[(size_t)ii * Cp + j] = from_f<CT>(qv[r]);
          cbr[rb][cb][r] = lo ? -hv[r] * x : 0.f;
        }
        store4<CT>(Q1T + (size_t)j * Cp + i, qv);
      });
    });
    __syncthreads();
    // Hbar = diag(A) dO W2 + diag(E) dO S2 - Q1 Hk ; Zbar = Hbar * s'(Z)
    for_blocks_n<CP, H, NWH>([&](int i0, int j0) {
      typedef CT ct4 __attribute__((ext_vector_type(4)));
      ct4 szv[BCH::RB][BCH::CB];  // s'(Z), requested ahead of the products
      blk_each4<BCH::RB, BCH::CB>(i0, j0, [&](int rb, int cb, int, int) {
        szv[rb][cb] = *reinterpret_cast<const ct4*>(Sz + frag_ofs<CP, H>(i0 + 16 * rb, j0 + 16 * cb, l));
      });
      f4 a1[BCH::RB][BCH::CB], a2[BCH::RB][BCH::CB], a3[BCH::RB][BCH::CB];
      zero_blk(a1);
      zero_blk(a2);
      zero_blk(a3);
      mma_blk<CT, KC, KC, BCH::RB, BCH::CB, D>(a1, dO, d, i0, W2T, d, j0);
      mma_blk<CT, KC, KC, BCH::RB, BCH::CB, D>(a2, dO, d, i0, S2T, d, j0);
      mma_blk<CT, KC, KC, BCH::RB, BCH::CB, CP>(a3, Q1, Cp, i0, HkT, Cp, j0);
      blk_each4<BCH::RB, BCH::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        f4 zv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = i + r;
          zv[r] = (cf.A[ii] * a1[rb][cb][r] + cf.E[ii] * a2[rb][cb][r] - a3[rb][cb][r]) *
                  to_f(szv[rb][cb][r]);
          Zb[(size_t)ii * h + j] = from_f<CT>(zv[r]);
        }
        store4<CT>(ZbT + (size_t)j * Cp + i, zv);
      });
    });
    __syncthreads();  // dO and Q1 are dead: their region takes Q2, Q2^T, Xbar, Xbar^T
    // dZD1 = Zbar D1^T ; Q2 = c o dZD1 ; cbar -= XK o dZD1, then cbar to the record
    for_blocks<CP, CP>([&](int i0, int j0) {
      f4 xkv[BCC::RB][BCC::CB];  // X K^T, requested ahead of the product
      blk_each4<BCC::RB, BCC::CB>(i0, j0, [&](int rb, int cb, int, int) {
        xkv[rb][cb] = load4<float>(fXK + frag_ofs<CP, CP>(i0 + 16 * rb, j0 + 16 * cb, l));
      });
      f4 acc[BCC::RB][BCC::CB];
      zero_blk(acc);
      mma_blk<CT, KC, KC, BCC::RB, BCC::CB, H>(acc, Zb, h, i0, D1, h, j0);
      blk_each4<BCC::RB, BCC::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        const f4 xk = xkv[rb][cb];
        f4 qv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = i + r;
          const float x = acc[rb][cb][r];
          const bool lo = j <= ii;
          qv[r] = lo ? cf.cc(ii, j) * x : 0.f;
          Q2[(size_t)ii * Cp + j] = from_f<CT>(qv[r]);
          if (lo) cbr[rb][cb][r] -= xk[r] * x;
          BRF_(Cb)[(size_t)ii * Cp + j] = cbr[rb][cb][r];
        }
        store4<CT>(Q2T + (size_t)j * Cp + i, qv);
      });
    });
    __syncthreads();
    // Xbar = diag(A) Zbar W1 + diag(E) Zbar S1 - Q2 K
    for_blocks<CP, D>([&](int i0, int j0) {
      typedef CT ct4 __attribute__((ext_vector_type(4)));
      ct4 xv4[BCD::RB][BCD::CB];  // X, the lane's four rows from X^T, ahead of the products
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        xv4[rb][cb] = *reinterpret_cast<const ct4*>(XT + (size_t)j * Cp + i);
      });
      f4 a1[BCD::RB][BCD::CB], a2[BCD::RB][BCD::CB], a3[BCD::RB][BCD::CB];
      zero_blk(a1);
      zero_blk(a2);
      zero_blk(a3);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, H>(a1, Zb, h, i0, W1T, h, j0);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, H>(a2, Zb, h, i0, S1T, h, j0);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, CP>(a3, Q2, Cp, i0, KT, Cp, j0);
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        f4 xv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = i + r;
          const float x = to_f(xv4[rb][cb][r]);
          xv[r] = cf.A[ii] * a1[rb][cb][r] + cf.E[ii] * a2[rb][cb][r] - a3[rb][cb][r];
          Xb[(size_t)ii * d + j] = from_f<CT>(xv[r]);
          if (!Dm.qk_proj && ii < C) dqp[(size_t)(tok0 + ii) * d + j] = xv[r];
          const float sa = sum16b(a1[rb][cb][r] * x), se = sum16b(a2[rb][cb][r] * x);
          if ((l & 15) == 0) {
            pA[(j >> 4) * Cp + ii] = sa;
            pE[(j >> 4) * Cp + ii] = se;
          }
        }
        store4<CT>(XbT + (size_t)j * Cp + i, xv);
      });
    });
    __syncthreads();  // Zbar is dead: its slot takes Kbar, Nbar
    // Kbar (retrieval part) = -Q2^T X
    for_blocks<CP, D>([&](int i0, int j0) {
      f4 a1[BCD::RB][BCD::CB];
      zero_blk(a1);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, CP>(a1, Q2T, Cp, i0, XT, Cp, j0);
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
        for (int r = 0; r < 4; ++r) fKb[(size_t)(i + r) * d + j] = -a1[rb][cb][r];
      });
    });
    __syncthreads();  // Q2, Q2^T are dead: their space takes dXN, dXN^T
    if (threadIdx.x < Cp) {
      const int i = threadIdx.x;
      float sa = 0.f, se = 0.f;
#pragma unroll
      for (int q = 0; q < (d >> 4); ++q) {
        sa += pA[q * Cp + i];
        se += pE[q * Cp + i];
      }
      BRF_(gA)[i] = gAi + sa;
      BRF_(gE)[i] = gEi + se;
    }
    if (Dm.qk_proj) {
      // dXN = tril(Xbar N^T)
      for_blocks<CP, CP>([&](int i0, int j0) {
        f4 acc[BCC::RB][BCC::CB];
        zero_blk(acc);
        mma_blk<CT, KC, KC, BCC::RB, BCC::CB, D>(acc, Xb, d, i0, N, d, j0);
        blk_each4<BCC::RB, BCC::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
          f4 y;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            y[r] = j <= i + r ? acc[rb][cb][r] : 0.f;
            dXN[(size_t)(i + r) * Cp + j] = from_f<CT>(y[r]);
          }
          store4<CT>(dXNT + (size_t)j * Cp + i, y);
        });
      });
      // Xbar^T Q for the carried Q-K state adjoint
      if (shard_qk)
        for_blocks<D, D>([&](int i0, int j0) {
          f4 a1[BDD::RB][BDD::CB];
          zero_blk(a1);
          mma_blk<CT, KC, KC, BDD::RB, BDD::CB, CP>(a1, XbT, Cp, i0, QT, Cp, j0);
          blk_each4<BDD::RB, BDD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
            for (int r = 0; r < 4; ++r) BRF_(XbQ)[(size_t)(i + r) * d + j] = a1[rb][cb][r];
          });
        });
      __syncthreads();
      // Qbar = Xbar M0 + tril(Xbar N^T) N ; Nbar (this chunk's terms) = Str^T Xbar + dXN^T Q
      for_blocks<CP, D>([&](int i0, int j0) {
        f4 q1[BCD::RB][BCD::CB], n1[BCD::RB][BCD::CB];
        zero_blk(q1);
        zero_blk(n1);
        if (shard_qk) mma_blk<CT, KC, KC, BCD::RB, BCD::CB, D>(q1, Xb, d, i0, McT, d, j0);
        mma_blk<CT, KC, KC, BCD::RB, BCD::CB, CP>(q1, dXN, Cp, i0, NT, Cp, j0);
        mma_blk<CT, KC, KC, BCD::RB, BCD::CB, CP>(n1, StrT, Cp, i0, XbT, Cp, j0);
        mma_blk<CT, KC, KC, BCD::RB, BCD::CB, CP>(n1, dXNT, Cp, i0, QT, Cp, j0);
        blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ii = i + r;
            if (ii < C) dqp[(size_t)(tok0 + ii) * d + j] = q1[rb][cb][r];
            fNb[(size_t)ii * d + j] = n1[rb][cb][r];
          }
        });
      });
      __syncthreads();
      // Kbar += (Nbar - N (N . Nbar)) / ||k||
      for (int i = wave_id(); i < C; i += num_waves()) {
        const float nr = knorm[i];
        float dt = 0.f;
        for (int j = l; j < d; j += WAVE) dt += to_f(N[(size_t)i * d + j]) * fNb[(size_t)i * d + j];
        dt = wave_sum(dt);
        if (nr > 0.f)
          for (int j = l; j < d; j += WAVE) {
            const size_t e = (size_t)i * d + j;
            fKb[e] += (fNb[e] - to_f(N[e]) * dt) / nr;
          }
      }
      __syncthreads();
    }
    for (int e = threadIdx.x * 4; e < C * d; e += blockDim.x * 4)
      *reinterpret_cast<f32x4*>(dkp + (size_t)tok0 * d + e) = *reinterpret_cast<const f32x4*>(fKb + e);
    __syncthreads();  // the next chunk reuses LDS and the temporaries
#undef FR_
#undef FRF_
#undef BR_
#undef BRF_
  }
}

// Two products sharing their A operand over all CP rows, for one 16-column strip
// j0 of the outputs: t0 += A B0[j0.., :]^T, t1 += A B1[j0.., :]^T (A rows and B rows
// contraction-contiguous, K long).  The K steps go in groups of G with every
// load of a group in flight before its MFMAs.  Alongside, the strip's share of
// the elementwise products with two compute-type matrices S0, S1 of the B
// operands' shape (layout SL: KC as the B operands, MC transposed, leading
// dimension lds), both sides as the MFMAs see them (compute type):
// pa += B0 . S0, pe += B0 . S1, pb += B1 . S1.
template <int RBN, int K, int G, int SL, int BL = KC, typename EB = float>
__device__ __forceinline__ void mma_pair_dots(f4 (&t0)[RBN], f4 (&t1)[RBN], const __bf16* A,
                                              int lda, const EB* B0, const EB* B1, int ldb,
                                              int j0, const __bf16* S0, const __bf16* S1,
                                              int lds, float& pa, float& pe, float& pb) {
  typedef Mma<__bf16> MM;
  const int l = lane_id_local();
  const int ko = MM::kofs(l), jr = j0 + (l & 15);
  constexpr int NS = K / MM::KS;
  static_assert(K % MM::KS == 0 && NS % G == 0, "whole groups of K steps");
#pragma unroll 1
  for (int g0 = 0; g0 < NS; g0 += G) {
    typename MM::frag fa[G][RBN], f0[G], f1[G], s0[G], s1[G];
#pragma unroll
    for (int st = 0; st < G; ++st) {
      const int k0 = (g0 + st) * MM::KS + ko;
#pragma unroll
      for (int r = 0; r < RBN; ++r)
        fa[st][r] = MM::template load<KC>(A, lda, 16 * r + (l & 15), k0, K, nullptr);
      f0[st] = MM::template load<BL>(B0, ldb, jr, k0, K, nullptr);
      f1[st] = MM::template load<BL>(B1, ldb, jr, k0, K, nullptr);
      s0[st] = MM::template load<SL>(S0, lds, jr, k0, K, nullptr);
      s1[st] = MM::template load<SL>(S1, lds, jr, k0, K, nullptr);
    }
#pragma unroll
    for (int st = 0; st < G; ++st) {
#pragma unroll
      for (int r = 0; r < RBN; ++r) {
        MM::mma(t0[r], fa[st][r], f0[st]);
        MM::mma(t1[r], fa[st][r], f1[st]);
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float x0 = (float)f0[st][q], x1 = (float)f1[st][q];
        const float y0 = (float)s0[st][q], y1 = (float)s1[st][q];
        pa += x0 * y0;
        pe += x0 * y1;
        pb += x1 * y1;
      }
    }
  }
}

// ===========================================================================
// pass B: the carried adjoint, walked back through a unit's chunks
// ===========================================================================
template <typename IO, typename CT, int ACT, int D, int H, int CP>
__global__ void __launch_bounds__(512) local_bwd_chain_kernel(LocalBwdArgs a, SplitPtrs P) {
  __shared__ float sC[MAXC], sB[MAXC], sc3[4];
  __shared__ float dpart[3][16];
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int d = D, h = H, Cp = CP;
  using LB = SplitBLds<CT, CP, D, H>;
  CT* slot1 = reinterpret_cast<CT*>(smem);  // Gbar (D1bar .. Rbar), then Zkbar (Hkbar .. Kbar)
  float* const fT3 = reinterpret_cast<float*>(smem + LB::t34);
  float* const fT4 = fT3 + CP * D;
  float* const fT5 = reinterpret_cast<float*>(smem + LB::t56);
  float* const fT6 = fT5 + CP * D;
  CT* const ZkbT = reinterpret_cast<CT*>(smem + LB::t56);  // T5, T6 are dead from phase 3 on
  CT* const Ykb = reinterpret_cast<CT*>(smem + LB::ykb);
  CT* const YkbT = reinterpret_cast<CT*>(smem + LB::ykbt);
  float* const pC = reinterpret_cast<float*>(smem + LB::pc);
  float* const pB = reinterpret_cast<float*>(smem + LB::pb);
  float* const pC2 = reinterpret_cast<float*>(smem + LB::pc2);
  float* const pB2 = reinterpret_cast<float*>(smem + LB::pb2);
  CT* const GbT = reinterpret_cast<CT*>(smem + LB::gbt);

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int nch = Dm.S / C;
  const int u = blockIdx.x;
  const int b = u / (Dm.H * nshard), hh = (u / nshard) % Dm.H, s = u % nshard;
  constexpr size_t hd = (size_t)h * d;
  constexpr SplitLayout Y = make_split_layout(CP, D, H);
  const float rscale = 2.0f / (float)d;
  const size_t cbase = ((size_t)b * Dm.H + hh) * Dm.L;
  float* dkp = a.dk_part + cbase * d;
  float* dvp = a.dv_part + cbase * d;
  float* const adj0 = a.adj + (size_t)u * 4 * hd;
  using BCH0 = Blk<CP, H>;
  static_assert(BCH0::NB <= 8, "each wave owns at most one C x h block");

  // the adjoint leaving the shard's last chunk is zero: that chunk skips every
  // product with it and writes the adjoint without reading it
  for (int n = P.n0 + P.nc - 1; n >= P.n0; --n) {
    const bool zadj = n == nch - 1;
    const size_t t = (size_t)u * nch + n;
    const CT* rc = (const CT*)a.frec + t * Y.r.fc.n;
    const float* rf = a.frec_f + t * Y.r.ff.n;
    CT* bq = (CT*)P.brec + t * Y.r.bc.n;
    float* bqf = P.brec_f + t * Y.r.bf.n;
    float* adj = adj0;
    rc = launder_global(rc);
    rf = launder_global(rf);
    bq = launder_global(bq);
    bqf = launder_global(bqf);
    adj = launder_global(adj);
#define R_(x) (rc + Y.r.fc.o[rec::x])
#define RF_(x) (rf + Y.r.ff.o[rec::x])
#define BQ_(x) (bq + Y.r.bc.o[rec::x])
#define BQF_(x) (bqf + Y.r.bf.o[rec::x])
    float *Wb1 = adj, *Wb2 = adj + hd, *Sb1 = adj + 2 * hd, *Sb2 = adj + 3 * hd;
    CT *Gb = slot1, *Zkb = slot1;
    // the Zkbar terms known after phase 1, kept by the wave that owns the block
    // until phase 3 (both phases walk the same C x h blocks)
    f4 zkp[BCH0::RB][BCH0::CB];
    const CT *Hk = R_(Hk), *HkT = R_(HkT), *D1 = R_(D1), *ZbT = BQ_(ZbT), *HT = R_(HT),
             *Sp = R_(Sp), *Spp = R_(Spp), *G = R_(G), *PzT = R_(PzT), *Q1T = BQ_(Q1T),
             *PoT = R_(PoT), *K = R_(K), *KT = R_(KT), *KcC = R_(KcC), *Kb = R_(Kb), *R = R_(R),
             *RT = R_(RT), *RcC = R_(RcC), *Rb = R_(Rb), *dOT = BQ_(dOT), *XAT = R_(XAT),
             *XET = R_(XET), *dOAT = BQ_(dOAT), *dOET = BQ_(dOET);
    const int tok0 = s * Dm.S + n * C;
    const int l = lane_id_local();
    const CT* pk = (const CT*)a.statesT + ((size_t)u * a.nslots + n) * (4 * hd + (size_t)d * d);
    const CT *W1T = pk, *W2T = pk + hd, *S1T = pk + 2 * hd, *S2T = pk + 3 * hd;
    using BCD = Blk<CP, D>;
    using BCH = Blk<CP, H>;
    auto fofs = [&](int i0, int j0, int rb, int cb) -> size_t {
      const int blk = (i0 / (BCH::RB * 16)) * BCH::NBN + j0 / (BCH::CB * 16);
      return ((size_t)((blk * BCH::RB + rb) * BCH::CB + cb) * WAVE + l) * 4;
    };
    auto fofsD = [&](int i0, int j0, int rb, int cb) -> size_t {  // C x d tiles, fragment-major
      const int blk = (i0 / (BCD::RB * 16)) * BCD::NBN + j0 / (BCD::CB * 16);
      return ((size_t)((blk * BCD::RB + rb) * BCD::CB + cb) * WAVE + l) * 4;
    };

    // ---- phase 1: chunk coefficients; T3..T6 with the adjoint . state dot products
    // (dA_C, dE_C, dB_C); D1bar -> Gbar; the first part of Hkbar
    if (threadIdx.x < Cp) {
      sC[threadIdx.x] = RF_(cC)[threadIdx.x];
      sB[threadIdx.x] = RF_(bb)[threadIdx.x];
    }
    if (threadIdx.x < 3) sc3[threadIdx.x] = RF_(sc)[threadIdx.x];
    // T3 = D1 W1bar', T4 = D1 S1bar' (waves 0-3), T5 = Hk W2bar'^T, T6 = Hk S2bar'^T (waves
    // 4-7), C x d each: a wave takes one 16-column strip of a pair over all rows, the pair
    // sharing its A fragments.  Kept in LDS at their fragment positions; the cC_bar / b_bar
    // row dots (-K.T3 - R.T5, -K.T4 - R.T6) as partial sums over each tile's 16 columns.
    // The strips of the adjoint's B operands cover it whole: the adjoint . state products
    // are taken from the same fragments, both sides as the MFMAs see them (the adjoint
    // read down its fp32 columns and rounded to the compute type, the state from its
    // transposed compute-type copy).
    {
      static_assert(D == 64, "two pairs of four column strips for eight waves");
      static_assert(sizeof(CT) == 2, "bf16 operands");
      constexpr int RBN = CP / 16;
      const int pair = wave_id() >> 2, j0 = 16 * (wave_id() & 3);
      f4 t0[RBN], t1[RBN];
#pragma unroll
      for (int r = 0; r < RBN; ++r) t0[r] = t1[r] = zero4();
      float pa = 0.f, pe = 0.f, pb = 0.f;
      // the row-dot factors (K for T3, T4; R for T5, T6), the lane's four rows of its
      // column from the transposed record, requested ahead of the products
      typedef CT ct4 __attribute__((ext_vector_type(4)));
      ct4 mxv[RBN];
      {
        const CT* MT = pair == 0 ? KT : RT;
#pragma unroll
        for (int rb = 0; rb < RBN; ++rb)
          mxv[rb] = *reinterpret_cast<const ct4*>(MT + (size_t)(j0 + (l & 15)) * Cp + 16 * rb + 4 * (l >> 4));
      }
      if (zadj) {
      } else if (pair == 0) {
        mma_pair_dots<RBN, H, 4, KC, MC>(t0, t1, D1, h, Wb1, Sb1, d, j0, W1T, S1T, h, pa, pe, pb);
      } else {
        mma_pair_dots<RBN, H, 4, MC>(t0, t1, Hk, h, Wb2, Sb2, h, j0, W2T, S2T, d, pa, pe, pb);
      }
      pa = wave_sum(pa);
      pe = wave_sum(pe);
      pb = wave_sum(pb);
      if (l == 0) {
        dpart[0][wave_id()] = pa;
        dpart[1][wave_id()] = pe;
        dpart[2][wave_id()] = pb;
      }
      float* const q0 = pair == 0 ? pC : pC2;
      float* const q1 = pair == 0 ? pB : pB2;
      float* const f0 = pair == 0 ? fT3 : fT5;
      float* const f1 = pair == 0 ? fT4 : fT6;
#pragma unroll
      for (int rb = 0; rb < RBN; ++rb) {
        const size_t fo = frag_ofs<CP, D>(16 * rb, j0, l);
        store4<float>(f0 + fo, t0[rb]);
        store4<float>(f1 + fo, t1[rb]);
        const int i = 16 * rb + 4 * (l >> 4), j = j0 + (l & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float mx = to_f(mxv[rb][r]);
          const float s0 = sum16b(mx * t0[rb][r]), s1 = sum16b(mx * t1[rb][r]);
          if ((l & 15) == 0) {
            q0[(j >> 4) * Cp + i + r] = s0;
            q1[(j >> 4) * Cp + i + r] = s1;
          }
        }
      }
    }
    // D1bar = -Pz^T Zbar - diag(cC) K W1bar'^T - diag(b) K S1bar'^T ; Gbar = D1bar * s'(Zk);
    // Hkbar so far = -Q1^T H - diag(cC) R W2bar' - diag(b) R S2bar' ; the Zkbar terms known
    // now, D1bar * G * s''(Zk) + Hkbar * s'(Zk), are kept per fragment
    for_blocks<CP, H>([&](int i0, int j0) {
      typedef CT ct4 __attribute__((ext_vector_type(4)));
      ct4 spv[BCH::RB][BCH::CB], gv4[BCH::RB][BCH::CB], sppv[BCH::RB][BCH::CB];  // ahead of the products
      blk_each4<BCH::RB, BCH::CB>(i0, j0, [&](int rb, int cb, int, int) {
        const size_t fo = fofs(i0, j0, rb, cb);
        spv[rb][cb] = *reinterpret_cast<const ct4*>(Sp + fo);
        gv4[rb][cb] = *reinterpret_cast<const ct4*>(G + fo);
        sppv[rb][cb] = *reinterpret_cast<const ct4*>(Spp + fo);
      });
      f4 a1[BCH::RB][BCH::CB], a2[BCH::RB][BCH::CB];
      zero_blk(a1);
      zero_blk(a2);
      mma_blk<CT, KC, KC, BCH::RB, BCH::CB, CP>(a1, PzT, Cp, i0, ZbT, Cp, j0);
      mma_blk<CT, KC, KC, BCH::RB, BCH::CB, CP>(a2, Q1T, Cp, i0, HT, Cp, j0);
      if (!zadj) {
        mma_blk<CT, KC, KC, BCH::RB, BCH::CB, D>(a1, KcC, d, i0, Wb1, d, j0);
        mma_blk<CT, KC, KC, BCH::RB, BCH::CB, D>(a1, Kb, d, i0, Sb1, d, j0);
        mma_blk<CT, KC, MC, BCH::RB, BCH::CB, D>(a2, RcC, d, i0, Wb2, h, j0);
        mma_blk<CT, KC, MC, BCH::RB, BCH::CB, D>(a2, Rb, d, i0, Sb2, h, j0);
      }
      blk_each4<BCH::RB, BCH::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        f4 gv, zp;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d1b = -a1[rb][cb][r], sp = to_f(spv[rb][cb][r]);
          gv[r] = d1b * sp;
          zp[r] = d1b * to_f(gv4[rb][cb][r]) * to_f(sppv[rb][cb][r]) - a2[rb][cb][r] * sp;
          Gb[(size_t)(i + r) * h + j] = from_f<CT>(gv[r]);
        }
        zkp[rb][cb] = zp;
        store4<CT>(GbT + (size_t)j * Cp + i, gv);
      });
    });
    __syncthreads();

    // ---- phase 2: cC_bar = -K.T3 - R.T5, b_bar = -K.T4 - R.T6 (row dots);
    // Rbar = -Po^T dO - diag(cC) T5 - diag(b) T6 + Gbar W2^T ; Ykbar = (2/d) Rbar ; Vbar = -Ykbar
    for (int i = threadIdx.x; i < Cp; i += blockDim.x) {
      float sc_ = 0.f, sb_ = 0.f;
#pragma unroll
      for (int q = 0; q < (d >> 4); ++q) {  // fixed order: deterministic
        sc_ += pC[q * Cp + i] + pC2[q * Cp + i];
        sb_ += pB[q * Cp + i] + pB2[q * Cp + i];
      }
      BQF_(gCC)[i] = -sc_;
      BQF_(gB)[i] = -sb_;
    }
    if (threadIdx.x < 3) {
      float x = 0.f;
#pragma unroll
      for (int w = 0; w < 8; ++w) x += dpart[threadIdx.x][w];
      BQF_(dots)[threadIdx.x] = x;
    }
    for_blocks<CP, D>([&](int i0, int j0) {
      f4 a1[BCD::RB][BCD::CB], a2[BCD::RB][BCD::CB];
      zero_blk(a1);
      zero_blk(a2);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, CP>(a1, PoT, Cp, i0, dOT, Cp, j0);
      mma_blk<CT, KC, MC, BCD::RB, BCD::CB, H>(a2, Gb, h, i0, W2T, d, j0);
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        const size_t fo = fofsD(i0, j0, rb, cb);
        const f4 t5 = load4<float>(fT5 + fo), t6 = load4<float>(fT6 + fo);
        f4 yv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = i + r;
          const size_t e = (size_t)ii * d + j;
          const float rb_ = -a1[rb][cb][r] - sC[ii] * t5[r] - sB[ii] * t6[r] + a2[rb][cb][r];
          yv[r] = (ii < C) ? rscale * rb_ : 0.f;
          Ykb[e] = from_f<CT>(yv[r]);
          if (ii < C) dvp[(size_t)(tok0 + ii) * d + j] = -yv[r];
        }
        store4<CT>(YkbT + (size_t)j * Cp + i, yv);
      });
    });
    __syncthreads();

    // ---- phase 3: Zkbar = (Hkbar + Ykbar W2) * s'(Zk) + D1bar * G * s''(Zk)  (slot: Gbar is dead)
    for_blocks<CP, H>([&](int i0, int j0) {
      typedef CT ct4 __attribute__((ext_vector_type(4)));
      ct4 spv[BCH::RB][BCH::CB];  // s'(Zk), requested ahead of the product
      blk_each4<BCH::RB, BCH::CB>(i0, j0, [&](int rb, int cb, int, int) {
        spv[rb][cb] = *reinterpret_cast<const ct4*>(Sp + fofs(i0, j0, rb, cb));
      });
      f4 a4[BCH::RB][BCH::CB];
      zero_blk(a4);
      mma_blk<CT, KC, KC, BCH::RB, BCH::CB, D>(a4, Ykb, d, i0, W2T, d, j0);
      blk_each4<BCH::RB, BCH::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        const f4 zp = zkp[rb][cb];
        f4 zv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          zv[r] = a4[rb][cb][r] * to_f(spv[rb][cb][r]) + zp[r];
          Zkb[(size_t)(i + r) * h + j] = from_f<CT>(zv[r]);
        }
        store4<CT>(ZkbT + (size_t)j * Cp + i, zv);
      });
    });
    __syncthreads();

    // ---- phase 4: Kbar (carried part) = -diag(cC) T3 - diag(b) T4 + Zkbar W1 ;
    // adjoint of the chunk-entry state (in place, fp32)
    for_blocks<CP, D>([&](int i0, int j0) {
      f4 kold[BCD::RB][BCD::CB];  // dk so far, requested ahead of the product
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          kold[rb][cb][r] = (i + r < C) ? dkp[(size_t)(tok0 + i + r) * d + j] : 0.f;
      });
      f4 a2[BCD::RB][BCD::CB];
      zero_blk(a2);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, H>(a2, Zkb, h, i0, W1T, h, j0);
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        const size_t fo = fofsD(i0, j0, rb, cb);
        const f4 t3 = load4<float>(fT3 + fo), t4 = load4<float>(fT4 + fo);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = i + r;
          if (ii < C)
            dkp[(size_t)(tok0 + ii) * d + j] =
                kold[rb][cb][r] + (-sC[ii] * t3[r] - sB[ii] * t4[r] + a2[rb][cb][r]);
        }
      });
    });
    const float AC = sc3[0], BC = sc3[1], EC = sc3[2];
    using BHD = Blk<H, D>;
    using BDH = Blk<D, H>;
    for_blocks<H, D>([&](int i0, int j0) {  // W1bar, S1bar : h x d
      f4 a1[BHD::RB][BHD::CB], a3[BHD::RB][BHD::CB], ow[BHD::RB][BHD::CB], os[BHD::RB][BHD::CB];
      zero_blk(ow);
      zero_blk(os);
      if (!zadj)
        blk_each4<BHD::RB, BHD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            ow[rb][cb][r] = Wb1[(size_t)(i + r) * d + j];
            os[rb][cb][r] = Sb1[(size_t)(i + r) * d + j];
          }
        });
      zero_blk(a1);
      zero_blk(a3);
      mma_blk_shared<CT, BHD::RB, BHD::CB, CP, true>(a1, a3, ZbT, ZbT, Cp, i0, XAT, XET, Cp, j0);
      mma_blk<CT, KC, KC, BHD::RB, BHD::CB, CP>(a1, ZkbT, Cp, i0, KT, Cp, j0);
      blk_each4<BHD::RB, BHD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        f4 nw, ns;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i + r) * d + j;
          const float w = ow[rb][cb][r], sv = os[rb][cb][r];
          nw[r] = AC * w + a1[rb][cb][r];
          ns[r] = EC * w + BC * sv + a3[rb][cb][r];
          Wb1[e] = nw[r];
          Sb1[e] = ns[r];
        }
      });
    });
    for_blocks<D, H>([&](int i0, int j0) {  // W2bar, S2bar : d x h
      f4 a1[BDH::RB][BDH::CB], a4[BDH::RB][BDH::CB], ow[BDH::RB][BDH::CB], os[BDH::RB][BDH::CB];
      zero_blk(ow);
      zero_blk(os);
      if (!zadj)
        blk_each4<BDH::RB, BDH::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            ow[rb][cb][r] = Wb2[(size_t)(i + r) * h + j];
            os[rb][cb][r] = Sb2[(size_t)(i + r) * h + j];
          }
        });
      zero_blk(a1);
      zero_blk(a4);
      mma_blk_shared<CT, BDH::RB, BDH::CB, CP, false>(a1, a4, dOAT, dOET, Cp, i0, HT, HT, Cp, j0);
      mma_blk<CT, KC, KC, BDH::RB, BDH::CB, CP>(a1, RT, Cp, i0, GbT, Cp, j0);
      mma_blk<CT, KC, KC, BDH::RB, BDH::CB, CP>(a1, YkbT, Cp, i0, HkT, Cp, j0);
      blk_each4<BDH::RB, BDH::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
        f4 nw, ns;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const size_t e = (size_t)(i + r) * h + j;
          const float w = ow[rb][cb][r], sv = os[rb][cb][r];
          nw[r] = AC * w + a1[rb][cb][r];
          ns[r] = EC * w + BC * sv + a4[rb][cb][r];
          Wb2[e] = nw[r];
          Sb2[e] = ns[r];
        }
      });
    });
    __syncthreads();
#undef R_
#undef RF_
#undef BQ_
#undef BQF_
  }
  // adjoint of the learned init for this unit (after the launch that walks chunk 0)
  if (P.n0 == 0) {
    float* dst = a.dWinit_part + (size_t)u * 2 * hd;
    for (size_t e = threadIdx.x; e < 2 * hd; e += blockDim.x) dst[e] = adj0[e];
  }
}

// ===========================================================================
// Q-K state adjoint: per unit, the suffix sums over later chunks of Xbar^T Q
// (in place: chunk n's slot ends up holding the sum over chunks m > n)
// ===========================================================================
__global__ void __launch_bounds__(256) split_madj_scan_kernel(float* rec_f, size_t rec_stride,
                                                              size_t off, int units, int nch, int dd) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t u = idx / dd, e = idx - u * dd;
  if (u >= (size_t)units) return;
  float run = 0.f;
  for (int n = nch - 1; n >= 0; --n) {
    float* p = rec_f + (u * nch + n) * rec_stride + off + e;
    const float x = *p;
    *p = run;
    run += x;
  }
}

// ===========================================================================
// pass C: gate adjoints and the carried Q-K term of dk, every chunk at once
// ===========================================================================
// Sized so that four workgroups share a CU: packed coefficients, Msym in the
// compute type, and the affine scan's rows U folded into their column sums in
// the registers of the wave that scans them.
template <typename CT, int D, int H, int CP>
__global__ void __launch_bounds__(512) local_bwd_gate_kernel(LocalBwdArgs a, SplitPtrs P) {
  __shared__ CoefGN<CP> cf;
  __shared__ float gA[CP], gE[CP], gCC[CP], gB[CP], dots[4];
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int d = D, Cp = CP;
  float* fCb = reinterpret_cast<float*>(smem);
  float* gpart = fCb + Cp * Cp;  // [5][8][Cp]
  float* fNb = fCb;              // Q-K term first: Nbar [Cp][d] fp32 (Mbar [d][d + 1]
  CT* sMs = reinterpret_cast<CT*>(fCb + D * (D + 1));  // fp32 before it), Msym [d][d] CT

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int nch = Dm.S / C;
  const int t = blockIdx.x;
  const int u = t / nch, n = t - u * nch;
  const int b = u / (Dm.H * nshard), hh = (u / nshard) % Dm.H, s = u % nshard;
  constexpr SplitLayout Y = make_split_layout(CP, D, H);
  const CT* rc = (const CT*)a.frec + (size_t)t * Y.r.fc.n;
  const float* rf = a.frec_f + (size_t)t * Y.r.ff.n;
  const float* bqf = P.brec_f + (size_t)t * Y.r.bf.n;
  const size_t cbase = ((size_t)b * Dm.H + hh) * Dm.L;
  const float* mom = a.mom + cbase;
  const float* dec = a.decay + cbase;
  const int tok0 = s * Dm.S + n * C;
  const int l = lane_id();
  const bool shard_qk = Dm.qk_proj && Dm.qk_scope == 0;

  // this thread's eight elements of a row of dk: rows i, columns c0 .. c0 + 7
  // (eight threads a row, one wave's lanes 8r .. 8r + 7)
  constexpr int CPR = D / 8, ITEMS = CP * CPR;
  static_assert(ITEMS <= 512 && 64 % CPR == 0, "one item per thread, a row's threads in one wave");
  const int qi = threadIdx.x / CPR, qc = (threadIdx.x % CPR) * 8;
  const bool qrow = threadIdx.x < ITEMS && qi < C;
  float* dkp = a.dk_part + (cbase + tok0) * d;
  const bool fuse = a.dk_out != nullptr;  // write the final dk (every other part is done)
  const bool qk_here = shard_qk && n < nch - 1;
  f32x4 k0v = {0.f, 0.f, 0.f, 0.f}, k1v = k0v;
  if (qk_here) {
    // Kbar += (Nbar' - N (N . Nbar')) / ||k||, Nbar' = N (Mbar + Mbar^T), Mbar the
    // suffix sum of Xbar^T Q over the shard's later chunks (Mbar + Mbar^T formed
    // through a padded LDS copy of Mbar and rounded to the compute type, where the
    // MFMA would round it)
    const CT* N = rc + Y.r.fc.o[rec::N];
    const float* Mb = bqf + Y.r.bf.o[rec::XbQ];
    float* const fMt = fCb;  // Mbar, rows padded to d + 1 (dead before Nbar is written)
    const float* kn = rf + Y.r.ff.o[rec::kn];
    // the row elements of dk and N, requested ahead of the product
    float nv[8];
    if (qrow) {
      k0v = *reinterpret_cast<const f32x4*>(dkp + (size_t)qi * d + qc);
      k1v = *reinterpret_cast<const f32x4*>(dkp + (size_t)qi * d + qc + 4);
      load8(N + (size_t)qi * d + qc, nv);
    }
    for (int e = threadIdx.x * 4; e < d * d; e += blockDim.x * 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(Mb + e);
      const int i = e / d, j = e - i * d;
#pragma unroll
      for (int q = 0; q < 4; ++q) fMt[i * (d + 1) + j + q] = v[q];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < d * d; e += blockDim.x) {
      const int i = e / d, j = e - i * d;
      sMs[e] = from_f<CT>(fMt[i * (d + 1) + j] + fMt[j * (d + 1) + i]);
    }
    __syncthreads();
    using BCD = Blk<CP, D>;
    for_blocks<CP, D>([&](int i0, int j0) {
      f4 n1[BCD::RB][BCD::CB];
      zero_blk(n1);
      mma_blk<CT, KC, KC, BCD::RB, BCD::CB, D>(n1, N, d, i0, sMs, d, j0);
      blk_each4<BCD::RB, BCD::CB>(i0, j0, [&](int rb, int cb, int i, int j) {
#pragma unroll
        for (int r = 0; r < 4; ++r) fNb[(size_t)(i + r) * d + j] = n1[rb][cb][r];
      });
    });
    __syncthreads();
    {
      float f8[8], dt = 0.f;
      if (qrow) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          f8[q] = fNb[(size_t)qi * d + qc + q];
          dt += nv[q] * f8[q];
        }
      }
#pragma unroll
      for (int o = 1; o < CPR; o <<= 1) dt += __shfl_xor(dt, o, WAVE);  // the row's threads
      if (qrow) {
        const float nr = kn[qi];
        if (nr > 0.f) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            k0v[q] += (f8[q] - nv[q] * dt) / nr;
            k1v[q] += (f8[q + 4] - nv[q + 4] * dt) / nr;
          }
          if (!fuse) {
            *reinterpret_cast<f32x4*>(dkp + (size_t)qi * d + qc) = k0v;
            *reinterpret_cast<f32x4*>(dkp + (size_t)qi * d + qc + 4) = k1v;
          }
        }
      }
    }
    __syncthreads();  // LDS is reused below
  }
  if (fuse && qrow) {
    // the final dk of the row: every memory's part in a fixed order (the order of
    // the separate sum), this memory's from the registers
    if (!qk_here) {
      k0v = *reinterpret_cast<const f32x4*>(dkp + (size_t)qi * d + qc);
      k1v = *reinterpret_cast<const f32x4*>(dkp + (size_t)qi * d + qc + 4);
    }
    const size_t e = (cbase + tok0 + qi) * d + qc;
    f32x4 s0 = k0v, s1 = k1v;
    for (int p = 0; p < a.dk_nparts; ++p) {
      f32x4 y0 = k0v, y1 = k1v;
      if (p != a.dk_self) {
        y0 = *reinterpret_cast<const f32x4*>(a.dk_parts + p * a.dk_stride + e);
        y1 = *reinterpret_cast<const f32x4*>(a.dk_parts + p * a.dk_stride + e + 4);
      }
      if (p == 0) {
        s0 = y0;
        s1 = y1;
      } else {
        s0 += y0;
        s1 += y1;
      }
    }
    bf16x8 ov;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ov[q] = (__bf16)s0[q];
      ov[q + 4] = (__bf16)s1[q];
    }
    *reinterpret_cast<bf16x8*>(reinterpret_cast<__bf16*>(a.dk_out) + e) = ov;
  }

  chunk_coefs_g(cf, a.lr + cbase, mom, dec, tok0, C, Cp);  // ends with a barrier
  for (int e = threadIdx.x * 4; e < Cp * Cp; e += blockDim.x * 4)
    *reinterpret_cast<f32x4*>(fCb + e) = *reinterpret_cast<const f32x4*>(bqf + Y.r.bf.o[rec::Cb] + e);
  if (threadIdx.x < Cp) {
    const int i = threadIdx.x;
    gA[i] = bqf[Y.r.bf.o[rec::gA] + i];
    gE[i] = bqf[Y.r.bf.o[rec::gE] + i];
    gCC[i] = bqf[Y.r.bf.o[rec::gCC] + i];
    gB[i] = bqf[Y.r.bf.o[rec::gB] + i];
  }
  if (threadIdx.x < 3) dots[threadIdx.x] = bqf[Y.r.bf.o[rec::dots] + threadIdx.x];
  __syncthreads();
  if (wave_id() == 0) {
    const int i = l;
    if (i < Cp) fCb[(C - 1) * Cp + i] += gCC[i];
    if (i == 0) {
      gA[C - 1] += dots[0];
      gE[C - 1] += dots[1];
    }
  }
  __syncthreads();
  {
    const int w = wave_id(), i = l;
    const int r0 = w * (Cp / 8), r1 = r0 + Cp / 8;
    // column sums of cbar o ct, cbar o c over rows r in this block (r >= i),
    // row sums of cbar o c over columns t in this block (t <= i)
    float eb = 0.f, cols = 0.f, rows = 0.f;
    if (i < Cp) {
#pragma unroll 4
      for (int r = r0; r < r1; ++r) {
        if (r >= i) {
          const float cb = fCb[r * Cp + i];
          eb += cb * cf.ctt(r, i);
          cols += cb * cf.cc(r, i);
        }
        if (r <= i) rows += fCb[i * Cp + r] * cf.cc(i, r);
      }
      gpart[(0 * 8 + w) * Cp + i] = eb;
      gpart[(1 * 8 + w) * Cp + i] = cols;
      gpart[(2 * 8 + w) * Cp + i] = rows;
    }
    // U_{i, j} = beta'_j U_{i, j-1} + cbar_{i j} eta_j (j <= i), beta'_j = e^{lb_j - lb_{j-1}},
    // for this wave's rows i, as an affine scan over the lanes j; each lane keeps
    // the column sums over those rows
    //   T_j = sum_{i >= j} e^{la_i - la_j} U_{i j},  Y_j = sum_{i >= j} e^{la_i - la_j} Ebar_i
    const int j = l;
    const float aj = (j < Cp) ? expf(cf.lb[j] - (j > 0 ? cf.lb[j - 1] : 0.f)) : 0.f;
    const float laj = (j < Cp) ? cf.la[j] : 0.f;
    float T = 0.f, Yv = 0.f;
    for (int ri = r0; ri < r1; ++ri) {
      float sa = aj, sx = (j <= ri && j < Cp) ? fCb[ri * Cp + j] * cf.eta[j] : 0.f;
#pragma unroll
      for (int o = 1; o < WAVE; o <<= 1) {
        const float pa_ = __shfl_up(sa, o, WAVE), px = __shfl_up(sx, o, WAVE);
        if (j >= o) {
          sx = sa * px + sx;
          sa = sa * pa_;
        }
      }
      if (j < C && ri >= j) {
        const float e = expf(cf.la[ri] - laj);
        T += e * sx;
        Yv += e * gE[ri];
      }
    }
    if (j < Cp) {
      gpart[(3 * 8 + w) * Cp + j] = T;
      gpart[(4 * 8 + w) * Cp + j] = Yv;
    }
  }
  __syncthreads();
  if (wave_id() == 0) {
    const int j = l;
    float sum[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
    if (j < Cp)
#pragma unroll
      for (int k = 0; k < 5; ++k)
#pragma unroll
        for (int w = 0; w < 8; ++w) sum[k] += gpart[(k * 8 + w) * Cp + j];
    const float eb = sum[0] + (j < Cp ? gB[j] * cf.ebt[j] : 0.f);
    const float cols = sum[1], rows = sum[2], T = sum[3], Yv = sum[4];
    float la_b = 0.f, lb_b = 0.f;
    const float dBC = dots[2];
    const float bsum = wave_sum(j < Cp ? gB[j] * cf.bb[j] : 0.f);
    if (j < C) {
      const float yl = Yv * expf(cf.lb[j]);
      la_b = gA[j] * cf.A[j] + gE[j] * cf.E[j] + rows - T - yl;
      lb_b = T - cols + yl - gB[j] * cf.bb[j];
      if (j == C - 1) lb_b += dBC * cf.BC + bsum;
    }
    // suffix sums over positions
    const float pla = wave_incl_sum(la_b), plb = wave_incl_sum(lb_b);
    const float tla = __shfl(pla, WAVE - 1, WAVE), tlb = __shfl(plb, WAVE - 1, WAVE);
    const float sla = tla - pla + la_b, slb = tlb - plb + lb_b;
    if (j < C) {
      const size_t tt = cbase + tok0 + j;
      const float al = a.decay[tt], be = a.mom[tt];
      a.dlr[tt] = eb;
      a.ddecay[tt] = -sla / (1.0f - al);
      a.dmom[tt] = (logf(be) > LOG_CLAMP) ? slb / be : 0.f;
    }
  }
}

// ===========================================================================
// host side
// ===========================================================================
namespace {

template <typename CT, int CP, int D, int H>
constexpr bool split_fits() {
  // pass C's static LDS is under 40 KB
  return split_a_lds<CT, CP, D, H>() + SPLIT_A_STATIC <= 160 * 1024 &&
         split_b_lds<CT, CP, D, H>() + 2 * 1024 <= 160 * 1024 &&
         split_c_lds<CT, CP, D>() + 40 * 1024 <= 160 * 1024;
}

struct SplitSizes {
  size_t rec_ct, rec_f;  // elements
};

template <typename CT, int CP, int D, int H>
SplitSizes split_sizes(int units, int nch) {
  constexpr SplitLayout Y = make_split_layout(CP, D, H);
  const size_t t = (size_t)units * nch;
  return SplitSizes{t * Y.r.bc.n, t * Y.r.bf.n};
}

size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

template <typename CT>
size_t total_bytes(const SplitSizes& z) {
  return up256(z.rec_ct * sizeof(CT)) + up256(z.rec_f * 4);
}

template <typename CT>
SplitPtrs carve(void* ws, const SplitSizes& z, int units) {
  char* p = (char*)ws;
  SplitPtrs P{};
  P.brec = p; p += up256(z.rec_ct * sizeof(CT));
  P.brec_f = (float*)p;
  P.units = units;
  return P;
}

template <typename IO, typename CT, int ACT, int D, int H, int CP>
bool split_match(const Dims& Dm) {
  return Dm.d == D && Dm.hid == H && Dm.Cp == CP && Dm.act == ACT && split_fits<CT, CP, D, H>();
}

// size query (ws == nullptr) or launch
// the gate pass over every chunk of every unit
template <typename CT, int D, int H, int CP>
void launch_gate(const LocalBwdArgs& a, int units, int nch, hipStream_t st) {
  SplitPtrs P = carve<CT>(a.split_ws, split_sizes<CT, CP, D, H>(units, nch), units);
  P.n0 = 0;
  P.nc = nch;
  auto kc = local_bwd_gate_kernel<CT, D, H, CP>;
  constexpr size_t lds = split_c_lds<CT, CP, D>();
  hipLaunchKernelGGL(kc, dim3(units * nch), dim3(512), lds, st, a, P);
}

template <typename IO, typename CT, int ACT, int D, int H, int CP>
bool try_split(const LocalBwdArgs* a, const Dims& Dm, int units, void* ws, hipStream_t st,
               hipError_t* err, size_t* bytes) {
  if (!split_match<IO, CT, ACT, D, H, CP>(Dm)) return false;
  const int nch = Dm.S / Dm.C;
  const SplitSizes z = split_sizes<CT, CP, D, H>(units, nch);
  if (bytes) *bytes = total_bytes<CT>(z);
  if (!a) return true;
  SplitPtrs P = carve<CT>(ws, z, units);
  constexpr SplitLayout Y = make_split_layout(CP, D, H);
  const int total = units * nch;
  // When the walks leave half the CUs free and are long (32 chunks or more), the
  // chunks are cut in two: passes A and B take the upper chunks first, and the
  // lower chunks' pass A runs on the second stream beside the walk of the upper
  // ones (the walk reaches the lower chunks only after them).  Each part's pass A
  // writes only its own records and dq, dk rows.  The second stream runs the
  // global chain after it, so with short walks the split only delays that chain.
  // The lower part is five eighths of the chunks: the walk of the upper three
  // eighths covers that part's pass A on half the chip (one half measured 0.04 ms
  // slower at 32 chunks, three quarters 0.04 ms slower too).
  const bool halves = a->aux && a->aux_mid && a->aux_done && a->pass_a_done && nch >= 32 &&
                      2 * units <= device_cus();
  const int nlo = halves ? nch * 5 / 8 : 0;
  P.n0 = nlo;
  P.nc = nch - nlo;
  auto ka = local_bwd_ret_kernel<IO, CT, ACT, D, H, CP>;
  auto kb = local_bwd_chain_kernel<IO, CT, ACT, D, H, CP>;
  auto kc = local_bwd_gate_kernel<CT, D, H, CP>;
  constexpr size_t lds_a = split_a_lds<CT, CP, D, H>(), lds_b = split_b_lds<CT, CP, D, H>(),
                   lds_c = split_c_lds<CT, CP, D>();
  if (!lds_fits((const void*)ka, lds_a) || !lds_fits((const void*)kb, lds_b) ||
      !lds_fits((const void*)kc, lds_c)) {  // the compiled static LDS, not the estimate
    *err = hipErrorInvalidConfiguration;
    return true;
  }
  set_lds_limit((const void*)ka);
  set_lds_limit((const void*)kb);
  set_lds_limit((const void*)kc);
  hipLaunchKernelGGL(ka, dim3(units * P.nc), dim3(512), lds_a, st, *a, P);
  auto fail = [&](hipError_t e) {
    *err = e;
    return true;
  };
  hipError_t e;
  if (a->pass_a_done && (e = hipEventRecord(a->pass_a_done, st)) != hipSuccess) return fail(e);
  SplitPtrs Plo = P;
  Plo.n0 = 0;
  Plo.nc = nlo;
  if (halves) {
    if ((e = hipStreamWaitEvent(a->aux, a->pass_a_done, 0)) != hipSuccess) return fail(e);
    hipLaunchKernelGGL(ka, dim3(units * nlo), dim3(512), lds_a, a->aux, *a, Plo);
    if ((e = hipEventRecord(a->aux_mid, a->aux)) != hipSuccess) return fail(e);
  }
  // the suffix sums of pass A's Xbar^T Q over later chunks (read by the gate
  // pass): on the second stream beside the walk when there is one
  const bool scan = Dm.qk_proj && Dm.qk_scope == 0;
  const bool on_aux = scan && a->aux && a->aux_done && a->pass_a_done;
  auto launch_scan = [&](hipStream_t s) {
    const size_t thr = (size_t)units * D * D;
    hipLaunchKernelGGL(split_madj_scan_kernel, dim3((unsigned)((thr + 255) / 256)), dim3(256), 0, s,
                       P.brec_f, Y.r.bf.n, Y.r.bf.o[rec::XbQ], units, nch, D * D);
  };
  if (on_aux) {
    if (!halves && (e = hipStreamWaitEvent(a->aux, a->pass_a_done, 0)) != hipSuccess) return fail(e);
    launch_scan(a->aux);
    if ((e = hipEventRecord(a->aux_done, a->aux)) != hipSuccess) return fail(e);
  }
  const int sec = section_begin("local_bwd_walk", st);  // the walk of the carried adjoint alone
  hipLaunchKernelGGL(kb, dim3(units), dim3(512), lds_b, st, *a, P);
  if (halves) {
    if ((e = hipStreamWaitEvent(st, a->aux_mid, 0)) != hipSuccess) return fail(e);
    hipLaunchKernelGGL(kb, dim3(units), dim3(512), lds_b, st, *a, Plo);
  }
  section_end(sec, st);
  if (a->pass_b_done && (e = hipEventRecord(a->pass_b_done, st)) != hipSuccess) return fail(e);
  if (a->defer_gate && a->gate_deferred && halves && (on_aux || !scan)) {
    // the caller launches the gate pass later (launch_local_bwd_gate)
    *a->gate_deferred = 1;
    *err = hipGetLastError();
    return true;
  }
  if (on_aux) {
    if ((e = hipStreamWaitEvent(st, a->aux_done, 0)) != hipSuccess) return fail(e);
  } else if (scan) {
    launch_scan(st);
  }
  launch_gate<CT, D, H, CP>(*a, units, nch, st);
  *err = hipGetLastError();
  return true;
}

template <typename IO, typename CT, int ACT, int D, int H, int CP>
bool try_gate(const LocalBwdArgs& a, const Dims& Dm, int units, hipStream_t st, hipError_t* err) {
  if (!split_match<IO, CT, ACT, D, H, CP>(Dm)) return false;
  // the suffix scan ran on the second stream (a deferral needs it there)
  if (Dm.qk_proj && Dm.qk_scope == 0 && (*err = hipStreamWaitEvent(st, a.aux_done, 0)) != hipSuccess)
    return true;
  launch_gate<CT, D, H, CP>(a, units, Dm.S / Dm.C, st);
  *err = hipGetLastError();
  return true;
}

// The shapes of the fixed-size bf16 forward (whose split passes write the forward
// records these passes read); other shapes take the one-walk kernels.
bool dispatch_split(const LocalBwdArgs* a, const Dims& Dm, int units, void* ws, hipStream_t st,
                    hipError_t* err, size_t* bytes) {
  if (!Dm.bf16) return false;
  return try_split<__bf16, __bf16, ACT_SILU, 64, 256, 64>(a, Dm, units, ws, st, err, bytes) ||
         try_split<__bf16, __bf16, ACT_SILU, 64, 256, 32>(a, Dm, units, ws, st, err, bytes) ||
         try_split<__bf16, __bf16, ACT_SILU, 64, 256, 16>(a, Dm, units, ws, st, err, bytes) ||
         try_split<__bf16, __bf16, ACT_GELU, 64, 256, 64>(a, Dm, units, ws, st, err, bytes);
}

bool dispatch_gate(const LocalBwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  const Dims& Dm = a.D;
  if (!Dm.bf16) return false;
  return try_gate<__bf16, __bf16, ACT_SILU, 64, 256, 64>(a, Dm, units, st, err) ||
         try_gate<__bf16, __bf16, ACT_SILU, 64, 256, 32>(a, Dm, units, st, err) ||
         try_gate<__bf16, __bf16, ACT_SILU, 64, 256, 16>(a, Dm, units, st, err) ||
         try_gate<__bf16, __bf16, ACT_GELU, 64, 256, 64>(a, Dm, units, st, err);
}

}  // namespace

hipError_t launch_local_bwd_gate(const LocalBwdArgs& a, int units, hipStream_t st) {
  hipError_t e = hipSuccess;
  return dispatch_gate(a, units, st, &e) ? e : hipErrorInvalidValue;
}

size_t local_bwd_split_bytes(const Dims& D, int units) {
  size_t bytes = 0;
  hipError_t e = hipSuccess;
  return dispatch_split(nullptr, D, units, nullptr, nullptr, &e, &bytes) ? bytes : 0;
}

bool launch_local_bwd_split(const LocalBwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (!a.split_ws || !a.frec || !a.frec_f) return false;  // needs the forward's records
  return dispatch_split(&a, a.D, units, a.split_ws, st, err, nullptr);
}

}  // namespace tnt
