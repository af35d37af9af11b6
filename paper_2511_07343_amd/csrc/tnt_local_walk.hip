// Forward walk of a local memory with the fp32 state held in registers.
//
// One workgroup (8 waves) walks the chunks of one unit (batch row, head,
// shard).  The state (W1, S1, W2, S2, and the shard-scoped Q-K sum M) never
// leaves the workgroup's registers: wave w owns hidden columns [32w, 32w+32)
// of every state matrix, held as 16 x 16 MFMA accumulator tiles
//
//     W1^T, S1^T : d x hid   (tile rows d, columns hid)
//     W2,   S2   : d x hid
//
// and the chunk step is organised around that ownership (Sec. 2.2 chunk rule,
// gates of App. D):
//
//   Zk = K W1^T     the wave's hidden columns, B operand straight from its
//                   W1^T tiles  -> Hk = s(Zk) (registers and LDS), s'(Zk)
//   Yk = Hk W2^T    contraction over all hidden columns: from LDS (Hk and a
//                   bf16 copy of W2 that the previous carry left there)
//   R  = (2/d)(Yk - V)
//   G  = R W2       the wave's hidden columns, B operand from its W2 tiles
//   D1 = G * s'(Zk)
//   carry           W1^T' = A_C W1^T + E_C S1^T - (cC K)^T D1,
//                   S1^T' = B_C S1^T - (b K)^T D1,
//                   W2'   = A_C W2 + E_C S2 - (cC R)^T Hk,
//                   S2'   = B_C S2 - (b R)^T Hk,
//                   the B operands D1 and Hk straight from the wave's own
//                   tiles, the A operands from LDS.
//
// An accumulator tile used as a B operand: lane l holds rows 4(l/16)+r of
// column l%16, so two tiles stacked along the contraction give lane l the
// contraction indices {4(l/16)+r} and {16+4(l/16)+r}.  The MFMA sums over its
// 32 operand slots in any order, so the A operand only has to present the
// same contraction index in the same slot: two 8-byte LDS reads at k0+4(l/16)
// and k0+16+4(l/16) instead of one 16-byte read.
//
// Per chunk the walk writes what the chunk-parallel retrieval and the
// backward read: the compute-type transposes of the next state slot, the Q-K
// sum (fp32 and transposed), D1^T and R of the chunk for the retrieval, and
// the forward record's Hk, Hk^T, D1, s'(Zk), s''(Zk) and G (without a record,
// Hk goes to the retrieval's buffer).  Nothing is read back from memory.
#include "tnt_local_common.h"
#include "tnt_local_record.h"
#include "tnt_regtile.h"

namespace tnt {

namespace {

constexpr int WMAXC = 64;
struct WalkCoef {
  float cC[WMAXC], bb[WMAXC], knorm[WMAXC];  // knorm: reciprocal key norms, 0 for padding
  float AC, BC, EC;
};

// LDS carve-up (bf16 elements).  Row strides are padded so that the sixteen
// rows one MFMA operand read touches fall in distinct banks: +4 elements
// (8 bytes) for the arrays read 8 bytes per lane (a_pair), +8 (16 bytes) for
// those read 16 bytes per lane.
template <int D, int HID, int CP>
struct WalkLds {
  static constexpr int LK = D + 4;            // sK, sR rows
  static constexpr int LT = CP + 4;           // the scaled transposes' rows
  static constexpr int LN = CP + 8;           // sNT rows
  static constexpr int LH = HID + 8;          // sHk, sW2 rows
  static constexpr int K = 0;                 // [CP][LK]   keys
  static constexpr int KcT = K + CP * LK;     // [D][LT]    -(cC K)^T
  static constexpr int KbT = KcT + D * LT;    // [D][LT]    -(b K)^T
  static constexpr int NT = KbT + D * LT;     // [D][LN]    (K / |K|)^T
  static constexpr int Hk = NT + D * LN;      // [CP][LH]   s(Zk)
  static constexpr int W2 = Hk + CP * LH;     // [D][LH]    chunk-entry W2
  static constexpr int R = W2 + D * LH;       // [CP][LK]
  static constexpr int RcT = R + CP * LK;     // [D][LT]    -(cC R)^T
  static constexpr int RbT = RcT + D * LT;    // [D][LT]    -(b R)^T
  static constexpr int Sp = RbT + D * LT;     // s'(Zk), each wave's tiles, lane-major
  static constexpr int total = Sp + CP * HID;
};

}  // namespace

template <int D, int HID, int CP>
constexpr size_t walk_lds_bytes() {
  return (size_t)WalkLds<D, HID, CP>::total * sizeof(__bf16);
}

template <typename IO, int ACT, int D, int HID, int CP>
__global__ void __launch_bounds__(512) local_walk_kernel(LocalFwdArgs a) {
  using CT = __bf16;
  using Ly = WalkLds<D, HID, CP>;
  constexpr int NW = 8;
  constexpr int HT = HID / (16 * NW);  // hidden tiles per wave
  constexpr int DT = D / 16;           // d tiles
  constexpr int TM = CP / 16;          // token tiles
  static_assert(HID % (16 * NW) == 0 && D % 32 == 0 && DT * DT == 2 * NW, "tile ownership");
  static_assert(CP <= WMAXC && (TM == 1 || TM % 2 == 0), "token tiles in pairs");
  constexpr int LK = Ly::LK, LT = Ly::LT, LN = Ly::LN, LH = Ly::LH;
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ WalkCoef cfs[2];
  CT* L = (CT*)smem;
  CT *sK = L + Ly::K, *sKcT = L + Ly::KcT, *sKbT = L + Ly::KbT, *sNT = L + Ly::NT,
     *sHk = L + Ly::Hk, *sW2 = L + Ly::W2, *sR = L + Ly::R, *sRcT = L + Ly::RcT,
     *sRbT = L + Ly::RbT, *sSp = L + Ly::Sp;

  const Dims Dm = a.D;
  const int C = Dm.C;
  const int nshard = Dm.L / Dm.S;
  const int nch = Dm.S / C;
  const int u = blockIdx.x;
  const int b = u / (Dm.H * nshard), hh = (u / nshard) % Dm.H, s = u % nshard;
  constexpr size_t hd = (size_t)HID * D;
  const size_t chain = (size_t)b * Dm.H + hh;
  const IO* k = (const IO*)a.k + chain * Dm.L * D;
  const IO* v = (const IO*)a.v + chain * Dm.L * D;
  const float* lr = a.lr + chain * Dm.L;
  const float* mom = a.mom + chain * Dm.L;
  const float* dec = a.decay + chain * Dm.L;
  constexpr size_t PS = 4 * hd + (size_t)D * D;  // CT elements per transposed slot
  CT* const pku = (CT*)a.statesT + (size_t)u * a.nslots * PS;
  float* const mst = a.mstates + (size_t)u * a.nslots * D * D;
  const bool shard_qk = Dm.qk_proj && Dm.qk_scope == 0;
  const float rscale = 2.0f / (float)D;
  const int l = lane_id(), w = wave_id_uniform(), g = l >> 4, lc = l & 15;
  constexpr size_t FS = 2 * (size_t)CP * HID + (size_t)CP * D;  // Hk, D1^T, R per chunk
  constexpr rec::RecLayout RL = rec::make_rec_layout(CP, D, HID);

  // ---- the state, at the shard start: (W1, W2) = init, S = 0, M = 0
  f4 W1T[DT][HT], S1T[DT][HT], W2[DT][HT], S2[DT][HT], M[2];
  {
    const float* W1i = a.W1i + hh * hd;  // [HID][D]
    const float* W2i = a.W2i + hh * hd;  // [D][HID]
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int ht = 0; ht < HT; ++ht) {
        const int h = (w * HT + ht) * 16 + lc, d0 = dt * 16 + 4 * g;
        const f32x4 x = *reinterpret_cast<const f32x4*>(W1i + (size_t)h * D + d0);
        W1T[dt][ht] = f4{x[0], x[1], x[2], x[3]};
#pragma unroll
        for (int r = 0; r < 4; ++r) W2[dt][ht][r] = W2i[(size_t)(d0 + r) * HID + h];
        S1T[dt][ht] = zero4();
        S2[dt][ht] = zero4();
      }
    M[0] = M[1] = zero4();
  }

  // compute-type transposes of the state into a slot, the fp32 Q-K sum, and
  // the LDS copy of W2 that the next chunk's Yk reads
  auto write_slot = [&](CT* pk, float* ms) {
    pk = launder_global(pk);
    ms = launder_global(ms);
    const int ll = lane_id_local(), lc = ll & 15, g = ll >> 4;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int ht = 0; ht < HT; ++ht) {
        const int h = (w * HT + ht) * 16 + lc, d0 = dt * 16 + 4 * g;
        // W1^T, S1^T [D][HID]: the lane holds four rows of one column.  For chunks of
        // up to 32 rows (many chunks per shard) a transpose within the lane's quad
        // gives it four columns of one row, one 8-byte store instead of four 2-byte
        // ones (fewer stores in flight when the next chunk waits for its keys); at 64
        // rows the four stores measured faster.
        if constexpr (CP < 64) {
          const int q = lc & 3;
          store4<CT>(pk + (size_t)(d0 + q) * HID + (h - q), quad_transpose(W1T[dt][ht]));
          store4<CT>(pk + 2 * hd + (size_t)(d0 + q) * HID + (h - q), quad_transpose(S1T[dt][ht]));
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            pk[(size_t)(d0 + r) * HID + h] = (CT)W1T[dt][ht][r];
            pk[2 * hd + (size_t)(d0 + r) * HID + h] = (CT)S1T[dt][ht][r];
          }
        }
        if constexpr (CP < 64) {
          const int q = lc & 3;
          *reinterpret_cast<bf16x4*>(sW2 + (size_t)(d0 + q) * LH + h - q) = cvt4(quad_transpose(W2[dt][ht]));
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) sW2[(size_t)(d0 + r) * LH + h] = (CT)W2[dt][ht][r];
        }
        store4<CT>(pk + hd + (size_t)h * D + d0, W2[dt][ht]);      // W2^T [HID][D]
        store4<CT>(pk + 3 * hd + (size_t)h * D + d0, S2[dt][ht]);  // S2^T [HID][D]
      }
    if (shard_qk)
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int t = 2 * w + x, i0 = (t / DT) * 16, j0 = (t % DT) * 16;
        store4<CT>(pk + 4 * hd + (size_t)(j0 + lc) * D + i0 + 4 * g, M[x]);  // M^T
        if constexpr (CP < 64) {  // by rows after the quad transpose, as the copies above
          const int q = lc & 3;
          store4<float>(ms + (size_t)(i0 + 4 * g + q) * D + j0 + lc - q, quad_transpose(M[x]));
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) ms[(size_t)(i0 + 4 * g + r) * D + j0 + lc] = M[x][r];
        }
      }
  };
  write_slot(pku, mst);

  // Loads of a chunk's inputs are issued ahead of the phase that uses them:
  // the keys and gates of chunk n + 1 during chunk n's carry (their round trip
  // overlaps the carry and the slot stores), the values of chunk n before its
  // coefficient scan (written to LDS after that scan's barrier).
  constexpr int VEC = 8;  // bf16 per 16-byte load
  static_assert(sizeof(IO) == 2, "the walk reads bf16 inputs");
  static_assert((CP * D / VEC) % WAVE == 0 && CP * D / VEC <= 512, "one 16-byte load per thread");
  const int e_in = threadIdx.x * VEC;  // this thread's element of a [CP][D] chunk array
  const bool ld_in = e_in < CP * D;
  auto load_rows = [&](const IO* base, int tok0) {
    bf16x8 x;
    const int i = e_in / D;
    if (ld_in && i < C) {
      x = *reinterpret_cast<const bf16x8*>(launder_global(base + (size_t)tok0 * D) + e_in);
    } else {
#pragma unroll
      for (int j = 0; j < VEC; ++j) x[j] = (__bf16)0.f;
    }
    return x;
  };
  float g_lr = 0.f, g_mom = 1.f, g_dec = 0.f;  // wave 0: lane i's gates of the next chunk
  auto load_gates = [&](int tok0) {
    if (w == 0 && lane_id() < C) {
      g_lr = lr[tok0 + lane_id()];
      g_mom = mom[tok0 + lane_id()];
      g_dec = dec[tok0 + lane_id()];
    }
  };
  bf16x8 k_next = load_rows(k, s * Dm.S);
  load_gates(s * Dm.S);
  // the carry's coefficients of a chunk from its gates (wave 0; the same suffix
  // scan as carry_coefs).  For chunks of up to 32 rows they are formed at the end
  // of the chunk before (gates loaded a chunk ahead), where they overlap the slot
  // stores instead of holding the chunk's first barrier; at 64 rows, where that
  // measured slower, at the chunk's start from the gates loaded during the carry
  // before.
  constexpr bool EARLY = CP < 64;
  auto scan_coefs = [&](WalkCoef& cf) {
    if (w == 0) {
      const int i = lane_id();
      const bool in = i < C;
      const float eta = in ? g_lr : 0.f;
      const float lmb = in ? log_mom(g_mom) : 0.f;
      const float lka = in ? log_keep(g_dec) : 0.f;
      const float la = wave_incl_sum(lka), lb = wave_incl_sum(lmb);
      const float laC = __shfl(la, C - 1, WAVE), lbC = __shfl(lb, C - 1, WAVE);
      const float lbn = __shfl_down(lb, 1, WAVE);
      float ya = in ? __expf(laC - la) : 0.f;
      float yb = (i + 1 < C) ? __expf(lbn - lb) : 0.f;
  #pragma unroll
      for (int o = 1; o < WAVE; o <<= 1) {
        const float pa = __shfl_down(ya, o, WAVE), pb = __shfl_down(yb, o, WAVE);
        if (i + o < WAVE) {
          ya = ya + yb * pa;
          yb = yb * pb;
        }
      }
      const float ec = wave_sum(in ? __expf(laC - la + lb) : 0.f);
      if (i < CP) {
        cf.cC[i] = in ? eta * ya : 0.f;
        cf.bb[i] = in ? eta * __expf(lbC - lb) : 0.f;
      }
      if (i == 0) {
        cf.AC = __expf(laC);
        cf.BC = __expf(lbC);
        cf.EC = ec;
      }
    }
  };
  if constexpr (EARLY) {
    scan_coefs(cfs[0]);
    if (nch > 1) load_gates(s * Dm.S + C);  // one chunk ahead of their scan
  }

  for (int n = 0; n < nch; ++n) {
    WalkCoef& cf = cfs[n & 1];
    const int tok0 = s * Dm.S + n * C;
    // per-chunk bases re-derived through opaque moves (and lane indices below
    // through lane_id_local), so that no per-lane address is kept live across
    // the chunk loop beside the register-resident state
    CT* const fsn = launder_global((CT*)a.fsplit + ((size_t)u * nch + n) * FS);
    CT* const fr = a.frec ? launder_global((CT*)a.frec + ((size_t)u * nch + n) * RL.fc.n) : nullptr;

    const bf16x8 v_cur = load_rows(v, tok0);
    // ---- keys (prefetched; rows >= C zero) and their reciprocal norms
    {
      constexpr int LPR = D / VEC;  // lanes per row
      if (ld_in) {
        const int i = e_in / D, jc = e_in - i * D;
        float ss = 0.f;
#pragma unroll
        for (int j = 0; j < VEC; ++j) ss += (float)k_next[j] * (float)k_next[j];
        *reinterpret_cast<bf16x8*>(sK + (size_t)i * LK + jc) = k_next;
#pragma unroll
        for (int o = 1; o < LPR; o <<= 1) ss += __shfl_xor(ss, o, WAVE);
        if ((threadIdx.x & (LPR - 1)) == 0) cf.knorm[i] = ss > 0.f ? __builtin_amdgcn_rsqf(ss) : 0.f;
      }
    }
    if constexpr (!EARLY) scan_coefs(cf);
    __syncthreads();
    // the chunk's values into sR (each Yk tile's owner reads them there and
    // overwrites them with R)
    if (ld_in) {
      const int i = e_in / D, jc = e_in - i * D;
      *reinterpret_cast<bf16x8*>(sR + (size_t)i * LK + jc) = v_cur;
    }

    // ---- -(cC K)^T, -(b K)^T and the normalised keys' transpose
    for (int e = threadIdx.x; e < D * CP; e += blockDim.x) {
      const int j = e / CP, i = e - j * CP;  // destination row j (of D), column i (of CP)
      const float kx = to_f(sK[(size_t)i * LK + j]);
      sKcT[(size_t)j * LT + i] = (CT)(-cf.cC[i] * kx);
      sKbT[(size_t)j * LT + i] = (CT)(-cf.bb[i] * kx);
      if (shard_qk) sNT[(size_t)j * LN + i] = (CT)(kx * cf.knorm[i]);
    }

    // ---- Zk = K W1^T on the wave's hidden tiles -> Hk (registers, LDS), s'(Zk)
    // (LDS, the wave's own slots: lane l's four values of tile (it, ht) at
    // 4 (64 ((w TM + it) HT + ht) + l))
    bf16x4 hk[TM][HT];
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      const int l = lane_id_local(), g = l >> 4, lc = l & 15;
      bf16x8 bw[DT / 2];
#pragma unroll
      for (int c = 0; c < DT / 2; ++c) bw[c] = join(cvt4(W1T[2 * c][ht]), cvt4(W1T[2 * c + 1][ht]));
      const int j0 = (w * HT + ht) * 16;
#pragma unroll
      for (int it = 0; it < TM; ++it) {
        f4 acc = zero4();
#pragma unroll
        for (int c = 0; c < DT / 2; ++c) mma32(acc, a_pair(sK, LK, it * 16 + lc, 32 * c, g), bw[c]);
        f4 hv, d1v, d2v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const ActVals av = act_all<ACT>(acc[r]);
          hv[r] = av.s;
          d1v[r] = av.d1;
          d2v[r] = av.d2;
          if constexpr (CP >= 64) sHk[(size_t)(it * 16 + 4 * g + r) * LH + j0 + lc] = (CT)av.s;
        }
        if constexpr (CP < 64) {  // one 8-byte LDS write by rows after the quad transpose
          const int q = lc & 3;
          *reinterpret_cast<bf16x4*>(sHk + (size_t)(it * 16 + 4 * g + q) * LH + j0 + lc - q) =
              cvt4(quad_transpose(hv));
        }
        hk[it][ht] = cvt4(hv);
        *reinterpret_cast<bf16x4*>(sSp + 4 * (64 * ((w * TM + it) * HT + ht) + l)) = cvt4(d1v);
        if (fr) {
          const size_t fo = frag_ofs<CP, HID>(it * 16, j0, l);
          store4<CT>(fr + RL.fc.o[rec::Sp] + fo, d1v);
          store4<CT>(fr + RL.fc.o[rec::Spp] + fo, d2v);
          // Hk^T [HID][CP]: the lane's four rows are contiguous
          store4<CT>(fr + RL.fc.o[rec::HkT] + (size_t)(j0 + lc) * CP + it * 16 + 4 * g, hv);
        }
      }
    }
    __syncthreads();  // Hk, the key transposes complete

    // ---- the Q-K sum: M' = M + N^T N (the wave's two tiles of M)
    if (shard_qk)
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int t = 2 * w + x, i0 = (t / DT) * 16, j0 = (t % DT) * 16;
        mma_tile<CT, KC, KC>(M[x], sNT, LN, i0, sNT, LN, j0, CP);
      }

    // ---- Yk = Hk W2^T -> R = (2/d)(Yk - V), its scaled transposes
    {
      constexpr int nt = TM * DT;
      const int l = lane_id_local(), g = l >> 4, lc = l & 15;
      for (int t = w; t < nt; t += NW) {
        const int i0 = (t / DT) * 16, j0 = (t % DT) * 16;
        float vv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) vv[r] = (float)sR[(size_t)(i0 + 4 * g + r) * LK + j0 + lc];
        f4 acc = zero4();
        {
          // K = HID in a rolled loop: two steps' operands live at a time
          const CT* pa = sHk + (size_t)(i0 + lc) * LH + 8 * g;
          const CT* pb = sW2 + (size_t)(j0 + lc) * LH + 8 * g;
#pragma unroll 2
          for (int k0 = 0; k0 < HID; k0 += 32)
            mma32(acc, *reinterpret_cast<const bf16x8*>(pa + k0),
                  *reinterpret_cast<const bf16x8*>(pb + k0));
        }
        f4 rc, rb;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + 4 * g + r;
          const CT rv = (CT)(i < C ? rscale * (acc[r] - vv[r]) : 0.f);
          sR[(size_t)i * LK + j0 + lc] = rv;
          rc[r] = -cf.cC[i] * (float)rv;
          rb[r] = -cf.bb[i] * (float)rv;
        }
        *reinterpret_cast<bf16x4*>(sRcT + (size_t)(j0 + lc) * LT + i0 + 4 * g) = cvt4(rc);
        *reinterpret_cast<bf16x4*>(sRbT + (size_t)(j0 + lc) * LT + i0 + 4 * g) = cvt4(rb);
      }
    }
    __syncthreads();  // R and its transposes complete

    // ---- G = R W2 on the wave's hidden tiles, D1 = G s'(Zk)
    bf16x4 d1[TM][HT];
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      const int l = lane_id_local(), g = l >> 4, lc = l & 15;
      bf16x8 bw[DT / 2];
#pragma unroll
      for (int c = 0; c < DT / 2; ++c) bw[c] = join(cvt4(W2[2 * c][ht]), cvt4(W2[2 * c + 1][ht]));
      const int j0 = (w * HT + ht) * 16;
#pragma unroll
      for (int it = 0; it < TM; ++it) {
        f4 acc = zero4();
#pragma unroll
        for (int c = 0; c < DT / 2; ++c) mma32(acc, a_pair(sR, LK, it * 16 + lc, 32 * c, g), bw[c]);
        const bf16x4 sp = *reinterpret_cast<const bf16x4*>(sSp + 4 * (64 * ((w * TM + it) * HT + ht) + l));
        f4 dv;
#pragma unroll
        for (int r = 0; r < 4; ++r) dv[r] = acc[r] * (float)sp[r];
        d1[it][ht] = cvt4(dv);
        if (fr) {
          store4<CT>(fr + RL.fc.o[rec::G] + frag_ofs<CP, HID>(it * 16, j0, l), acc);
          if constexpr (CP < 64) {  // [CP][HID]: one row of four columns after the quad transpose
            const int q = lc & 3;
            store4<CT>(fr + RL.fc.o[rec::D1] + (size_t)(it * 16 + 4 * g + q) * HID + j0 + lc - q,
                       quad_transpose(dv));
          } else {
            CT* const d1r = fr + RL.fc.o[rec::D1] + (size_t)(it * 16 + 4 * g) * HID + j0 + lc;
#pragma unroll
            for (int r = 0; r < 4; ++r) d1r[(size_t)r * HID] = (CT)dv[r];
          }
        }
        // D1^T [HID][CP] for the retrieval: the lane's four rows are contiguous
        store4<CT>(fsn + (size_t)CP * HID + (size_t)(j0 + lc) * CP + it * 16 + 4 * g, dv);
      }
    }
    // Hk [CP][HID] (into the forward record when there is one, else the
    // retrieval's buffer) and R [CP][D] for the retrieval (LDS -> 16-byte stores)
    CT* const hkd = fr ? fr + RL.fc.o[rec::Hk] : fsn;
    for (int e = threadIdx.x * 8; e < CP * HID; e += blockDim.x * 8) {
      const int i = e / HID, j = e - i * HID;
      *reinterpret_cast<bf16x8*>(hkd + e) = *reinterpret_cast<const bf16x8*>(sHk + (size_t)i * LH + j);
    }
    for (int e = threadIdx.x * 8; e < CP * D; e += blockDim.x * 8) {
      const int i = e / D, j = e - i * D;
      *reinterpret_cast<bf16x8*>(fsn + 2 * (size_t)CP * HID + e) =
          *reinterpret_cast<const bf16x8*>(sR + (size_t)i * LK + j);
    }

    // ---- the next chunk's keys and gates (in flight during the carry)
    if (n + 1 < nch) {
      k_next = load_rows(k, tok0 + C);
      if constexpr (!EARLY) load_gates(tok0 + C);
    }
    // ---- the carry into the next state
    const float AC = cf.AC, BC = cf.BC, EC = cf.EC;
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      const int l = lane_id_local(), g = l >> 4, lc = l & 15;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int row = dt * 16 + lc;
        f4 w1 = AC * W1T[dt][ht] + EC * S1T[dt][ht];
        f4 s1 = BC * S1T[dt][ht];
        f4 w2 = AC * W2[dt][ht] + EC * S2[dt][ht];
        f4 s2 = BC * S2[dt][ht];
        if constexpr (TM == 1) {
          const bf16x4 z = zero_bf4();
          const bf16x8 bd = join(d1[0][ht], z), bh = join(hk[0][ht], z);
          mma32(w1, a_pair(sKcT, LT, row, 0, g, false), bd);
          mma32(s1, a_pair(sKbT, LT, row, 0, g, false), bd);
          mma32(w2, a_pair(sRcT, LT, row, 0, g, false), bh);
          mma32(s2, a_pair(sRbT, LT, row, 0, g, false), bh);
        } else {
#pragma unroll
          for (int c = 0; c < TM / 2; ++c) {
            const bf16x8 bd = join(d1[2 * c][ht], d1[2 * c + 1][ht]);
            const bf16x8 bh = join(hk[2 * c][ht], hk[2 * c + 1][ht]);
            mma32(w1, a_pair(sKcT, LT, row, 32 * c, g), bd);
            mma32(s1, a_pair(sKbT, LT, row, 32 * c, g), bd);
            mma32(w2, a_pair(sRcT, LT, row, 32 * c, g), bh);
            mma32(s2, a_pair(sRbT, LT, row, 32 * c, g), bh);
          }
        }
        W1T[dt][ht] = w1;
        S1T[dt][ht] = s1;
        W2[dt][ht] = w2;
        S2[dt][ht] = s2;
      }
    }
    write_slot(pku + (size_t)(n + 1) * PS, mst + (size_t)(n + 1) * D * D);
    if (EARLY && n + 1 < nch) {  // the next chunk's coefficients (its buffer was chunk n - 1's)
      scan_coefs(cfs[(n + 1) & 1]);
      if (n + 2 < nch) load_gates(tok0 + 2 * C);
    }
  }
}

// Launches the walk for the fixed-size shapes it is built for; false when
// `a` is not one of them.
template <typename IO, int ACT, int D, int HID, int CP>
static bool try_walk(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  if (a.D.d != D || a.D.hid != HID || a.D.Cp != CP || a.D.act != ACT) return false;
  constexpr size_t lds = walk_lds_bytes<D, HID, CP>();
  static_assert(lds + 2 * sizeof(WalkCoef) <= 160 * 1024, "LDS of one CU");
  auto kern = local_walk_kernel<IO, ACT, D, HID, CP>;
  if (!lds_fits((const void*)kern, lds)) {  // the compiled static LDS, not the estimate
    *err = hipErrorInvalidConfiguration;
    return true;
  }
  set_lds_limit((const void*)kern);
  hipLaunchKernelGGL(kern, dim3(units), dim3(512), lds, st, a);
  *err = hipGetLastError();
  return true;
}

bool launch_local_walk(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err) {
  // the walk writes the compute-type state copies only: families whose backward
  // reads the fp32 slots (fslots == 0) take the other walk
  if (!a.D.bf16 || !a.statesT || !a.fsplit || a.fslots == 0 || a.nslots <= a.D.S / a.D.C)
    return false;
  return try_walk<__bf16, ACT_SILU, 64, 256, 64>(a, units, st, err) ||
         try_walk<__bf16, ACT_SILU, 64, 256, 32>(a, units, st, err) ||
         try_walk<__bf16, ACT_SILU, 64, 256, 16>(a, units, st, err) ||
         try_walk<__bf16, ACT_GELU, 64, 256, 64>(a, units, st, err) ||
         try_walk<__bf16, ACT_GELU, 64, 256, 16>(a, units, st, err);
}

}  // namespace tnt
