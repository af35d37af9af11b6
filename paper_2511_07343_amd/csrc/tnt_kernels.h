// Kernel argument blocks and host-side launchers shared by the C ABI and the
// kernel translation units.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tnt {

// Header at the start of a saved buffer (tnt_mem_fwd -> tnt_mem_bwd): which
// layout, kernel family, ring sizes and configuration wrote it.
constexpr uint32_t SAVED_MAGIC = 0x544e5453u;  // "STNT"
constexpr uint32_t SAVED_LAYOUT_VERSION = 4;
constexpr size_t SAVED_HEADER_BYTES = 256;
struct SavedHeader {
  uint32_t magic, layout_version, family, pad;
  uint32_t fslots[4];
  uint64_t cfg_hash, bytes;
};
static_assert(sizeof(SavedHeader) <= SAVED_HEADER_BYTES, "header fits its reserved bytes");
hipError_t launch_write_header(void* dst, const SavedHeader& h, hipStream_t st);

// Sizes of one memory's pass, shared by every kernel.
struct Dims {
  int B, H, L, d, hid;
  int C;      // chunk size of this memory
  int Cp;     // C rounded up to a multiple of 16 (local memories)
  int S;      // shard length (local) or L (global)
  int act;    // ACT_GELU / ACT_SILU
  int bf16;   // 1: q/k/v/o are bf16 and MFMA operands are bf16
  int qk_proj, qk_scope;
  int gsub;   // > 1: gradients of every gsub consecutive chunks are taken at the state
              // entering the first of them (the global memory's intra-chunk reading
              // walked in sub-chunks, runtime-sized kernels only); 0 or 1 otherwise
};

// Per-unit scratch of the local memory kernels (element offsets into a CT
// array); filled by local_scratch_plan.
struct LocalPlan {
  size_t elems;  // CT elements per unit
  size_t Q, K, N, NT, X, KcT, KbT, R, RT, RcT, RbT, S, P;           // forward, small
  size_t Hk, HkT, Sp, D1T, H;                                      // forward, C x hid
  // backward extras
  size_t Spp, G, D1, Sz, HT, dZ, dZT, dGT, dZkT, dYkT, dXT, QT, KT, XT, XAT, XET,
      dOT, dOAT, dOET, PzT, PoT, Q1T, Q2T, dXN, dXNT, ST, Rb, small_f32;
  size_t f32_elems;  // fp32 elements per unit (dX, dK, dQ, dR, dN, dc, U, ...)
};

struct LocalFwdArgs {
  const void* q; const void* k; const void* v;
  const float* lr; const float* mom; const float* decay;  // this memory, [B][H][L]
  const float* W1i; const float* W2i;                    // this memory, [H][hid][d], [H][d][hid]
  float* o_part;                                         // [B][H][L][d]
  float* states;                                         // [units][nslots][4*hid*d]
  float* mstates;                                        // [units][nslots][d*d]
  void* statesT;                                         // null, or CT [units][nslots][4*hid*d + d*d]:
                                                         // W1^T, W2^T, S1^T, S2^T, M^T of every slot
  void* fsplit;                                          // null, or local_fwd_split_bytes(D, units)
                                                         // bytes: the split forward (saved states only)
  void* frec; float* frec_f;                             // null, or the forward records (saved
                                                         // buffer) the backward passes read
  int nslots;
  int fslots;                                            // 0: the walk writes every fp32 slot
                                                         // ([units][nslots][4*hid*d]); else
                                                         // `states` is [units][fslots][4*hid*d],
                                                         // a ring the walk cycles through (the
                                                         // backward then reads only statesT)
  void* scratch;                                         // units * plan.elems CT
  LocalPlan plan;
  Dims D;
  int force_generic;                                     // 1: skip fixed-size kernels
};

struct LocalBwdArgs {
  const void* q; const void* k; const void* v; const void* dO;
  const float* lr; const float* mom; const float* decay;
  const float* states;                                   // saved chunk-entry states
  const float* mstates;
  const void* statesT;                                   // CT [units][nslots][4*hid*d + d*d]:
                                                         // W1^T, W2^T, S1^T, S2^T, M^T
  int nslots;
  int fslots;                                            // nonzero: `states` holds only the walk's
                                                         // ring, not every chunk-entry state
  float* adj;                                            // [units][4*hid*d] adjoint state
  float* madj;                                           // [units][2][d*d]
  float* hadj;                                           // D.gsub > 1: [units][2*hid*d], the
                                                         // adjoint of the gradient-point state
  float* dq_part; float* dk_part; float* dv_part;        // [B][H][L][d] fp32
  float* dlr; float* dmom; float* ddecay;                // this memory, [B][H][L]
  float* dWinit_part;                                    // [units][2*hid*d]
  void* scratch;
  float* scratch_f32;                                    // units * plan.f32_elems
  LocalPlan plan;
  Dims D;
  const void* frec; const float* frec_f;                 // forward records (written by the split
                                                         // forward; required by the split backward)
  void* split_ws;                                        // null, or local_bwd_split_bytes(D, units)
                                                         // bytes for the three-pass fixed-size kernels
  int single_walk;                                       // 1: the one-walk fixed-size kernel
  hipEvent_t pass_a_done;                                // null, or recorded on the stream once the
                                                         // chunk-parallel pass is done (at once when
                                                         // the backward has no such pass)
  hipEvent_t pass_b_done;                                // null, or recorded on the stream once dq,
                                                         // dv and dWinit_part are final (after the
                                                         // walk; before the gate pass, which adds
                                                         // only to dk and the gate adjoints)
  hipStream_t aux;                                       // null, or a second stream for work that
  hipEvent_t aux_done;                                   // needs pass A only (with pass_a_done set):
                                                         // it waits for pass_a_done there, and the
                                                         // gate pass waits for aux_done
  hipEvent_t aux_mid;                                    // with aux: recorded there once the lower
                                                         // half of the chunks has its pass A
  int force_generic;                                     // 1: skip fixed-size kernels
  // Host side: with defer_gate set, the three-pass kernels may leave their gate
  // pass out (setting *gate_deferred) for launch_local_bwd_gate to run later.
  int defer_gate;
  int* gate_deferred;
  // The final dk, when every other memory's dk part is done before the gate pass:
  // the gate pass writes dk_out (I/O dtype) = the fixed-order sum of dk_nparts fp32
  // parts dk_stride elements apart, this memory's (part dk_self) from registers.
  void* dk_out;
  const float* dk_parts;
  size_t dk_stride;
  int dk_nparts, dk_self;
};

struct GlobalArgs {
  const void* q; const void* k; const void* v; const void* dO;
  const float* lr; const float* mom; const float* decay;  // memory 0, [B][H][L]
  const float* W1i; const float* W2i;                    // memory 0, [H][hid][d], ...
  float* o_part;                                         // [B][H][L][d]
  float* states;                                         // [B*H][nslots][4*hid*d]
  int nslots;
  float* tokc;                                           // [B*H][L][TKS] cC, b, la, lb, s, e^{lb_C-lb}
  float* chunkc;                                         // [B*H][L/C][4] A_C, B_C, E_C, 0
  float* Rbuf;                                           // [B*H][C][d]
  // backward
  float* adj;                                            // [B*H][2][4*hid*d] ping-pong
  float* dRbuf;                                          // [B*H][C][d]
  float* dtok;                                           // [B*H][L][4]  d cC_t, d b_t
  float* dchunk;                                         // [B*H][L/C][nsl][4] partials
  float* dq_part; float* dk_part; float* dv_part;
  float* dlr; float* dmom; float* ddecay;
  float* dWinit;                                         // [B*H][2*hid*d] (reduced later)
  void* scratch;                                         // phase-A scratch of the backward
  size_t scratch_f32_off;
  float* part;                                           // [B*H][nsplit][4*hid*d] split partials
  void* packT;                                           // CT [B*H][4*hid*d]: W1^T, W2^T, W1, W2
  void* packA;                                           // CT [B*H][8*hid*d]: the adjoint's four
                                                         // matrices transposed, then as they are
  void* opT;                                             // CT per-chain transposed chunk operands
  Dims D;
  int force_generic;                                     // 1: skip fixed-size kernels
  int skip_final_carry;                                  // 1: the state after the last chunk
                                                         // is not read (no final-state output)
  // Forward, the last chunk's retrieval-only tile (skip_final_carry): with o_final
  // set it writes the layer output of its tokens (I/O dtype) = the fixed-order sum
  // of o_nparts fp32 parts o_stride elements apart, the global memory's (part 0)
  // from registers, after waiting on its stream for parts_ready; *o_fused is set
  // when that tile was launched.  tile_done (host side): recorded after the tile of
  // chunk tile_done_n.
  void* o_final;
  size_t o_stride;
  int o_nparts;
  hipEvent_t parts_ready, tile_done;
  int tile_done_n;
  int* o_fused;
  int* tile_recorded;  // set when tile_done was recorded
};

constexpr int TKS = 8;  // floats per token in GlobalArgs::tokc

// Compute units of the current device (0 if the query fails).
inline int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return n;
}

// Allow a kernel the whole LDS of a CU for its dynamic shared memory.
inline void set_lds_limit(const void* fn) {
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) !=
      hipSuccess)
    (void)hipGetLastError();
}

// Whether a compiled kernel's static LDS (as the runtime reports it) plus `dyn`
// bytes of dynamic LDS fit one CU's 160 KB: checked before every launch of a
// fixed-size kernel, so that a layout change that outgrows the LDS is refused
// (hipErrorInvalidConfiguration) instead of launched.
inline bool lds_fits(const void* fn, size_t dyn) {
  hipFuncAttributes at{};
  if (hipFuncGetAttributes(&at, fn) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return at.sharedSizeBytes + dyn <= 160 * 1024;
}

size_t local_plan(const Dims& D, LocalPlan* p, bool backward);

hipError_t launch_local_fwd(const LocalFwdArgs& a, int units, hipStream_t st);
size_t local_fwd_split_bytes(const Dims& D, int units);  // 0: no fixed-size forward for D
bool launch_local_fwd_fast(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err);
// the register-resident forward walk (saved states, fixed sizes); false: not built for `a`
bool launch_local_walk(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err);
// the retrieval of every (unit, chunk) after the walk (same shapes); false: not built for `a`
bool launch_local_ret(const LocalFwdArgs& a, int units, hipStream_t st, hipError_t* err);
hipError_t launch_pack_states(const float* states, const float* mstates, void* out, int units,
                               int nslots, int d, int hid, int with_m, int bf16, hipStream_t st);
hipError_t launch_local_bwd(const LocalBwdArgs& a, int units, hipStream_t st);
bool launch_local_bwd_blk(const LocalBwdArgs& a, int units, hipStream_t st, hipError_t* err);
size_t local_bwd_split_bytes(const Dims& D, int units);  // 0: no three-pass kernels for D
bool launch_local_bwd_split(const LocalBwdArgs& a, int units, hipStream_t st, hipError_t* err);
// the gate pass that launch_local_bwd_split deferred (same arguments)
hipError_t launch_local_bwd_gate(const LocalBwdArgs& a, int units, hipStream_t st);
hipError_t launch_global_scan(const GlobalArgs& a, hipStream_t st);
hipError_t launch_global_init(const GlobalArgs& a, hipStream_t st);
hipError_t launch_global_fwd_chunk(const GlobalArgs& a, int n, hipStream_t st);
hipError_t launch_global_bwd_chunk(const GlobalArgs& a, int n, hipStream_t st);
hipError_t launch_global_bwd_zero(const GlobalArgs& a, int slot, hipStream_t st);
hipError_t launch_reduce_global_init(const float* part, int B, int H, size_t hd, float* dW1,
                                     float* dW2, hipStream_t st);
size_t global_bwd_scratch_bytes(const Dims& D, size_t* f32_off);
int global_fwd_splits(const Dims& D);
int global_blk_splits(const Dims& D);
hipError_t launch_global_carry_reduce(const GlobalArgs& a, int n, int nsplit, hipStream_t st);
hipError_t launch_gbwd_state_reduce(const GlobalArgs& a, int n, int nsplit, hipStream_t st);
bool launch_global_fwd_blk(const GlobalArgs& a, int n, hipStream_t st, hipError_t* err);
// Opt-in timing of one step inside a composite launch (the global state-carry
// GEMMs and their reduction): section_begin records a start event on `st` and
// returns a handle (-1 while launch timing is off); section_end records the
// matching stop event.  The pair is reported under `name` with the launches.
int section_begin(const char* name, hipStream_t st);
void section_end(int handle, hipStream_t st);
bool launch_global_bwd_blk(const GlobalArgs& a, int n, hipStream_t st, hipError_t* err);
int global_bwd_splits(const Dims& D);
constexpr int GRED_BLOCKS = 16;  // blocks per chain of the split reductions

// Step-wise forward from a carried state (tnt_mem_step).  Memory m's chunk is
// C[m] and, for a local memory, its shard S[m].  state: per (memory, chain) a
// block of mem_stride fp32 = W^1, W^2 (chunk-entry), W1, W2, S1, S2 (each
// hid*d) and the Q-K sum M (d*d).
struct StepArgs {
  int B, H, T, d, hid, M, has_global, act, qk_proj, qk_scope, bf16;
  long long pos;       // tokens the state has consumed before this call
  int C[9], S[9];
  const void *q, *k, *v;                      // [B][H][T][d]
  const float *lr, *mom, *decay;              // [M][B][H][T]
  const float *W1i, *W2i;                     // [M][H][hid][d], [M][H][d][hid]
  float* state;
  void* o;                                    // [B][H][T][d]
  size_t mem_stride;
  // per-token launches: hidden units split into G slices of HS; the scratch
  // area (after every state block) holds sc_stride floats per (memory, chain)
  int G, HS, t;
  float* scratch;
  size_t sc_stride;
};
size_t step_state_floats(int d, int hid);
size_t step_scratch_floats(int d, int hid);
hipError_t launch_step_init(const StepArgs& a, hipStream_t st);
hipError_t launch_step_from_final(const StepArgs& a, const float* fin, hipStream_t st);
hipError_t launch_step(const StepArgs& a, hipStream_t st);
hipError_t launch_global_gate_bwd(const GlobalArgs& a, hipStream_t st);

// tnt_dbg_chunk_grads: one chunk (tokens tok0 .. tok0 + C of a chain's rows in
// k, v) at the weights W1 [hid][d], W2 [d][hid]
struct DbgArgs {
  int d, hid, C, act, bf16;
  size_t tok0;         // row of the chunk's first token in the [B*H*L][d] arrays
  const void *k, *v;
  const float *W1, *W2;
  float *Zk, *R, *D1;  // [C][hid], [C][d], [C][hid]
};
hipError_t launch_dbg_chunk_grads(const DbgArgs& a, hipStream_t st);
struct SumJobs {  // up to three (partials, output) pairs summed by one launch
  const float* parts[3];
  void* out[3];
};
hipError_t launch_sum_outs(const SumJobs& jobs, int njobs, int nparts, size_t stride, size_t n,
                           int bf16, hipStream_t st);
hipError_t launch_sum_out(const float* parts, int nparts, size_t stride, size_t n, void* out,
                          int bf16, hipStream_t st);
// the same sum over the first `seg` of every `per` elements (nseq runs; seg and per
// multiples of 8)
hipError_t launch_sum_out_runs(const float* parts, int nparts, size_t stride, size_t nseq, size_t per,
                               size_t seg, void* out, int bf16, hipStream_t st);
hipError_t launch_reduce_init(const float* parts, int B, int H, int nshard, size_t hd2,
                              float* dW1, float* dW2, int d, int hid, int accumulate,
                              hipStream_t st);
hipError_t launch_copy_final(const float* states, int nslots, int nchains, size_t slot_elems,
                             int last, float* out, hipStream_t st);

}  // namespace tnt
