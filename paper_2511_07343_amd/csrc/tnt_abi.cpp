// C ABI of the TNT memory layer: validation, workspace layout and the launch
// sequence of the forward and backward passes.  See include/tnt.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/tnt.h"
#include "tnt_entry.h"
#include "tnt_kernels.h"
#include "tnt_local_bwd_layout.h"
#include "tnt_local_record.h"

using namespace tnt;

namespace {

constexpr size_t ALIGN = 256;
inline size_t up(size_t x) { return (x + ALIGN - 1) & ~(ALIGN - 1); }

bool one_of(int x, std::initializer_list<int> v) {
  for (int y : v)
    if (x == y) return true;
  return false;
}

// need_L = false: the step-wise entry points, where the sequence is open-ended
// and L is ignored
tnt_status validate(const tnt_config* c, bool need_L = true) {
  if (!c) return TNT_ERR_NULL;
  if (c->act < 0 || c->act > 1 || c->qk_proj < 0 || c->qk_proj > 1 || c->qk_scope < 0 ||
      c->qk_scope > 1 || c->dtype < 0 || c->dtype > 1 || c->has_global < 0 || c->has_global > 1 ||
      c->global_intra < 0 || c->global_intra > 1)
    return TNT_ERR_ARG;
  if (c->B <= 0 || c->H <= 0 || (need_L && c->L <= 0) || c->d <= 0 || c->hid <= 0)
    return TNT_ERR_SHAPE;
  if (c->n_local < 0 || c->n_local > TNT_MAX_LOCAL) return TNT_ERR_SHAPE;
  if (c->has_global + c->n_local < 1) return TNT_ERR_SHAPE;
  if (c->has_global) {
    if (c->C_G <= 0 || (need_L && c->L % c->C_G)) return TNT_ERR_SHAPE;
  }
  for (int i = 0; i < c->n_local; ++i) {
    if (c->C_L[i] <= 0 || c->S_L[i] <= 0) return TNT_ERR_SHAPE;
    if (c->S_L[i] % c->C_L[i] || (need_L && c->L % c->S_L[i])) return TNT_ERR_SHAPE;
  }
  if (!one_of(c->d, {16, 32, 64, 128})) return TNT_ERR_UNSUPPORTED;
  if (!one_of(c->hid, {16, 32, 64, 128, 256, 512})) return TNT_ERR_UNSUPPORTED;
  for (int i = 0; i < c->n_local; ++i)
    if (c->C_L[i] > 64) return TNT_ERR_UNSUPPORTED;
  // the intra-chunk reading of the global memory runs as one more local-style
  // memory (see effective()): chunk-parallel calls only, one slot to spare
  if (c->has_global && c->global_intra && (c->n_local >= TNT_MAX_LOCAL || !need_L))
    return TNT_ERR_UNSUPPORTED;
  return TNT_OK;
}

// The global memory under the intra-chunk reading (each token read at V_t
// after its own update, gradients at the chunk-entry state) is the local rule
// with C_L = C_G, no reset within the sequence and no Q-K projection (a pinned
// identity of the oracle).  It is walked as local memory 0 in sub-chunks of
// csub <= 64 tokens (the largest divisor of C_G up to 64) whose gradients are
// all taken at the state entering their C_G chunk (gsub = C_G / csub
// sub-chunks per gradient point); the locals follow it.
struct Eff {
  tnt_config c;
  int gsub;  // > 0: local 0 of `c` is the global memory under the intra-chunk reading
};

Eff effective(const tnt_config* c) {
  Eff e{*c, 0};
  if (!(c->has_global && c->global_intra)) return e;
  int cs = c->C_G < 64 ? c->C_G : 64;
  while (c->C_G % cs) --cs;
  e.gsub = c->C_G / cs;
  e.c.has_global = 0;
  e.c.n_local = c->n_local + 1;
  for (int i = TNT_MAX_LOCAL - 1; i >= 1; --i) {
    e.c.C_L[i] = c->C_L[i - 1];
    e.c.S_L[i] = c->S_L[i - 1];
  }
  e.c.C_L[0] = cs;
  e.c.S_L[0] = c->L;
  return e;
}

Dims dims_of(const tnt_config* c, int C, int S) {
  Dims D{};
  D.B = c->B; D.H = c->H; D.L = c->L; D.d = c->d; D.hid = c->hid;
  D.C = C; D.Cp = (C + 15) / 16 * 16; D.S = S;
  D.act = c->act; D.bf16 = c->dtype == TNT_BF16;
  D.qk_proj = c->qk_proj; D.qk_scope = c->qk_scope;
  return D;
}

// Byte offsets of every buffer.  Offsets are relative to the workspace, or to
// the saved buffer for the chunk-entry states.
struct Layout {
  int M, BH;
  int gsub0;  // > 0: local 0 is the global memory under the intra-chunk reading
  size_t hd, io_elems, gates;
  // saved (or workspace-resident) chunk states
  size_t sv_g, sv_l[TNT_MAX_LOCAL], sv_m[TNT_MAX_LOCAL], sv_t[TNT_MAX_LOCAL],
      sv_fr[TNT_MAX_LOCAL], sv_frf[TNT_MAX_LOCAL], saved_bytes;
  int g_chunks, l_units[TNT_MAX_LOCAL], l_chunks[TNT_MAX_LOCAL];
  int l_fslots[TNT_MAX_LOCAL];  // 0: every fp32 chunk-entry state saved; else the walk's ring
  // forward workspace
  size_t w_opart, w_tokc, w_chunkc, w_R, w_part, w_gpack, w_gop, w_scr[TNT_MAX_LOCAL],
      w_fsplit[TNT_MAX_LOCAL], w_ring,
      fwd_bytes;
  // without a saved buffer, the two-pass local forward's every-slot compute-type
  // state copies and fp32 Q-K states (SIZE_MAX: that memory walks in one pass)
  size_t w_nt[TNT_MAX_LOCAL], w_nm[TNT_MAX_LOCAL], fwd_two_bytes;
  size_t ring_g, ring_l[TNT_MAX_LOCAL], ring_m[TNT_MAX_LOCAL];
  LocalPlan lplan[TNT_MAX_LOCAL];
  // backward workspace
  size_t b_dparts, b_adj_g, b_dR, b_dtok, b_dchunk, b_dWg, b_gscr, b_gscr_f32, b_gpackA, b_gop,
      b_adj_l[TNT_MAX_LOCAL], b_madj[TNT_MAX_LOCAL], b_hadj[TNT_MAX_LOCAL], b_dWl[TNT_MAX_LOCAL],
      b_scr[TNT_MAX_LOCAL], b_scrf[TNT_MAX_LOCAL], b_split[TNT_MAX_LOCAL], b_states, bwd_bytes,
      bwd_re_bytes;
  BwdLayout blay[TNT_MAX_LOCAL];
};

// Kernel family (tnt_set_kernel_family): which of the kernel families the
// calls take; fixed per saved buffer (recorded in its header).
std::atomic<int> g_family{TNT_FAMILY_DEFAULT};
int generic_only() { return g_family.load() == TNT_FAMILY_GENERIC ? 1 : 0; }
int single_walk_only() { return g_family.load() == TNT_FAMILY_SINGLE_WALK ? 1 : 0; }

// Sizes of local memory i's pass (the intra-reading global memory, local 0
// when gsub0 > 0, has no Q-K projection and takes its gradients per group).
Dims mem_dims(const tnt_config* c, int gsub0, int i) {
  Dims D = dims_of(c, c->C_L[i], c->S_L[i]);
  if (i == 0 && gsub0 > 0) {
    D.qk_proj = 0;
    D.qk_scope = 0;
    D.gsub = gsub0;
  }
  return D;
}

Layout layout_of(const tnt_config* c, int gsub0 = 0) {
  Layout y{};
  y.gsub0 = gsub0;
  y.M = c->has_global + c->n_local;
  y.BH = c->B * c->H;
  y.hd = (size_t)c->hid * c->d;
  y.io_elems = (size_t)y.BH * c->L * c->d;
  y.gates = (size_t)y.BH * c->L;
  const size_t cts = c->dtype == TNT_BF16 ? 2 : 4;
  const size_t f = sizeof(float);
  const size_t dd = (size_t)c->d * c->d;

  // saved states, behind the buffer's header
  size_t off = SAVED_HEADER_BYTES;
  if (c->has_global) {
    y.g_chunks = c->L / c->C_G;
    y.sv_g = off;
    off += up((size_t)y.BH * (y.g_chunks + 1) * 4 * y.hd * f);
  }
  for (int i = 0; i < c->n_local; ++i) {
    y.l_units[i] = y.BH * (c->L / c->S_L[i]);
    y.l_chunks[i] = c->S_L[i] / c->C_L[i];
    // Shapes with both chunk-parallel kernels save forward records, and their
    // backward reads the states only through the compute-type transposes: the
    // walk then cycles its fp32 carry through two slots per unit instead of
    // writing every slot, and only those two are reserved.  The families that
    // recompute from the fp32 states (one-walk, runtime-sized) keep every slot.
    const Dims D = mem_dims(c, gsub0, i);
    const bool recs = !(i == 0 && gsub0) && local_fwd_split_bytes(D, y.l_units[i]) &&
                      local_bwd_split_bytes(D, y.l_units[i]);
    y.l_fslots[i] = (recs && !single_walk_only() && !generic_only()) ? 2 : 0;
    y.sv_l[i] = off;
    off += up((size_t)y.l_units[i] * (y.l_fslots[i] ? y.l_fslots[i] : y.l_chunks[i] + 1) * 4 *
              y.hd * f);
    y.sv_m[i] = off;
    off += up((size_t)y.l_units[i] * (y.l_chunks[i] + 1) * dd * f);
    y.sv_t[i] = off;  // CT transposes of every slot, written by the forward
    off += up((size_t)y.l_units[i] * (y.l_chunks[i] + 1) * (4 * y.hd + dd) * cts);
    // forward records of the chunk-parallel passes (shapes with both split kernels)
    y.sv_fr[i] = y.sv_frf[i] = SIZE_MAX;
    if (recs) {
      const rec::RecLayout R = rec::make_rec_layout(D.Cp, D.d, D.hid);
      const size_t items = (size_t)y.l_units[i] * y.l_chunks[i];
      y.sv_fr[i] = off; off += up(items * R.fc.n * cts);
      y.sv_frf[i] = off; off += up(items * R.ff.n * f);
    }
  }
  y.saved_bytes = off;

  // forward workspace
  off = 0;
  y.w_opart = off; off += up((size_t)y.M * y.io_elems * f);
  if (c->has_global) {
    y.w_tokc = off; off += up(y.gates * TKS * f);
    y.w_chunkc = off; off += up((size_t)y.BH * y.g_chunks * 4 * f);
    y.w_R = off; off += up((size_t)y.BH * c->C_G * c->d * f);
    const Dims D = dims_of(c, c->C_G, c->L);
    const int ns = std::max({global_fwd_splits(D), global_bwd_splits(D), global_blk_splits(D), 1});
    y.w_part = off; off += up((size_t)y.BH * ns * 4 * y.hd * f);
    // transposed state copies and the chunk operands of the fixed-size global kernels
    y.w_gpack = off; off += up((size_t)y.BH * 4 * y.hd * cts);
    y.w_gop = off; off += up((size_t)y.BH * (2 * (size_t)c->hid + 4 * (size_t)c->d) * c->C_G * cts);
  }
  for (int i = 0; i < c->n_local; ++i) {
    const Dims D = mem_dims(c, gsub0, i);
    local_plan(D, &y.lplan[i], false);
    y.w_scr[i] = off; off += up((size_t)y.l_units[i] * y.lplan[i].elems * cts);
    const size_t fb = local_fwd_split_bytes(D, y.l_units[i]);
    y.w_fsplit[i] = fb ? off : SIZE_MAX;
    off += up(fb);
  }
  const size_t fwd_core = off;
  // two-slot state rings, used when no saved buffer is given
  y.w_ring = off;
  if (c->has_global) { y.ring_g = off; off += up((size_t)y.BH * 2 * 4 * y.hd * f); }
  for (int i = 0; i < c->n_local; ++i) {
    // a two-slot ring, or every slot for the grouped gradient points
    const size_t ns = (i == 0 && gsub0) ? (size_t)y.l_chunks[i] + 1 : 2;
    y.ring_l[i] = off; off += up((size_t)y.l_units[i] * ns * 4 * y.hd * f);
    y.ring_m[i] = off; off += up((size_t)y.l_units[i] * ns * dd * f);
  }
  y.fwd_bytes = off;
  (void)fwd_core;
  // the two-pass local forward without a saved buffer: past the smallest forward
  // workspace (the backward workspace may reuse this space: it never runs a
  // forward without saving)
  for (int i = 0; i < c->n_local; ++i) {
    y.w_nt[i] = y.w_nm[i] = SIZE_MAX;
    if (!y.l_fslots[i]) continue;  // the memories whose forward has both passes
    y.w_nt[i] = off; off += up((size_t)y.l_units[i] * (y.l_chunks[i] + 1) * (4 * y.hd + dd) * cts);
    y.w_nm[i] = off; off += up((size_t)y.l_units[i] * (y.l_chunks[i] + 1) * dd * f);
  }
  y.fwd_two_bytes = off;

  // backward workspace (shares the forward's front part for recomputation)
  off = y.fwd_bytes;
  y.b_dparts = off; off += up(3 * (size_t)y.M * y.io_elems * f);
  if (c->has_global) {
    y.b_adj_g = off; off += up((size_t)y.BH * 2 * 4 * y.hd * f);
    y.b_dR = off; off += up((size_t)y.BH * c->C_G * c->d * f);
    y.b_dtok = off; off += up(y.gates * 4 * f);
    y.b_dchunk = off; off += up((size_t)y.BH * y.g_chunks * GRED_BLOCKS * 4 * f);
    y.b_dWg = off; off += up((size_t)y.BH * 2 * y.hd * f);
    const Dims D = dims_of(c, c->C_G, c->L);
    y.b_gscr = off;
    off += up(global_bwd_scratch_bytes(D, &y.b_gscr_f32));
    y.b_gpackA = off; off += up((size_t)y.BH * 8 * y.hd * cts);  // transposed and as they are
    y.b_gop = off; off += up((size_t)y.BH * 5 * ((size_t)c->hid + c->d) * c->C_G * cts);
  }
  for (int i = 0; i < c->n_local; ++i) {
    const Dims D = mem_dims(c, gsub0, i);
    bwd_layout(D.Cp, D.d, D.hid, &y.blay[i]);
    y.b_adj_l[i] = off; off += up((size_t)y.l_units[i] * 4 * y.hd * f);
    y.b_madj[i] = off; off += up((size_t)y.l_units[i] * dd * f);
    y.b_hadj[i] = off;
    if (i == 0 && gsub0) off += up((size_t)y.l_units[i] * 2 * y.hd * f);
    y.b_dWl[i] = off; off += up((size_t)y.l_units[i] * 2 * y.hd * f);
    y.b_scr[i] = off; off += up((size_t)y.l_units[i] * y.blay[i].ct_elems * cts);
    y.b_scrf[i] = off; off += up((size_t)y.l_units[i] * y.blay[i].f32_elems * f);
    const size_t sb = local_bwd_split_bytes(D, y.l_units[i]);
    y.b_split[i] = sb ? off : SIZE_MAX;
    off += up(sb);
  }
  y.bwd_bytes = off;
  y.b_states = off;
  y.bwd_re_bytes = off + y.saved_bytes;
  return y;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

// ---- the saved buffer's header: what wrote it and for which call.  The
// forward writes it into the first SAVED_HEADER_BYTES of `saved` (device) and
// records it per buffer on the host; the backward compares the host record
// with its own call before it enqueues anything.
uint64_t config_hash(const tnt_config* c) {
  tnt_config n = *c;  // entries the call does not use do not count
  for (int i = n.n_local; i < TNT_MAX_LOCAL; ++i) n.C_L[i] = n.S_L[i] = 0;
  if (!n.has_global) n.C_G = n.global_intra = 0;
  uint64_t h = 1469598103934665603ull;  // FNV-1a over the configuration's bytes
  const unsigned char* p = (const unsigned char*)&n;
  for (size_t i = 0; i < sizeof(tnt_config); ++i) h = (h ^ p[i]) * 1099511628211ull;
  return h;
}

SavedHeader header_of(const tnt_config* c, const Layout& y) {
  SavedHeader h{};
  h.magic = SAVED_MAGIC;
  h.layout_version = SAVED_LAYOUT_VERSION;
  h.family = (uint32_t)g_family.load();
  for (int i = 0; i < TNT_MAX_LOCAL; ++i) h.fslots[i] = (uint32_t)y.l_fslots[i];  // 0 past the memories
  h.cfg_hash = config_hash(c);
  h.bytes = y.saved_bytes;
  return h;
}

bool same_header(const SavedHeader& a, const SavedHeader& b) {
  return std::memcmp(&a, &b, sizeof(SavedHeader)) == 0;
}

std::mutex g_saved_mu;
std::vector<std::pair<const void*, SavedHeader>> g_saved;  // most recent last
constexpr size_t SAVED_RECORDS = 4096;

void remember_saved(const void* p, const SavedHeader& h) {
  std::lock_guard<std::mutex> lk(g_saved_mu);
  for (size_t i = 0; i < g_saved.size(); ++i)
    if (g_saved[i].first == p) {
      g_saved.erase(g_saved.begin() + i);
      break;
    }
  if (g_saved.size() >= SAVED_RECORDS) g_saved.erase(g_saved.begin());
  g_saved.emplace_back(p, h);
}

bool recorded_saved(const void* p, SavedHeader* out) {
  std::lock_guard<std::mutex> lk(g_saved_mu);
  for (size_t i = g_saved.size(); i-- > 0;)
    if (g_saved[i].first == p) {
      *out = g_saved[i].second;
      return true;
    }
  return false;
}

// ---- opt-in launch timing (hipEvent pairs per launch)
struct TimedLaunch {
  const char* name;
  hipEvent_t a, b;
};
struct Timing {
  bool on = false;
  std::vector<TimedLaunch> rec;
  std::vector<hipEvent_t> pool;
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Timing g_timing;
constexpr size_t TIMING_CAP = 65536;

template <typename F>
hipError_t timed(const char* name, hipStream_t st, F&& launch) {
  if (!g_timing.on || g_timing.rec.size() >= TIMING_CAP) return launch();
  TimedLaunch t{name, g_timing.get(), g_timing.get()};
  if (!t.a || !t.b) return launch();
  hipEventRecord(t.a, st);
  const hipError_t e = launch();
  hipEventRecord(t.b, st);
  g_timing.rec.push_back(t);
  return e;
}

// ---- helper stream per device: the global memory's chain runs on it while
// the local shards run on the caller's stream (they only meet at the sums).
// Default priority; events are reused under a lock, so concurrent host
// threads serialise their enqueues here.
struct Fork {
  hipStream_t side = nullptr, side2 = nullptr;  // side2: local memories after the first
  hipEvent_t e0 = nullptr, e1 = nullptr, ea = nullptr, eb = nullptr, eg = nullptr, es = nullptr,
            ec = nullptr, er = nullptr, et = nullptr, e2 = nullptr;
};
constexpr int MAX_DEV = 64;
Fork g_fork[MAX_DEV];
std::mutex g_fork_mu;

hipError_t fork_of(Fork** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEV) return hipErrorInvalidDevice;
  Fork& f = g_fork[dev];
  if (!f.side) {
    if ((e = hipStreamCreateWithFlags(&f.side, hipStreamNonBlocking)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.e0, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.e1, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.ea, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.eb, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.eg, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.es, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.ec, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.er, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.et, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipStreamCreateWithFlags(&f.side2, hipStreamNonBlocking)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&f.e2, hipEventDisableTiming)) != hipSuccess) return e;
  }
  *out = &f;
  return hipSuccess;
}

#define HIP_TRY(x)                         \
  do {                                     \
    if ((x) != hipSuccess) return TNT_ERR_HIP; \
  } while (0)
#define HIP_TIMED(name, x) HIP_TRY(timed(name, st, [&]() { return (x); }))

// forward pass into a given state area (`sv` = saved buffer, or nullptr to use
// the two-slot rings in the workspace)
// `fork`: false keeps every launch on `st` (no helper stream is created or used).
tnt_status run_forward(const tnt_config* c, const Layout& y, const void* q, const void* k,
                       const void* v, const float* lr, const float* mom, const float* decay,
                       const float* W1i, const float* W2i, void* o, float* final_state,
                       char* sv, char* ws, hipStream_t st, bool fork = true,
                       size_t ws_bytes = 0) {
  // no saved buffer: the two-pass local forward still runs when the workspace
  // holds its state copies
  const bool two = !sv && ws_bytes >= y.fwd_two_bytes;
  const size_t G = y.gates;
  float* opart = (float*)(ws + y.w_opart);
  int m = 0;
  std::unique_lock<std::mutex> lock(g_fork_mu);
  Fork* fk = nullptr;
  const hipStream_t main_st = st;
  if (fork && c->has_global && c->n_local) {
    HIP_TRY(fork_of(&fk));
    HIP_TRY(hipEventRecord(fk->e0, main_st));
    HIP_TRY(hipStreamWaitEvent(fk->side, fk->e0, 0));
    st = fk->side;
  }
  // the local walks first: their workgroups are the critical path, and the
  // dispatcher places work in the order it is enqueued (the global chain's
  // tile grids would otherwise take the CUs before the walk starts).  With two or
  // more local memories (none of them the grouped global memory) every one after
  // the first runs on a second helper stream beside the first: they share nothing
  // (each has its own workspace and saved regions and its own output part).
  const bool conc = fk && c->n_local >= 2 && !y.gsub0;
  if (conc) HIP_TRY(hipStreamWaitEvent(fk->side2, fk->e0, 0));
  m = c->has_global;
  for (int i = 0; i < c->n_local; ++i, ++m) {
    st = (conc && i > 0) ? fk->side2 : main_st;
    LocalFwdArgs a{};
    a.q = q; a.k = k; a.v = v;
    a.lr = lr + m * G; a.mom = mom + m * G; a.decay = decay + m * G;
    a.W1i = W1i + (size_t)m * c->H * y.hd;
    a.W2i = W2i + (size_t)m * c->H * y.hd;
    a.o_part = opart + (size_t)m * y.io_elems;
    const bool two_i = two && y.w_nt[i] != SIZE_MAX;
    a.states = sv ? (float*)(sv + y.sv_l[i]) : (float*)(ws + y.ring_l[i]);
    a.mstates = sv ? (float*)(sv + y.sv_m[i]) : two_i ? (float*)(ws + y.w_nm[i]) : (float*)(ws + y.ring_m[i]);
    a.statesT = sv ? (void*)(sv + y.sv_t[i]) : two_i ? (void*)(ws + y.w_nt[i]) : nullptr;
    a.frec = (sv && y.sv_fr[i] != SIZE_MAX) ? (void*)(sv + y.sv_fr[i]) : nullptr;
    a.frec_f = (sv && y.sv_frf[i] != SIZE_MAX) ? (float*)(sv + y.sv_frf[i]) : nullptr;
    const bool grouped = i == 0 && y.gsub0;
    a.nslots = (sv || grouped || two_i) ? y.l_chunks[i] + 1 : 2;
    a.fslots = sv ? y.l_fslots[i] : two_i ? 2 : 0;  // two_i: the two-slot fp32 ring
    a.scratch = ws + y.w_scr[i];
    a.fsplit = y.w_fsplit[i] != SIZE_MAX ? (void*)(ws + y.w_fsplit[i]) : nullptr;
    a.plan = y.lplan[i];
    a.D = mem_dims(c, y.gsub0, i);
    a.force_generic = generic_only() || grouped;
    HIP_TIMED(grouped ? "global_intra_fwd" : "local_fwd", launch_local_fwd(a, y.l_units[i], st));
    if (grouped && final_state)  // the global memory's state after the last token
      HIP_TIMED("copy_final", launch_copy_final(a.states, a.nslots, y.l_units[i], 4 * y.hd,
                                                y.l_chunks[i], final_state, st));
  }
  // With the helper stream and no final state: the last global chunk's tile writes
  // the layer output of its tokens, and the caller's stream sums the other tokens'
  // parts once the tile of the chunk before it is done (beside the last carry).
  st = main_st;
  if (conc) {
    HIP_TRY(hipEventRecord(fk->e2, fk->side2));
    HIP_TRY(hipStreamWaitEvent(main_st, fk->e2, 0));
  }
  int o_fused = 0, tile_rec = 0;
  const bool fuse_o = fk && o && !final_state;
  if (fuse_o) HIP_TRY(hipEventRecord(fk->er, main_st));
  if (c->has_global) {
    st = fk ? fk->side : main_st;
    GlobalArgs g{};
    g.q = q; g.k = k; g.v = v;
    g.lr = lr; g.mom = mom; g.decay = decay;
    g.W1i = W1i; g.W2i = W2i;
    g.o_part = opart;
    g.states = sv ? (float*)(sv + y.sv_g) : (float*)(ws + y.ring_g);
    g.nslots = sv ? y.g_chunks + 1 : 2;
    g.tokc = (float*)(ws + y.w_tokc);
    g.chunkc = (float*)(ws + y.w_chunkc);
    g.Rbuf = (float*)(ws + y.w_R);
    g.part = (float*)(ws + y.w_part);
    g.packT = ws + y.w_gpack;
    g.opT = ws + y.w_gop;
    g.D = dims_of(c, c->C_G, c->L);
    g.force_generic = generic_only();
    g.skip_final_carry = final_state == nullptr;
    if (fuse_o) {
      g.o_final = o;
      g.o_stride = y.io_elems;
      g.o_nparts = y.M;
      g.parts_ready = fk->er;
      g.tile_done = fk->et;
      g.tile_done_n = y.g_chunks - 2;
      g.o_fused = &o_fused;
      g.tile_recorded = &tile_rec;
    }
    HIP_TIMED("global_scan", launch_global_scan(g, st));
    HIP_TIMED("global_init", launch_global_init(g, st));
    for (int n = 0; n < y.g_chunks; ++n) HIP_TIMED("global_fwd_chunk", launch_global_fwd_chunk(g, n, st));
    if (final_state)
      HIP_TIMED("copy_final", launch_copy_final(g.states, g.nslots, y.BH, 4 * y.hd, y.g_chunks % g.nslots,
                                final_state, st));
  }
  st = main_st;
  const int bf = c->dtype == TNT_BF16;
  if (o_fused && y.g_chunks >= 2) {
    // the tokens of every global chunk but the last (the last tile wrote the rest)
    const hipEvent_t ready = tile_rec ? fk->et : fk->e1;
    if (!tile_rec) HIP_TRY(hipEventRecord(fk->e1, fk->side));
    HIP_TRY(hipStreamWaitEvent(main_st, ready, 0));
    const size_t per = (size_t)c->L * c->d, seg = (size_t)(y.g_chunks - 1) * c->C_G * c->d;
    HIP_TIMED("sum_out", launch_sum_out_runs(opart, y.M, y.io_elems, y.BH, per, seg, o, bf, st));
  }
  if (fk) {
    HIP_TRY(hipEventRecord(fk->e1, fk->side));
    HIP_TRY(hipStreamWaitEvent(main_st, fk->e1, 0));
  }
  if (o && !o_fused) HIP_TIMED("sum_out", launch_sum_out(opart, y.M, y.io_elems, y.io_elems, o, bf, st));
  return TNT_OK;
}

tnt_status run_backward(const tnt_config* c, const Layout& y, const void* q, const void* k,
                        const void* v, const float* lr, const float* mom, const float* decay,
                        const float* W1i, const float* W2i, const void* dO, char* sv,
                        void* dq, void* dk, void* dv, float* dlr, float* dmom, float* ddecay,
                        float* dW1, float* dW2, char* ws, hipStream_t st) {
  const size_t G = y.gates;
  float* dparts = (float*)(ws + y.b_dparts);
  float* dqp = dparts;
  float* dkp = dparts + (size_t)y.M * y.io_elems;
  float* dvp = dparts + 2 * (size_t)y.M * y.io_elems;
  std::unique_lock<std::mutex> lock(g_fork_mu);
  Fork* fk = nullptr;
  const hipStream_t main_st = st;
  // The local memories go first on the caller's stream; the global chain runs on
  // the helper stream from the moment the first local memory's chunk-parallel
  // pass is done (that pass fills the chip; the walk after it leaves half the
  // CUs to the global chain).
  if (c->has_global && c->n_local) HIP_TRY(fork_of(&fk));
  // the last local memory's gate pass, when its walk ran beside the global chain:
  // launched after that chain (and the separate dk sum folded into it)
  int gate_deferred = 0;
  LocalBwdArgs last_local{};
  // two or more local memories: every one after the first on a second helper
  // stream beside the first (as in the forward)
  const bool conc = fk && c->n_local >= 2 && !y.gsub0;
  if (conc) {
    HIP_TRY(hipEventRecord(fk->e0, main_st));
    HIP_TRY(hipStreamWaitEvent(fk->side2, fk->e0, 0));
  }
  for (int i = 0, m = c->has_global; i < c->n_local; ++i, ++m) {
    st = (conc && i > 0) ? fk->side2 : main_st;
    LocalBwdArgs a{};
    a.q = q; a.k = k; a.v = v; a.dO = dO;
    a.lr = lr + m * G; a.mom = mom + m * G; a.decay = decay + m * G;
    a.states = (const float*)(sv + y.sv_l[i]);
    a.mstates = (const float*)(sv + y.sv_m[i]);
    a.nslots = y.l_chunks[i] + 1;
    a.fslots = y.l_fslots[i];
    a.statesT = sv + y.sv_t[i];
    a.frec = y.sv_fr[i] != SIZE_MAX ? (const void*)(sv + y.sv_fr[i]) : nullptr;
    a.frec_f = y.sv_frf[i] != SIZE_MAX ? (const float*)(sv + y.sv_frf[i]) : nullptr;
    a.adj = (float*)(ws + y.b_adj_l[i]);
    a.madj = (float*)(ws + y.b_madj[i]);
    a.dq_part = dqp + (size_t)m * y.io_elems;
    a.dk_part = dkp + (size_t)m * y.io_elems;
    a.dv_part = dvp + (size_t)m * y.io_elems;
    a.dlr = dlr + m * G; a.dmom = dmom + m * G; a.ddecay = ddecay + m * G;
    a.dWinit_part = (float*)(ws + y.b_dWl[i]);
    a.scratch = ws + y.b_scr[i];
    a.scratch_f32 = (float*)(ws + y.b_scrf[i]);
    a.split_ws = y.b_split[i] != SIZE_MAX ? (void*)(ws + y.b_split[i]) : nullptr;
    a.single_walk = single_walk_only();
    a.D = mem_dims(c, y.gsub0, i);
    const bool grouped = i == 0 && y.gsub0;
    a.force_generic = generic_only() || grouped;
    a.hadj = grouped ? (float*)(ws + y.b_hadj[i]) : nullptr;
    a.pass_a_done = (fk && i == 0) ? fk->ea : nullptr;
    a.aux = (fk && i == 0) ? fk->side : nullptr;  // ahead of the global chain there
    a.aux_done = (fk && i == 0) ? fk->es : nullptr;
    a.aux_mid = (fk && i == 0) ? fk->ec : nullptr;
    // the last local memory's walk is the point after which dq, dv and every dW_init
    // part are final: the helper stream reduces them beside its gate pass
    const bool last = i == c->n_local - 1;
    a.pass_b_done = (fk && last && !conc) ? fk->eb : nullptr;
    a.defer_gate = fk && last && !grouped && !conc;
    a.gate_deferred = &gate_deferred;
    HIP_TIMED(grouped ? "global_intra_bwd" : "local_bwd", launch_local_bwd(a, y.l_units[i], st));
    if (last) last_local = a;
    if (!(fk && last))
      HIP_TIMED("reduce_init", launch_reduce_init(a.dWinit_part, c->B, c->H, c->L / c->S_L[i], 2 * y.hd,
                                 dW1 + (size_t)m * c->H * y.hd, dW2 + (size_t)m * c->H * y.hd,
                                 c->d, c->hid, 0, st));
  }
  st = main_st;
  if (conc) {  // dq, dv and every dW_init part are final once both streams are done
    HIP_TRY(hipEventRecord(fk->e2, fk->side2));
    HIP_TRY(hipStreamWaitEvent(main_st, fk->e2, 0));
    HIP_TRY(hipEventRecord(fk->eb, main_st));
  }
  if (c->has_global) {
    if (fk) {
      HIP_TRY(hipStreamWaitEvent(fk->side, fk->ea, 0));
      st = fk->side;
    }
    GlobalArgs g{};
    g.q = q; g.k = k; g.v = v; g.dO = dO;
    g.lr = lr; g.mom = mom; g.decay = decay;
    g.W1i = W1i; g.W2i = W2i;
    g.states = (float*)(sv + y.sv_g);
    g.nslots = y.g_chunks + 1;
    g.tokc = (float*)(ws + y.w_tokc);
    g.chunkc = (float*)(ws + y.w_chunkc);
    g.Rbuf = (float*)(ws + y.w_R);
    g.part = (float*)(ws + y.w_part);
    g.adj = (float*)(ws + y.b_adj_g);
    g.dRbuf = (float*)(ws + y.b_dR);
    g.dtok = (float*)(ws + y.b_dtok);
    g.dchunk = (float*)(ws + y.b_dchunk);
    g.dWinit = (float*)(ws + y.b_dWg);
    g.scratch = ws + y.b_gscr;
    g.scratch_f32_off = y.b_gscr_f32;
    g.dq_part = dqp; g.dk_part = dkp; g.dv_part = dvp;
    g.dlr = dlr; g.dmom = dmom; g.ddecay = ddecay;
    g.packT = ws + y.w_gpack;
    g.packA = ws + y.b_gpackA;
    g.opT = ws + y.b_gop;
    g.D = dims_of(c, c->C_G, c->L);
    g.force_generic = generic_only();
    HIP_TIMED("global_scan", launch_global_scan(g, st));
    HIP_TIMED("global_bwd_zero", launch_global_bwd_zero(g, y.g_chunks & 1, st));
    for (int n = y.g_chunks - 1; n >= 0; --n) HIP_TIMED("global_bwd_chunk", launch_global_bwd_chunk(g, n, st));
    // the global memory's dq, dk, dv are final here (the main stream sums dk after its
    // gate pass); its gate adjoints and dW_init follow while the local walk still runs
    if (fk) HIP_TRY(hipEventRecord(fk->eg, fk->side));
    HIP_TIMED("global_gate_bwd", launch_global_gate_bwd(g, st));
    HIP_TIMED("reduce_init", launch_reduce_global_init(g.dWinit, c->B, c->H, y.hd, dW1, dW2, st));
    if (fk) {
      // dq and dv are final once the last local memory's walk is done too
      HIP_TRY(hipStreamWaitEvent(fk->side, fk->eb, 0));
      SumJobs side{};
      side.parts[0] = dqp; side.out[0] = dq;
      side.parts[1] = dvp; side.out[1] = dv;
      HIP_TIMED("sum_grads", launch_sum_outs(side, 2, y.M, y.io_elems, y.io_elems,
                                             c->dtype == TNT_BF16, st));
    }
  }
  const int bf = c->dtype == TNT_BF16;
  if (fk) {
    // helper stream, last: the last local memory's dW_init reduction (its walk is done)
    const int i = c->n_local - 1, m = c->has_global + i;
    HIP_TIMED("reduce_init", launch_reduce_init((float*)(ws + y.b_dWl[i]), c->B, c->H, c->L / c->S_L[i],
                               2 * y.hd, dW1 + (size_t)m * c->H * y.hd,
                               dW2 + (size_t)m * c->H * y.hd, c->d, c->hid, 0, st));
    HIP_TRY(hipEventRecord(fk->e1, fk->side));
    st = main_st;
    HIP_TRY(hipStreamWaitEvent(main_st, fk->eg, 0));
    if (gate_deferred) {
      // every other memory's dk part is final: the gate pass writes dk itself
      LocalBwdArgs a = last_local;
      a.dk_out = dk;
      a.dk_parts = dkp;
      a.dk_stride = y.io_elems;
      a.dk_nparts = y.M;
      a.dk_self = c->has_global + c->n_local - 1;
      HIP_TIMED("local_bwd_gate", launch_local_bwd_gate(a, y.l_units[c->n_local - 1], st));
    } else {
      SumJobs mainj{};
      mainj.parts[0] = dkp; mainj.out[0] = dk;
      HIP_TIMED("sum_grads", launch_sum_outs(mainj, 1, y.M, y.io_elems, y.io_elems, bf, st));
    }
    HIP_TRY(hipStreamWaitEvent(main_st, fk->e1, 0));
    return TNT_OK;
  }
  st = main_st;
  SumJobs jobs{};
  jobs.parts[0] = dqp; jobs.out[0] = dq;
  jobs.parts[1] = dkp; jobs.out[1] = dk;
  jobs.parts[2] = dvp; jobs.out[2] = dv;
  HIP_TIMED("sum_grads", launch_sum_outs(jobs, 3, y.M, y.io_elems, y.io_elems, bf, st));
  return TNT_OK;
}

}  // namespace

namespace tnt {
int section_begin(const char* name, hipStream_t st) {
  if (!g_timing.on || g_timing.rec.size() >= TIMING_CAP) return -1;
  TimedLaunch t{name, g_timing.get(), g_timing.get()};
  if (!t.a || !t.b) return -1;
  if (hipEventRecord(t.a, st) != hipSuccess) return -1;
  g_timing.rec.push_back(t);
  return (int)g_timing.rec.size() - 1;
}

void section_end(int handle, hipStream_t st) {
  if (handle >= 0 && handle < (int)g_timing.rec.size()) hipEventRecord(g_timing.rec[handle].b, st);
}
}  // namespace tnt

extern "C" {

int32_t tnt_abi_version(void) { return 2; }

int32_t tnt_set_kernel_family(int32_t family) {
  if (family < TNT_FAMILY_DEFAULT || family > TNT_FAMILY_SINGLE_WALK) return -1;
  return g_family.exchange(family);
}

int32_t tnt_timing_enable(int32_t on) {
  const int32_t prev = g_timing.on ? 1 : 0;
  g_timing.on = on != 0;
  return prev;
}

int32_t tnt_timing_read(int32_t max, char* names, double* total_ms, int32_t* launches) {
  std::vector<std::string> keys;
  std::vector<double> ms;
  std::vector<int32_t> cnt;
  int32_t status = 0;
  for (const TimedLaunch& t : g_timing.rec) {
    float e = 0.f;
    if (hipEventSynchronize(t.b) != hipSuccess || hipEventElapsedTime(&e, t.a, t.b) != hipSuccess)
      status = -1;
    size_t i = 0;
    while (i < keys.size() && keys[i] != t.name) ++i;
    if (i == keys.size()) {
      keys.emplace_back(t.name);
      ms.push_back(0.0);
      cnt.push_back(0);
    }
    ms[i] += e;
    cnt[i] += 1;
    g_timing.pool.push_back(t.a);
    g_timing.pool.push_back(t.b);
  }
  g_timing.rec.clear();
  if (status) return status;
  const int32_t n = std::min<int32_t>(max, (int32_t)keys.size());
  for (int32_t i = 0; i < n; ++i) {
    if (names) {
      std::strncpy(names + 32 * i, keys[i].c_str(), 31);
      names[32 * i + 31] = 0;
    }
    if (total_ms) total_ms[i] = ms[i];
    if (launches) launches[i] = cnt[i];
  }
  return n;
}

const char* tnt_strerror(tnt_status s) {
  switch (s) {
    case TNT_OK: return "ok";
    case TNT_ERR_NULL: return "null pointer";
    case TNT_ERR_SHAPE: return "invalid shape or divisibility";
    case TNT_ERR_UNSUPPORTED: return "unsupported size";
    case TNT_ERR_WORKSPACE: return "workspace too small";
    case TNT_ERR_ALIGN: return "pointer not 16-byte aligned";
    case TNT_ERR_HIP: return "HIP runtime error";
    case TNT_ERR_ARG: return "invalid enum argument";
  }
  return "unknown status";
}

size_t tnt_mem_workspace_size(const tnt_config* cfg, int kind) {
  if (validate(cfg) != TNT_OK) return 0;
  const Eff E = effective(cfg);
  const Layout y = layout_of(&E.c, E.gsub);
  if (kind == TNT_WS_FWD) return y.fwd_two_bytes;
  if (kind == TNT_WS_FWD_MIN) return y.fwd_bytes;
  if (kind == TNT_WS_BWD) return y.bwd_bytes;
  if (kind == TNT_WS_BWD_RECOMPUTE) return y.bwd_re_bytes;
  return 0;
}

size_t tnt_mem_saved_size(const tnt_config* cfg) {
  if (validate(cfg) != TNT_OK) return 0;
  const Eff E = effective(cfg);
  return layout_of(&E.c, E.gsub).saved_bytes;
}

tnt_status tnt_mem_fwd(const tnt_config* cfg, const void* q, const void* k, const void* v,
                       const float* lr, const float* mom, const float* decay,
                       const float* W1_init, const float* W2_init, void* o, float* final_state,
                       void* saved, size_t saved_bytes, void* workspace, size_t ws_bytes,
                       void* stream) {
  return tnt::forward_entry(cfg, q, k, v, lr, mom, decay, W1_init, W2_init, o, final_state,
                            saved, saved_bytes, workspace, ws_bytes, true, (hipStream_t)stream);
}
}  // extern "C"

namespace tnt {
tnt_status forward_entry(const tnt_config* cfg, const void* q, const void* k, const void* v,
                         const float* lr, const float* mom, const float* decay,
                         const float* W1_init, const float* W2_init, void* o,
                         float* final_state, void* saved, size_t saved_bytes, void* workspace,
                         size_t ws_bytes, bool fork, hipStream_t stream) {
  tnt_status s = validate(cfg);
  if (s != TNT_OK) return s;
  if (!q || !k || !v || !lr || !mom || !decay || !W1_init || !W2_init || !o || !workspace)
    return TNT_ERR_NULL;
  if (final_state && !cfg->has_global) return TNT_ERR_SHAPE;
  for (const void* p : {(const void*)q, (const void*)k, (const void*)v, (const void*)lr,
                        (const void*)mom, (const void*)decay, (const void*)W1_init,
                        (const void*)W2_init, (const void*)o, (const void*)final_state,
                        (const void*)saved, (const void*)workspace})
    if (p && misaligned(p)) return TNT_ERR_ALIGN;
  const Eff E = effective(cfg);
  const Layout y = layout_of(&E.c, E.gsub);
  if (ws_bytes < y.fwd_bytes) return TNT_ERR_WORKSPACE;
  if (saved && saved_bytes < y.saved_bytes) return TNT_ERR_WORKSPACE;
  const SavedHeader hdr = header_of(cfg, y);
  s = run_forward(&E.c, y, q, k, v, lr, mom, decay, W1_init, W2_init, o, final_state,
                  (char*)saved, (char*)workspace, stream, fork, ws_bytes);
  if (s != TNT_OK || !saved) return s;
  if (launch_write_header(saved, hdr, stream) != hipSuccess) return TNT_ERR_HIP;
  remember_saved(saved, hdr);
  return TNT_OK;
}
}  // namespace tnt

extern "C" {

tnt_status tnt_mem_bwd(const tnt_config* cfg, const void* q, const void* k, const void* v,
                       const float* lr, const float* mom, const float* decay,
                       const float* W1_init, const float* W2_init, const void* dO,
                       const void* saved, size_t saved_bytes, void* dq, void* dk, void* dv,
                       float* dlr, float* dmom, float* ddecay, float* dW1_init,
                       float* dW2_init, void* workspace, size_t ws_bytes, void* stream) {
  tnt_status s = validate(cfg);
  if (s != TNT_OK) return s;
  if (!q || !k || !v || !lr || !mom || !decay || !W1_init || !W2_init || !dO || !dq || !dk ||
      !dv || !dlr || !dmom || !ddecay || !dW1_init || !dW2_init || !workspace)
    return TNT_ERR_NULL;
  for (const void* p : {(const void*)q, (const void*)k, (const void*)v, (const void*)lr,
                        (const void*)mom, (const void*)decay, (const void*)W1_init,
                        (const void*)W2_init, (const void*)dO, (const void*)saved,
                        (const void*)dq, (const void*)dk, (const void*)dv, (const void*)dlr,
                        (const void*)dmom, (const void*)ddecay, (const void*)dW1_init,
                        (const void*)dW2_init, (const void*)workspace})
    if (p && misaligned(p)) return TNT_ERR_ALIGN;
  const Eff E = effective(cfg);
  const Layout y = layout_of(&E.c, E.gsub);
  if (ws_bytes < (saved ? y.bwd_bytes : y.bwd_re_bytes)) return TNT_ERR_WORKSPACE;
  if (saved) {
    // the buffer must hold what a forward of this very configuration and
    // kernel family wrote (its layout and which slots were written depend on both)
    SavedHeader rec{};
    if (!recorded_saved(saved, &rec) || !same_header(rec, header_of(cfg, y))) return TNT_ERR_ARG;
    if (saved_bytes < y.saved_bytes) return TNT_ERR_WORKSPACE;
  }
  char* ws = (char*)workspace;
  char* sv = saved ? (char*)saved : ws + y.b_states;
  hipStream_t st = (hipStream_t)stream;
  if (!saved) {
    s = run_forward(&E.c, y, q, k, v, lr, mom, decay, W1_init, W2_init, nullptr, nullptr, sv, ws,
                    st);
    if (s != TNT_OK) return s;
  }
  return run_backward(&E.c, y, q, k, v, lr, mom, decay, W1_init, W2_init, dO, sv, dq, dk, dv,
                      dlr, dmom, ddecay, dW1_init, dW2_init, ws, st);
}

size_t tnt_mem_state_size(const tnt_config* cfg) {
  if (validate(cfg, false) != TNT_OK) return 0;
  const size_t M = (size_t)cfg->has_global + cfg->n_local;
  return M * cfg->B * cfg->H *
         (step_state_floats(cfg->d, cfg->hid) + step_scratch_floats(cfg->d, cfg->hid)) *
         sizeof(float);
}

}  // extern "C"

namespace {
StepArgs step_args(const tnt_config* c) {
  static_assert(1 + TNT_MAX_LOCAL <= (int)(sizeof(StepArgs::C) / sizeof(int)), "StepArgs::C");
  StepArgs a{};
  a.B = c->B; a.H = c->H; a.d = c->d; a.hid = c->hid;
  a.M = c->has_global + c->n_local;
  a.has_global = c->has_global; a.act = c->act; a.qk_proj = c->qk_proj;
  a.qk_scope = c->qk_scope; a.bf16 = c->dtype == TNT_BF16;
  int m = 0;
  if (c->has_global) { a.C[m] = c->C_G; a.S[m] = 0; ++m; }
  for (int i = 0; i < c->n_local; ++i, ++m) { a.C[m] = c->C_L[i]; a.S[m] = c->S_L[i]; }
  a.mem_stride = step_state_floats(c->d, c->hid);
  a.HS = c->hid < 64 ? c->hid : 64;
  a.G = c->hid / a.HS;
  a.sc_stride = step_scratch_floats(c->d, c->hid);
  return a;
}
}  // namespace

extern "C" {

tnt_status tnt_mem_state_init(const tnt_config* cfg, const float* W1_init, const float* W2_init,
                              void* state, void* stream) {
  tnt_status s = validate(cfg, false);
  if (s != TNT_OK) return s;
  if (!W1_init || !W2_init || !state) return TNT_ERR_NULL;
  for (const void* p : {(const void*)W1_init, (const void*)W2_init, (const void*)state})
    if (misaligned(p)) return TNT_ERR_ALIGN;
  StepArgs a = step_args(cfg);
  a.W1i = W1_init; a.W2i = W2_init; a.state = (float*)state;
  return launch_step_init(a, (hipStream_t)stream) == hipSuccess ? TNT_OK : TNT_ERR_HIP;
}

tnt_status tnt_dbg_chunk_grads(const tnt_config* cfg, int32_t b, int32_t h, int32_t t0,
                               int32_t C, const void* k, const void* v, const float* W1,
                               const float* W2, float* Zk, float* R, float* D1, void* stream) {
  tnt_status s = validate(cfg);
  if (s != TNT_OK) return s;
  if (b < 0 || b >= cfg->B || h < 0 || h >= cfg->H || t0 < 0 || C < 1 || C > 64 ||
      t0 > cfg->L - C)
    return TNT_ERR_SHAPE;
  if (!k || !v || !W1 || !W2 || !Zk || !R || !D1) return TNT_ERR_NULL;
  for (const void* p : {(const void*)k, (const void*)v, (const void*)W1, (const void*)W2,
                        (const void*)Zk, (const void*)R, (const void*)D1})
    if (misaligned(p)) return TNT_ERR_ALIGN;
  DbgArgs a{};
  a.d = cfg->d; a.hid = cfg->hid; a.C = C; a.act = cfg->act; a.bf16 = cfg->dtype == TNT_BF16;
  a.tok0 = ((size_t)b * cfg->H + h) * cfg->L + t0;
  a.k = k; a.v = v; a.W1 = W1; a.W2 = W2; a.Zk = Zk; a.R = R; a.D1 = D1;
  return launch_dbg_chunk_grads(a, (hipStream_t)stream) == hipSuccess ? TNT_OK : TNT_ERR_HIP;
}

tnt_status tnt_mem_state_from_fwd(const tnt_config* cfg, const float* final_state,
                                  const float* W1_init, const float* W2_init, void* state,
                                  void* stream) {
  tnt_status s = validate(cfg);  // L: the prefix the forward ran over
  if (s != TNT_OK) return s;
  if (cfg->has_global && cfg->global_intra) return TNT_ERR_UNSUPPORTED;
  if (!W1_init || !W2_init || !state || (cfg->has_global && !final_state)) return TNT_ERR_NULL;
  for (const void* p : {(const void*)W1_init, (const void*)W2_init, (const void*)state,
                        (const void*)final_state})
    if (p && misaligned(p)) return TNT_ERR_ALIGN;
  StepArgs a = step_args(cfg);
  a.W1i = W1_init; a.W2i = W2_init; a.state = (float*)state;
  a.scratch = a.state + (size_t)a.M * a.B * a.H * a.mem_stride;
  return launch_step_from_final(a, final_state, (hipStream_t)stream) == hipSuccess ? TNT_OK
                                                                                   : TNT_ERR_HIP;
}

tnt_status tnt_mem_step(const tnt_config* cfg, int64_t pos, int32_t T, const void* q,
                        const void* k, const void* v, const float* lr, const float* mom,
                        const float* decay, const float* W1_init, const float* W2_init,
                        void* state, void* o, void* stream) {
  tnt_status s = validate(cfg, false);
  if (s != TNT_OK) return s;
  if (pos < 0 || T < 0) return TNT_ERR_SHAPE;
  if (T == 0) return TNT_OK;
  if (!q || !k || !v || !lr || !mom || !decay || !W1_init || !W2_init || !state || !o)
    return TNT_ERR_NULL;
  for (const void* p : {(const void*)q, (const void*)k, (const void*)v, (const void*)lr,
                        (const void*)mom, (const void*)decay, (const void*)W1_init,
                        (const void*)W2_init, (const void*)state, (const void*)o})
    if (misaligned(p)) return TNT_ERR_ALIGN;
  StepArgs a = step_args(cfg);
  a.T = T; a.pos = pos;
  a.q = q; a.k = k; a.v = v; a.lr = lr; a.mom = mom; a.decay = decay;
  a.W1i = W1_init; a.W2i = W2_init; a.state = (float*)state; a.o = o;
  a.scratch = a.state + (size_t)a.M * a.B * a.H * a.mem_stride;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = timed("step", st, [&]() { return launch_step(a, st); });
  return e == hipSuccess ? TNT_OK : TNT_ERR_HIP;
}

}  // extern "C"
