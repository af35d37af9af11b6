/*
 * tnt.h -- C ABI of the TNT hierarchical memory layer (forward and backward)
 * on one AMD Instinct MI355X (gfx950).
 *
 * Method: "TNT: Improving Chunkwise Training for Test-Time Memorization"
 * (arXiv 2511.07343).  One layer holds one global deep memory (Sec. 4.1.1,
 * global update equation; App. E) updated in chunks of C_G tokens, and
 * n_local local deep memories (Sec. 4.1.1, local update equation; App. E),
 * each updated in chunks of C_L[i] tokens and reset to its learned initial
 * state every S_L[i] tokens.  Every memory is the MLP f(W, x) = W2 s(W1 x)
 * (W1: hid x d, W2: d x hid, s = GELU or SiLU) trained at test time by
 * gradient steps on the recall loss (1/d) ||f(W, k_t) - v_t||^2, the mean
 * squared error of Sec. 2.1.  All
 * gradients of a chunk are taken at the chunk-entry weights (Sec. 2.2) and
 * accumulated with momentum and decay (App. D):
 *     S_t = mom_t * S_{t-1} - lr_t * u_t,     W_t = (1 - decay_t) * W_{t-1} + S_t.
 * The output is o_t = f(V_{xi(t,C_G)}, q_t) + sum_i f(W^(i)_t, M^(i)_t q_t)
 * (Sec. 4.1.2 retrieval box; App. E), where V_{xi(t,C_G)} is the global state
 * entering t's chunk and M^(i)_t = sum over tau in [shard start, t] of
 * k_tau k_tau^T / ||k_tau||^2 is the Q-K projection (Sec. 4.1.2; App. C).
 *
 * Conventions shared by every entry point
 *  - All tensor pointers are DEVICE pointers owned by the caller.  The
 *    library never allocates, frees or synchronises; all work is enqueued on
 *    `stream` (a hipStream_t; NULL = the default stream) and the call returns
 *    after the enqueue.  Outputs and gradients are overwritten, never
 *    accumulated.
 *  - Layouts are contiguous row-major:
 *      q, k, v, o, dO, dq, dk, dv : [B][H][L][d]         (dtype: fp32 or bf16)
 *      lr, mom, decay (and grads) : [M][B][H][L]         (fp32)  eta, beta, alpha
 *      W1_init, dW1_init          : [M][H][hid][d]       (fp32)
 *      W2_init, dW2_init          : [M][H][d][hid]       (fp32)
 *      final_state                : [B][H][4][hid*d]     (fp32) V1 [hid][d], V2 [d][hid],
 *                                                        S1 [hid][d], S2 [d][hid]
 *    with M = has_global + n_local memories; memory 0 is the global memory
 *    when has_global, local memory i is memory has_global + i.  The initial
 *    weights are per memory and per head, shared by every batch row and every
 *    shard; their gradients are summed over both.
 *  - Every pointer must be 16-byte aligned (TNT_ERR_ALIGN otherwise).
 *  - Validation happens before anything is enqueued; a failing call enqueues
 *    nothing.  Asynchronous faults surface at the caller's synchronisation.
 *  - Gates: mom must lie in (0, 1] and decay in [0, 1); logarithms of mom are
 *    clamped at -80, so mom below e^-80 acts as e^-80.
 *  - The global memory's chunk chain runs on a helper stream that the library
 *    creates (default priority) on first use for each device, forked from and
 *    joined back into `stream` with events, so it overlaps the local memories;
 *    local memories after the first run on a second such stream.
 *    Calls from several host threads serialise their enqueue on a lock; calls
 *    on different streams with distinct workspaces may run concurrently.
 *  - tnt_mem_fwd and tnt_mem_bwd can be captured into a HIP graph on `stream`
 *    (they enqueue no memset or copy; the fork and join become graph edges) and
 *    replayed while the buffers they were captured with stay allocated.
 */
#ifndef TNT_H_
#define TNT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TNT_OK = 0,
  TNT_ERR_NULL = 1,        /* a required pointer is NULL                      */
  TNT_ERR_SHAPE = 2,       /* non-positive size or a divisibility rule broken */
  TNT_ERR_UNSUPPORTED = 3, /* size outside what the kernels are built for     */
  TNT_ERR_WORKSPACE = 4,   /* workspace smaller than tnt_mem_workspace_size   */
  TNT_ERR_ALIGN = 5,       /* pointer not 16-byte aligned                     */
  TNT_ERR_HIP = 6,         /* the HIP runtime reported an error at launch     */
  TNT_ERR_ARG = 7          /* an enum field holds an unknown value            */
} tnt_status;

typedef enum { TNT_F32 = 0, TNT_BF16 = 1 } tnt_dtype;       /* dtype of q,k,v,o and their grads */
typedef enum { TNT_GELU = 0, TNT_SILU = 1 } tnt_act;         /* GELU = exact erf form            */
typedef enum { TNT_QK_SHARD = 0, TNT_QK_CHUNK = 1 } tnt_qk_scope;

#define TNT_MAX_LOCAL 4

typedef struct {
  int32_t B, H, L, d, hid; /* batch, heads, sequence length, head dim, MLP hidden width    */
  int32_t has_global;      /* 1: global memory present (memory 0); 0: locals only          */
  int32_t C_G;             /* global chunk size; L % C_G == 0                              */
  int32_t n_local;         /* number of local memories, 0..TNT_MAX_LOCAL                   */
  int32_t C_L[TNT_MAX_LOCAL]; /* local chunk sizes; S_L[i] % C_L[i] == 0                   */
  int32_t S_L[TNT_MAX_LOCAL]; /* local shard lengths (reset period); L % S_L[i] == 0       */
  int32_t act;             /* tnt_act                                                      */
  int32_t qk_proj;         /* 1: query the locals at M_t q_t (Sec. 4.1.2); 0: at q_t       */
  int32_t qk_scope;        /* TNT_QK_SHARD: M_t sums from the shard start (App. C);
                              TNT_QK_CHUNK: from the chunk start (retrieval box literal)    */
  int32_t dtype;           /* tnt_dtype of q, k, v, o, dO, dq, dk, dv                      */
  int32_t global_intra;    /* retrieval of the global memory: 0 = at the chunk-entry state
                              V_xi (Sec. 4.1.2 retrieval box; App. E); 1 = at V_t after
                              token t's own update, the chunkwise retrieval rule of
                              Sec. 2.2 applied to the global memory (gradients still at
                              the chunk-entry state).  Ignored without a global memory.    */
} tnt_config;

/* Supported sizes: d in {16, 32, 64, 128}, hid in {16, 32, 64, 128, 256, 512},
 * C_L in {1..64} (rounded up internally to a multiple of 16 when below 16 is
 * not a multiple), C_G any divisor of L with C_G >= 1, B*H >= 1. */

/* Which workspace to size. */
typedef enum {
  TNT_WS_FWD = 0,          /* tnt_mem_fwd                                       */
  TNT_WS_BWD = 1,          /* tnt_mem_bwd given the forward's saved buffer     */
  TNT_WS_BWD_RECOMPUTE = 2,/* tnt_mem_bwd with saved == NULL                   */
  TNT_WS_FWD_MIN = 3       /* the least tnt_mem_fwd accepts: with saved == NULL
                              and less than TNT_WS_FWD, each local memory's
                              forward runs as one walk per shard instead of the
                              walk plus the chunk-parallel retrieval (same
                              results to rounding, slower)                      */
} tnt_ws_kind;

/* Bytes of device workspace the call needs (0 if the config is invalid). */
size_t tnt_mem_workspace_size(const tnt_config* cfg, int kind);

/* Kernel families.  TNT_FAMILY_DEFAULT takes the fixed-size kernels where a
 * shape has them (the local backward in three passes); TNT_FAMILY_GENERIC
 * runs every shape on the runtime-sized kernels; TNT_FAMILY_SINGLE_WALK keeps
 * the fixed-size local backward in one reverse walk per unit.  All three
 * compute the same function (to rounding); the non-default ones exist to test
 * one family against another.  The family is process-wide. */
typedef enum {
  TNT_FAMILY_DEFAULT = 0,
  TNT_FAMILY_GENERIC = 1,
  TNT_FAMILY_SINGLE_WALK = 2
} tnt_kernel_family;

/* Selects the kernel family of later calls; returns the previous one, or -1
 * (nothing changed) for an unknown value.  Sizes (tnt_mem_saved_size,
 * tnt_mem_workspace_size) depend on the family: size buffers after choosing
 * it.  A saved buffer can only be used by a tnt_mem_bwd under the family (and
 * configuration) of the tnt_mem_fwd that wrote it (TNT_ERR_ARG otherwise). */
int32_t tnt_set_kernel_family(int32_t family);

/* Bytes of the optional saved-state buffer: a header, then the chunk-entry
 * states of every memory (fp32, plus transposed copies of the local memories'
 * states in the compute type) and, for the local shapes whose backward runs
 * chunk-parallel, the forward records, written by tnt_mem_fwd and read by
 * tnt_mem_bwd so that the backward does not recompute the forward.  Opaque
 * layout.  For those shapes the backward reads the local states only through
 * their compute-type copies, and only the forward walk's two-slot fp32 ring is
 * reserved for them (the runtime-sized and single-walk families keep every
 * fp32 slot).  The header records the configuration, the kernel family and
 * the layout; tnt_mem_fwd also keeps that record per buffer on the host, and
 * tnt_mem_bwd refuses (TNT_ERR_ARG, before enqueuing anything) a buffer that
 * no tnt_mem_fwd of this process wrote for the same configuration and family. */
size_t tnt_mem_saved_size(const tnt_config* cfg);

/* Forward pass: o = TNT layer output (see the file comment).
 *   final_state : may be NULL; else receives the global memory's (V1, V2, S1, S2)
 *                 after the last token (requires has_global).
 *   saved       : may be NULL; else saved_bytes >= tnt_mem_saved_size(cfg)
 *                 (TNT_ERR_WORKSPACE otherwise) that receive the header and the
 *                 chunk-entry states for a later tnt_mem_bwd.
 *   workspace   : ws_bytes >= tnt_mem_workspace_size(cfg, TNT_WS_FWD_MIN); with
 *                 saved == NULL, ws_bytes >= tnt_mem_workspace_size(cfg, TNT_WS_FWD)
 *                 lets the local memories take the two-pass forward. */
tnt_status tnt_mem_fwd(const tnt_config* cfg, const void* q, const void* k, const void* v,
                       const float* lr, const float* mom, const float* decay,
                       const float* W1_init, const float* W2_init, void* o,
                       float* final_state, void* saved, size_t saved_bytes, void* workspace,
                       size_t ws_bytes, void* stream);

/* Backward pass: gradients of sum(dO * o) with respect to every input of the
 * forward, exact (second-order terms through the inner gradient included).
 *   saved : the buffer filled by tnt_mem_fwd on the same inputs (same
 *           configuration and kernel family; TNT_ERR_ARG otherwise), or NULL to
 *           recompute the states (then ws_bytes must cover TNT_WS_BWD_RECOMPUTE).
 * dq, dk, dv have the I/O dtype; the others are fp32 in the layouts above. */
tnt_status tnt_mem_bwd(const tnt_config* cfg, const void* q, const void* k, const void* v,
                       const float* lr, const float* mom, const float* decay,
                       const float* W1_init, const float* W2_init, const void* dO,
                       const void* saved, size_t saved_bytes, void* dq, void* dk, void* dv,
                       float* dlr, float* dmom, float* ddecay, float* dW1_init,
                       float* dW2_init, void* workspace, size_t ws_bytes, void* stream);

/* ---- Forward pass without a caller-provided workspace --------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the forward
 * of tnt_mem_fwd with no workspace and no saved buffer arguments.  Its
 * workspace is a device array of TNT_NOALLOC_WORKSPACE_BYTES that the library
 * holds on each GPU it runs on from the first call there until the process
 * ends; configurations whose smallest forward workspace (tnt_mem_workspace_size(cfg,
 * TNT_WS_FWD_MIN)) is larger get TNT_ERR_WORKSPACE (the forward takes the faster
 * two-pass local path when TNT_WS_FWD also fits).  The call allocates nothing
 * (no hipMalloc / hipFree, no helper stream: every launch is on `stream`), and
 * the forward writes every part of that array it reads, so the previous
 * call's contents do not matter.  All calls on one GPU share the array: calls
 * that overlap on one GPU (other streams, other host threads) race, and the
 * caller must serialise them.  Results equal tnt_mem_fwd's (same kernels). */
#define TNT_NOALLOC_WORKSPACE_BYTES (128u << 20)
tnt_status tnt_mem_fwd_noalloc(const tnt_config* cfg, const void* q, const void* k,
                               const void* v, const float* lr, const float* mom,
                               const float* decay, const float* W1_init, const float* W2_init,
                               void* o, float* final_state, void* stream);

/* ---- Step-wise forward (prefill / decode) from a carried state ----------
 * Within a chunk every gradient is taken at the chunk-entry weights W^ and
 * folded in with momentum and decay (Sec. 2.2; App. D), so the chunkwise rule
 * runs token by token once W^ is carried beside the running weights:
 *     S_t = mom_t S_{t-1} - lr_t grad l(W^; k_t, v_t),  W_t = (1 - decay_t) W_{t-1} + S_t,
 * with W^ <- W at each chunk start.  The global memory answers f(V^, q_t)
 * (entry state, Sec. 4.1.2 retrieval box); a local memory resets (W^, W, S, M)
 * to (W_init, W_init, 0, 0) at each shard start and answers f(W_t, M_t q_t)
 * after the update (Sec. 4.1.1 local update, Sec. 4.1.2; App. C).  Feeding a
 * sequence through tnt_mem_step in pieces of any length gives, token for
 * token, the o of tnt_mem_fwd on the whole sequence (to rounding).  cfg->L is
 * ignored by these three calls (the sequence is open-ended); every other
 * field is validated as for tnt_mem_fwd.  The state is device memory owned by
 * the caller: per memory m and per (batch row, head) chain, fp32
 *     W^1 [hid][d], W^2 [d][hid], W1 [hid][d], W2 [d][hid], S1 [hid][d],
 *     S2 [d][hid], M [d][d]       (M unused for the global memory),
 * blocks ordered [M][B][H], followed by a scratch area of M*B*H blocks of
 * 2*hid + d + 3*G*d floats (G = hid / min(64, hid)), each rounded up to a
 * multiple of 64 floats, whose contents are undefined between calls.  Calls
 * on one state must be serialised (same stream).  Each token takes three
 * launches over (hidden-unit slice, chain, memory) workgroups; the work is
 * matrix-vector products and rank-one updates of the fp32 state. */

/* Bytes of the carried state (0 if the config is invalid). */
size_t tnt_mem_state_size(const tnt_config* cfg);

/* Sets `state` to the start of a sequence: every memory at its initial
 * weights (W^ = W = W_init of the chain's head), zero momenta and Q-K sums. */
tnt_status tnt_mem_state_init(const tnt_config* cfg, const float* W1_init,
                              const float* W2_init, void* state, void* stream);

/* Carried state after tnt_mem_fwd over a prefix of cfg->L tokens (a multiple
 * of C_G and of every S_L, as tnt_mem_fwd requires), for decoding on from
 * pos = cfg->L: the global memory takes the forward's final_state (V1, V2,
 * S1, S2; required when has_global), each local memory is set as by
 * tnt_mem_state_init (it resets at the next token, a shard start, anyway).
 * The chunk-parallel forward then serves as the prefill of tnt_mem_step. */
tnt_status tnt_mem_state_from_fwd(const tnt_config* cfg, const float* final_state,
                                  const float* W1_init, const float* W2_init, void* state,
                                  void* stream);

/* Forward over T >= 0 further tokens of every chain, advancing `state`.
 *   pos   : tokens `state` has consumed so far (0 after tnt_mem_state_init);
 *           chunk and shard boundaries are taken from pos + t.  A pos that
 *           does not match the state's history gives undefined outputs.
 *   q, k, v, o : [B][H][T][d] (I/O dtype);  lr, mom, decay : [M][B][H][T] fp32;
 *   W1_init, W2_init : as for tnt_mem_fwd (read at local shard starts).
 * T == 0 enqueues nothing.  TNT_ERR_SHAPE for pos < 0 or T < 0. */
tnt_status tnt_mem_step(const tnt_config* cfg, int64_t pos, int32_t T, const void* q,
                        const void* k, const void* v, const float* lr, const float* mom,
                        const float* decay, const float* W1_init, const float* W2_init,
                        void* state, void* o, void* stream);

/* Debug: the per-token quantities of one chunk's inner gradient (the chain
 * rule of the recall loss, Sec. 2.1; every token of the chunk at the same
 * weights, Sec. 2.2) for the chain (b, h), tokens [t0, t0 + C):
 *     Zk = K W1^T (C x hid),  R = (2/d) (s(Zk) W2^T - V) (C x d),
 *     D1 = (R W2) * s'(Zk) (C x hid),
 * so that token t's gradients are u1_t = D1_t^T k_t and u2_t = R_t^T s(Zk_t).
 *   k, v   : [B][H][L][d] as for tnt_mem_fwd (cfg->dtype);
 *   W1, W2 : [hid][d], [d][hid] fp32, the weights the gradients are taken at;
 *   Zk, D1 : [C][hid] fp32;  R : [C][d] fp32 (device, caller-owned).
 * 1 <= C <= 64 and t0 + C <= L (TNT_ERR_SHAPE otherwise).  fp32 arithmetic,
 * one workgroup: a check of the gradient math, not a fast path. */
tnt_status tnt_dbg_chunk_grads(const tnt_config* cfg, int32_t b, int32_t h, int32_t t0,
                               int32_t C, const void* k, const void* v, const float* W1,
                               const float* W2, float* Zk, float* R, float* D1, void* stream);

/* Human-readable name of a status code (static storage). */
const char* tnt_strerror(tnt_status status);

/* Version of this ABI (bumped on any incompatible change). */
int32_t tnt_abi_version(void);

/* Opt-in kernel timing, for benchmarks.  While enabled (on != 0), every
 * kernel launch of tnt_mem_fwd / tnt_mem_bwd / tnt_mem_step (and the
 * state-carry section of each global chunk step) is bracketed by a pair of
 * hipEvents recorded on the launch stream (at most 65536 launches are kept).
 * tnt_timing_read synchronises on the recorded events, writes one entry per
 * kernel name (names: 32-byte NUL-terminated slots; total_ms: summed event
 * time; launches: number of launches), clears the record, and returns the
 * number of entries (at most max), or -1 on a HIP error.  Not thread-safe:
 * use from one host thread while enabled.  Returns the previous setting. */
int32_t tnt_timing_enable(int32_t on);
int32_t tnt_timing_read(int32_t max, char* names, double* total_ms, int32_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* TNT_H_ */
