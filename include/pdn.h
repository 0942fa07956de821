/*
 * pdn.h -- C ABI of the chunkwise preconditioned delta rule on MI355X (gfx950).
 *
 * Computes, for every batch b and head h independently, the recurrence of
 * "Preconditioned DeltaNet" (arXiv 2604.21100), Sec. 3.5, Eq. precond_end2end,
 * in its three instantiations (PDN: no decay; PGDN: scalar decay; PKDA:
 * per-key-channel decay -- the decayed forms of Sec. 3.5 and App. D):
 *
 *   A_t  = exp(gP_t) A_{t-1} + betaP_t (k_t * k_t)            diagonal key Gram
 *   r_t  = log(A_t) - exp(logAScale_h)
 *   B_t  = exp(-log(x) * r_t / (1 + |r_t|))                    in [1/x, x]
 *   kt_t = B_t * k_t                                           write key
 *   S_t  = alpha_t S_{t-1} + beta_t (v_t - alpha_t S_{t-1} k_t) kt_t^T
 *   o_t  = scale * S_t q_t
 *
 * with S_t in R^{dv x dk} (the paper's orientation), alpha_t = exp(g_t) a
 * scalar (PGDN) or a dk-vector acting as S Diag(alpha_t) (PKDA).  The library
 * evaluates it with the chunkwise-parallel form of Eq. chunkwise_atk_form /
 * App. D (UT transform T = (I + tril(Diag(beta) K Kt^T, -1))^{-1} Diag(beta),
 * W = T K, U = T V, inter-chunk state scan, chunk output).
 *
 * Conventions
 *   - Every tensor argument is a DEVICE pointer to dense row-major memory owned
 *     by the caller.  The library never allocates or frees device memory; all
 *     scratch lives in a caller-provided workspace (pdn_workspace_size), except
 *     for pdn_chunk_fwd_noalloc's fixed per-device array (see there).
 *   - Layouts: q, k, ktilde, dq, dk: [B, T, H, dk];  v, o, dO, dv: [B, T, H, dv];
 *     beta, betaP, gP and a scalar gate g: [B, T, H];  a per-channel gate g:
 *     [B, T, H, dk];  logAScale: [H];  A0, A_T: [B, H, dk];
 *     S0, S_T, dS_T, dS0: [B, H, dk, dv] holding S^T (the transpose of the
 *     paper's S), i.e. element (b, h, i, j) is S[j][i].
 *   - q, k, v, o, ktilde and their gradients use the problem's io dtype
 *     (IEEE fp32 or bfloat16); every other tensor is fp32.
 *   - Calls are asynchronous on the given HIP stream (a hipStream_t passed as
 *     void*; NULL = the null stream).  Inputs, outputs and workspace must stay
 *     valid until the stream work completes.
 *   - Errors: every argument is validated on the host BEFORE any HIP call;
 *     on a validation failure the function returns the first failing code
 *     and writes nothing.  A failed kernel launch returns PDN_ERR_HIP and
 *     leaves the outputs undefined.  Values are not inspected: NaN / Inf in
 *     the inputs propagate.  No exception, abort or printf crosses the ABI.
 *   - Apart from pdn_chunk_fwd_noalloc (which shares one fixed scratch array
 *     per device), the library keeps no mutable global state: calls are
 *     re-entrant and may run concurrently on different streams with
 *     distinct workspaces.
 */
#ifndef PDN_H
#define PDN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PDN_ABI_VERSION 5

typedef enum {
  PDN_OK = 0,
  PDN_ERR_NULL = 1,        /* a required pointer is NULL                       */
  PDN_ERR_SHAPE = 2,       /* B, T, H negative or sizes overflow               */
  PDN_ERR_DTYPE = 3,       /* unknown io dtype                                 */
  PDN_ERR_UNSUPPORTED = 4, /* dk, dv or chunk outside the built kernels (dk, dv
                              in {64, 128}, chunk in {32, 64}), or a mode
                              the entry point does not cover                 */
  PDN_ERR_ALIGN = 5,       /* a tensor is not 16-byte aligned                  */
  PDN_ERR_ALIAS = 6,       /* an output overlaps an input or another output    */
  PDN_ERR_WORKSPACE = 7,   /* workspace NULL, too small or misaligned          */
  PDN_ERR_VALUE = 8,       /* bad scalar (x < 1, non-finite x/scale, ridge <= 0
                              for DIAG_SM / ATQ) or enum (knorm other than
                              NONE without SQUASH), or a gate pointer
                              inconsistent with the gate kind               */
  PDN_ERR_HIP = 9,         /* a HIP launch failed                              */
  PDN_ERR_SCRATCH = 10     /* pdn_chunk_fwd_noalloc: the problem's workspace
                              exceeds PDN_NOALLOC_SCRATCH_BYTES              */
} pdn_status;

typedef enum { PDN_F32 = 0, PDN_BF16 = 1 } pdn_dtype;

typedef enum {
  PDN_GATE_NONE = 0,    /* PDN:  alpha_t = 1                        */
  PDN_GATE_SCALAR = 1,  /* PGDN: alpha_t = exp(g_t), g [B,T,H]      */
  PDN_GATE_CHANNEL = 2  /* PKDA: alpha_t = exp(g_t), g [B,T,H,dk]   */
} pdn_gate;

/* Admissible per-channel decay (PDN_GATE_CHANNEL).  Inside a chunk the
 * decay between tokens t <= r of one channel, exp(G_r - G_t) with G the
 * in-chunk prefix sum of that channel's g, is applied as the product of two
 * fp32 factors split at a reference row of each 16-token block (forward
 * interaction matrices and the backward's intra-chunk products).  One of
 * the two is the exponential of up to 15 consecutive log-decays with the
 * sign flipped, so every run of 15 consecutive g of a channel must sum to
 * more than -87 (a mean log-decay above -5.8 per token, alpha above 0.003);
 * below that the factor overflows and outputs and gradients hold Inf / NaN.
 * Nothing checks the range.  The scalar gate has no such limit.           */

typedef enum {
  PDN_PRECOND_SQUASH = 0,   /* write key of Eq. precond_end2end (the method) */
  PDN_PRECOND_IDENTITY = 1, /* kt = k: plain DeltaNet / GDN / KDA            */
  PDN_PRECOND_EXTERNAL = 2, /* kt supplied by the caller in `ktilde`         */
  /* Unstable ATK (App. D, "ATK (unstable) preconditioner recurrence"; the
   * Sherman-Morrison form of Sec. 3.4): with the same A recurrence and
   * P_t = Diag(A_{t-1} + ridge)^{-1} (the state BEFORE token t),
   *   kt_t = P_t k_t / (1 + k_t^T P_t k_t)
   * and the delta rule above.  Forward only.                               */
  PDN_PRECOND_DIAG_SM = 3,
  /* Preconditioned linear attention, apply-to-query (Sec. 3.3 chunkwise PLA
   * form; App. D, "ATQ preconditioner recurrence"; P-Mamba-2 with a scalar
   * gate, PGLA with a per-channel gate): no delta rule,
   *   S_t = alpha_t S_{t-1} + beta_t v_t k_t^T
   *   o_t = scale * S_t (q_t / (A_t + ridge))          (A_t: current state)
   * ktilde is unused (write key = read key).  Forward only.                */
  PDN_PRECOND_ATQ = 4
} pdn_precond;

/* Normalisation factor on the SQUASH write key (the ablation of App. E,
 * "Stable parameterization", table of normalisation factors): with
 * m_t = k_t^T B_t k_t,
 *   kt_t = B_t k_t * { 1 | 1 / m_t | 1 / (1 + m_t) | beta_t / (alpha_t + beta_t m_t) }
 * alpha_t = exp(g_t) for a scalar gate, 1 without a gate.  NONE is the
 * method; the others are forward only, SQUASH only, and BETA is not
 * defined for a per-channel gate (PDN_ERR_UNSUPPORTED).                    */
typedef enum {
  PDN_KNORM_NONE = 0,
  PDN_KNORM_M = 1,      /* 1 / m_t                                          */
  PDN_KNORM_1PM = 2,    /* 1 / (1 + m_t)                                    */
  PDN_KNORM_BETA = 3    /* beta_t / (alpha_t + beta_t m_t)                  */
} pdn_knorm;

typedef struct {
  int64_t B, T, H;     /* batch, sequence length, heads; 0 is allowed      */
  int32_t dk, dv;      /* head dims: each 64 or 128                         */
  int32_t chunk;       /* chunk length C: 32 or 64 (the paper's form for
                          any C; results differ only by rounding)        */
  pdn_dtype io;        /* dtype of q, k, v, o, ktilde and their gradients   */
  pdn_gate gate;
  pdn_precond precond;
  float x;             /* squash range [1/x, x]; x >= 1 (paper: 1.5)        */
  float scale;         /* output scale (paper: 1.0)                         */
  float ridge;         /* DIAG_SM and ATQ: the ridge lambda > 0 added to A
                          before the elementwise inverse; ignored otherwise */
  pdn_knorm knorm;     /* SQUASH write-key normalisation; NONE otherwise    */
} pdn_problem;

typedef struct {
  const void* q;             /* [B,T,H,dk] io                                */
  const void* k;             /* [B,T,H,dk] io  (read key)                    */
  const void* v;             /* [B,T,H,dv] io                                */
  const float* beta;         /* [B,T,H]                                      */
  const float* g;            /* NULL for GATE_NONE, else [B,T,H] / [B,T,H,dk] */
  const float* beta_p;       /* [B,T,H]; SQUASH, DIAG_SM, ATQ               */
  const float* g_p;          /* [B,T,H] or NULL (alpha^P = 1); as beta_p     */
  const float* log_a_scale;  /* [H]; mu_h = exp(.); SQUASH only              */
  const float* A0;           /* [B,H,dk] or NULL (= 0); as beta_p            */
  const float* S0;           /* [B,H,dk,dv] (S^T) or NULL (= 0)              */
  const void* ktilde;        /* [B,T,H,dk] io; EXTERNAL only                 */
} pdn_inputs;

typedef struct {
  void* o;      /* [B,T,H,dv] io                                             */
  float* S_T;   /* [B,H,dk,dv] final state S_T^T, or NULL                    */
  float* A_T;   /* [B,H,dk] final preconditioner state, or NULL (SQUASH,
                   DIAG_SM, ATQ)                                             */
} pdn_fwd_out;

typedef struct {
  void* dq;              /* [B,T,H,dk] io                                    */
  void* dk;              /* [B,T,H,dk] io                                    */
  void* dv;              /* [B,T,H,dv] io                                    */
  float* dbeta;          /* [B,T,H]                                          */
  float* dg;             /* [B,T,H] / [B,T,H,dk]; NULL iff GATE_NONE         */
  float* dS0;            /* [B,H,dk,dv] or NULL                              */
  float* dbeta_p;        /* [B,T,H] or NULL (SQUASH)                         */
  float* dg_p;           /* [B,T,H] or NULL (SQUASH)                         */
  float* dlog_a_scale;   /* [H] or NULL (SQUASH)                             */
  float* dA0;            /* [B,H,dk] or NULL (SQUASH)                        */
  void* dktilde;         /* [B,T,H,dk] io, EXTERNAL only, or NULL            */
} pdn_bwd_out;

/* Bytes of workspace pdn_chunk_fwd (with_bwd = 0) or pdn_chunk_bwd
 * (with_bwd = 1) needs for this problem.  Host-only, no HIP call.
 * Returns PDN_ERR_NULL / SHAPE / DTYPE / UNSUPPORTED / VALUE for a bad
 * problem; *bytes is written only on PDN_OK. */
pdn_status pdn_workspace_size(const pdn_problem* problem, int with_bwd,
                              size_t* bytes);

/* Number of sequence segments the forward state scan of this problem runs
 * in (1: one pass over the chunks).  A scan workgroup holds one head's
 * 32-column state slab on one compute unit, so with few heads (B * H *
 * dv / 32 far below the 256 compute units of MI355X) most of the chip
 * would idle.  The chunks are then cut into S >= 3 segments: segment 0
 * runs from S0 while every middle segment runs from zero and, with its
 * values zeroed, from the identity (giving its d_k x d_k transition Phi,
 * S_end^T = Phi S_start^T + local end, the chunkwise recurrence being
 * affine in the state); the exact start of each segment is composed from
 * those, and segments 1 .. S - 1 run again from it.  The result is the same
 * recurrence up to fp32 rounding.  S depends only on the problem's sizes,
 * as does the workspace (which holds the segment states).  Host-only, no
 * HIP call; errors as pdn_workspace_size. */
pdn_status pdn_scan_segments(const pdn_problem* problem, int* segments);

/* Forward pass (Eq. chunkwise_atk_form with the preconditioner of Eq.
 * precond_end2end; decayed forms of App. D).  Writes o and, when non-NULL,
 * S_T and A_T.  `ws` must be 256-byte aligned and at least
 * pdn_workspace_size(problem, 0) bytes.  Asynchronous on `hip_stream`. */
pdn_status pdn_chunk_fwd(const pdn_problem* problem, const pdn_inputs* in,
                         pdn_fwd_out* out, void* ws, size_t ws_bytes,
                         void* hip_stream);

/* pdn_chunk_fwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It computes exactly what pdn_chunk_fwd
 * computes, with the same kernels, using as its workspace a fixed scratch
 * array of PDN_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds in
 * every device it runs on, from the library's loading on that device until
 * the process ends.  It calls no hipMalloc / hipFree or other allocating
 * routine; its first call on a device looks up that device's array once.
 *
 * Limit: pdn_workspace_size(problem, 0, &n) must give n <=
 * PDN_NOALLOC_SCRATCH_BYTES, else PDN_ERR_SCRATCH (returned, like every
 * other validation failure, before any HIP call).  For example, bf16 with
 * d_k = d_v = 128 and a scalar gate needs about 0.53 KB per token-head:
 * B*T*H up to about 120k (B=1, T=8192, H=14).
 *
 * Sharing: every call on one device uses that device's single array, which
 * keeps the last call's contents (the forward overwrites every byte it reads
 * before reading it, so nothing needs clearing).  Calls that overlap in time
 * on one device -- on different streams, or from different host threads
 * without ordering -- race on the array and give undefined results; order
 * them on one stream.  Arguments, outputs and errors otherwise as
 * pdn_chunk_fwd. */
#define PDN_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
pdn_status pdn_chunk_fwd_noalloc(const pdn_problem* problem, const pdn_inputs* in,
                                 pdn_fwd_out* out, void* hip_stream);

/* PDN_NOALLOC_SCRATCH_BYTES of the built library. */
size_t pdn_noalloc_scratch_bytes(void);

/* pdn_chunk_fwd that also records caller-created HIP events (hipEvent_t
 * handles passed as void*) on `hip_stream` at the stage boundaries, for
 * timing individual kernels:
 *   stage_events[0]  before the preconditioner scan (k1_*; empty unless
 *                    SQUASH)
 *   stage_events[1]  after it / before the per-chunk prep kernel (k2)
 *   stage_events[2]  after k2 / before the inter-chunk scan + output (k3)
 *   stage_events[3]  after k3
 * n_events must be 4 (else PDN_ERR_VALUE); a NULL entry is not recorded
 * (each record costs a few microseconds of GPU time between kernels, so a
 * caller timing one stage passes only its two boundaries).  The events stay
 * owned by the caller; results are identical to pdn_chunk_fwd. */
#define PDN_FWD_STAGE_EVENTS 4
pdn_status pdn_chunk_fwd_events(const pdn_problem* problem, const pdn_inputs* in,
                                pdn_fwd_out* out, void* ws, size_t ws_bytes,
                                void* hip_stream, void* const* stage_events,
                                int n_events);

/* Backward pass: gradients of <dO, o> + <dS_T, S_T> with respect to every
 * input of pdn_chunk_fwd (App. C, backward pseudocode).  dO is [B,T,H,dv]
 * io; dS_T is [B,H,dk,dv] fp32 or NULL (= 0).  The forward intermediates are
 * recomputed; `ws` must hold pdn_workspace_size(problem, 1) bytes.  The
 * output pointers dbeta_p, dg_p, dlog_a_scale, dA0 and dS0 may be NULL to
 * skip them.  SQUASH, IDENTITY and EXTERNAL only (DIAG_SM, ATQ:
 * PDN_ERR_UNSUPPORTED), and knorm NONE only. */
pdn_status pdn_chunk_bwd(const pdn_problem* problem, const pdn_inputs* in,
                         const void* dO, const float* dS_T, pdn_bwd_out* out,
                         void* ws, size_t ws_bytes, void* hip_stream);

/* pdn_chunk_bwd that also records caller-created HIP events on `hip_stream`
 * at its stage boundaries (n_events must be PDN_BWD_STAGE_EVENTS):
 *   [0] start  [1] after the preconditioner recompute (k1_*)
 *   [2] after the per-chunk prep recompute (k2, backward mode)
 *   [3] after the state-saving forward scan (k3)
 *   [4] after the reverse state-adjoint scan (r1)
 *   [5] after the per-chunk adjoints and gradients (p12)
 *   [6] after the preconditioner's reverse scan (pc_*) or the key combine
 * NULL entries are not recorded.  Results are identical to pdn_chunk_bwd. */
#define PDN_BWD_STAGE_EVENTS 7
pdn_status pdn_chunk_bwd_events(const pdn_problem* problem, const pdn_inputs* in,
                                const void* dO, const float* dS_T, pdn_bwd_out* out,
                                void* ws, size_t ws_bytes, void* hip_stream,
                                void* const* stage_events, int n_events);

/* Training pair.  pdn_chunk_fwd_train computes exactly what pdn_chunk_fwd
 * computes and also leaves in `ws` the forward intermediates the backward
 * reads (per-chunk solve factors, chunk-start states, the X and E rows, the
 * write-key rows, ...), so that pdn_chunk_bwd_train can skip the
 * recompute of the forward that pdn_chunk_bwd performs.  This trades memory
 * for time: `ws` must hold at least pdn_workspace_size(problem, 1, &bytes) bytes
 * (the backward's workspace) for both calls.
 *
 * Contract: pdn_chunk_bwd_train must receive the same problem, the same
 * input pointers with unchanged contents and the same `ws` as the preceding
 * pdn_chunk_fwd_train, with no other call writing `ws` in between (the
 * library cannot detect a violation; results are then undefined, but every
 * access stays inside the declared buffers).  pdn_chunk_bwd_train leaves the
 * saved intermediates intact, so it may be called again for another dO.
 * The backward's restrictions apply to both calls (fp32 io only with
 * d_k = d_v = 64; no DIAG_SM or ATQ; knorm NONE: PDN_ERR_UNSUPPORTED).
 *
 * stage_events: NULL with n_events = 0, or PDN_FWD_STAGE_EVENTS /
 * PDN_BWD_STAGE_EVENTS caller-created events recorded as in the _events
 * variants (the backward's recompute stages are then empty). */
pdn_status pdn_chunk_fwd_train(const pdn_problem* problem, const pdn_inputs* in,
                               pdn_fwd_out* out, void* ws, size_t ws_bytes,
                               void* hip_stream, void* const* stage_events,
                               int n_events);
pdn_status pdn_chunk_bwd_train(const pdn_problem* problem, const pdn_inputs* in,
                               const void* dO, const float* dS_T, pdn_bwd_out* out,
                               void* ws, size_t ws_bytes, void* hip_stream,
                               void* const* stage_events, int n_events);

/* Static, NUL-terminated description of a status code. */
const char* pdn_status_string(pdn_status status);

/* PDN_ABI_VERSION of the built library. */
int pdn_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PDN_H */
