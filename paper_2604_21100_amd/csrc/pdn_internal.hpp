// Host/device shared parameter blocks and launchers (internal to libpdn).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pdn {

// chunk lengths C the kernels are built for
constexpr bool chunk_supported(int c) { return c == 32 || c == 64; }

enum GateKind { kGateNone = 0, kGateScalar = 1, kGateChannel = 2 };
enum PrecondKind { kSquash = 0, kIdentity = 1, kExternal = 2, kDiagSM = 3, kATQ = 4 };
enum KnormKind { kKnormNone = 0, kKnormM = 1, kKnorm1pm = 2, kKnormBeta = 3 };

// the write key (or, for ATQ, the query) comes from the diagonal Gram
// recurrence A_t = exp(gP_t) A_{t-1} + betaP_t k_t^2
constexpr bool has_gram(int precond) {
  return precond == kSquash || precond == kDiagSM || precond == kATQ;
}

// Everything the forward kernels read or write.  Per-token tensors use the
// ABI layout [B, T, H, d]; workspace tensors are head-major and padded to
// whole chunks (T_pad = NT * C rows).
struct FwdArgs {
  int64_t B, T, H, BH;
  int chunk;     // chunk length C (32 or 64)
  int NT;        // number of chunks, ceil(T / C)
  int64_t Tpad;  // NT * C
  int dk, dv;
  int gate, precond;
  float lnx;     // log(x)
  float scale;
  float ridge;   // DIAG_SM / ATQ: lambda added to A before the inverse
  int knorm;     // SQUASH write-key normalisation (pdn_knorm)
  // inputs
  const void* q;
  const void* k;
  const void* v;
  const void* ktilde;
  const float* beta;
  const float* g;
  const float* beta_p;
  const float* g_p;
  const float* log_a_scale;
  const float* A0;
  const float* S0;
  // outputs
  void* o;
  float* S_T;
  float* A_T;
  // workspace
  float* sumL;    // [BH, NT, dk]   in-chunk decayed sum of betaP k^2
  float* sumD;    // [BH, NT]       in-chunk sum of gP (log of the decay)
  float* Abound;  // [BH, NT+1, dk] preconditioner state before each chunk
  void* KtG;      // [BH, NT, dk, C] (Kt * Gamma)^T per chunk, io dtype
  void* Tm;       // [BH, NT, C, C]  T = (I + At)^{-1} Diag(beta), io dtype
  void* Pm;       // [BH, NT, C, C]  causal (Q*Lam)(Kt/Lam)^T, io dtype
  float* G;       // scalar gate: [BH, Tpad] in-chunk log-decay prefix; per-channel
                  // gate: [BH, NT, dk], its chunk-end row only
  void* Qt;       // [BH, Tpad, dk] io   ATQ: preconditioned query rows q / (A + ridge)
  void* QL;       // [BH, Tpad, dk] io   per-channel gate: Lam o (the query the scan reads)
  void* KL;       // [BH, Tpad, dk] io   per-channel gate: Lam o K
  // backward only (NULL in the forward): forward intermediates kept for the
  // adjoint kernels.  lam_r = exp(G_r), w_r = exp(G_{C-1} - G_r).
  void* Hs;       // [BH, NT, dk, dv] io  chunk-start states S^T
  void* Er;       // [BH, Tpad, dv] io    E = T X rows
  void* PtT;      // [BH, NT, C, C] io    P^T
  void* MtT;      // [BH, NT, C, C] io    M^T, M = (I + At)^{-1} (T = M Diag(beta))
  void* Ktr;      // [BH, Tpad, dk] io    write key rows
  void* Kw;       // [BH, Tpad, dk] io    w_r o write key rows (per-channel gate; else NULL)
  void* QlT;      // [BH, NT, dk, C] io   (Diag(lam) Q)^T per chunk
  void* KnT;      // [BH, NT, dk, C] io   -(Diag(lam) K)^T per chunk
  // sequence split of the state scan (see scan_split): seg_phase 0 = one
  // pass over all chunks from S0; 1 = segment 0 from S0 next to the local
  // scans (from zero) and transitions (from the identity, no values) of the
  // middle segments; 3 = segments 1 .. seg_cnt - 1 from seg_start
  int seg_phase, seg_len, seg_cnt;
  float* seg_end;    // [S, BH, dk, dv] phase-1 end states (segment 0: exact; others: local)
  float* seg_phi;    // [S, BH, dk, dk] segment transitions, S_end^T = Phi S_start^T + local
  float* seg_start;  // [S, BH, dk, dv] exact start states of segments 1 .. S - 1
};

// Sequence split of the state scan.  A scan workgroup holds one head's
// 32-column state slab (one per compute unit); with few heads most of the
// chip idles through the sequential chunk loop.  The chunks are then cut
// into S segments of L: segment 0 runs from S0 while each middle segment
// runs from zero (its local end state) and, on d_k / 32 more workgroups,
// from the identity with the values zeroed (its d_k x d_k transition); a
// short sequential pass composes the exact start of every segment, and
// segments 1 .. S - 1 run again from it.  The critical path drops from NT
// steps to about 2 NT / S; S is the largest count whose first pass still
// fits one workgroup per compute unit of the target device, with at least
// kSegMinChunks chunks per segment.
constexpr int kScanCUs = 256;       // compute units of MI355X
constexpr int kSegMinChunks = 4;
constexpr int kSegMax = 16;
struct ScanSplit {
  int S, L;   // segments (1: no split) and chunks per segment
};
inline ScanSplit scan_split(int64_t BH, int NT, int dk, int dv) {
  const int64_t ns = dv / 32, np = dk / 32;
  ScanSplit r{1, NT};
  for (int s = 3; s <= kSegMax; ++s) {
    if (BH * (ns + (s - 2) * (ns + np)) > kScanCUs) break;
    const int L = (NT + s - 1) / s;
    if (L < kSegMinChunks) break;
    r.S = (NT + L - 1) / L;
    r.L = L;
  }
  if (r.S < 3) r = ScanSplit{1, NT};
  return r;
}

// Backward-only arguments and workspace (the forward recompute uses f).
struct BwdArgs {
  FwdArgs f;
  const void* dO;       // [B, T, H, dv] io
  const float* dS_T;    // [B, H, dk, dv] or NULL
  // outputs
  void* dq;
  void* dk;
  void* dv;
  float* dbeta;
  float* dg;
  float* dS0;
  float* dbeta_p;
  float* dg_p;
  float* dlog_a_scale;
  float* dA0;
  void* dktilde;
  // workspace
  void* dHs;      // [BH, NT, dk, dv] io  state adjoint entering each chunk from the right
  void* Zr;       // [BH, Tpad, dv] io    Z = M^T dE rows (dX = dV = Diag(beta) Z)
  void* dKt;      // [BH, Tpad, dk] io    gradient of the write key
  void* dKm;      // [BH, Tpad, dk] io    gradient of the read key (main recurrence)
  float* pcL;     // [BH, NT, dk]         preconditioner: in-chunk adjoint at chunk start
  float* pcS;     // [BH, NT, C/16, dk]   preconditioner: per 16-token segment, the in-segment adjoint it sends left
  float* pcA;     // [BH, NT, C/16, dk]   preconditioner: per 16-token segment, the state before it
  float* pcC;     // [BH, NT + 1, dk]     preconditioner: adjoint carried into each chunk
  float* pcMu;    // [BH, NT]             preconditioner: partial d mu
};

// The composition pass of a split scan (seg_compose): the exact segment
// starts from the first pass's end states and transitions, forward or (rev)
// for the reverse state-adjoint scan.
hipError_t launch_seg_compose(const FwdArgs& a, bool rev, hipStream_t s);

struct WsLayout {
  size_t sumL, sumD, Abound, KtG, Tm, Pm, G, Qt, QL, KL, seg_end, seg_phi, seg_start, total;
  ScanSplit split;
};

WsLayout fwd_ws_layout(int64_t BH, int NT, int dk, int dv, int esz, int gate, int precond, int C);

struct BwdWsLayout {
  WsLayout f;
  size_t Hs, Er, PtT, MtT, Ktr, Kw, QlT, KnT;
  size_t dHs, Zr, dKt, dKm, pcL, pcS, pcA, pcC, pcMu, total;
};

BwdWsLayout bwd_ws_layout(int64_t BH, int NT, int dk, int dv, int esz, int gate, int precond, int C);

// ev: NULL or 8 events recorded at the stage boundaries (see
// pdn_chunk_bwd_events).  recompute = false: the forward intermediates are
// already in the workspace (left there by the training forward).
hipError_t launch_backward(const BwdArgs& a, int io_bf16, hipStream_t stream,
                           hipEvent_t const* ev = nullptr, bool recompute = true);

// Fixed scratch of pdn_chunk_fwd_noalloc (PDN_NOALLOC_SCRATCH_BYTES): a
// static device array in pdn_fwd.hip, one copy per device.
constexpr size_t kNoallocScratchBytes = static_cast<size_t>(64) << 20;
constexpr int kNoallocMaxDevices = 64;

// Device address of the current device's scratch array, looked up with
// hipGetSymbolAddress on the first call made with that device current and
// cached per device (thread-safe).  Fails for device ids >= 64.
hipError_t noalloc_scratch(void** ptr);

// ev: NULL or 4 events recorded at the stage boundaries (see
// pdn_chunk_fwd_events).  train: also leave the backward's intermediates in
// the workspace (a's backward fields set).
hipError_t launch_forward(const FwdArgs& a, int io_bf16, hipStream_t stream,
                          hipEvent_t const* ev = nullptr, bool train = false);

}  // namespace pdn
