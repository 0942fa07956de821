// Host/device shared parameter blocks and launchers (internal to libpdn).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pdn {

constexpr int kChunk = 64;  // chunk length C

enum GateKind { kGateNone = 0, kGateScalar = 1, kGateChannel = 2 };
enum PrecondKind { kSquash = 0, kIdentity = 1, kExternal = 2 };

// Everything the forward kernels read or write.  Per-token tensors use the
// ABI layout [B, T, H, d]; workspace tensors are head-major and padded to
// whole chunks (T_pad = NT * C rows).
struct FwdArgs {
  int64_t B, T, H, BH;
  int NT;        // number of chunks, ceil(T / C)
  int64_t Tpad;  // NT * C
  int dk, dv;
  int gate, precond;
  float lnx;     // log(x)
  float scale;
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
  float* G;       // [BH, Tpad] or [BH, Tpad, dk] in-chunk log-decay prefix
};

struct WsLayout {
  size_t sumL, sumD, Abound, KtG, Tm, Pm, G, total;
};

WsLayout fwd_ws_layout(int64_t BH, int NT, int dk, int esz, int gate, int precond);

// ev: NULL or 4 events recorded at the stage boundaries (see
// pdn_chunk_fwd_events)
hipError_t launch_forward(const FwdArgs& a, int io_bf16, hipStream_t stream,
                          hipEvent_t const* ev = nullptr);

}  // namespace pdn
