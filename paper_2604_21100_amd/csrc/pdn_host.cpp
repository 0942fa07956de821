// C ABI of libpdn: argument validation (host only, before any HIP call),
// workspace sizing and kernel sequencing.  See include/pdn.h.
#include "../../include/pdn.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <vector>

#include "pdn_internal.hpp"

namespace {


static_assert(PDN_NOALLOC_SCRATCH_BYTES == pdn::kNoallocScratchBytes,
              "the header's scratch size and the library's must agree");

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

bool overlap(const Range& a, const Range& b) {
  return a.lo < b.hi && b.lo < a.hi;
}

// checked multiply of non-negative sizes
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

struct Sizes {
  int64_t BH, NT, tok;        // tok = B*T*H
  int64_t nq, nv, nscal, ngate, nS, nA;
  int esz;
};

pdn_status check_problem(const pdn_problem* p, Sizes* sz) {
  if (!p) return PDN_ERR_NULL;
  if (p->B < 0 || p->T < 0 || p->H < 0) return PDN_ERR_SHAPE;
  if (p->io != PDN_F32 && p->io != PDN_BF16) return PDN_ERR_DTYPE;
  if ((p->dk != 64 && p->dk != 128) || (p->dv != 64 && p->dv != 128)) return PDN_ERR_UNSUPPORTED;
  if (!pdn::chunk_supported(p->chunk)) return PDN_ERR_UNSUPPORTED;
  if (p->gate != PDN_GATE_NONE && p->gate != PDN_GATE_SCALAR && p->gate != PDN_GATE_CHANNEL)
    return PDN_ERR_VALUE;
  if (p->precond != PDN_PRECOND_SQUASH && p->precond != PDN_PRECOND_IDENTITY &&
      p->precond != PDN_PRECOND_EXTERNAL && p->precond != PDN_PRECOND_DIAG_SM &&
      p->precond != PDN_PRECOND_ATQ)
    return PDN_ERR_VALUE;
  if (!std::isfinite(p->x) || !(p->x >= 1.0f) || !std::isfinite(p->scale)) return PDN_ERR_VALUE;
  if ((p->precond == PDN_PRECOND_DIAG_SM || p->precond == PDN_PRECOND_ATQ) &&
      (!std::isfinite(p->ridge) || !(p->ridge > 0.0f)))
    return PDN_ERR_VALUE;
  if (p->knorm < PDN_KNORM_NONE || p->knorm > PDN_KNORM_BETA) return PDN_ERR_VALUE;
  if (p->knorm != PDN_KNORM_NONE && p->precond != PDN_PRECOND_SQUASH) return PDN_ERR_VALUE;
  if (p->knorm == PDN_KNORM_BETA && p->gate == PDN_GATE_CHANNEL) return PDN_ERR_UNSUPPORTED;
  Sizes s{};
  int64_t bt;
  if (!mul_ok(p->B, p->H, &s.BH) || !mul_ok(p->B, p->T, &bt) || !mul_ok(bt, p->H, &s.tok))
    return PDN_ERR_SHAPE;
  s.NT = (p->T + p->chunk - 1) / p->chunk;
  int64_t tpad;
  if (!mul_ok(s.NT, p->chunk, &tpad)) return PDN_ERR_SHAPE;
  // every element count used below must fit in int64 (with a generous margin
  // for the workspace's byte counts)
  int64_t tmp;
  if (!mul_ok(s.tok, 128, &s.nq) || !mul_ok(s.BH, tpad, &tmp) || !mul_ok(tmp, 128 * 8, &tmp) ||
      !mul_ok(s.BH, 128 * 128 * 4, &tmp))
    return PDN_ERR_SHAPE;
  if (s.NT > (int64_t)1 << 30 || s.BH * s.NT > (int64_t)INT32_MAX) return PDN_ERR_SHAPE;
  s.nq = s.tok * p->dk;
  s.nv = s.tok * p->dv;
  s.nscal = s.tok;
  s.ngate = p->gate == PDN_GATE_NONE ? 0 : (p->gate == PDN_GATE_SCALAR ? s.tok : s.tok * p->dk);
  s.nS = s.BH * p->dk * p->dv;
  s.nA = s.BH * p->dk;
  s.esz = p->io == PDN_BF16 ? 2 : 4;
  *sz = s;
  return PDN_OK;
}

Range rng(const void* p, int64_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Range{a, a + static_cast<uintptr_t>(bytes)};
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Buf {
  const void* p;
  int64_t bytes;
};

// outputs must not overlap inputs, each other or the workspace; the workspace
// must not overlap inputs
pdn_status check_aliasing(const std::vector<Buf>& ins, const std::vector<Buf>& outs, Buf ws) {
  for (size_t i = 0; i < outs.size(); ++i) {
    if (!outs[i].p || outs[i].bytes == 0) continue;
    const Range ro = rng(outs[i].p, outs[i].bytes);
    for (const Buf& in : ins)
      if (in.p && in.bytes && overlap(ro, rng(in.p, in.bytes))) return PDN_ERR_ALIAS;
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (outs[j].p && outs[j].bytes && overlap(ro, rng(outs[j].p, outs[j].bytes))) return PDN_ERR_ALIAS;
    if (ws.p && ws.bytes && overlap(ro, rng(ws.p, ws.bytes))) return PDN_ERR_ALIAS;
  }
  if (ws.p && ws.bytes)
    for (const Buf& in : ins)
      if (in.p && in.bytes && overlap(rng(ws.p, ws.bytes), rng(in.p, in.bytes))) return PDN_ERR_ALIAS;
  return PDN_OK;
}

pdn_status check_inputs(const pdn_problem* p, const pdn_inputs* in, const Sizes& s,
                        std::vector<Buf>* bufs) {
  if (!in) return PDN_ERR_NULL;
  const bool empty = s.tok == 0;
  // per-token tensors are only dereferenced when there are tokens
  if (!empty) {
    if (!in->q || !in->k || !in->v || !in->beta) return PDN_ERR_NULL;
    if (p->gate != PDN_GATE_NONE && !in->g) return PDN_ERR_NULL;
    if (pdn::has_gram(p->precond) && !in->beta_p) return PDN_ERR_NULL;
    if (p->precond == PDN_PRECOND_SQUASH && !in->log_a_scale) return PDN_ERR_NULL;
    if (p->precond == PDN_PRECOND_EXTERNAL && !in->ktilde) return PDN_ERR_NULL;
  }
  if (p->gate == PDN_GATE_NONE && in->g) return PDN_ERR_VALUE;
  const int64_t e = s.esz;
  std::vector<Buf> b = {
      {in->q, s.nq * e}, {in->k, s.nq * e}, {in->v, s.nv * e}, {in->beta, s.nscal * 4},
      {in->g, s.ngate * 4}, {in->S0, s.nS * 4},
  };
  if (pdn::has_gram(p->precond)) {
    b.push_back({in->beta_p, s.nscal * 4});
    b.push_back({in->g_p, s.nscal * 4});
    b.push_back({in->A0, s.nA * 4});
  }
  if (p->precond == PDN_PRECOND_SQUASH) b.push_back({in->log_a_scale, p->H * 4});
  if (p->precond == PDN_PRECOND_EXTERNAL) b.push_back({in->ktilde, s.nq * e});
  for (const Buf& x : b)
    if (x.p && !aligned16(x.p)) return PDN_ERR_ALIGN;
  *bufs = b;
  return PDN_OK;
}

// the backward covers every gate kind and the SQUASH / IDENTITY / EXTERNAL
// write keys; fp32 io at head dims 64
pdn_status check_bwd_support(const pdn_problem* p) {
  if (p->io == PDN_F32 && (p->dk != 64 || p->dv != 64)) return PDN_ERR_UNSUPPORTED;
  if (p->precond == PDN_PRECOND_DIAG_SM || p->precond == PDN_PRECOND_ATQ) return PDN_ERR_UNSUPPORTED;
  if (p->knorm != PDN_KNORM_NONE) return PDN_ERR_UNSUPPORTED;
  return PDN_OK;
}

}  // namespace

extern "C" {

const char* pdn_status_string(pdn_status st) {
  switch (st) {
    case PDN_OK: return "ok";
    case PDN_ERR_NULL: return "a required pointer is NULL";
    case PDN_ERR_SHAPE: return "invalid or overflowing shape";
    case PDN_ERR_DTYPE: return "unknown io dtype";
    case PDN_ERR_UNSUPPORTED: return "head dimension, chunk size or mode not supported (dk, dv in {64, 128}; chunk 32 or 64)";
    case PDN_ERR_ALIGN: return "a tensor is not 16-byte aligned";
    case PDN_ERR_ALIAS: return "an output overlaps an input, another output or the workspace";
    case PDN_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case PDN_ERR_VALUE: return "invalid scalar, enum or gate pointer";
    case PDN_ERR_HIP: return "HIP launch failed";
    case PDN_ERR_SCRATCH:
      return "problem needs more workspace than the no-allocation entry point's fixed scratch "
             "(pdn_noalloc_scratch_bytes(), 64 MiB per device)";
  }
  return "unknown status";
}

int pdn_abi_version(void) { return PDN_ABI_VERSION; }

pdn_status pdn_workspace_size(const pdn_problem* p, int with_bwd, size_t* bytes) {
  if (!bytes) return PDN_ERR_NULL;
  Sizes s;
  const pdn_status st = check_problem(p, &s);
  if (st != PDN_OK) return st;
  if (with_bwd) {
    const pdn_status sb = check_bwd_support(p);
    if (sb != PDN_OK) return sb;
    *bytes = pdn::bwd_ws_layout(s.BH, static_cast<int>(s.NT), p->dk, p->dv, s.esz, p->gate, p->precond, p->chunk).total;
    return PDN_OK;
  }
  const pdn::WsLayout L = pdn::fwd_ws_layout(s.BH, static_cast<int>(s.NT), p->dk, p->dv, s.esz, p->gate,
                                             p->precond, p->chunk);
  *bytes = L.total;
  return PDN_OK;
}

pdn_status pdn_scan_segments(const pdn_problem* p, int* segments) {
  if (!segments) return PDN_ERR_NULL;
  Sizes s;
  const pdn_status st = check_problem(p, &s);
  if (st != PDN_OK) return st;
  *segments = s.tok > 0 ? pdn::scan_split(s.BH, static_cast<int>(s.NT), p->dk, p->dv).S : 1;
  return PDN_OK;
}

// Forward intermediates the backward kernels read: the forward workspace
// plus the residual arrays of the backward layout.
static void set_forward_ws(pdn::FwdArgs& a, const pdn::WsLayout& L, const pdn_problem* p, char* w) {
  if (p->precond == PDN_PRECOND_ATQ) a.Qt = w + L.Qt;
  if (p->gate == PDN_GATE_CHANNEL) {
    a.QL = w + L.QL;
    a.KL = w + L.KL;
  }
  if (pdn::has_gram(p->precond)) {
    a.sumL = reinterpret_cast<float*>(w + L.sumL);
    a.sumD = reinterpret_cast<float*>(w + L.sumD);
    a.Abound = reinterpret_cast<float*>(w + L.Abound);
  }
  a.KtG = w + L.KtG;
  a.Tm = w + L.Tm;
  a.Pm = w + L.Pm;
  if (p->gate != PDN_GATE_NONE) a.G = reinterpret_cast<float*>(w + L.G);
  if (L.split.S > 1) {
    a.seg_cnt = L.split.S;
    a.seg_len = L.split.L;
    a.seg_end = reinterpret_cast<float*>(w + L.seg_end);
    a.seg_phi = reinterpret_cast<float*>(w + L.seg_phi);
    a.seg_start = reinterpret_cast<float*>(w + L.seg_start);
  }
}

static void set_residuals(pdn::FwdArgs& f, const pdn::BwdWsLayout& L, char* w) {
  f.Hs = w + L.Hs; f.Er = w + L.Er; f.PtT = w + L.PtT; f.MtT = w + L.MtT;
  f.Ktr = w + L.Ktr; f.Kw = L.Kw ? w + L.Kw : nullptr; f.QlT = w + L.QlT; f.KnT = w + L.KnT;
}

// train: the training forward (also leaves the backward's intermediates in
// the workspace, which then has the backward's size).  noalloc: ws and
// ws_bytes are ignored; the workspace is the device's fixed scratch array,
// looked up only after every argument has been validated.
static pdn_status chunk_fwd_impl(const pdn_problem* p, const pdn_inputs* in, pdn_fwd_out* out,
                                 void* ws, size_t ws_bytes, void* hip_stream,
                                 hipEvent_t const* ev, bool train, bool noalloc = false) {
  Sizes s;
  pdn_status st = check_problem(p, &s);
  if (st != PDN_OK) return st;
  std::vector<Buf> ins;
  if ((st = check_inputs(p, in, s, &ins)) != PDN_OK) return st;
  if (train && (st = check_bwd_support(p)) != PDN_OK) return st;
  if (!out) return PDN_ERR_NULL;
  if (s.tok > 0 && !out->o) return PDN_ERR_NULL;
  if (!pdn::has_gram(p->precond) && out->A_T) return PDN_ERR_VALUE;
  const std::vector<Buf> outs = {{out->o, s.nv * s.esz}, {out->S_T, s.nS * 4}, {out->A_T, s.nA * 4}};
  for (const Buf& x : outs)
    if (x.p && !aligned16(x.p)) return PDN_ERR_ALIGN;
  const pdn::WsLayout L = pdn::fwd_ws_layout(s.BH, static_cast<int>(s.NT), p->dk, p->dv, s.esz, p->gate,
                                             p->precond, p->chunk);
  const pdn::BwdWsLayout LB =
      pdn::bwd_ws_layout(s.BH, static_cast<int>(s.NT), p->dk, p->dv, s.esz, p->gate, p->precond, p->chunk);
  const size_t need_bytes = train ? LB.total : L.total;
  const bool need_ws = s.tok > 0;
  if (noalloc) {
    ws = nullptr;
    ws_bytes = 0;
    if (need_ws && need_bytes > pdn::kNoallocScratchBytes) return PDN_ERR_SCRATCH;
  }
  // the whole declared workspace range must be disjoint from inputs/outputs;
  // its size is checked last
  if ((st = check_aliasing(ins, outs, Buf{ws, need_ws ? static_cast<int64_t>(ws_bytes) : 0})) != PDN_OK)
    return st;
  if (noalloc && need_ws) {
    // every argument is valid: the first HIP call of this entry point (the
    // scratch array belongs to the library, so it overlaps no caller buffer)
    if (pdn::noalloc_scratch(&ws) != hipSuccess) return PDN_ERR_HIP;
    ws_bytes = pdn::kNoallocScratchBytes;
  }
  if (need_ws && (!ws || ws_bytes < need_bytes || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0))
    return PDN_ERR_WORKSPACE;

  pdn::FwdArgs a{};
  a.B = p->B; a.T = p->T; a.H = p->H; a.BH = s.BH;
  a.chunk = p->chunk;
  a.NT = static_cast<int>(s.NT);
  a.Tpad = s.NT * p->chunk;
  a.dk = p->dk; a.dv = p->dv;
  a.gate = p->gate; a.precond = p->precond;
  a.lnx = std::log(p->x);
  a.scale = p->scale;
  a.ridge = p->ridge;
  a.knorm = p->knorm;
  a.q = in->q; a.k = in->k; a.v = in->v; a.ktilde = in->ktilde;
  a.beta = in->beta; a.g = in->g; a.beta_p = in->beta_p; a.g_p = in->g_p;
  a.log_a_scale = in->log_a_scale; a.A0 = in->A0; a.S0 = in->S0;
  a.o = out->o; a.S_T = out->S_T; a.A_T = out->A_T;
  char* w = static_cast<char*>(ws);
  if (need_ws) {
    set_forward_ws(a, train ? LB.f : L, p, w);
    if (train) set_residuals(a, LB, w);
  }
  const hipError_t e =
      pdn::launch_forward(a, p->io == PDN_BF16, static_cast<hipStream_t>(hip_stream), ev, train);
  return e == hipSuccess ? PDN_OK : PDN_ERR_HIP;
}

pdn_status pdn_chunk_fwd(const pdn_problem* p, const pdn_inputs* in, pdn_fwd_out* out, void* ws,
                         size_t ws_bytes, void* hip_stream) {
  return chunk_fwd_impl(p, in, out, ws, ws_bytes, hip_stream, nullptr, false);
}

pdn_status pdn_chunk_fwd_noalloc(const pdn_problem* p, const pdn_inputs* in, pdn_fwd_out* out,
                                 void* hip_stream) {
  return chunk_fwd_impl(p, in, out, nullptr, 0, hip_stream, nullptr, false, true);
}

size_t pdn_noalloc_scratch_bytes(void) { return pdn::kNoallocScratchBytes; }

pdn_status pdn_chunk_fwd_events(const pdn_problem* p, const pdn_inputs* in, pdn_fwd_out* out,
                                void* ws, size_t ws_bytes, void* hip_stream,
                                void* const* stage_events, int n_events) {
  if (!stage_events) return PDN_ERR_NULL;
  if (n_events != PDN_FWD_STAGE_EVENTS) return PDN_ERR_VALUE;
  return chunk_fwd_impl(p, in, out, ws, ws_bytes, hip_stream,
                        reinterpret_cast<hipEvent_t const*>(stage_events), false);
}

// saved: the forward intermediates are in ws already (training forward)
static pdn_status chunk_bwd_impl(const pdn_problem* p, const pdn_inputs* in, const void* dO,
                                 const float* dS_T, pdn_bwd_out* out, void* ws, size_t ws_bytes,
                                 void* hip_stream, hipEvent_t const* ev, bool saved) {
  Sizes s;
  pdn_status st = check_problem(p, &s);
  if (st != PDN_OK) return st;
  std::vector<Buf> ins;
  if ((st = check_inputs(p, in, s, &ins)) != PDN_OK) return st;
  if ((st = check_bwd_support(p)) != PDN_OK) return st;
  if (!out) return PDN_ERR_NULL;
  const bool tok = s.tok > 0;
  if (tok && (!dO || !out->dq || !out->dk || !out->dv || !out->dbeta)) return PDN_ERR_NULL;
  if (tok && p->gate != PDN_GATE_NONE && !out->dg) return PDN_ERR_NULL;
  if (p->gate == PDN_GATE_NONE && out->dg) return PDN_ERR_VALUE;
  const bool sq = p->precond == PDN_PRECOND_SQUASH;
  if (!sq && (out->dbeta_p || out->dg_p || out->dlog_a_scale || out->dA0)) return PDN_ERR_VALUE;
  if (p->precond != PDN_PRECOND_EXTERNAL && out->dktilde) return PDN_ERR_VALUE;
  ins.push_back({dO, s.nv * s.esz});
  ins.push_back({dS_T, s.nS * 4});
  const int64_t e = s.esz;
  const std::vector<Buf> outs = {
      {out->dq, s.nq * e},        {out->dk, s.nq * e},          {out->dv, s.nv * e},
      {out->dbeta, s.nscal * 4},  {out->dg, s.ngate * 4},       {out->dS0, s.nS * 4},
      {out->dbeta_p, s.nscal * 4}, {out->dg_p, s.nscal * 4},    {out->dlog_a_scale, p->H * 4},
      {out->dA0, s.nA * 4},       {out->dktilde, s.nq * e}};
  for (const Buf& x : outs)
    if (x.p && !aligned16(x.p)) return PDN_ERR_ALIGN;
  for (const Buf& x : ins)
    if (x.p && !aligned16(x.p)) return PDN_ERR_ALIGN;
  const pdn::BwdWsLayout L =
      pdn::bwd_ws_layout(s.BH, static_cast<int>(s.NT), p->dk, p->dv, s.esz, p->gate, p->precond, p->chunk);
  if ((st = check_aliasing(ins, outs, Buf{ws, tok ? static_cast<int64_t>(ws_bytes) : 0})) != PDN_OK)
    return st;
  if (tok && (!ws || ws_bytes < L.total || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0))
    return PDN_ERR_WORKSPACE;
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  if (s.BH == 0 || !tok) {
    if (ev)  // nothing to time: the stage events still mark the empty stages
      for (int k = 0; k < PDN_BWD_STAGE_EVENTS; ++k)
        if (ev[k] && hipEventRecord(ev[k], stream) != hipSuccess) return PDN_ERR_HIP;
  }
  if (s.BH == 0) return PDN_OK;
  if (!tok) {
    // T == 0: the state passes through unchanged
    pdn::FwdArgs f{};
    f.BH = s.BH; f.dk = p->dk; f.dv = p->dv;
    f.S0 = dS_T; f.S_T = out->dS0; f.A0 = nullptr; f.A_T = out->dA0;
    const hipError_t he = pdn::launch_forward(f, p->io == PDN_BF16, stream);
    return he == hipSuccess ? PDN_OK : PDN_ERR_HIP;
  }
  pdn::BwdArgs a{};
  pdn::FwdArgs& f = a.f;
  f.B = p->B; f.T = p->T; f.H = p->H; f.BH = s.BH;
  f.chunk = p->chunk;
  f.NT = static_cast<int>(s.NT);
  f.Tpad = s.NT * p->chunk;
  f.dk = p->dk; f.dv = p->dv;
  f.gate = p->gate; f.precond = p->precond;
  f.lnx = std::log(p->x);
  f.scale = p->scale;
  f.q = in->q; f.k = in->k; f.v = in->v; f.ktilde = in->ktilde;
  f.beta = in->beta; f.g = in->g; f.beta_p = in->beta_p; f.g_p = in->g_p;
  f.log_a_scale = in->log_a_scale; f.A0 = in->A0; f.S0 = in->S0;
  f.o = nullptr; f.S_T = nullptr; f.A_T = nullptr;
  char* w = static_cast<char*>(ws);
  set_forward_ws(f, L.f, p, w);
  set_residuals(f, L, w);
  a.dO = dO; a.dS_T = dS_T;
  a.dq = out->dq; a.dk = out->dk; a.dv = out->dv; a.dbeta = out->dbeta; a.dg = out->dg;
  a.dS0 = out->dS0; a.dbeta_p = out->dbeta_p; a.dg_p = out->dg_p; a.dlog_a_scale = out->dlog_a_scale;
  a.dA0 = out->dA0; a.dktilde = out->dktilde;
  a.dHs = w + L.dHs; a.Zr = w + L.Zr;
  a.dKt = w + L.dKt;
  a.dKm = w + L.dKm;
  a.pcL = reinterpret_cast<float*>(w + L.pcL);
  a.pcS = reinterpret_cast<float*>(w + L.pcS);
  a.pcA = reinterpret_cast<float*>(w + L.pcA);
  a.pcC = reinterpret_cast<float*>(w + L.pcC);
  a.pcMu = reinterpret_cast<float*>(w + L.pcMu);
  const hipError_t he = pdn::launch_backward(a, p->io == PDN_BF16, stream, ev, !saved);
  return he == hipSuccess ? PDN_OK : PDN_ERR_HIP;
}

pdn_status pdn_chunk_bwd(const pdn_problem* p, const pdn_inputs* in, const void* dO,
                         const float* dS_T, pdn_bwd_out* out, void* ws, size_t ws_bytes,
                         void* hip_stream) {
  return chunk_bwd_impl(p, in, dO, dS_T, out, ws, ws_bytes, hip_stream, nullptr, false);
}

pdn_status pdn_chunk_bwd_events(const pdn_problem* p, const pdn_inputs* in, const void* dO,
                                const float* dS_T, pdn_bwd_out* out, void* ws, size_t ws_bytes,
                                void* hip_stream, void* const* stage_events, int n_events) {
  if (!stage_events) return PDN_ERR_NULL;
  if (n_events != PDN_BWD_STAGE_EVENTS) return PDN_ERR_VALUE;
  return chunk_bwd_impl(p, in, dO, dS_T, out, ws, ws_bytes, hip_stream,
                        reinterpret_cast<hipEvent_t const*>(stage_events), false);
}

// stage_events: NULL (n_events 0) or an array of n_events == n entries
// (NULL entries are skipped)
static pdn_status check_events(void* const* ev, int n_events, int n) {
  if (!ev) return n_events == 0 ? PDN_OK : PDN_ERR_NULL;
  if (n_events != n) return PDN_ERR_VALUE;
  return PDN_OK;
}

pdn_status pdn_chunk_fwd_train(const pdn_problem* p, const pdn_inputs* in, pdn_fwd_out* out,
                               void* ws, size_t ws_bytes, void* hip_stream,
                               void* const* stage_events, int n_events) {
  const pdn_status st = check_events(stage_events, n_events, PDN_FWD_STAGE_EVENTS);
  if (st != PDN_OK) return st;
  return chunk_fwd_impl(p, in, out, ws, ws_bytes, hip_stream,
                        reinterpret_cast<hipEvent_t const*>(stage_events), true);
}

pdn_status pdn_chunk_bwd_train(const pdn_problem* p, const pdn_inputs* in, const void* dO,
                               const float* dS_T, pdn_bwd_out* out, void* ws, size_t ws_bytes,
                               void* hip_stream, void* const* stage_events, int n_events) {
  const pdn_status st = check_events(stage_events, n_events, PDN_BWD_STAGE_EVENTS);
  if (st != PDN_OK) return st;
  return chunk_bwd_impl(p, in, dO, dS_T, out, ws, ws_bytes, hip_stream,
                        reinterpret_cast<hipEvent_t const*>(stage_events), true);
}

}  // extern "C"
