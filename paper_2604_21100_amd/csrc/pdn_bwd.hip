// Backward kernels of the chunkwise preconditioned delta rule for gfx950
// (PDN, PGDN and PKDA: no gate, a scalar or a per-channel gate).
//
// The gradient is the exact adjoint of the chunkwise forward (Eq.
// chunkwise_atk_form with the decayed forms of App. D).  Per chunk, with
// lam_r = exp(G_r) (G the in-chunk prefix of the log-decay), w_r =
// exp(G_{C-1} - G_r), Gam_rt = exp(G_r - G_t) (r >= t), S^T the chunk-start
// state (dk x dv), M = (I + At)^{-1}, T = M Diag(beta):
//   X  = V - Diag(lam) K S^T            E = T X
//   O  = scale [ Diag(lam) Q S^T + (Gam o Q Kt^T)_causal E ]
//   S'^T = lam_C S^T + Kt^T Diag(w) E
//   At = strict_lower(Diag(beta) (Gam o K Kt^T))
// and the adjoint, given dO and dS'^T (the state adjoint from the right):
//   dE  = (Gam o Q Kt^T)_causal^T dO_s + Diag(w) Kt dS'^T      dO_s = scale dO
//   Z   = M^T dE                      dX = T^T dE = Diag(beta) Z,  dV = dX
//   dS^T = lam_C dS'^T + Q^T Diag(lam) dO_s - K^T Diag(lam) dX
//   dQ  = Diag(lam) dO_s S + dSqk Kt  dK = -Diag(lam) dX S + dSkk Kt
//   dKt = dSqk^T Q + Diag(w) E dS' + dSkk^T K
//   dSqk = Gam o (dO_s E^T)_causal
// The inverse's adjoint collapses: with dM = dE X^T Diag(beta) the gradient
// of L = (I + At)^{-1} is dL = -M^T dM M^T = -(M^T dE)(M Diag(beta) X)^T =
// -Z E^T, one C x C product of stored rows, so
//   dAt = strict_lower(-Z E^T),  dSkk = Gam o Diag(beta) dAt
//   dbeta_t = sum_v Z_tv X_tv + sum_{s<t} dAt_ts (Gam o K Kt^T)_ts
// with sum_v Z_tv X_tv = Z_t . V_t - lam_t K_t . (Z S)_t, where Z S is the
// product p2 forms anyway (dX S = Diag(beta) Z S), so X is never stored.
// plus the gate terms (gradients of lam, w, lam_C and Gam, reverse-summed
// over the chunk) and the preconditioner's reverse scan.
//
//   r1_state_adjoint   sequential over chunks (reverse): dS^T carry, dE, Z,
//                      dX (= dv)
//   p12_chunk_grads    per chunk: the C x C adjoints (dSqk, dSkk), dq, the
//                      read- and write-key gradients, dbeta, dg
//   p12c_chunk_grads   the same for the per-channel gate (decay inside the
//                      key contractions; dg per channel)
//   pc_*               preconditioner: reverse scan over tokens of the
//                      diagonal Gram recurrence (dk, dbetaP, dgP, dlogAScale,
//                      dA0)
#include "pdn_device.hpp"
#include "pdn_internal.hpp"

namespace pdn {

constexpr int BVB = 32;  // value columns per workgroup in the reverse scan

// Every kernel here takes the chunk length C (32 or 64) as a template
// parameter.  Wave w owns the chunk's row block w (16 tokens); at C = 32
// waves 2 and 3 skip the row work and take part in the column-wise and
// cooperative work only.  Guards written (NB == 4 || ...) are compile-time
// true at C = 64.

// A thread's share of a [NR rows] x BVB slab in 16-byte vectors: vector j
// of thread tid is idx = tid + 256 j (idx < kN), row idx / kSegs
template <typename T, int NR>
struct Slab {
  static constexpr int kVec = 16 / static_cast<int>(sizeof(T));
  static constexpr int kSegs = BVB / kVec;
  static constexpr int kN = NR * kSegs;
  static constexpr int kPer = (kN + 255) / 256;
  static constexpr bool kWhole = kN % 256 == 0;
};

// sw() for LDS slabs whose rows hold COLS token columns: the XOR stays
// inside the COLS columns (COLS = 64: the same permutation as sw())
template <int COLS, typename T>
__device__ __forceinline__ T* swc(T* base, int ld, int row, int col) {
  return base + row * ld + (col ^ (((row >> 3) & (COLS / 16 - 1) & 3) << 4));
}
template <int COLS, typename T>
__device__ __forceinline__ const T* swc(const T* base, int ld, int row, int col) {
  return base + row * ld + (col ^ (((row >> 3) & (COLS / 16 - 1) & 3) << 4));
}

__device__ __forceinline__ void lds_barrier_b() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// [v][t] (or [v][c]) LDS slab -> rows 0 .. NROWS-1 of a [rows][ld] tensor
// (16-byte stores), rows < n unless ALL; a fixed count per thread, so no
// loop or branch around the stores inside the scan step
template <int NROWS, bool ALL, typename T>
__device__ __forceinline__ void slab_to_rows(T* dst, int64_t ld, const T* src, int lds, int n, int tid) {
  using SM = Slab<T, NROWS>;
#pragma unroll
  for (int j = 0; j < SM::kPer; ++j) {
    const int idx = tid + 256 * j;
    if (!SM::kWhole && idx >= SM::kN) break;
    const int row = idx / SM::kSegs, c0 = (idx % SM::kSegs) * SM::kVec;
    float4 pk;
    T* e = reinterpret_cast<T*>(&pk);
#pragma unroll
    for (int s2 = 0; s2 < SM::kVec; ++s2) e[s2] = *swc<NROWS>(src, lds, c0 + s2, row);
    if (ALL || row < n) *reinterpret_cast<float4*>(dst + row * ld + c0) = pk;
  }
}

// ------------------------------------------------------------ r1
template <typename T, int DK, int GATE, int C>
struct RevFrags {
  static constexpr int KK = DK / 32, CT = DK / 64, KC = C / 32;
  Frag8<T> Pt[KC], Kw[KK], Mt[KC], Ql[CT][KC], Kn[CT][KC];
  float4 dO[Slab<T, C>::kPer];   // dO slab of the chunk before this one
  // log decay at the chunk end: scalar, or per channel of the state rows
  // c = 16 (w CT + ct) + 4 lg + ii this lane holds
  float gC[GATE == kGateChannel ? CT : 1][GATE == kGateChannel ? 4 : 1];
  float beta[4];   // beta of rows 16w + 4lg + ii (raw: past the end masked at use)
  float gw[GATE == kGateScalar ? 4 : 1];   // scalar gate: G of rows 16w + 4lg + ii
};

struct RevCtx {
  int64_t b, h, bh;
  int v0, w, lr, lg, tid;
  float dscale;   // scale, or 0 for a transition workgroup (dO zeroed)
};

// dO slab of chunk i (rows past the sequence end re-read its last row; the
// staging zeroes them)
template <typename T, int C, int NPER = Slab<T, C>::kPer>
__device__ __forceinline__ void rev_load_dO(float4 (&d)[NPER], const BwdArgs& ba, int i,
                                            const RevCtx& x) {
  using SM = Slab<T, C>;
  constexpr uint32_t E = sizeof(T);
  const FwdArgs& a = ba.f;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int last = static_cast<int>(min<int64_t>(C, a.T - t0)) - 1;
  const int64_t HV = a.H * (int64_t)a.dv;
  const T* dob = static_cast<const T*>(ba.dO) + (x.b * a.T + t0) * HV + x.h * a.dv + x.v0;
#pragma unroll
  for (int j = 0; j < SM::kPer; ++j) {
    const int idx = x.tid + 256 * j;
    if (!SM::kWhole && idx >= SM::kN) break;
    const uint32_t row = static_cast<uint32_t>(min(idx / SM::kSegs, last));
    const uint32_t off = (row * static_cast<uint32_t>(HV) + (idx % SM::kSegs) * SM::kVec) * E;
    d[j] = *reinterpret_cast<const float4*>(at_bytes(dob, off));
  }
}

template <typename T, int DK, int GATE, int C>
__device__ __forceinline__ void rev_load(RevFrags<T, DK, GATE, C>& f, const BwdArgs& ba, int i,
                                         const RevCtx& x) {
  constexpr int KK = DK / 32, CT = DK / 64, KC = C / 32, NB = C / 16;
  constexpr uint32_t E = sizeof(T);
  const bool rows = NB == 4 || x.w < NB;
  const FwdArgs& a = ba.f;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int last = static_cast<int>(min<int64_t>(C, a.T - t0)) - 1;
  const int64_t cc = (x.bh * a.NT + i) * (int64_t)(C * C);
  const int64_t ck = (x.bh * a.NT + i) * (int64_t)(DK * C);
  const T* pt = static_cast<const T*>(a.PtT) + cc;
  const T* mt = static_cast<const T*>(a.MtT) + cc;
  // decayed write-key rows w_r Kt: stored for the per-channel gate; with a
  // scalar gate (or none) the plain rows, w_r applied to the product's rows
  const T* kw = static_cast<const T*>(GATE == kGateChannel ? a.Kw : a.Ktr) + (x.bh * a.Tpad + t0) * DK;
  const T* ql = static_cast<const T*>(a.QlT) + ck;
  const T* kn = static_cast<const T*>(a.KnT) + ck;
  const int ra = 16 * x.w + x.lr;
  if (rows) {
    const uint32_t ocr = static_cast<uint32_t>(ra * C + 8 * x.lg) * E;
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) {
      f.Pt[k2] = ld8(at_bytes(pt, ocr + k2 * 32 * E));
      f.Mt[k2] = ld8(at_bytes(mt, ocr + k2 * 32 * E));
    }
    const uint32_t okw = static_cast<uint32_t>(ra * DK + 8 * x.lg) * E;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) f.Kw[kk] = ld8(at_bytes(kw, okw + kk * 32 * E));
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) {
      const uint32_t o = static_cast<uint32_t>((16 * (x.w * CT + ct) + x.lr) * C + 8 * x.lg + k2 * 32) * E;
      f.Ql[ct][k2] = ld8(at_bytes(ql, o));
      f.Kn[ct][k2] = ld8(at_bytes(kn, o));
    }
  // the dO slab staged at the end of this chunk's step: that of the chunk
  // before it (reverse order), so it has two steps to arrive
  rev_load_dO<T, C>(f.dO, ba, max(i - 1, 0), x);
  if (GATE == kGateScalar) {
    f.gC[0][0] = a.G[x.bh * a.Tpad + t0 + C - 1];
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) f.gw[ii] = rows ? a.G[x.bh * a.Tpad + t0 + 16 * x.w + 4 * x.lg + ii] : 0.f;
  }
  if (GATE == kGateChannel) {
    const float* gl = a.G + (x.bh * a.NT + i) * DK;   // G at the chunk end
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) f.gC[ct][ii] = gl[16 * (x.w * CT + ct) + 4 * x.lg + ii];
  }
  const float* bb = a.beta + (x.b * a.T + t0) * a.H + x.h;
#pragma unroll
  for (int ii = 0; ii < 4; ++ii) f.beta[ii] = bb[min(16 * x.w + 4 * x.lg + ii, last) * a.H];
}

// scale * dO of one chunk -> sDO[v][r]; rows past the sequence end are zero
template <typename T, int C>
__device__ __forceinline__ void rev_stage_dO(const float4 (&v)[Slab<T, C>::kPer], T* sDO, int n,
                                             float scale, int tid) {
  using SM = Slab<T, C>;
  constexpr int LDE = C + 8;
#pragma unroll
  for (int j = 0; j < SM::kPer; ++j) {
    const int idx = tid + 256 * j;
    if (!SM::kWhole && idx >= SM::kN) break;
    const int row = idx / SM::kSegs, c0 = (idx % SM::kSegs) * SM::kVec;
    const float4 raw = pin_here(v[j]);
    const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int s2 = 0; s2 < SM::kVec; ++s2)
      *swc<C>(sDO, LDE, c0 + s2, row) = from_f<T>(row < n ? scale * to_f(e[s2]) : 0.f);
  }
}

// WR = false: the step leaves no rows behind (dHs, Z and dv are not
// written): a run that only needs its end state
template <bool FULL, typename T, int DK, int GATE, int C, bool WR = true>
__device__ __forceinline__ void rev_step(RevFrags<T, DK, GATE, C>& f, bool stage_next,
                                         floatx4 (&st)[DK / 64][2], const BwdArgs& ba, int i,
                                         const RevCtx& x, T* sH, T* sDOc, T* sDOn, T* sE, T* sX,
                                         T* sZ) {
  constexpr int KK = DK / 32, CT = DK / 64, KC = C / 32, NB = C / 16;
  constexpr int LDH = DK + 8, LDE = C + 8;
  const FwdArgs& a = ba.f;
  const int w = x.w, lr = x.lr, lg = x.lg;
  const bool rows = NB == 4 || w < NB;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = FULL ? C : static_cast<int>(min<int64_t>(C, a.T - t0));
  // ---- dE = P^T dO_s + Diag(w) Kt dS'^T   (rows t of this wave)
  float wr[4];
#pragma unroll
  for (int ii = 0; ii < 4; ++ii) wr[ii] = GATE == kGateScalar ? fast_exp(f.gC[0][0] - f.gw[ii]) : 1.f;
  Frag8<T> bO[2][KC], bS[2][KK];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt) {
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) bO[vt][k2] = ld8(swc<C>(sDOc, LDE, 16 * vt + lr, k2 * 32 + 8 * lg));
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) bS[vt][kk] = ld8(sw(sH, LDH, 16 * vt + lr, kk * 32 + 8 * lg));
  }
  // state adjoint entering this chunk from the right, rows c, slab columns
  // (its LDS reads after the operand reads: LDS reads complete in issue order)
  if (WR)
    slab_to_rows<DK, true>(static_cast<T*>(ba.dHs) + (x.bh * a.NT + i) * (int64_t)DK * a.dv + x.v0, a.dv,
                           sH, LDH, DK, x.tid);
  if (rows) {
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f}, acw = acc;
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) mma(acc, f.Pt[k2], bO[vt][k2]);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) mma(acw, f.Kw[kk], bS[vt][kk]);
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) acc[ii] += wr[ii] * acw[ii];
      st4<T>(swc<C>(sE, LDE, 16 * vt + lr, 16 * w + 4 * lg), acc[0], acc[1], acc[2], acc[3]);
    }
  }
  lds_barrier_b();
  // ---- Z = M^T dE;  dX = Diag(beta) Z   (rows t = 16w + 4lg + ii)
  if (rows) {
    float bt[4];
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) bt[ii] = (FULL || 16 * w + 4 * lg + ii < n) ? f.beta[ii] : 0.f;
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) mma(acc, f.Mt[k2], ld8(swc<C>(sE, LDE, 16 * vt + lr, k2 * 32 + 8 * lg)));
      st4<T>(swc<C>(sZ, LDE, 16 * vt + lr, 16 * w + 4 * lg), acc[0], acc[1], acc[2], acc[3]);
      st4<T>(swc<C>(sX, LDE, 16 * vt + lr, 16 * w + 4 * lg), bt[0] * acc[0], bt[1] * acc[1],
             bt[2] * acc[2], bt[3] * acc[3]);
    }
  }
  lds_barrier_b();
  // ---- dS^T <- Diag(lam_C) dS'^T + (Lam o Q)^T dO_s - (Lam o K)^T dX
  const float gam = GATE == kGateScalar ? fast_exp(f.gC[0][0]) : 1.f;
  Frag8<T> bX[2][KC];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt)
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) bX[vt][k2] = ld8(swc<C>(sX, LDE, 16 * vt + lr, k2 * 32 + 8 * lg));
  if (WR) {
    // Z and dv rows (their LDS reads after the operand reads)
    const int64_t r0 = (x.bh * a.Tpad + t0) * a.dv + x.v0;
    slab_to_rows<C, true>(static_cast<T*>(ba.Zr) + r0, a.dv, sZ, LDE, C, x.tid);
    const int64_t HV = a.H * (int64_t)a.dv;
    slab_to_rows<C, FULL>(static_cast<T*>(ba.dv) + (x.b * a.T + t0) * HV + x.h * a.dv + x.v0, HV, sX, LDE,
                          n, x.tid);
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        st[ct][vt][ii] *= GATE == kGateChannel ? fast_exp(f.gC[ct][ii]) : gam;
      }
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) {
        mma(st[ct][vt], f.Ql[ct][k2], bO[vt][k2]);
        mma(st[ct][vt], f.Kn[ct][k2], bX[vt][k2]);
      }
      st4<T>(sw(sH, LDH, 16 * vt + lr, 16 * (w * CT + ct) + 4 * lg), st[ct][vt][0], st[ct][vt][1],
             st[ct][vt][2], st[ct][vt][3]);
    }
  if (stage_next) rev_stage_dO<T, C>(f.dO, sDOn, C, x.dscale, x.tid);  // earlier chunks are full
  lds_barrier_b();
}

// One workgroup's run of the reverse scan: chunks [c0, c1) of head x.bh
// from the top down, from the start state its role gives (dS_T, a composed
// segment start, zero, or for a transition slab the identity columns
// pv0 ..), ending with the end state written where its role sends it.
template <typename T, int DK, int GATE, int C, bool WR>
__device__ __forceinline__ void r1_body(const BwdArgs& ba, const RevCtx& x, int seg, bool probe, int pv0,
                                        int c0, int c1, T* sH, T* sDO0, T* sDO1, T* sE, T* sX, T* sZ) {
  constexpr int CT = DK / 64;
  constexpr int LDH = DK + 8;
  const FwdArgs& a = ba.f;
  const int S = a.seg_cnt;
  const int64_t bh = x.bh;
  T* sDO[2] = {sDO0, sDO1};
  const int w = x.w, lr = x.lr, lg = x.lg;
  const int DV = a.dv;
  const int64_t BHDK = a.BH * static_cast<int64_t>(DK);
  floatx4 st[CT][2];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int c = 16 * (w * CT + ct) + 4 * lg + ii, v = 16 * vt + lr;
        float s0 = 0.f;   // middle segments' local runs start from zero
        if (a.seg_phase == 0 || (a.seg_phase == 1 && seg == S - 1))
          s0 = ba.dS_T ? ba.dS_T[(bh * DK + c) * DV + x.v0 + v] : 0.f;
        else if (a.seg_phase == 3)
          s0 = a.seg_start[(seg * BHDK + bh * DK + c) * DV + x.v0 + v];
        else if (probe)
          s0 = c == pv0 + v ? 1.f : 0.f;
        st[ct][vt][ii] = s0;
      }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      st4<T>(sw(sH, LDH, 16 * vt + lr, 16 * (w * CT + ct) + 4 * lg), st[ct][vt][0], st[ct][vt][1],
             st[ct][vt][2], st[ct][vt][3]);
  // reverse order over the run [c0, c1): its top chunk first (the ragged
  // last chunk of the sequence, if the run ends there), then full chunks two
  // per trip with a branch-free body; dO slabs double-buffered
  const int top = c1 - 1;
  RevFrags<T, DK, GATE, C> fA, fB;
  float4 dlast[Slab<T, C>::kPer];
  rev_load_dO<T, C>(dlast, ba, top, x);
  rev_load<T, DK, GATE, C>(fA, ba, top, x);
  rev_load<T, DK, GATE, C>(fB, ba, max(top - 1, c0), x);
  rev_stage_dO<T, C>(dlast, sDO[0], static_cast<int>(min<int64_t>(C, a.T - static_cast<int64_t>(top) * C)),
                     x.dscale, x.tid);
  __syncthreads();
  rev_step<false, T, DK, GATE, C, WR>(fA, top > c0, st, ba, top, x, sH, sDO[0], sDO[1], sE, sX, sZ);
  int i = top - 1, buf = 1;
  for (; i >= c0 + 1; i -= 2) {
    rev_load<T, DK, GATE, C>(fA, ba, i - 1, x);
    rev_step<true, T, DK, GATE, C, WR>(fB, true, st, ba, i, x, sH, sDO[buf], sDO[buf ^ 1], sE, sX, sZ);
    buf ^= 1;
    rev_load<T, DK, GATE, C>(fB, ba, max(i - 2, c0), x);
    rev_step<true, T, DK, GATE, C, WR>(fA, true, st, ba, i - 1, x, sH, sDO[buf], sDO[buf ^ 1], sE, sX, sZ);
    buf ^= 1;
  }
  if (i == c0) rev_step<true, T, DK, GATE, C, WR>(fB, false, st, ba, c0, x, sH, sDO[buf], sDO[buf ^ 1], sE, sX, sZ);
  // the end state: dS0 after chunk 0; phase 1: the last segment's exact
  // end, a middle segment's local end or its transition
  float* dst = nullptr;
  int64_t ld = DV;
  int col0 = x.v0;
  if (a.seg_phase == 1) {
    if (probe) {
      dst = a.seg_phi + (seg * BHDK + bh * DK) * DK;
      ld = DK;
      col0 = pv0;
    } else {
      dst = a.seg_end + (seg * BHDK + bh * DK) * DV;
    }
  } else if (c0 == 0 && ba.dS0) {
    dst = ba.dS0 + bh * DK * DV;
  }
  if (dst) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int vt = 0; vt < 2; ++vt)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int c = 16 * (w * CT + ct) + 4 * lg + ii;
          dst[c * ld + col0 + 16 * vt + lr] = st[ct][vt][ii];
        }
  }
}

template <typename T, int DK, int GATE, int C>
__global__ __launch_bounds__(256) void r1_state_adjoint(BwdArgs ba) {
  constexpr int CT = DK / 64;
  constexpr int LDH = DK + 8, LDE = C + 8;
  __shared__ __attribute__((aligned(16))) T sH[BVB * LDH];
  __shared__ __attribute__((aligned(16))) T sDO[2][BVB * LDE];
  __shared__ __attribute__((aligned(16))) T sE[BVB * LDE];
  __shared__ __attribute__((aligned(16))) T sX[BVB * LDE];
  __shared__ __attribute__((aligned(16))) T sZ[BVB * LDE];
  const FwdArgs& a = ba.f;
  // workgroup -> (head, role, slab) as in the forward scan, mirrored: phase
  // 1 runs the last segment from dS_T beside the middle segments' local
  // runs (from zero) and transitions (from the identity, dO zeroed); phase
  // 3 runs segments 0 .. S - 2 from their composed starts
  const int nslab = a.dv / BVB, npslab = DK / BVB;
  const int S = a.seg_cnt;
  const int nrole = a.seg_phase == 0 ? nslab
                  : a.seg_phase == 1 ? nslab + (S - 2) * (nslab + npslab)
                                     : (S - 1) * nslab;
  const int64_t bid = blockIdx.x;
  const int xcd = static_cast<int>(bid & 7);
  const int64_t j8 = bid >> 3;
  const int role = static_cast<int>(j8 % nrole);
  const int64_t bh = (j8 / nrole) * 8 + xcd;
  if (bh >= a.BH) return;
  int seg = S - 1, slab = role;
  bool probe = false;
  if (a.seg_phase == 1 && role >= nslab) {
    const int r = role - nslab;
    seg = 1 + r / (nslab + npslab);
    slab = r % (nslab + npslab);
    probe = slab >= nslab;
  } else if (a.seg_phase == 3) {
    seg = role / nslab;
    slab = role % nslab;
  }
  const int c0 = a.seg_phase == 0 ? 0 : seg * a.seg_len;
  const int c1 = a.seg_phase == 0 ? a.NT : min(a.NT, c0 + a.seg_len);
  RevCtx x;
  x.bh = bh;
  x.b = bh / a.H;
  x.h = bh % a.H;
  x.tid = threadIdx.x;
  x.w = x.tid >> 6;
  x.lr = x.tid & 15;
  x.lg = (x.tid & 63) >> 4;
  x.v0 = probe ? 0 : slab * BVB;
  x.dscale = probe ? 0.f : a.scale;
  const int pv0 = probe ? (slab - nslab) * BVB : 0;
  // middle segments of the first pass need only their end states
  if (a.seg_phase == 1 && seg < S - 1) {
    r1_body<T, DK, GATE, C, false>(ba, x, seg, probe, pv0, c0, c1, sH, sDO[0], sDO[1], sE, sX, sZ);
    return;
  }
  r1_body<T, DK, GATE, C, true>(ba, x, seg, probe, pv0, c0, c1, sH, sDO[0], sDO[1], sE, sX, sZ);
}

// ------------------------------------------------------------ p1
// Rows [C][DD] of a workspace tensor -> LDS rows [C][DD + 8] (16-byte copies,
// bank-spread addressing: read back through sw()), in two halves, so the
// loads can be issued early and other work done before the LDS store waits
// for them
template <typename T, int DD, int C>
struct RowStage {
  static constexpr int kVec = 16 / static_cast<int>(sizeof(T)), kVpr = DD / kVec;
  static constexpr int kPer = C * kVpr / 256;
  static_assert(C * kVpr % 256 == 0 && kPer >= 1 && kPer <= 4, "one to four vectors per thread");
  float4 v0, v1, v2, v3;   // named registers: a private array here is placed in memory
  __device__ __forceinline__ void load(const T* src, int tid) {
    auto get = [&](int j, float4& x) {
      const int idx = tid + 256 * j, r = idx / kVpr, cv = idx % kVpr;
      x = *reinterpret_cast<const float4*>(src + r * DD + cv * kVec);
    };
    get(0, v0);
    if constexpr (kPer > 1) get(1, v1);
    if constexpr (kPer > 2) get(2, v2);
    if constexpr (kPer > 3) get(3, v3);
  }
  __device__ __forceinline__ void store(T* dst, int tid) const {
    constexpr int LD = DD + 8;
    auto put = [&](int j, float4 x) {
      const int idx = tid + 256 * j, r = idx / kVpr, cv = idx % kVpr;
      *reinterpret_cast<float4*>(sw(dst, LD, r, cv * kVec)) = x;
    };
    put(0, v0);
    if constexpr (kPer > 1) put(1, v1);
    if constexpr (kPer > 2) put(2, v2);
    if constexpr (kPer > 3) put(3, v3);
  }
};

// A [C][HC] tile held in registers between its load and its transposed
// store to dst[HC][C + 8].  (Named registers, not an array: a private array
// here is moved to LDS.)
// (C = 32 in bf16: 128 vectors, so half the threads hold one: kN guards)
template <typename T, int HC, int C>
struct HeldTile {
  static constexpr int kVec = 16 / static_cast<int>(sizeof(T)), kVpr = HC / kVec;
  static constexpr int kN = C * kVpr;
  static constexpr int kPer = (kN + 255) / 256;
  static_assert(kPer == 1 || kPer == 2, "one or two vectors per thread");
  float4 v0, v1;
};
template <typename T, int HC, int C>
__device__ __forceinline__ void tile_t_put(T* dst, float4 x, int j, int tid) {
  using HT = HeldTile<T, HC, C>;
  constexpr int LDT = C + 8;
  const int idx = tid + 256 * j, r = idx / HT::kVpr, cv = idx % HT::kVpr;
  if (HT::kN % 256 != 0 && idx >= HT::kN) return;
  const T* e = reinterpret_cast<const T*>(&x);
#pragma unroll
  for (int s2 = 0; s2 < HT::kVec; ++s2) *swc<C>(dst, LDT, cv * HT::kVec + s2, r) = e[s2];
}
template <typename T, int HC, int C>
__device__ __forceinline__ void tile_t_store(T* dst, const HeldTile<T, HC, C>& held, int tid) {
  tile_t_put<T, HC, C>(dst, held.v0, 0, tid);
  if constexpr (HeldTile<T, HC, C>::kPer == 2) tile_t_put<T, HC, C>(dst, held.v1, 1, tid);
}
// One pass's tile (rows [C], columns HC from src) into registers, a pass
// ahead of its transposed LDS store (tile_t_store); rows >= nvalid are zero
template <typename T, int HC, int C>
__device__ __forceinline__ void load_tile_regs(HeldTile<T, HC, C>& t, const T* src, int64_t lds, int nvalid,
                                               int tid) {
  using HT = HeldTile<T, HC, C>;
  auto get = [&](int j, float4& v) {
    const int idx = tid + 256 * j, r = idx / HT::kVpr, cv = idx % HT::kVpr;
    v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < nvalid && (HT::kN % 256 == 0 || idx < HT::kN))
      v = *reinterpret_cast<const float4*>(src + r * lds + cv * HT::kVec);
  };
  get(0, t.v0);
  if constexpr (HT::kPer == 2) get(1, t.v1);
}

// Dot product of two 16-byte vectors of T, on the packed words (no
// element-addressed copy, which the compiler would place in memory)
template <typename T>
__device__ __forceinline__ float dot16(const float4& a, const float4& b);
template <>
__device__ __forceinline__ float dot16<float>(const float4& a, const float4& b) {
  return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
}
template <>
__device__ __forceinline__ float dot16<bf16>(const float4& a, const float4& b) {
  // a 32-bit word holds two bf16: the low one is the high half of its float
  auto w2 = [](float x, float y) {
    const uint32_t u = __float_as_uint(x), v = __float_as_uint(y);
    return __uint_as_float(u << 16) * __uint_as_float(v << 16) +
           __uint_as_float(u & 0xffff0000u) * __uint_as_float(v & 0xffff0000u);
  };
  return w2(a.x, b.x) + w2(a.y, b.y) + w2(a.z, b.z) + w2(a.w, b.w);
}

// Two adjacent passes' tiles at once (columns [0, HC) into `now`, [HC, 2 HC)
// into `held`), so every row segment fetched is a whole 128-byte line
template <typename T, int HC, int C>
__device__ __forceinline__ void load_pair_regs(HeldTile<T, HC, C>& now, HeldTile<T, HC, C>& held, const T* src,
                                               int64_t lds, int nvalid, int tid) {
  load_tile_regs<T, HC, C>(now, src, lds, nvalid, tid);
  load_tile_regs<T, HC, C>(held, src + HC, lds, nvalid, tid);
}

// One phase-B pass's rows of the chunk-start state S^T and of its adjoint
// ([HC][DV] each), loaded a pass ahead into named registers and written to
// LDS ([HC][DV + 8], bank-spread) when the pass starts.
template <typename T, int HC, int DV>
struct StateRows {
  static constexpr int kVec = 16 / static_cast<int>(sizeof(T)), kVpr = DV / kVec;
  static constexpr int kPer = HC * kVpr / 256;
  static_assert(HC * kVpr % 256 == 0 && (kPer == 1 || kPer == 2), "one or two vectors per thread");
  float4 h0, h1, d0, d1;
  __device__ __forceinline__ void load(const T* Hs, const T* dHs, int tid) {
    auto get = [&](int j, float4& h, float4& d) {
      const int idx = tid + 256 * j, c = idx / kVpr, cv = idx % kVpr;
      h = *reinterpret_cast<const float4*>(Hs + c * DV + cv * kVec);
      d = *reinterpret_cast<const float4*>(dHs + c * DV + cv * kVec);
    };
    get(0, h0, d0);
    if constexpr (kPer == 2) get(1, h1, d1);
  }
  __device__ __forceinline__ void store(T* sS, T* sdS, int tid) const {
    constexpr int LDV = DV + 8;
    auto put = [&](int j, float4 h, float4 d) {
      const int idx = tid + 256 * j, c = idx / kVpr, cv = idx % kVpr;
      *reinterpret_cast<float4*>(sw(sS, LDV, c, cv * kVec)) = h;
      *reinterpret_cast<float4*>(sw(sdS, LDV, c, cv * kVec)) = d;
    };
    put(0, h0, d0);
    if constexpr (kPer == 2) put(1, h1, d1);
  }
  // sum of S o dS' over vector J's elements (state row (tid + 256 J) / kVpr)
  template <int J>
  __device__ __forceinline__ float dot() const {
    return J == 0 ? dot16<T>(h0, d0) : dot16<T>(h1, d1);
  }
};

// ------------------------------------------------------------ p12
// Per chunk, every gradient after the reverse scan except the
// preconditioner's, in one pass over the chunk's rows:
//   phase A  dP = dO E^T, dLn = Z E^T (dL = -dLn), Sqk = Q Kt^T,
//            Skk = K Kt^T and their elementwise adjoint algebra: dSqk,
//            dSkk, the At term of dbeta, Z . V, the Gam terms of dG
//   phase B  (HC key columns at a time)
//            A1 = dO_s S, A2' = Z S, A3 = E dS'       (C x dk, over dv;
//            dX S = Diag(beta) A2')
//            dq = Diag(lam) A1 + dSqk Kt,  dK = -Diag(lam beta) A2' + dSkk Kt,
//            dKt = Diag(w) A3 + dSqk^T Q + dSkk^T K
//   then     dbeta's T term -lam K . A2', dG and its reverse cumsum -> dg
// Wave w owns rows 16w .. 16w + 15.  Its A operands (dO, Z, E, V, Q, K rows)
// are private and load straight into fragments; shared B operands (E and Kt
// rows; the chunk-start state and its adjoint as rows [c][v]; Kt, Q, K
// transposed to [c][t]) are staged in LDS.  The C x C adjoints pass from
// the C accumulator layout to A fragments (rows and, across waves,
// transposed rows) through LDS once, then stay in registers.  Token rows
// past the sequence end re-read the last row: their dP rows are masked,
// their other products meet a zero factor (Z and beta vanish there), and
// their outputs are not stored.
// 16-byte store through a raw buffer resource: offsets at or past its byte
// range are dropped by the hardware's range check (no branch).
__device__ __forceinline__ void buf_store16(__amdgpu_buffer_rsrc_t r, uint32_t off, float4 v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  u32x4 u;
  __builtin_memcpy(&u, &v, 16);
  __builtin_amdgcn_raw_buffer_store_b128(u, r, static_cast<int>(off), 0, 0);
}

// One wave's 16 output rows x HC columns of dq, dK and dKt, from its LDS
// staging (the wave reads back only what it wrote: no barrier needed):
// 16-byte stores, a fixed count per lane.  dq is the chunk's rows of the
// caller's [B,T,H,dk] tensor as a buffer ending with its last valid row, so
// rows past the sequence end are dropped; dKm / dKt are padded workspace.
template <typename T, int HC, int LDO, int DK>
__device__ __forceinline__ void p12_flush_rows(const T* so, __amdgpu_buffer_rsrc_t dqr, int64_t HD,
                                               int c0, T* dKm, T* dKt, int w, int l) {
  constexpr int VEC = 16 / sizeof(T), SPR = HC / VEC;
  static_assert(16 * SPR % 64 == 0, "whole rounds of the wave");
#pragma unroll
  for (int u = 0; u < 16 * SPR / 64; ++u) {
    const int idx = l + 64 * u;
    const int rr = idx / SPR, sgc = (idx % SPR) * VEC, r = 16 * w + rr;
    const float4 vq = *reinterpret_cast<const float4*>(so + rr * LDO + sgc);
    const float4 vk = *reinterpret_cast<const float4*>(so + (16 + rr) * LDO + sgc);
    const float4 vt = *reinterpret_cast<const float4*>(so + (32 + rr) * LDO + sgc);
    buf_store16(dqr, static_cast<uint32_t>((r * HD + c0 + sgc) * static_cast<int64_t>(sizeof(T))), vq);
    *reinterpret_cast<float4*>(dKm + r * DK + c0 + sgc) = vk;
    *reinterpret_cast<float4*>(dKt + r * DK + c0 + sgc) = vt;
  }
}

template <typename T, int DK, int DV, int C>
struct P12Smem {
  static constexpr int HC = 32;                 // key columns per phase-B pass
  static constexpr int LDE = DV + 8, LDK = DK + 8, LDV = DV + 8, LDT = C + 8;
  static constexpr int LDO = HC + 16;           // output staging rows (bank-spread)
  static constexpr size_t kA = sizeof(T) * (C * LDE + C * LDK + 4 * C * LDT);
  // phase B: state rows, the pass's Q^T and K^T tiles, output staging, then
  // the whole transposed write-key tile [DK][C] (written once, after phase A
  // has read its C x C adjoints, from phase A's row-major copy, which lies
  // below it)
  static constexpr size_t kKtT = 2 * HC * LDV + 2 * HC * LDT + 4 * 3 * 16 * LDO;   // elements
  static constexpr size_t kB = sizeof(T) * (kKtT + DK * LDT);
  static_assert(kKtT >= static_cast<size_t>(C * LDE + C * LDK), "the K~^T tile lies above phase A's K~ tile");
  static constexpr size_t kMain = kA > kB ? kA : kB;
  static constexpr size_t kTotal = kMain + sizeof(float) * (12 * C + 4);
};

template <typename T, int DK, int DV, int GATE, int C>
__global__ __launch_bounds__(256, 2) void p12_chunk_grads(BwdArgs ba) {
  using SM = P12Smem<T, DK, DV, C>;
  constexpr int NB = C / 16, KC = C / 32;
  constexpr int HC = SM::HC, LDE = SM::LDE, LDK = SM::LDK, LDV = SM::LDV, LDT = SM::LDT;
  constexpr int LDO = SM::LDO;
  constexpr int KV = DV / 32, KD = DK / 32, NPASS = DK / HC;
  constexpr uint32_t E = sizeof(T);
  __shared__ __attribute__((aligned(16))) char smem[SM::kTotal];
  // phase A
  T* sE = reinterpret_cast<T*>(smem);
  T* sKt = sE + C * LDE;
  T* sSq = sKt + C * LDK;     // dSqk rows [r][t]
  T* sSk = sSq + C * LDT;     // dSkk rows
  T* sSqT = sSk + C * LDT;    // dSqk^T rows [t][r]
  T* sSkT = sSqT + C * LDT;   // dSkk^T rows
  // phase B (reuses the same memory)
  T* sS = reinterpret_cast<T*>(smem);   // S^T rows c0 .. c0 + HC - 1
  T* sdS = sS + HC * LDV;               // dS'^T rows
  T* sQT = sdS + HC * LDV;
  T* sKT = sQT + HC * LDT;
  T* sOut = sKT + HC * LDT;             // per wave: dq, dK, dKt rows [3][16][LDO]
  T* sKtT = reinterpret_cast<T*>(smem) + SM::kKtT;   // K~^T, all DK rows [c][t]
  float* sG = reinterpret_cast<float*>(smem + SM::kMain);
  float* sBeta = sG + C;
  float* sDb = sBeta + C;    // At term of dbeta
  float* sZV = sDb + C;      // Z_r . V_r
  float* sRs = sZV + C;      // row sums of the Gam products, then dG from them
  float* sCs = sRs + C;      // [4][C] their column sums per wave
  float* sDl = sCs + 4 * C;  // d lam_r
  float* sDw = sDl + C;      // d w_r
  float* sKZ = sDw + C;      // K_r . A2'_r
  float* sRed = sKZ + C;     // 4 wave partials of sum(dS' o S)

  const FwdArgs& a = ba.f;
  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const bool rows = NB == 4 || w < NB;   // this wave owns rows of the chunk
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  const int64_t HV = a.H * (int64_t)DV, HD = a.H * (int64_t)DK;
  const int64_t rv = (bh * a.Tpad + t0) * DV, rk = (bh * a.Tpad + t0) * DK;
  const int64_t cs = (bh * a.NT + i) * (int64_t)DK * DV;

  // ---- A operands of row ra (wave-private)
  const int ra = 16 * w + lr;
  const uint32_t rc = static_cast<uint32_t>(min(ra, n - 1));
  Frag8<T> fO[KV], fZ[KV], fE[KV];
  Frag8<T> fV[KV], fQ[KD], fK[KD];    // phase A only
  const T* dob = static_cast<const T*>(ba.dO) + (b * a.T + t0) * HV + h * DV;
  const T* eb = static_cast<const T*>(a.Er) + rv;
  // phase A's loads in two groups: the Gram products' operands (q, k rows,
  // the Kt tile) first, then dO, V, Z rows and the E tile, which stay in
  // flight while the Gram products run
  RowStage<T, DK, C> stKt;
  RowStage<T, DV, C> stE;
  {
    const T* qb = static_cast<const T*>(a.q) + (b * a.T + t0) * HD + h * DK;
    const T* kb = static_cast<const T*>(a.k) + (b * a.T + t0) * HD + h * DK;
#pragma unroll
    for (int kk = 0; kk < KD; ++kk) {
      const uint32_t o = (rc * static_cast<uint32_t>(HD) + 32 * kk + 8 * lg) * E;
      fQ[kk] = ld8(at_bytes(qb, o));
      fK[kk] = ld8(at_bytes(kb, o));
    }
    stKt.load(static_cast<const T*>(a.Ktr) + rk, tid);
    const T* vb = static_cast<const T*>(a.v) + (b * a.T + t0) * HV + h * DV;
    const T* zb = static_cast<const T*>(ba.Zr) + rv;
#pragma unroll
    for (int kk = 0; kk < KV; ++kk) {
      const uint32_t o = (rc * static_cast<uint32_t>(HV) + 32 * kk + 8 * lg) * E;
      const uint32_t ow = (static_cast<uint32_t>((rows ? ra : 0) * DV) + 32 * kk + 8 * lg) * E;
      fO[kk] = ld8(at_bytes(dob, o));
      fV[kk] = ld8(at_bytes(vb, o));
      fZ[kk] = ld8(at_bytes(zb, ow));
    }
    stE.load(eb, tid);
  }
  // per-row scalars, with the tiles: every wave loads the chunk's rows and
  // stores the same values (no branch, so the loads issue with the rest)
  const int rs = tid % C;
  const float vG = GATE == kGateScalar ? a.G[bh * a.Tpad + t0 + rs] : 0.f;
  const float vB = a.beta[(b * a.T + t0 + min(rs, n - 1)) * a.H + h];
  // ---- phase A: shared B operands (Kt now, E after the Gram products) and
  // per-row scalars
  stKt.store(sKt, tid);
  sG[rs] = vG;
  sBeta[rs] = rs < n ? vB : 0.f;
  __syncthreads();
  // the Gram products (Q and K rows die here)
  floatx4 Sqk[NB], Skk[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    Sqk[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    Skk[j] = Sqk[j];
    if (rows && j <= w) {
#pragma unroll
      for (int kk = 0; kk < KD; ++kk) {
        const Frag8<T> fk = ld8(sw(sKt, LDK, 16 * j + lr, 32 * kk + 8 * lg));
        mma(Sqk[j], fQ[kk], fk);
        mma(Skk[j], fK[kk], fk);
      }
    }
  }
  // phase B's first state rows: in flight through the rest of phase A
  StateRows<T, HC, DV> srows;
  srows.load(static_cast<const T*>(a.Hs) + cs, static_cast<const T*>(ba.dHs) + cs, tid);
  // and its transposed write-key, query and key tiles
  const T* qtile = static_cast<const T*>(a.q) + (b * a.T + t0) * HD + h * DK;
  const T* ktile = static_cast<const T*>(a.k) + (b * a.T + t0) * HD + h * DK;
  // (the tiles of two passes at a time: whole lines)
  static_assert(NPASS % 2 == 0, "phase B passes come in pairs");
  HeldTile<T, HC, C> tQ, tK, hQ, hK;
  load_pair_regs<T, HC, C>(tQ, hQ, qtile, HD, n, tid);
  load_pair_regs<T, HC, C>(tK, hK, ktile, HD, n, tid);
  stE.store(sE, tid);
  __syncthreads();
  {
    // Z_r . V_r for row ra (Z vanishes on rows past the end)
    float zv = 0.f;
#pragma unroll
    for (int kk = 0; kk < KV; ++kk)
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) zv += fZ[kk].get(s2) * fV[kk].get(s2);
    zv += __shfl_xor(zv, 16, 64);
    zv += __shfl_xor(zv, 32, 64);
    if (lg == 0 && rows) sZV[ra] = zv;
  }
  if (rows) {
    // dP and dL tile by tile straight into the elementwise algebra
    float dbA[4] = {0.f, 0.f, 0.f, 0.f}, rs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      floatx4 dP = {0.f, 0.f, 0.f, 0.f}, dL = dP;
      if (j <= w) {
#pragma unroll
        for (int kk = 0; kk < KV; ++kk) {
          const Frag8<T> fe = ld8(sw(sE, LDE, 16 * j + lr, 32 * kk + 8 * lg));
          mma(dP, fO[kk], fe);
          mma(dL, fZ[kk], fe);
        }
      }
      floatx4 dq, dk;
      float csum = 0.f;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int r = 16 * w + 4 * lg + ii, t = 16 * j + lr;
        const bool ca = r >= t && r < n, sl = r > t;
        const float gm = GATE == kGateScalar ? fast_exp(r >= t ? sG[r] - sG[t] : 0.f) : 1.f;
        dq[ii] = ca ? gm * a.scale * dP[ii] : 0.f;
        const float dA = sl ? -dL[ii] : 0.f;          // strict_lower(dL)
        dk[ii] = gm * sBeta[r] * dA;
        dbA[ii] += dA * gm * Skk[j][ii];              // dbeta through At
        // (dSkk o S_kk) + (dSqk o S_qk): row minus column sums give dG
        const float R = dk[ii] * Skk[j][ii] + dq[ii] * Sqk[j][ii];
        rs[ii] += R;
        csum += R;
      }
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        *swc<C>(sSq, LDT, 16 * w + 4 * lg + ii, 16 * j + lr) = from_f<T>(dq[ii]);
        *swc<C>(sSk, LDT, 16 * w + 4 * lg + ii, 16 * j + lr) = from_f<T>(dk[ii]);
      }
      st4<T>(swc<C>(sSqT, LDT, 16 * j + lr, 16 * w + 4 * lg), dq[0], dq[1], dq[2], dq[3]);
      st4<T>(swc<C>(sSkT, LDT, 16 * j + lr, 16 * w + 4 * lg), dk[0], dk[1], dk[2], dk[3]);
      csum += __shfl_xor(csum, 16, 64);
      csum += __shfl_xor(csum, 32, 64);
      if (lg == 0) sCs[w * C + 16 * j + lr] = csum;
    }
#pragma unroll
    for (int ii = 0; ii < 4; ++ii)
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        dbA[ii] += __shfl_xor(dbA[ii], off, 64);
        rs[ii] += __shfl_xor(rs[ii], off, 64);
      }
    if (lr == 0) {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        sDb[16 * w + 4 * lg + ii] = dbA[ii];
        sRs[16 * w + 4 * lg + ii] = rs[ii];
      }
    }
  }
  // E rows of this wave (phase B's A operand of A3), from the staged copy
  // (a wave without rows of the chunk reads row 0: its results are unused)
  const int rw = rows ? ra : 0;
#pragma unroll
  for (int kk = 0; kk < KV; ++kk) fE[kk] = ld8(sw(sE, LDE, rw, 32 * kk + 8 * lg));
  __syncthreads();
  // the C x C adjoints as A fragments of this wave's rows (k = 32 k2 + 8 lg)
  Frag8<T> fSq[KC], fSk[KC], fSqT[KC], fSkT[KC];
#pragma unroll
  for (int k2 = 0; k2 < KC; ++k2) {
    const int o = 32 * k2 + 8 * lg;
    fSq[k2] = ld8(swc<C>(sSq, LDT, rw, o));
    fSk[k2] = ld8(swc<C>(sSk, LDT, rw, o));
    fSqT[k2] = ld8(swc<C>(sSqT, LDT, rw, o));
    fSkT[k2] = ld8(swc<C>(sSkT, LDT, rw, o));
  }
  if (tid < C) {
    // Gam_rt = exp(G_r - G_t): d/dG_r of sum R_rt = row sum, d/dG_t = -column sum
    float cs4 = 0.f;
#pragma unroll
    for (int q = 0; q < NB; ++q) cs4 += sCs[q * C + tid];
    sRs[tid] = GATE == kGateScalar ? sRs[tid] - cs4 : 0.f;
  }
  __syncthreads();   // every wave holds its adjoint fragments
  {
    // K~^T for all of phase B, once, from the row-major tile phase A staged
    // (so phase B reads no write-key rows from HBM)
    static_assert(DK * C / 8 % 256 == 0, "whole rounds of 256 threads");
#pragma unroll
    for (int jj = 0; jj < DK * C / 8 / 256; ++jj) {
      const int idx = tid + 256 * jj;
      const int c = idx / (C / 8), t8 = (idx % (C / 8)) * 8;
      Frag8<T> f;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) f.set(s2, to_f(*sw(sKt, LDK, t8 + s2, c)));
      st8(swc<C>(sKtT, LDT, c, t8), f);
    }
  }
  // phase B computes its tiles transposed (every product with its operands
  // swapped), so a lane holds row ra = 16 w + lr at columns 16 j + 4 lg + ii
  const float lam = GATE == kGateScalar ? fast_exp(sG[rw]) : 1.f;
  const float wr = GATE == kGateScalar ? fast_exp(sG[C - 1] - sG[rw]) : 1.f;
  const float bt = sBeta[rw];

  // ---- phase B
  float pq = 0.f, pk = 0.f, pw = 0.f;
  float red = 0.f;
  T* dq = static_cast<T*>(ba.dq) + (b * a.T + t0) * HD + h * DK;
  // the chunk's dq rows as a raw buffer ending with row n - 1: a row r >= n
  // starts at r HD >= (n - 1) HD + DK elements, past the range
  const __amdgpu_buffer_rsrc_t dqr = __builtin_amdgcn_make_buffer_rsrc(
      dq, 0, static_cast<int>(((n - 1) * HD + DK) * static_cast<int64_t>(sizeof(T))), kBufWord3);
  T* dKm = static_cast<T*>(ba.dKm) + rk;
  T* dKt = static_cast<T*>(ba.dKt) + rk;
#pragma unroll 1
  for (int p = 0; p < NPASS; ++p) {
    const int c0 = p * HC;
    __syncthreads();   // phase A (or the previous pass) is done with the LDS
    srows.store(sS, sdS, tid);
    if (GATE == kGateScalar) {   // sum(dS' o S) over this pass's rows
      red += srows.template dot<0>();
      if constexpr (StateRows<T, HC, DV>::kPer == 2) red += srows.template dot<1>();
    }
    // transposed Kt, Q, K tiles (loaded during an earlier pass)
    if ((p & 1) == 0) {
      tile_t_store<T, HC, C>(sQT, tQ, tid);
      tile_t_store<T, HC, C>(sKT, tK, tid);
    } else {
      tile_t_store<T, HC, C>(sQT, hQ, tid);
      tile_t_store<T, HC, C>(sKT, hK, tid);
    }
    __syncthreads();
    {
      // the next pass's state rows load during this pass (the last pass
      // reloads its own rows, unused)
      const int cn = min(p + 1, NPASS - 1) * HC;
      srows.load(static_cast<const T*>(a.Hs) + cs + cn * DV, static_cast<const T*>(ba.dHs) + cs + cn * DV, tid);
      if ((p & 1) == 1 && p + 1 < NPASS) {   // the next two passes' tiles
        load_pair_regs<T, HC, C>(tQ, hQ, qtile + cn, HD, n, tid);
        load_pair_regs<T, HC, C>(tK, hK, ktile + cn, HD, n, tid);
      }
    }
#pragma unroll 1
    for (int j = 0; j < HC / 16 && rows; ++j) {
      // A1 = dO_s S, A2' = Z S, A3 = E dS' (transposed tiles)
      floatx4 A1 = {0.f, 0.f, 0.f, 0.f}, A2 = A1, A3 = A1;
#pragma unroll
      for (int kk = 0; kk < KV; ++kk) {
        const Frag8<T> fh = ld8(sw(sS, LDV, 16 * j + lr, 32 * kk + 8 * lg));
        const Frag8<T> fd = ld8(sw(sdS, LDV, 16 * j + lr, 32 * kk + 8 * lg));
        mma(A1, fh, fO[kk]);
        mma(A2, fh, fZ[kk]);
        mma(A3, fd, fE[kk]);
      }
      // row partials: Q_r . A1_r, K_r . A2'_r (gate and dbeta), Kt_r . A3_r
      const int cb = 16 * j + 4 * lg;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        A1[ii] *= a.scale;
        pq += to_f(*swc<C>(sQT, LDT, cb + ii, ra)) * A1[ii];
        pk += to_f(*swc<C>(sKT, LDT, cb + ii, ra)) * A2[ii];
        pw += to_f(*swc<C>(sKtT, LDT, c0 + cb + ii, ra)) * A3[ii];
      }
      floatx4 aq, ak, at;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        aq[ii] = lam * A1[ii];
        ak[ii] = -lam * bt * A2[ii];
        at[ii] = wr * A3[ii];
      }
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) {
        const Frag8<T> fk = ld8(swc<C>(sKtT, LDT, c0 + 16 * j + lr, 32 * k2 + 8 * lg));
        mma(aq, fk, fSq[k2]);
        mma(ak, fk, fSk[k2]);
        mma(at, ld8(swc<C>(sQT, LDT, 16 * j + lr, 32 * k2 + 8 * lg)), fSqT[k2]);
        mma(at, ld8(swc<C>(sKT, LDT, 16 * j + lr, 32 * k2 + 8 * lg)), fSkT[k2]);
      }
      // to this wave's output rows in LDS: row lr, four adjacent columns
      T* so = sOut + w * 3 * 16 * LDO + lr * LDO + cb;
      st4<T>(so, aq[0], aq[1], aq[2], aq[3]);
      st4<T>(so + 16 * LDO, ak[0], ak[1], ak[2], ak[3]);
      st4<T>(so + 32 * LDO, at[0], at[1], at[2], at[3]);
    }
    if (rows) p12_flush_rows<T, HC, LDO, DK>(sOut + w * 3 * 16 * LDO, dqr, HD, c0, dKm, dKt, w, l);
  }
#pragma unroll
  for (int off = 16; off < 64; off <<= 1) {
    pq += __shfl_xor(pq, off, 64);
    pk += __shfl_xor(pk, off, 64);
    pw += __shfl_xor(pw, off, 64);
  }
  if (lg == 0 && rows) {
    // dlam_r = Q_r . A1_r - beta_r K_r . A2'_r ;  dw_r = Kt_r . A3_r
    sDl[ra] = ra < n ? pq - bt * pk : 0.f;
    sDw[ra] = ra < n ? pw : 0.f;
    sKZ[ra] = pk;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) red += __shfl_xor(red, off, 64);
  if (l == 0) sRed[w] = red;
  __syncthreads();
  // ---- dbeta = At term + Z . V - lam K . A2'
  if (tid < n) {
    const float lamr = GATE == kGateScalar ? fast_exp(sG[tid]) : 1.f;
    ba.dbeta[(b * a.T + t0 + tid) * a.H + h] = sDb[tid] + sZV[tid] - lamr * sKZ[tid];
  }
  // ---- gate: dG_r, then the reverse in-chunk cumsum -> dg
  if (GATE == kGateScalar && w == 0) {
    // lanes r >= C (C = 32) carry zeros through the sums
    const int r = l, rr = min(l, C - 1);
    const bool in = r < C;
    const float lamr = fast_exp(sG[rr]);
    const float wrr = fast_exp(sG[C - 1] - sG[rr]);
    float wdw = in ? wrr * sDw[rr] : 0.f;
    float dG = in ? sRs[rr] + lamr * sDl[rr] - wdw : 0.f;
    // lam_C and the w_r all depend on G_{C-1}
    float tot = wdw;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) tot += __shfl_xor(tot, off, 64);
    if (r == C - 1) dG += tot + fast_exp(sG[C - 1]) * (sRed[0] + sRed[1] + sRed[2] + sRed[3]);
    // dg_j = sum_{r >= j} dG_r
    float x = dG;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_down(x, off, 64);
      if (r + off < 64) x += y;
    }
    if (r < n) ba.dg[(b * a.T + t0 + r) * a.H + h] = x;
  }
}

// ------------------------------------------------------------ p12c
// p12 for the per-channel gate (PKDA).  The decay now sits inside the key
// contractions: with Lam_r = exp(G_r) per channel, the chunk forward reads
// Lam o Q, Lam o K, Kt / Lam and Kt o (Lam_C / Lam), so
//   dq  = Lam o (dO_s S + dSqk (Kt / Lam))
//   dK  = Diag(beta) Lam o (-Z S + dAt (Kt / Lam))          (read key)
//   dKt = (dSqk^T (Lam o Q) + (Diag(beta) dAt)^T (Lam o K)) / Lam
//         + (Lam_C / Lam) o E dS'
// with dSqk = causal(dO_s E^T) and dAt = strict_lower(-Z E^T) carrying no
// decay.  A decay ratio exp(G_r - G_t) (r >= t) is split at a reference
// row per 16-row output block (its first row for dq and dK, its last for
// dKt), so every factor applied to an operand or an output is at most 1
// except inside the block itself; operand entries that only meet zeros of
// the causal masks are set to zero rather than scaled.  The gate gradient
// needs no C x C product: every place Lam enters is a product with one of
// the outputs, so per channel
//   dG_r = q_r dq_r + k_r dK_r - kt_r dKt_r
//          + [r = C - 1] (sum_t kt_t (Lam_C / Lam_t) (E dS')_t
//                         + Lam_C sum_v S dS')
// and dg is its reverse in-chunk cumsum.  dbeta_r = Z_r . V_r +
// sum_c k_rc (dK_rc / beta_r) takes the bracket before the beta factor.
template <typename T, int DK, int DV, int C>
struct P12cSmem {
  static constexpr int HC = 32;
  static constexpr int LDE = DV + 8, LDV = DV + 8, LDT = C + 8, LDO = HC + 16, LDG = C + 4;
  static constexpr size_t kA = sizeof(T) * (C * LDE + 4 * C * LDT);
  static constexpr size_t kStage = sizeof(T) * (2 * HC * LDV + 3 * HC * LDT + 4 * 3 * 16 * LDO);
  static constexpr size_t kB = kStage + sizeof(float) * (HC * LDG + C * (HC + 1));
  static constexpr size_t kMain = kA > kB ? kA : kB;
  static constexpr size_t kTotal = kMain + sizeof(float) * (3 * C + 4 * HC + HC + 8 * HC);
};

template <typename T, int DK, int DV, int C>
__global__ __launch_bounds__(256, 2) void p12c_chunk_grads(BwdArgs ba) {
  using SM = P12cSmem<T, DK, DV, C>;
  constexpr int NB = C / 16, KC = C / 32;
  constexpr int HC = SM::HC, LDE = SM::LDE, LDV = SM::LDV, LDT = SM::LDT, LDO = SM::LDO, LDG = SM::LDG;
  constexpr int KV = DV / 32, NPASS = DK / HC;
  constexpr uint32_t E = sizeof(T);
  __shared__ __attribute__((aligned(16))) char smem[SM::kTotal];
  // phase A
  T* sE = reinterpret_cast<T*>(smem);
  T* sSq = sE + C * LDE;      // dSqk rows [r][t]
  T* sSk = sSq + C * LDT;     // dAt rows
  T* sSqT = sSk + C * LDT;    // dSqk^T rows [t][r]
  T* sSkT = sSqT + C * LDT;   // (Diag(beta) dAt)^T rows
  // phase B
  T* sS = reinterpret_cast<T*>(smem);
  T* sdS = sS + HC * LDV;
  T* sKtT = sdS + HC * LDV;
  T* sQT = sKtT + HC * LDT;
  T* sKT = sQT + HC * LDT;
  T* sOut = sKT + HC * LDT;
  float* sGT = reinterpret_cast<float*>(smem + SM::kStage);   // G^T [c][t]
  float* sDG = sGT + HC * LDG;                                  // dG [t][c]
  float* sBeta = reinterpret_cast<float*>(smem + SM::kMain);
  float* sZV = sBeta + C;
  float* sDb = sZV + C;
  float* sXc = sDb + C;       // [4][HC] per-wave column sums of the last-row term
  float* sRedC = sXc + 4 * HC;   // [HC] sum_v S dS' per channel
  float* sSeg = sRedC + HC;      // [8][HC] segment totals of the cumsum

  const FwdArgs& a = ba.f;
  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const bool rows = NB == 4 || w < NB;   // this wave owns rows of the chunk
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  const int64_t HV = a.H * (int64_t)DV, HD = a.H * (int64_t)DK;
  const int64_t rv = (bh * a.Tpad + t0) * DV, rk = (bh * a.Tpad + t0) * DK;
  const int64_t cs = (bh * a.NT + i) * (int64_t)DK * DV;

  const int ra = 16 * w + lr;
  const uint32_t rc = static_cast<uint32_t>(min(ra, n - 1));
  Frag8<T> fO[KV], fZ[KV], fE[KV];
  const T* dob = static_cast<const T*>(ba.dO) + (b * a.T + t0) * HV + h * DV;
  {
    Frag8<T> fV[KV];
    const T* vb = static_cast<const T*>(a.v) + (b * a.T + t0) * HV + h * DV;
    const T* zb = static_cast<const T*>(ba.Zr) + rv;
#pragma unroll
    for (int kk = 0; kk < KV; ++kk) {
      const uint32_t o = (rc * static_cast<uint32_t>(HV) + 32 * kk + 8 * lg) * E;
      const uint32_t ow = (static_cast<uint32_t>((rows ? ra : 0) * DV) + 32 * kk + 8 * lg) * E;
      fO[kk] = ld8(at_bytes(dob, o));
      fV[kk] = ld8(at_bytes(vb, o));
      fZ[kk] = ld8(at_bytes(zb, ow));
    }
    // Z_r . V_r (Z vanishes on rows past the end)
    float zv = 0.f;
#pragma unroll
    for (int kk = 0; kk < KV; ++kk)
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) zv += fZ[kk].get(s2) * fV[kk].get(s2);
    zv += __shfl_xor(zv, 16, 64);
    zv += __shfl_xor(zv, 32, 64);
    if (lg == 0 && rows) sZV[ra] = zv;
  }
  RowStage<T, DV, C> stE;
  stE.load(static_cast<const T*>(a.Er) + rv, tid);
  // phase B's first state rows: in flight through the rest of phase A
  StateRows<T, HC, DV> srows;
  srows.load(static_cast<const T*>(a.Hs) + cs, static_cast<const T*>(ba.dHs) + cs, tid);
  // and its transposed write-key, query and key tiles
  const T* qtile = static_cast<const T*>(a.q) + (b * a.T + t0) * HD + h * DK;
  const T* ktile = static_cast<const T*>(a.k) + (b * a.T + t0) * HD + h * DK;
  const T* kttile = static_cast<const T*>(a.Ktr) + rk;
  // (the tiles of two passes at a time: whole lines)
  static_assert(NPASS % 2 == 0, "phase B passes come in pairs");
  HeldTile<T, HC, C> tKt, tQ, tK, hKt, hQ, hK;
  load_pair_regs<T, HC, C>(tKt, hKt, kttile, DK, C, tid);
  load_pair_regs<T, HC, C>(tQ, hQ, qtile, HD, n, tid);
  load_pair_regs<T, HC, C>(tK, hK, ktile, HD, n, tid);
  const int rs = tid % C;
  const float vB = a.beta[(b * a.T + t0 + min(rs, n - 1)) * a.H + h];
  stE.store(sE, tid);
  sBeta[rs] = rs < n ? vB : 0.f;   // every wave stores the same values
  __syncthreads();
  // ---- phase A: dSqk = causal(dO_s E^T), dAt = strict_lower(-Z E^T)
#pragma unroll
  for (int j = 0; j < NB && rows; ++j) {
    floatx4 dP = {0.f, 0.f, 0.f, 0.f}, dL = dP;
    if (j <= w) {
#pragma unroll
      for (int kk = 0; kk < KV; ++kk) {
        const Frag8<T> fe = ld8(sw(sE, LDE, 16 * j + lr, 32 * kk + 8 * lg));
        mma(dP, fO[kk], fe);
        mma(dL, fZ[kk], fe);
      }
    }
    floatx4 dq, dA, dAb;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int r = 16 * w + 4 * lg + ii, t = 16 * j + lr;
      dq[ii] = (r >= t && r < n) ? a.scale * dP[ii] : 0.f;
      dA[ii] = r > t ? -dL[ii] : 0.f;
      dAb[ii] = sBeta[r] * dA[ii];
      *swc<C>(sSq, LDT, r, t) = from_f<T>(dq[ii]);
      *swc<C>(sSk, LDT, r, t) = from_f<T>(dA[ii]);
    }
    st4<T>(swc<C>(sSqT, LDT, 16 * j + lr, 16 * w + 4 * lg), dq[0], dq[1], dq[2], dq[3]);
    st4<T>(swc<C>(sSkT, LDT, 16 * j + lr, 16 * w + 4 * lg), dAb[0], dAb[1], dAb[2], dAb[3]);
  }
  // (a wave without rows of the chunk reads row 0: its results are unused)
  const int rw = rows ? ra : 0;
#pragma unroll
  for (int kk = 0; kk < KV; ++kk) fE[kk] = ld8(sw(sE, LDE, rw, 32 * kk + 8 * lg));
  __syncthreads();
  Frag8<T> fSq[KC], fSk[KC], fSqT[KC], fSkT[KC];
#pragma unroll
  for (int k2 = 0; k2 < KC; ++k2) {
    const int o = 32 * k2 + 8 * lg;
    fSq[k2] = ld8(swc<C>(sSq, LDT, rw, o));
    fSk[k2] = ld8(swc<C>(sSk, LDT, rw, o));
    fSqT[k2] = ld8(swc<C>(sSqT, LDT, rw, o));
    fSkT[k2] = ld8(swc<C>(sSkT, LDT, rw, o));
  }
  float bt[4];
#pragma unroll
  for (int ii = 0; ii < 4; ++ii) bt[ii] = rows ? sBeta[16 * w + 4 * lg + ii] : 0.f;

  // ---- phase B
  float pdb[4] = {0.f, 0.f, 0.f, 0.f};
  T* dq = static_cast<T*>(ba.dq) + (b * a.T + t0) * HD + h * DK;
  // the chunk's dq rows as a raw buffer ending with row n - 1: a row r >= n
  // starts at r HD >= (n - 1) HD + DK elements, past the range
  const __amdgpu_buffer_rsrc_t dqr = __builtin_amdgcn_make_buffer_rsrc(
      dq, 0, static_cast<int>(((n - 1) * HD + DK) * static_cast<int64_t>(sizeof(T))), kBufWord3);
  T* dKm = static_cast<T*>(ba.dKm) + rk;
  T* dKt = static_cast<T*>(ba.dKt) + rk;
  // the per-channel log-decays g of the pass's channels: C / 8 segments of
  // 8 rows, one thread per (channel, segment)
  constexpr int NSG = C / 8;
  const int gc = tid & (HC - 1), gsg = tid / HC;
  const bool gseg = NSG == 8 || gsg < NSG;
  const float* gin = a.g + ((b * a.T + t0) * a.H + h) * DK;   // row stride HD
#pragma unroll 1
  for (int p = 0; p < NPASS; ++p) {
    const int c0 = p * HC;
    __syncthreads();   // phase A (or the previous pass) is done with the LDS
    if (gseg) {
      // raw g of the pass's channels, transposed (rows past the end: 0);
      // the in-chunk prefix is rebuilt from it below rather than read back
      float gr[8];
#pragma unroll
      for (int q = 0; q < 8; ++q)
        gr[q] = *at_bytes(gin, static_cast<uint32_t>(min(8 * gsg + q, n - 1) * HD + c0 + gc) * 4u);
#pragma unroll
      for (int q = 0; q < 8; ++q) sGT[gc * LDG + 8 * gsg + q] = 8 * gsg + q < n ? gr[q] : 0.f;
    }
    srows.store(sS, sdS, tid);
    {
      // sum_v S dS' per channel of the pass, from the rows just stored: the
      // kVpr lanes of a channel are adjacent
      using SR = StateRows<T, HC, DV>;
      auto chan = [&](float r2, int jj) {
#pragma unroll
        for (int off = 1; off < SR::kVpr; off <<= 1) r2 += __shfl_xor(r2, off, 64);
        if (tid % SR::kVpr == 0) sRedC[(tid + 256 * jj) / SR::kVpr] = r2;
      };
      chan(srows.template dot<0>(), 0);
      if constexpr (SR::kPer == 2) chan(srows.template dot<1>(), 1);
    }
    // the in-chunk prefix G, in place: each segment is summed, then re-walked
    // from the total of the segments before it
    __syncthreads();
    if (gseg) {
      float x = 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q) x += sGT[gc * LDG + 8 * gsg + q];
      sSeg[gsg * HC + gc] = x;
    }
    __syncthreads();
    if (gseg) {
      float x = 0.f;
      for (int q = 0; q < gsg; ++q) x += sSeg[q * HC + gc];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        float* gp = sGT + gc * LDG + 8 * gsg + q;
        x += *gp;
        *gp = x;
      }
    }
    if ((p & 1) == 0) {
      tile_t_store<T, HC, C>(sKtT, tKt, tid);
      tile_t_store<T, HC, C>(sQT, tQ, tid);
      tile_t_store<T, HC, C>(sKT, tK, tid);
    } else {
      tile_t_store<T, HC, C>(sKtT, hKt, tid);
      tile_t_store<T, HC, C>(sQT, hQ, tid);
      tile_t_store<T, HC, C>(sKT, hK, tid);
    }
    __syncthreads();
    {
      // the next pass's state rows load during this pass (the last pass
      // reloads its own rows, unused)
      const int cn = min(p + 1, NPASS - 1) * HC;
      srows.load(static_cast<const T*>(a.Hs) + cs + cn * DV, static_cast<const T*>(ba.dHs) + cs + cn * DV, tid);
      if ((p & 1) == 1 && p + 1 < NPASS) {   // the next two passes' tiles
        load_pair_regs<T, HC, C>(tKt, hKt, kttile + cn, DK, C, tid);
        load_pair_regs<T, HC, C>(tQ, hQ, qtile + cn, HD, n, tid);
        load_pair_regs<T, HC, C>(tK, hK, ktile + cn, HD, n, tid);
      }
    }
#pragma unroll 1
    for (int j = 0; j < HC / 16 && rows; ++j) {
      const int c = 16 * j + lr;
      const float* gcol = sGT + c * LDG;
      floatx4 A1 = {0.f, 0.f, 0.f, 0.f}, A2 = A1, A3 = A1;
#pragma unroll
      for (int kk = 0; kk < KV; ++kk) {
        const Frag8<T> fh = ld8(sw(sS, LDV, c, 32 * kk + 8 * lg));
        const Frag8<T> fd = ld8(sw(sdS, LDV, c, 32 * kk + 8 * lg));
        mma(A1, fO[kk], fh);
        mma(A2, fZ[kk], fh);
        mma(A3, fE[kk], fd);
      }
      // intra-chunk products with the decay split at the block's reference rows
      const float gref = gcol[16 * w], gref2 = gcol[16 * w + 15];
      floatx4 aqi = {0.f, 0.f, 0.f, 0.f}, aki = aqi, ati = aqi;
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) {
        const int tb = 32 * k2 + 8 * lg;
        const float4 g0 = *reinterpret_cast<const float4*>(gcol + tb);
        const float4 g1 = *reinterpret_cast<const float4*>(gcol + tb + 4);
        const float gt[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        Frag8<T> fk = ld8(swc<C>(sKtT, LDT, c, tb));
        Frag8<T> fq = ld8(swc<C>(sQT, LDT, c, tb));
        Frag8<T> fr = ld8(swc<C>(sKT, LDT, c, tb));
#pragma unroll
        for (int s2 = 0; s2 < 8; ++s2) {
          const int t = tb + s2;
          // columns t > 16w + 15 meet only zeros of dSqk / dAt rows of this block;
          // rows r < 16w only zeros of their transposes
          const float e1 = t < 16 * w + 16 ? fast_exp(gref - gt[s2]) : 0.f;
          const float e2 = t >= 16 * w ? fast_exp(gt[s2] - gref2) : 0.f;
          fk.set(s2, e1 * fk.get(s2));
          fq.set(s2, e2 * fq.get(s2));
          fr.set(s2, e2 * fr.get(s2));
        }
        mma(aqi, fSq[k2], fk);
        mma(aki, fSk[k2], fk);
        mma(ati, fSqT[k2], fq);
        mma(ati, fSkT[k2], fr);
      }
      const float gend = gcol[C - 1];
      const float4 g4 = *reinterpret_cast<const float4*>(gcol + 16 * w + 4 * lg);
      const float gr4[4] = {g4.x, g4.y, g4.z, g4.w};
      const typename Vec4<T>::type q4 = *reinterpret_cast<const typename Vec4<T>::type*>(swc<C>(sQT, LDT, c, 16 * w + 4 * lg));
      const typename Vec4<T>::type k4 = *reinterpret_cast<const typename Vec4<T>::type*>(swc<C>(sKT, LDT, c, 16 * w + 4 * lg));
      const typename Vec4<T>::type t4 = *reinterpret_cast<const typename Vec4<T>::type*>(swc<C>(sKtT, LDT, c, 16 * w + 4 * lg));
      floatx4 oq, ok, ot;
      float xk = 0.f;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int r = 16 * w + 4 * lg + ii;
        const float lam = fast_exp(gr4[ii]);
        const float wr = fast_exp(gend - gr4[ii]);
        const float akp = fast_exp(gr4[ii] - gref) * aki[ii] - lam * A2[ii];
        oq[ii] = lam * a.scale * A1[ii] + fast_exp(gr4[ii] - gref) * aqi[ii];
        ok[ii] = bt[ii] * akp;
        const float wa3 = wr * A3[ii];
        ot[ii] = wa3 + fast_exp(gref2 - gr4[ii]) * ati[ii];
        const float qv = to_f(q4[ii]), kv = to_f(k4[ii]), tv = to_f(t4[ii]);
        pdb[ii] += kv * akp;
        xk += tv * wa3;
        sDG[r * (HC + 1) + c] = qv * oq[ii] + kv * ok[ii] - tv * ot[ii];
      }
      xk += __shfl_xor(xk, 16, 64);
      xk += __shfl_xor(xk, 32, 64);
      if (lg == 0) sXc[w * HC + c] = xk;
      T* so = sOut + w * 3 * 16 * LDO;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        so[(4 * lg + ii) * LDO + c] = from_f<T>(oq[ii]);
        so[(16 + 4 * lg + ii) * LDO + c] = from_f<T>(ok[ii]);
        so[(32 + 4 * lg + ii) * LDO + c] = from_f<T>(ot[ii]);
      }
    }
    if (rows) p12_flush_rows<T, HC, LDO, DK>(sOut + w * 3 * 16 * LDO, dqr, HD, c0, dKm, dKt, w, l);
    __syncthreads();
    {
      // dg_j = sum_{r >= j} dG_r + the last-row term, per channel: C / 8
      // segments of 8 rows, then the totals of the later segments
      const int c = tid & (HC - 1), sg = tid / HC;
      const bool seg = NSG == 8 || sg < NSG;
      float x = 0.f;
      float v[8];
#pragma unroll
      for (int q = 7; q >= 0; --q) {
        if (seg) x += sDG[(8 * sg + q) * (HC + 1) + c];
        v[q] = x;
      }
      if (seg) sSeg[sg * HC + c] = x;
      __syncthreads();
      if (seg) {
        float add = fast_exp(sGT[c * LDG + C - 1]) * sRedC[c];
#pragma unroll
        for (int q = 0; q < NB; ++q) add += sXc[q * HC + c];
        for (int q = sg + 1; q < NSG; ++q) add += sSeg[q * HC + c];
        float* dg = ba.dg + ((b * a.T + t0) * a.H + h) * DK + c0 + c;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int r = 8 * sg + q;
          if (r < n) dg[r * HD] = v[q] + add;
        }
      }
    }
  }
#pragma unroll
  for (int ii = 0; ii < 4; ++ii)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) pdb[ii] += __shfl_xor(pdb[ii], off, 64);
  if (lr == 0 && rows) {
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) sDb[16 * w + 4 * lg + ii] = pdb[ii];
  }
  __syncthreads();
  if (tid < n) ba.dbeta[(b * a.T + t0 + tid) * a.H + h] = sDb[tid] + sZV[tid];
}

// ------------------------------------------------------------ preconditioner
// Reverse scan of A_t = aP_t A_{t-1} + bP_t k_t^2, kt_t = B(A_t) k_t over the
// tokens.  With D_t the adjoint of A_t: D_t = inj_t + aP_{t+1} D_{t+1},
// inj_t = (dB/dA)(A_t) (dkt_t o k_t).  Chunk-parallel in three passes:
// pc_chunk<false> computes each chunk's local adjoint (zero carry), pc_carry
// chains the chunks (adjoint entering each chunk from the right), and
// pc_chunk<true> runs the exact recurrences and writes dk, dbetaP, dgP and
// the partial d mu.
// Sum of each of 16 per-row values over the 64 lanes of a wave; lane l
// returns the total of value l >> 2.  Static indices only: a per-lane
// choice between array elements gets merged into a runtime index by the
// compiler, which then lowers it to compare / select chains.
__device__ __forceinline__ float pc_wave_sum16(const float (&v)[16], int l) {
  // reduce-scatter: each of the lane bits 5..2 halves the values a lane
  // keeps (the half named by the bit), bits 1, 0 finish the sum, so lane l
  // ends with the total of value l >> 2
  float u[8];
  const bool b5 = l & 32, b4 = l & 16, b3 = l & 8, b2 = l & 4;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float keep = b5 ? v[k + 8] : v[k], send = b5 ? v[k] : v[k + 8];
    u[k] = keep + __shfl_xor(send, 32, 64);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float keep = b4 ? u[k + 4] : u[k], send = b4 ? u[k] : u[k + 4];
    u[k] = keep + __shfl_xor(send, 16, 64);
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float keep = b3 ? u[k + 2] : u[k], send = b3 ? u[k] : u[k + 2];
    u[k] = keep + __shfl_xor(send, 8, 64);
  }
  float x = (b2 ? u[1] : u[0]) + __shfl_xor(b2 ? u[0] : u[1], 4, 64);
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 1, 64);
  return x;
}

// One block per (b, h, chunk), one wave per segment of G = 16 tokens; lane l
// holds the CPL = d_k / 64 adjacent key channels CPL l .. CPL l + CPL - 1 of
// every token row of its segment, so each row of k, dkt, dk is one
// contiguous wave access (256 bytes for d_k = 128 in bf16) straight from
// HBM, all of a segment's rows in flight at once, and a token's sums over
// channels are reductions within one wave.  Both recurrences are
// first-order linear with a per-token factor aP_r shared by all channels.
// The summary pass (FINAL = false) scans each segment from zero and
// composes the segments through LDS:
//   forward  A_r = Ahat_r + (prod_{s0 <= j <= r} aP_j) A_in
//   reverse  send = aP_{s0} Dhat_{s0}   (what the segment sends left)
// (s0 the segment's first token, A_in the preconditioner state before it).
// It stores every segment's A_in and send; the final pass starts each
// segment from its exact A_in and from the exact adjoint entering it from
// the right (the chunk carry composed with the later segments' sends), so
// it runs one forward and one reverse recurrence and writes its outputs as
// the reverse one goes.  The per-token products come from the in-chunk
// prefix of gP.  Loop bodies are branch-free.
constexpr int PCG = 16;   // tokens per segment (one wave sum of 16 values)

template <typename T, int N>
struct alignas(sizeof(T) * N) PcPack {
  T x[N];
};

// Pins a packed row fragment to this point of the program, so that its
// unpacking is redone here instead of the unpacked values being kept alive
// from an earlier use (twice the registers).
template <typename P>
__device__ __forceinline__ P pc_pin(P p) {
  if constexpr (sizeof(P) % 4 == 0) {
    uint32_t u[sizeof(P) / 4];
    __builtin_memcpy(u, &p, sizeof(P));
#pragma unroll
    for (int i = 0; i < static_cast<int>(sizeof(P) / 4); ++i) asm volatile("" : "+v"(u[i]));
    __builtin_memcpy(&p, u, sizeof(P));
  }
  return p;
}

// A wave-uniform value (here a per-token factor read from LDS) moved to a
// scalar register: held in a vector register for every token of a segment
// it would cost one register per token.
__device__ __forceinline__ float pc_uni(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

// CPL values rounded to the row type; a bf16 pair is one packed conversion.
template <typename T, int N>
__device__ __forceinline__ PcPack<T, N> pc_pack(const float (&x)[N]) {
  PcPack<T, N> o;
  if constexpr (sizeof(T) == 2 && N == 2) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef T t16x2 __attribute__((ext_vector_type(2)));
    const f32x2 f = {x[0], x[1]};
    const t16x2 v = __builtin_convertvector(f, t16x2);
    __builtin_memcpy(&o, &v, sizeof(o));
  } else {
#pragma unroll
    for (int q = 0; q < N; ++q) o.x[q] = from_f<T>(x[q]);
  }
  return o;
}

// Stores a 2, 4 or 8 byte row fragment through a raw buffer resource.
// Offsets at or past the resource's byte range are dropped by the
// hardware's range check (no branch, so no per-row control flow for the
// compiler to schedule around).
template <typename P>
__device__ __forceinline__ void pc_store(__amdgpu_buffer_rsrc_t r, uint32_t off, const P& v) {
  if constexpr (sizeof(P) == 2) {
    unsigned short u;
    __builtin_memcpy(&u, &v, 2);
    __builtin_amdgcn_raw_buffer_store_b16(u, r, static_cast<int>(off), 0, 0);
  } else if constexpr (sizeof(P) == 4) {
    unsigned u;
    __builtin_memcpy(&u, &v, 4);
    __builtin_amdgcn_raw_buffer_store_b32(u, r, static_cast<int>(off), 0, 0);
  } else {
    static_assert(sizeof(P) == 8, "row fragment of 2, 4 or 8 bytes");
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    u32x2 u;
    __builtin_memcpy(&u, &v, 8);
    __builtin_amdgcn_raw_buffer_store_b64(u, r, static_cast<int>(off), 0, 0);
  }
}

// The adjoint injection at one token and channel, divided by -log x:
//   (dB/dA)(A) (dkt o k) / (-log x) = B(A) / A * s'(rho) dkt k,
// B(A) = exp(-log x s(rho)), rho = log A - mu, s = rho / (1 + |rho|),
// s' = 1 / (1 + |rho|)^2; zero where A <= 0 (B = x there, constant).
// B(A) / A is one exp2 of (-log x log2 e) s - log2 A.  Returns the
// injection and sets BoA = B(A) / A (finite for A > 0).
struct PcInj {
  float inj, BoA;
};
__device__ __forceinline__ PcInj pc_injection(float Ar, float gk, float kv, float mu, float nlx2) {
  // max(A, 1e-30) as an integer max: positive floats order as their bits,
  // and every A <= 0 (sign bit set, or +0) maps to the bound
  const float Ac = __int_as_float(max(__float_as_int(Ar), __float_as_int(1e-30f)));
  const float l2 = __builtin_amdgcn_logf(Ac);
  const float rr = fmaf(l2, kLn2, -mu);
  const float qd = fast_rcp(1.f + fabsf(rr));
  const float BoA = exp2_hw(fmaf(rr * qd, nlx2, -l2));
  PcInj r;
  r.inj = Ar > 0.f ? BoA * (gk * kv) * (qd * qd) : 0.f;
  r.BoA = BoA;
  return r;
}

template <typename T, int DK, bool FINAL, int C>
__global__ __launch_bounds__(64 * (C / PCG)) void pc_chunk(BwdArgs ba) {
  constexpr int PCS = C / PCG;   // segments (waves) per chunk
  constexpr int CPL = DK / 64;
  using Pk = PcPack<float, CPL>;
  using Pt = PcPack<T, CPL>;
  // per-token factors, one entry per lane (entries from C on unused)
  __shared__ float sEgp[64], sBp[64], sFf[64];
  __shared__ float sEnd[PCS][DK];          // summary pass: per-segment end values (A, then adjoint)
  // the states A_r of each wave's segment, read back in the reverse
  // recurrence (a wave reads only its own rows; kept here rather than in
  // registers, which leaves room for more waves)
  __shared__ Pk sA[PCS][PCG][64];
  __shared__ float sMu[PCS];
  const FwdArgs& a = ba.f;
  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, l = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // segment, wave-uniform
  const int s0 = PCG * w, c0 = CPL * l;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  // row bases are wave-uniform; a lane adds a 32-bit byte offset
  constexpr uint32_t E = sizeof(T);
  const uint32_t kstb = static_cast<uint32_t>(a.H * DK) * E, lo = static_cast<uint32_t>(c0) * E;
  const T* kb = static_cast<const T*>(a.k) + ((b * a.T + t0) * a.H + h) * DK;
  const T* gb = static_cast<const T*>(ba.dKt) + (bh * a.Tpad + t0) * DK;
  const T* mb = static_cast<const T*>(ba.dKm) + (bh * a.Tpad + t0) * DK;
  // per-segment values of this chunk: [BH, NT, PCS, DK]
  const int64_t segb = ((bh * a.NT + i) * PCS) * DK;
  // the per-token inputs first (lane = token; every wave loads them, so no
  // branch holds them back), then every row of the segment; rows past the
  // sequence end re-read the last row (keys are zeroed at use, dkt and dkm
  // rows there are zero)
  const int64_t lidx = (b * a.T + t0 + min(l, n - 1)) * a.H + h;
  const float vgp = a.g_p ? a.g_p[lidx] : 0.f;
  const float vbp = a.beta_p[lidx];
  // FINAL: the exact state before the segment and the adjoints the later
  // segments send (zero carry), then the chunk's carry from the right
  Pk A_seg, S_seg[PCS - 1], kap_chunk;
  if (FINAL) {
    A_seg = *reinterpret_cast<const Pk*>(ba.pcA + segb + w * DK + c0);
#pragma unroll
    for (int s = 1; s < PCS; ++s)
      if (s > w) S_seg[s - 1] = *reinterpret_cast<const Pk*>(ba.pcS + segb + s * DK + c0);
    kap_chunk = *reinterpret_cast<const Pk*>(ba.pcC + (bh * (a.NT + 1) + i + 1) * DK + c0);
  } else {
    A_seg = *reinterpret_cast<const Pk*>(a.Abound + (bh * (a.NT + 1) + i) * DK + c0);
  }
  Pt kr[PCG], gr[PCG], mr[FINAL ? PCG : 1];
#pragma unroll
  for (int j = 0; j < PCG; ++j) {
    const uint32_t rr = static_cast<uint32_t>(min(s0 + j, n - 1));
    const uint32_t ow = static_cast<uint32_t>((s0 + j) * DK) * E + lo;
    kr[j] = *reinterpret_cast<const Pt*>(at_bytes(kb, rr * kstb + lo));
    gr[j] = *reinterpret_cast<const Pt*>(at_bytes(gb, ow));
  }
  {
    // per-token factors; padded tokens: aP = 1 (gP = 0), bP = 0; x is the
    // in-chunk inclusive prefix of gP (shuffle scan over the lanes).  Every
    // wave computes and stores the same values: without a branch the
    // compiler keeps their loads ahead of the segment rows'
    const bool ok = l < n;
    const float gp = ok ? vgp : 0.f;
    float x = gp;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(x, off, 64);
      if (l >= off) x += y;
    }
    // segment composition factor prod_{s0 <= j <= r} aP_j
    const int q0 = l & ~(PCG - 1);
    const float gb = __shfl(x, q0 - 1, 64);
    sEgp[l] = fast_exp(gp);
    sBp[l] = ok ? vbp : 0.f;
    sFf[l] = fast_exp(x - (q0 > 0 ? gb : 0.f));
  }
  if (s0 + PCG > n) {   // wave-uniform: only the last chunk's tail segments
#pragma unroll
    for (int j = 0; j < PCG; ++j)
#pragma unroll
      for (int q = 0; q < CPL; ++q)
        if (s0 + j >= n) kr[j].x[q] = from_f<T>(0.f);   // keys past the end are zero
  }
  __syncthreads();
  // ---- forward: the summary pass scans from zero and composes the
  // segments; the final pass starts from the stored exact state
  // (summary pass: these are the states from zero, Ahat; the reverse
  // recurrence adds the composition term as it reads them)
  float A_in[CPL];
  {
    Pk x;
#pragma unroll
    for (int q = 0; q < CPL; ++q) x.x[q] = FINAL ? A_seg.x[q] : 0.f;
#pragma unroll
    for (int j = 0; j < PCG; ++j) {
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        const float kv = to_f(kr[j].x[q]);
        x.x[q] = fmaf(sEgp[s0 + j], x.x[q], sBp[s0 + j] * (kv * kv));
      }
      sA[w][j][l] = x;
    }
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!FINAL) sEnd[w][c0 + q] = x.x[q];
      A_in[q] = A_seg.x[q];
    }
  }
  if (!FINAL) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      float x = A_seg.x[q];
      for (int s = 0; s < w; ++s) x = sEnd[s][c0 + q] + sFf[PCG * s + PCG - 1] * x;   // segment product
      A_in[q] = x;
    }
    Pk st;
#pragma unroll
    for (int q = 0; q < CPL; ++q) st.x[q] = A_in[q];
    *reinterpret_cast<Pk*>(ba.pcA + segb + w * DK + c0) = st;
  }
  // ---- reverse.  The adjoint is carried divided by -log x (every
  // injection has that factor and the recurrence is linear), here, in the
  // segment and chunk summaries and in the carries; it is applied where
  // values leave: dk, dbetaP, dgP, d mu, dA0.
  const float mu = fast_exp(a.log_a_scale[h]);
  const float nlx = -a.lnx, nlx2 = nlx * kLog2e;
  if (!FINAL) {
    // local adjoint from zero; only what the segment sends left is kept
    Pk send;
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      float D = 0.f, aNext = 1.f;
#pragma unroll
      for (int j = PCG - 1; j >= 0; --j) {
        const float Ar = fmaf(sFf[s0 + j], A_in[q], sA[w][j][l].x[q]);
        const PcInj r = pc_injection(Ar, to_f(gr[j].x[q]), to_f(kr[j].x[q]), mu, nlx2);
        D = fmaf(aNext, D, r.inj);
        aNext = sEgp[s0 + j];
      }
      send.x[q] = aNext * D;   // aP_{s0} Dhat_{s0}
    }
    *reinterpret_cast<Pk*>(ba.pcS + segb + w * DK + c0) = send;
    __syncthreads();   // every wave is done with sEnd (forward)
#pragma unroll
    for (int q = 0; q < CPL; ++q) sEnd[w][c0 + q] = send.x[q];
    __syncthreads();
    // the adjoint this chunk sends to the left, with zero carry: aP_0 D_0
    if (w == 0)
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        float x = 0.f;
        for (int s = PCS - 1; s >= 0; --s) x = sEnd[s][c0 + q] + sFf[PCG * s + PCG - 1] * x;
        ba.pcL[(bh * a.NT + i) * DK + c0 + q] = x;
      }
    return;
  }
  // ---- final: the exact adjoint entering this segment from the right,
  // then one reverse recurrence writing dk = dKm + B dkt + 2 bP k D (times
  // the -log x the adjoint is kept divided by) and, per token, the sums
  // over channels of D k^2 and D A_{r-1}
  float D[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    float x = kap_chunk.x[q];
#pragma unroll
    for (int s = PCS - 1; s >= 1; --s)
      if (s > w) x = S_seg[s - 1].x[q] + sFf[PCG * s + PCG - 1] * x;
    D[q] = x;
  }
  // the read-key gradient rows are needed only here (fewer registers held
  // through the forward recurrence)
  // (the lane offset is pinned here too, or the compiler forms the sixteen
  // addresses before the forward recurrence and holds them through it; the
  // rows are steps of one pointer, so they become immediate offsets)
  const Pt* mrow = reinterpret_cast<const Pt*>(at_bytes(mb + s0 * DK, pc_pin(lo)));
#pragma unroll
  for (int j = 0; j < PCG; ++j) mr[j] = mrow[j * (DK / CPL)];
  const float xB = exp2_hw(-nlx2);   // B where A <= 0: x
  float sb[PCG], sg[PCG];
  float muPart = 0.f;
  T* dkb = static_cast<T*>(ba.dk) + ((b * a.T + t0) * a.H + h) * DK;
  // this (b, h, chunk)'s dk rows as a raw buffer ending with row n - 1:
  // a row r >= n starts at r kstb >= (n - 1) kstb + DK E, past the range
  const __amdgpu_buffer_rsrc_t dkr = __builtin_amdgcn_make_buffer_rsrc(
      dkb, 0, static_cast<int>((n - 1) * kstb + DK * E), kBufWord3);
  Pk Acur = sA[w][PCG - 1][l];
#pragma unroll
  for (int j = PCG - 1; j >= 0; --j) {
    const float f2 = 2.f * nlx * pc_uni(sBp[s0 + j]);
    const float aNext = j < PCG - 1 ? pc_uni(sEgp[s0 + j + 1]) : 1.f;
    Pk Aprev;
    if (j > 0) Aprev = sA[w][j - 1][l];
    else
#pragma unroll
      for (int q = 0; q < CPL; ++q) Aprev.x[q] = A_in[q];
    float o[CPL];
    const Pt kj = pc_pin(kr[j]);
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      const float Ar = Acur.x[q], kv = to_f(kj.x[q]), gk = to_f(gr[j].x[q]);
      const PcInj r = pc_injection(Ar, gk, kv, mu, nlx2);
      D[q] = fmaf(aNext, D[q], r.inj);
      const float Bv = Ar > 0.f ? r.BoA * Ar : xB;
      muPart = fmaf(-r.inj, Ar, muPart);   // -dB/dmu term: -(injection) A
      o[q] = fmaf(f2 * kv, D[q], fmaf(Bv, gk, to_f(mr[j].x[q])));
      sb[j] = q == 0 ? D[q] * (kv * kv) : fmaf(D[q], kv * kv, sb[j]);
      sg[j] = q == 0 ? D[q] * Aprev.x[q] : fmaf(D[q], Aprev.x[q], sg[j]);
    }
    Acur = Aprev;
    pc_store(dkr, static_cast<uint32_t>(s0 + j) * kstb + lo, pc_pack<T, CPL>(o));
  }
  // lane 4 j carries token s0 + j's sums
  const int jl = l >> 2;
  const int64_t sidx = (b * a.T + t0 + s0 + jl) * a.H + h;
  const bool tok = (l & 3) == 0 && s0 + jl < n;
  const float tb = pc_wave_sum16(sb, l);
  const float tg = pc_wave_sum16(sg, l);
  if (tok && ba.dbeta_p) ba.dbeta_p[sidx] = nlx * tb;
  if (tok && ba.dg_p) ba.dg_p[sidx] = nlx * sEgp[s0 + jl] * tg;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) muPart += __shfl_xor(muPart, off, 64);
  if (l == 0) sMu[w] = muPart;
  __syncthreads();
  if (tid == 0) {
    float m = 0.f;
#pragma unroll
    for (int s = 0; s < PCS; ++s) m += sMu[s];
    ba.pcMu[bh * a.NT + i] = nlx * m;
  }
}

// carry_{i-1} = L_i + exp(sumD_i) carry_i, from the last chunk (carry 0);
// summaries and carries are adjoints divided by -log x, as in pc_chunk
// The chunks' local adjoints chained from the right, carry_i = L_i +
// exp(D_i) carry_{i+1} (zero past the last chunk); pcC[i + 1] holds the
// carry entering chunk i.  16 channels x 16 chunk segments a workgroup:
// each segment reduces to its affine map, a segment's entering carry chains
// the maps of the segments to its right, and each segment re-walks its
// chunks writing the carries.
constexpr int kPcCh = 16, kPcSeg = 16;
template <int DK>
__global__ __launch_bounds__(256) void pc_carry(BwdArgs ba) {
  __shared__ float sE[kPcSeg][kPcCh], sP[kPcSeg][kPcCh];
  const FwdArgs& a = ba.f;
  const int64_t bh = blockIdx.x / (DK / kPcCh);
  const int ch = threadIdx.x % kPcCh, sg = threadIdx.x / kPcCh;
  const int c = static_cast<int>(blockIdx.x % (DK / kPcCh)) * kPcCh + ch;
  const int NT = a.NT, Ls = (NT + kPcSeg - 1) / kPcSeg;
  const int i0 = min(NT, sg * Ls), i1 = min(NT, i0 + Ls);
  float* out = ba.pcC + bh * (NT + 1) * DK + c;
  const float* L = ba.pcL + bh * NT * DK + c;
  const float* D = a.sumD + bh * NT;
  float E = 1.f, P = 0.f;
#pragma unroll 8
  for (int i = i1 - 1; i >= i0; --i) {
    const float e = fast_exp(D[i]);
    E *= e;
    P = L[(int64_t)i * DK] + e * P;
  }
  sE[sg][ch] = E;
  sP[sg][ch] = P;
  __syncthreads();
  float carry = 0.f;
  if (sg == kPcSeg - 1) out[(int64_t)NT * DK] = 0.f;
  for (int q = kPcSeg - 1; q > sg; --q) carry = sP[q][ch] + sE[q][ch] * carry;
#pragma unroll 8
  for (int i = i1 - 1; i >= i0; --i) {
    out[(int64_t)(i + 1) * DK] = carry;
    carry = L[(int64_t)i * DK] + fast_exp(D[i]) * carry;
  }
  // carries are kept divided by -log x
  if (ba.dA0 && sg == 0) ba.dA0[bh * DK + c] = -a.lnx * carry;
}

// d logAScale_h = mu_h * sum over batches and chunks of the partial d mu
__global__ void pc_mu(BwdArgs ba) {
  const FwdArgs& a = ba.f;
  const int64_t h = blockIdx.x;
  float s = 0.f;
  for (int64_t idx = threadIdx.x; idx < a.B * a.NT; idx += blockDim.x) {
    const int64_t b = idx / a.NT, i = idx % a.NT;
    s += ba.pcMu[(b * a.H + h) * a.NT + i];
  }
  __shared__ float red[256];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (static_cast<int>(threadIdx.x) < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) ba.dlog_a_scale[h] = fast_exp(a.log_a_scale[h]) * red[0];
}

// identity / external write key: dk = dKm (+ dKt), dktilde = dKt
template <typename T, int DK>
__global__ __launch_bounds__(256) void combine_dk(BwdArgs ba) {
  const FwdArgs& a = ba.f;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t tot = a.B * a.T * a.H * DK;
  if (idx >= tot) return;
  const int c = static_cast<int>(idx % DK);
  const int64_t tok = idx / DK;
  const int64_t h = tok % a.H, t = (tok / a.H) % a.T, b = tok / (a.H * a.T);
  const int64_t w = ((b * a.H + h) * a.Tpad + t) * DK + c;
  const float km = to_f(static_cast<const T*>(ba.dKm)[w]), kt = to_f(static_cast<const T*>(ba.dKt)[w]);
  if (a.precond == kIdentity) {
    static_cast<T*>(ba.dk)[idx] = from_f<T>(km + kt);
  } else {
    static_cast<T*>(ba.dk)[idx] = from_f<T>(km);
    if (ba.dktilde) static_cast<T*>(ba.dktilde)[idx] = from_f<T>(kt);
  }
}

// ------------------------------------------------------------ host side
static size_t align256b(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

BwdWsLayout bwd_ws_layout(int64_t BH, int NT, int dk, int dv, int esz, int gate, int precond, int C) {
  const int PCS = C / PCG;
  BwdWsLayout L{};
  L.f = fwd_ws_layout(BH, NT, dk, dv, esz, gate, precond, C);
  size_t off = L.f.total;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256b(off + bytes); return o; };
  const size_t bh = static_cast<size_t>(BH), nt = static_cast<size_t>(NT), tp = nt * C;
  L.Hs = take(bh * nt * dk * dv * esz);
  L.Er = take(bh * tp * dv * esz);
  L.PtT = take(bh * nt * C * C * esz);
  L.MtT = take(bh * nt * C * C * esz);
  L.Ktr = take(bh * tp * dk * esz);
  L.Kw = gate == kGateChannel ? take(bh * tp * dk * esz) : 0;   // = w_r Kt rows, per-channel gate only
  L.QlT = take(bh * nt * dk * C * esz);
  L.KnT = take(bh * nt * dk * C * esz);
  L.dHs = take(bh * nt * dk * dv * esz);
  L.Zr = take(bh * tp * dv * esz);
  L.dKt = take(bh * tp * dk * esz);
  L.dKm = take(bh * tp * dk * esz);
  L.pcL = take(bh * nt * dk * 4);
  L.pcS = take(bh * nt * PCS * dk * 4);
  L.pcA = take(bh * nt * PCS * dk * 4);
  L.pcC = take(bh * (nt + 1) * dk * 4);
  L.pcMu = take(bh * nt * 4);
  L.total = off;
  return L;
}

hipError_t launch_forward_parts(const FwdArgs& a, int io_bf16, hipStream_t s, hipEvent_t const* ev);

template <typename T, int DK, int DV, int GATE, int C>
static hipError_t launch_bwd_typed(const BwdArgs& ba, hipStream_t s, hipEvent_t const* ev) {
  constexpr int PCS = C / PCG;
  const FwdArgs& a = ba.f;
  hipError_t e;
  auto mark = [&](int i) { return ev && ev[i] ? hipEventRecord(ev[i], s) : hipSuccess; };
  const int nslab = DV / BVB, npslab = DK / BVB;
  auto grid_scan = [&](int nrole) { return dim3(static_cast<unsigned>(((a.BH + 7) / 8) * 8 * nrole)); };
  const unsigned grid_chunk = static_cast<unsigned>(a.BH * a.NT);
  if (a.seg_cnt < 3) {
    BwdArgs b0 = ba;
    b0.f.seg_phase = 0;
    hipLaunchKernelGGL((r1_state_adjoint<T, DK, GATE, C>), grid_scan(nslab), dim3(256), 0, s, b0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else {
    // split reverse scan: the last segment beside the middle segments'
    // local runs and transitions, the composed starts, then segments
    // 0 .. S - 2 (the first pass's middle runs also write dHs, Z and dv rows
    // for their chunks from the wrong start; the third pass overwrites them)
    const int S = a.seg_cnt;
    BwdArgs b1 = ba;
    b1.f.seg_phase = 1;
    hipLaunchKernelGGL((r1_state_adjoint<T, DK, GATE, C>), grid_scan(nslab + (S - 2) * (nslab + npslab)),
                       dim3(256), 0, s, b1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_seg_compose(b1.f, true, s)) != hipSuccess) return e;
    b1.f.seg_phase = 3;
    hipLaunchKernelGGL((r1_state_adjoint<T, DK, GATE, C>), grid_scan((S - 1) * nslab), dim3(256), 0, s, b1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if ((e = mark(4)) != hipSuccess) return e;
  if constexpr (GATE == kGateChannel)
    hipLaunchKernelGGL((p12c_chunk_grads<T, DK, DV, C>), dim3(grid_chunk), dim3(256), 0, s, ba);
  else
    hipLaunchKernelGGL((p12_chunk_grads<T, DK, DV, GATE, C>), dim3(grid_chunk), dim3(256), 0, s, ba);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = mark(5)) != hipSuccess) return e;
  if (a.precond == kSquash) {
    hipLaunchKernelGGL((pc_chunk<T, DK, false, C>), dim3(grid_chunk), dim3(64 * PCS), 0, s, ba);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((pc_carry<DK>), dim3(static_cast<unsigned>(a.BH * (DK / kPcCh))), dim3(256), 0, s, ba);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((pc_chunk<T, DK, true, C>), dim3(grid_chunk), dim3(64 * PCS), 0, s, ba);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ba.dlog_a_scale) {
      hipLaunchKernelGGL(pc_mu, dim3(static_cast<unsigned>(a.H)), dim3(256), 0, s, ba);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  } else {
    const int64_t tot = a.B * a.T * a.H * DK;
    hipLaunchKernelGGL((combine_dk<T, DK>), dim3(static_cast<unsigned>((tot + 255) / 256)), dim3(256), 0,
                       s, ba);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return mark(6);
}

template <typename T, int DK, int DV, int C>
static hipError_t launch_bwd_gate_c(const BwdArgs& ba, hipStream_t s, hipEvent_t const* ev) {
  switch (ba.f.gate) {
    case kGateNone: return launch_bwd_typed<T, DK, DV, kGateNone, C>(ba, s, ev);
    case kGateScalar: return launch_bwd_typed<T, DK, DV, kGateScalar, C>(ba, s, ev);
    default: return launch_bwd_typed<T, DK, DV, kGateChannel, C>(ba, s, ev);
  }
}

template <typename T, int DK, int DV>
static hipError_t launch_bwd_gate(const BwdArgs& ba, hipStream_t s, hipEvent_t const* ev) {
  return ba.f.chunk == 32 ? launch_bwd_gate_c<T, DK, DV, 32>(ba, s, ev)
                          : launch_bwd_gate_c<T, DK, DV, 64>(ba, s, ev);
}

// fp32 io: head dims 64 only (LDS); the host validates this
static hipError_t launch_bwd_f32(const BwdArgs& ba, hipStream_t s, hipEvent_t const* ev) {
  return launch_bwd_gate<float, 64, 64>(ba, s, ev);
}

template <typename T>
static hipError_t launch_bwd_dims(const BwdArgs& ba, hipStream_t s, hipEvent_t const* ev) {
  const FwdArgs& a = ba.f;
  if (a.dk == 128 && a.dv == 128) return launch_bwd_gate<T, 128, 128>(ba, s, ev);
  if (a.dk == 128 && a.dv == 64) return launch_bwd_gate<T, 128, 64>(ba, s, ev);
  if (a.dk == 64 && a.dv == 128) return launch_bwd_gate<T, 64, 128>(ba, s, ev);
  return launch_bwd_gate<T, 64, 64>(ba, s, ev);
}

hipError_t launch_backward(const BwdArgs& ba, int io_bf16, hipStream_t s, hipEvent_t const* ev,
                           bool recompute) {
  hipError_t e = hipSuccess;
  if (recompute) {
    e = launch_forward_parts(ba.f, io_bf16, s, ev);
  } else if (ev) {   // no recompute: its stages are empty
    for (int k = 0; k < 4 && e == hipSuccess; ++k)
      if (ev[k]) e = hipEventRecord(ev[k], s);
  }
  if (e != hipSuccess) return e;
  return io_bf16 ? launch_bwd_dims<bf16>(ba, s, ev) : launch_bwd_f32(ba, s, ev);
}

}  // namespace pdn
