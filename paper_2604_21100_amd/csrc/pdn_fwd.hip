// Forward kernels of the chunkwise preconditioned delta rule for gfx950.
//
//   k1_precond_summary  per chunk: decayed in-chunk sum of betaP k^2 and the
//                       chunk's total log-decay (the affine summary of the
//                       diagonal Gram recurrence over one chunk, App. D Eq.
//                       precond_from_boundary)
//   k1_precond_carry    per head: chains the summaries into the state before
//                       every chunk (d_k-wide, sequential over chunks)
//   k2_chunk_prep       per (head, chunk): in-chunk preconditioner prefix and
//                       write key (Eq. precond_end2end), gate prefix, the
//                       interaction matrices At (strict lower) and P (causal)
//                       on MFMA, the unit-lower inverse T = (I+At)^{-1}Diag(beta)
//                       (Eq. T_two_key) and the decayed write keys for the
//                       state update
//   k3_chunk_scan       per (head, 32-column value slab): the sequential
//                       inter-chunk state scan with the chunk output fused in
//                       (Eq. chunkwise_atk_form; decayed forms of App. D),
//                       using E = U - W S^T = T (V - (Lam*K) S^T)
#include "pdn_device.hpp"
#include "pdn_internal.hpp"

namespace pdn {

constexpr int C = kChunk;

// ---------------------------------------------------------------- K1
template <typename T, int DK>
__global__ __launch_bounds__(DK) void k1_precond_summary(FwdArgs a) {
  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int c = threadIdx.x;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  const T* k = static_cast<const T*>(a.k);
  float L = 0.f, D = 0.f;
  for (int r = 0; r < n; ++r) {
    const int64_t sidx = (b * a.T + t0 + r) * a.H + h;
    const float gp = a.g_p ? a.g_p[sidx] : 0.f;
    const float kv = to_f(k[sidx * DK + c]);
    L = fast_exp(gp) * L + a.beta_p[sidx] * kv * kv;
    D += gp;
  }
  a.sumL[(bh * a.NT + i) * DK + c] = L;
  if (c == 0) a.sumD[bh * a.NT + i] = D;
}

template <int DK>
__global__ __launch_bounds__(DK) void k1_precond_carry(FwdArgs a) {
  const int64_t bh = blockIdx.x;
  const int c = threadIdx.x;
  float A = a.A0 ? a.A0[bh * DK + c] : 0.f;
  float* out = a.Abound + bh * (a.NT + 1) * DK + c;
  const float* L = a.sumL + bh * a.NT * DK + c;
  const float* D = a.sumD + bh * a.NT;
  out[0] = A;
  int i = 0;
  for (; i + 8 <= a.NT; i += 8) {
    float d[8], l[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) { d[u] = D[i + u]; l[u] = L[(int64_t)(i + u) * DK]; }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      A = fast_exp(d[u]) * A + l[u];
      out[(int64_t)(i + u + 1) * DK] = A;
    }
  }
  for (; i < a.NT; ++i) {
    A = fast_exp(D[i]) * A + L[(int64_t)i * DK];
    out[(int64_t)(i + 1) * DK] = A;
  }
  if (a.A_T) a.A_T[bh * DK + c] = A;
}

// ---------------------------------------------------------------- K2
template <typename T, int DK, int GATE>
struct K2Smem {
  static constexpr int LDK = DK + 8;          // padded row (elements)
  static constexpr int LDA = C + 4;           // fp32 C x C rows
  static constexpr size_t kRow = sizeof(T) * C * LDK;
  static constexpr size_t kFloatCC = sizeof(float) * C * LDA;
  static constexpr size_t kR1 = kRow > kFloatCC ? kRow : kFloatCC;  // sK, later sA
  static constexpr size_t kR2 = kR1;                                // sQ, later sX
  static constexpr size_t kR3 = kRow;                               // sKt
  static constexpr size_t kGc = GATE == kGateChannel ? sizeof(float) * C * (DK + 4) : 0;
  static constexpr size_t kY = sizeof(float) * 4 * 16 * 17;
  static constexpr size_t kScal = sizeof(float) * 5 * C;
  static constexpr size_t kTotal = kR1 + kR2 + kR3 + kGc + kY + kScal;
};

template <typename T, int DK, int GATE, int PREC>
__global__ __launch_bounds__(256) void k2_chunk_prep(FwdArgs a) {
  using SM = K2Smem<T, DK, GATE>;
  constexpr int LDK = SM::LDK, LDA = SM::LDA;
  __shared__ __attribute__((aligned(16))) char smem[SM::kTotal];
  T* sK = reinterpret_cast<T*>(smem);
  float* sA = reinterpret_cast<float*>(smem);
  T* sQ = reinterpret_cast<T*>(smem + SM::kR1);
  float* sX = reinterpret_cast<float*>(smem + SM::kR1);
  T* sKt = reinterpret_cast<T*>(smem + SM::kR1 + SM::kR2);
  float* sGc = reinterpret_cast<float*>(smem + SM::kR1 + SM::kR2 + SM::kR3);
  float* sY = reinterpret_cast<float*>(smem + SM::kR1 + SM::kR2 + SM::kR3 + SM::kGc);
  float* sBeta = sY + 4 * 16 * 17;
  float* sBp = sBeta + C;
  float* sEgp = sBp + C;
  float* sG = sEgp + C;
  float* sGraw = sG + C;

  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  constexpr int VEC = 16 / sizeof(T);
  constexpr int VPR = DK / VEC;  // vectors per row

  // ---- load key, query (and external write key) tiles, zero-padded
  {
    const T* kp = static_cast<const T*>(a.k);
    const T* qp = static_cast<const T*>(a.q);
    const T* xp = static_cast<const T*>(a.ktilde);
    for (int idx = tid; idx < C * VPR; idx += 256) {
      const int r = idx / VPR, cv = idx % VPR;
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), qv = kv, xv = kv;
      if (r < n) {
        const int64_t off = ((b * a.T + t0 + r) * a.H + h) * DK + cv * VEC;
        kv = *reinterpret_cast<const float4*>(kp + off);
        qv = *reinterpret_cast<const float4*>(qp + off);
        if (PREC == kExternal) xv = *reinterpret_cast<const float4*>(xp + off);
      }
      *reinterpret_cast<float4*>(sK + r * LDK + cv * VEC) = kv;
      *reinterpret_cast<float4*>(sQ + r * LDK + cv * VEC) = qv;
      // identity write key: a copy of the key tile (the key tile's memory is
      // reused by the solve)
      if (PREC == kIdentity) *reinterpret_cast<float4*>(sKt + r * LDK + cv * VEC) = kv;
      if (PREC == kExternal) *reinterpret_cast<float4*>(sKt + r * LDK + cv * VEC) = xv;
    }
    if (tid < C) {
      const int r = tid;
      const bool ok = r < n;
      const int64_t sidx = (b * a.T + t0 + r) * a.H + h;
      sBeta[r] = ok ? a.beta[sidx] : 0.f;
      if (PREC == kSquash) {
        sBp[r] = ok ? a.beta_p[sidx] : 0.f;
        sEgp[r] = (ok && a.g_p) ? fast_exp(a.g_p[sidx]) : 1.f;
      }
      if (GATE == kGateScalar) sGraw[r] = ok ? a.g[sidx] : 0.f;
    }
    if (GATE == kGateChannel) {
      for (int idx = tid; idx < C * (DK / 4); idx += 256) {
        const int r = idx / (DK / 4), c4 = idx % (DK / 4);
        float4 gv = make_float4(0.f, 0.f, 0.f, 0.f);
        if (r < n)
          gv = *reinterpret_cast<const float4*>(a.g + ((b * a.T + t0 + r) * a.H + h) * DK + c4 * 4);
        *reinterpret_cast<float4*>(sGc + r * (DK + 4) + c4 * 4) = gv;
      }
    }
  }
  __syncthreads();

  // ---- gate prefix and preconditioner prefix
  if (GATE == kGateScalar && w == 0) {
    float x = sGraw[l];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(x, off, 64);
      if (l >= off) x += y;
    }
    sG[l] = x;
    a.G[bh * a.Tpad + t0 + l] = x;
  }
  if (tid < DK) {
    const int c = tid;
    if (GATE == kGateChannel) {
      float acc = 0.f;
      float* gout = a.G + (bh * a.Tpad + t0) * DK + c;
      for (int r = 0; r < C; ++r) {
        acc += sGc[r * (DK + 4) + c];
        sGc[r * (DK + 4) + c] = acc;
        gout[(int64_t)r * DK] = acc;
      }
    }
    if (PREC == kSquash) {
      float A = a.Abound[(bh * (a.NT + 1) + i) * DK + c];
      const float mu = fast_exp(a.log_a_scale[h]);
      for (int r = 0; r < C; ++r) {
        const float kv = to_f(sK[r * LDK + c]);
        A = sEgp[r] * A + sBp[r] * kv * kv;
        sKt[r * LDK + c] = from_f<T>(squash_gain(A, mu, a.lnx) * kv);
      }
    }
  }
  __syncthreads();

  // ---- interaction matrices on MFMA: wave w owns row block w
  floatx4 accA[4], accP[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) { accA[j] = floatx4{0.f, 0.f, 0.f, 0.f}; accP[j] = accA[j]; }
  {
    const int r = 16 * w + lr;  // A-operand row of this lane
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j > w) break;
      const int t = 16 * j + lr;  // B-operand column of this lane
#pragma unroll
      for (int kk = 0; kk < DK / 32; ++kk) {
        const int c0 = kk * 32 + 8 * lg;
        Frag8<T> fk = ld8(sK + r * LDK + c0);
        Frag8<T> fq = ld8(sQ + r * LDK + c0);
        Frag8<T> fb = ld8(sKt + t * LDK + c0);
        if (GATE == kGateChannel) {
          // reference point: first row of the row block keeps both factors
          // bounded for a non-increasing prefix
          const float* gr = sGc + r * (DK + 4) + c0;
          const float* gref = sGc + (16 * w) * (DK + 4) + c0;
          const float* gt = sGc + t * (DK + 4) + c0;
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            const float fa = fast_exp(gr[s] - gref[s]);
            fk.set(s, fk.get(s) * fa);
            fq.set(s, fq.get(s) * fa);
            fb.set(s, fb.get(s) * fast_exp(gref[s] - gt[s]));
          }
        }
        mma(accA[j], fk, fb);
        mma(accP[j], fq, fb);
      }
    }
  }
  // masks, beta and scalar decay; P goes straight to the workspace
  {
    T* P = static_cast<T*>(a.Pm) + (bh * a.NT + i) * (int64_t)(C * C);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = 16 * j + lr;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int r = 16 * w + 4 * lg + ii;
        float fac = 1.f;
        if (GATE == kGateScalar) fac = fast_exp(sG[r] - sG[t]);
        const float pv = (j <= w && r >= t) ? accP[j][ii] * fac : 0.f;
        accA[j][ii] = (j <= w && r > t) ? sBeta[r] * accA[j][ii] * fac : 0.f;
        P[r * C + t] = from_f<T>(pv);
      }
    }
  }
  __syncthreads();  // sK / sQ are free from here on
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j > w) break;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) sA[(16 * w + 4 * lg + ii) * LDA + 16 * j + lr] = accA[j][ii];
  }
  __syncthreads();

  // ---- X = (I + At)^{-1}: diagonal 16x16 blocks by forward substitution
  if (lg == 0) {
    const int col = lr;
    const float* Ab = sA + (16 * w) * LDA + 16 * w;
    float x[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float s = (r == col) ? 1.f : 0.f;
#pragma unroll
      for (int t = 0; t < r; ++t) s -= Ab[r * LDA + t] * x[t];
      x[r] = s;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) sX[(16 * w + r) * LDA + 16 * w + col] = x[r];
  }
  __syncthreads();
  // off-diagonal blocks, by distance from the diagonal:
  //   X_ij = -X_ii * sum_{j <= m < i} At_im X_mj
  float* Yw = sY + w * 16 * 17;
  for (int d = 1; d < 4; ++d) {
    const int j = w, ib = w + d;
    const bool active = ib < 4;
    floatx4 y = {0.f, 0.f, 0.f, 0.f};
    if (active) {
      for (int kb = 0; kb < 4 * d; ++kb) {
        const float av = sA[(16 * ib + lr) * LDA + 16 * j + 4 * kb + lg];
        const float bv = sX[(16 * j + 4 * kb + lg) * LDA + 16 * j + lr];
        mma4(y, av, bv);
      }
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) Yw[(4 * lg + ii) * 17 + lr] = y[ii];
    }
    __syncthreads();
    if (active) {
      floatx4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const float av = sX[(16 * ib + lr) * LDA + 16 * ib + 4 * kb + lg];
        const float bv = Yw[(4 * kb + lg) * 17 + lr];
        mma4(z, av, bv);
      }
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) sX[(16 * ib + 4 * lg + ii) * LDA + 16 * j + lr] = -z[ii];
    }
    __syncthreads();
  }

  // ---- T = X Diag(beta) (block-lower; upper blocks are zero)
  {
    T* Tout = static_cast<T*>(a.Tm) + (bh * a.NT + i) * (int64_t)(C * C);
    for (int idx = tid; idx < C * C / 8; idx += 256) {
      const int r = idx / (C / 8), t0v = (idx % (C / 8)) * 8;
      Frag8<T> f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = t0v + s;
        const bool lower = (t >> 4) < (r >> 4) || ((t >> 4) == (r >> 4) && t <= r);
        f.set(s, lower ? sX[r * LDA + t] * sBeta[t] : 0.f);
      }
      st8(Tout + r * C + t0v, f);
    }
  }
  // ---- decayed write keys, transposed per chunk: (Kt * Lam_C / Lam_t)^T
  {
    T* Kout = static_cast<T*>(a.KtG) + (bh * a.NT + i) * (int64_t)(DK * C);
    for (int idx = tid; idx < DK * C / 8; idx += 256) {
      const int c = idx / (C / 8), tv = (idx % (C / 8)) * 8;
      Frag8<T> f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = tv + s;
        float val = to_f(sKt[t * LDK + c]);
        if (GATE == kGateScalar) val *= fast_exp(sG[C - 1] - sG[t]);
        if (GATE == kGateChannel) val *= fast_exp(sGc[(C - 1) * (DK + 4) + c] - sGc[t * (DK + 4) + c]);
        f.set(s, val);
      }
      st8(Kout + c * C + tv, f);
    }
  }
}

// ---------------------------------------------------------------- K3
constexpr int BV = 32;  // value columns per workgroup

template <typename T, int DK, int GATE>
__global__ __launch_bounds__(256) void k3_chunk_scan(FwdArgs a) {
  constexpr int CT = DK / 64;       // state row tiles per wave
  constexpr int KK = DK / 32;       // contraction slabs over d_k
  constexpr int LDH = DK + 8, LDE = C + 8;
  __shared__ __attribute__((aligned(16))) T sH[BV * LDH];  // bf16/fp32 copy of S^T slab, [v][c]
  __shared__ __attribute__((aligned(16))) T sX[BV * LDE];  // X = V - Lam K S^T, [v][t]
  __shared__ __attribute__((aligned(16))) T sE[BV * LDE];  // E = T X, [v][t]

  const int nslab = a.dv / BV;
  const int64_t bid = blockIdx.x;
  const int xcd = static_cast<int>(bid & 7);
  const int64_t j8 = bid >> 3;
  const int slab = static_cast<int>(j8 % nslab);
  const int64_t bh = (j8 / nslab) * 8 + xcd;  // slabs of one head share an XCD (and its L2)
  if (bh >= a.BH) return;
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const int v0 = slab * BV;
  const int DV = a.dv;
  const T* qp = static_cast<const T*>(a.q);
  const T* kp = static_cast<const T*>(a.k);
  const T* vp = static_cast<const T*>(a.v);
  T* op = static_cast<T*>(a.o);
  const T* Tm = static_cast<const T*>(a.Tm);
  const T* Pm = static_cast<const T*>(a.Pm);
  const T* KtG = static_cast<const T*>(a.KtG);

  // state slab: rows c = 16*(w*CT+ct) + 4*lg + ii, column v0 + 16*vt + lr
  floatx4 st[CT][2];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int c = 16 * (w * CT + ct) + 4 * lg + ii;
        st[ct][vt][ii] = a.S0 ? a.S0[(bh * DK + c) * DV + v0 + 16 * vt + lr] : 0.f;
      }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      st4<T>(sH + (16 * vt + lr) * LDH + 16 * (w * CT + ct) + 4 * lg, st[ct][vt][0],
             st[ct][vt][1], st[ct][vt][2], st[ct][vt][3]);
  __syncthreads();

  const int rr = 16 * w + lr;  // A-operand row (token in chunk) of this lane
  for (int i = 0; i < a.NT; ++i) {
    const int64_t t0 = static_cast<int64_t>(i) * C;
    const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
    // ---- operand fragments for this wave
    Frag8<T> fK[KK], fQ[KK], fT[2], fP[2], fG[CT][2];
    const bool rok = rr < n;
    const int64_t rowoff = ((b * a.T + t0 + rr) * a.H + h) * DK;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (rok) {
        fK[kk] = ld8(kp + rowoff + kk * 32 + 8 * lg);
        fQ[kk] = ld8(qp + rowoff + kk * 32 + 8 * lg);
      } else {
        fK[kk] = frag_zero<T>();
        fQ[kk] = frag_zero<T>();
      }
    }
    const int64_t cc = (bh * a.NT + i) * (int64_t)(C * C);
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      fT[k2] = ld8(Tm + cc + rr * C + k2 * 32 + 8 * lg);
      fP[k2] = ld8(Pm + cc + rr * C + k2 * 32 + 8 * lg);
    }
    const int64_t kg = (bh * a.NT + i) * (int64_t)(DK * C);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
        fG[ct][k2] = ld8(KtG + kg + (16 * (w * CT + ct) + lr) * C + k2 * 32 + 8 * lg);
    // values in accumulator layout: rows 16w + 4lg + ii, column v0 + 16vt + lr
    float vv[2][4], lam[4];
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int t = 16 * w + 4 * lg + ii;
      lam[ii] = 1.f;
      if (GATE == kGateScalar) lam[ii] = fast_exp(a.G[bh * a.Tpad + t0 + t]);
#pragma unroll
      for (int vt = 0; vt < 2; ++vt)
        vv[vt][ii] = t < n ? to_f(vp[((b * a.T + t0 + t) * a.H + h) * DV + v0 + 16 * vt + lr]) : 0.f;
    }
    if (GATE == kGateChannel) {
      // Lam = exp(G) per (token, channel) on the read key and the query
      const float* gr = a.G + (bh * a.Tpad + t0 + rr) * DK;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const float e = fast_exp(gr[kk * 32 + 8 * lg + s]);
          fK[kk].set(s, fK[kk].get(s) * e);
          fQ[kk].set(s, fQ[kk].get(s) * e);
        }
    }

    // ---- (Lam K) S^T and (Lam Q) S^T
    floatx4 accX[2], accO[2];
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
      accX[vt] = floatx4{0.f, 0.f, 0.f, 0.f};
      accO[vt] = accX[vt];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const Frag8<T> bH = ld8(sH + (16 * vt + lr) * LDH + kk * 32 + 8 * lg);
        mma(accX[vt], fK[kk], bH);
        mma(accO[vt], fQ[kk], bH);
      }
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        accX[vt][ii] = vv[vt][ii] - lam[ii] * accX[vt][ii];
        accO[vt][ii] *= lam[ii];
      }
      st4<T>(sX + (16 * vt + lr) * LDE + 16 * w + 4 * lg, accX[vt][0], accX[vt][1], accX[vt][2],
             accX[vt][3]);
    }
    __syncthreads();

    // ---- E = T X
    floatx4 accE[2];
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
      accE[vt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
        mma(accE[vt], fT[k2], ld8(sX + (16 * vt + lr) * LDE + k2 * 32 + 8 * lg));
      st4<T>(sE + (16 * vt + lr) * LDE + 16 * w + 4 * lg, accE[vt][0], accE[vt][1], accE[vt][2],
             accE[vt][3]);
    }
    __syncthreads();

    // ---- O = scale [ (Lam Q) S^T + P E ];  S^T <- Diag(gamma_C) S^T + (Kt Gamma)^T E
    Frag8<T> fE[2][2];
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) fE[vt][k2] = ld8(sE + (16 * vt + lr) * LDE + k2 * 32 + 8 * lg);
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
      mma(accO[vt], fP[0], fE[vt][0]);
      if (w >= 2) mma(accO[vt], fP[1], fE[vt][1]);
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int t = 16 * w + 4 * lg + ii;
        if (t < n) op[((b * a.T + t0 + t) * a.H + h) * DV + v0 + 16 * vt + lr] = from_f<T>(a.scale * accO[vt][ii]);
      }
    }
    float gam[CT][4];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        gam[ct][ii] = 1.f;
        if (GATE == kGateScalar) gam[ct][ii] = fast_exp(a.G[bh * a.Tpad + t0 + C - 1]);
        if (GATE == kGateChannel)
          gam[ct][ii] = fast_exp(a.G[(bh * a.Tpad + t0 + C - 1) * DK + 16 * (w * CT + ct) + 4 * lg + ii]);
      }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int vt = 0; vt < 2; ++vt) {
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) st[ct][vt][ii] *= gam[ct][ii];
        mma(st[ct][vt], fG[ct][0], fE[vt][0]);
        mma(st[ct][vt], fG[ct][1], fE[vt][1]);
        st4<T>(sH + (16 * vt + lr) * LDH + 16 * (w * CT + ct) + 4 * lg, st[ct][vt][0], st[ct][vt][1],
               st[ct][vt][2], st[ct][vt][3]);
      }
    __syncthreads();
  }
  if (a.S_T) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int vt = 0; vt < 2; ++vt)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int c = 16 * (w * CT + ct) + 4 * lg + ii;
          a.S_T[(bh * DK + c) * DV + v0 + 16 * vt + lr] = st[ct][vt][ii];
        }
  }
}

// ---------------------------------------------------------------- T == 0
__global__ void k0_copy_states(FwdArgs a, int64_t nS, int64_t nA) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (a.S_T && idx < nS) a.S_T[idx] = a.S0 ? a.S0[idx] : 0.f;
  if (a.A_T && idx < nA) a.A_T[idx] = a.A0 ? a.A0[idx] : 0.f;
}

// ---------------------------------------------------------------- host side
static size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

WsLayout fwd_ws_layout(int64_t BH, int NT, int dk, int esz, int gate, int precond) {
  WsLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256(off + bytes); return o; };
  const size_t bh = static_cast<size_t>(BH), nt = static_cast<size_t>(NT);
  if (precond == kSquash) {
    L.sumL = take(bh * nt * dk * 4);
    L.sumD = take(bh * nt * 4);
    L.Abound = take(bh * (nt + 1) * dk * 4);
  }
  L.KtG = take(bh * nt * dk * C * esz);
  L.Tm = take(bh * nt * C * C * esz);
  L.Pm = take(bh * nt * C * C * esz);
  if (gate == kGateScalar) L.G = take(bh * nt * C * 4);
  if (gate == kGateChannel) L.G = take(bh * nt * C * dk * 4);
  L.total = off;
  return L;
}

template <typename T, int DK, int GATE, int PREC>
static hipError_t launch_k2(const FwdArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k2_chunk_prep<T, DK, GATE, PREC>), dim3(static_cast<unsigned>(a.BH * a.NT)),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int DK, int GATE>
static hipError_t launch_k2_prec(const FwdArgs& a, hipStream_t s) {
  switch (a.precond) {
    case kSquash: return launch_k2<T, DK, GATE, kSquash>(a, s);
    case kIdentity: return launch_k2<T, DK, GATE, kIdentity>(a, s);
    default: return launch_k2<T, DK, GATE, kExternal>(a, s);
  }
}

template <typename T, int DK>
static hipError_t launch_all(const FwdArgs& a, hipStream_t s, hipEvent_t const* ev) {
  hipError_t e;
  auto mark = [&](int i) { return ev ? hipEventRecord(ev[i], s) : hipSuccess; };
  if ((e = mark(0)) != hipSuccess) return e;
  if (a.precond == kSquash) {
    hipLaunchKernelGGL((k1_precond_summary<T, DK>), dim3(static_cast<unsigned>(a.BH * a.NT)), dim3(DK),
                       0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((k1_precond_carry<DK>), dim3(static_cast<unsigned>(a.BH)), dim3(DK), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if ((e = mark(1)) != hipSuccess) return e;
  switch (a.gate) {
    case kGateNone: e = launch_k2_prec<T, DK, kGateNone>(a, s); break;
    case kGateScalar: e = launch_k2_prec<T, DK, kGateScalar>(a, s); break;
    default: e = launch_k2_prec<T, DK, kGateChannel>(a, s); break;
  }
  if (e != hipSuccess) return e;
  if ((e = mark(2)) != hipSuccess) return e;
  const int64_t nslab = a.dv / BV;
  const unsigned grid = static_cast<unsigned>(((a.BH + 7) / 8) * 8 * nslab);
  switch (a.gate) {
    case kGateNone:
      hipLaunchKernelGGL((k3_chunk_scan<T, DK, kGateNone>), dim3(grid), dim3(256), 0, s, a); break;
    case kGateScalar:
      hipLaunchKernelGGL((k3_chunk_scan<T, DK, kGateScalar>), dim3(grid), dim3(256), 0, s, a); break;
    default:
      hipLaunchKernelGGL((k3_chunk_scan<T, DK, kGateChannel>), dim3(grid), dim3(256), 0, s, a); break;
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return mark(3);
}

hipError_t launch_forward(const FwdArgs& a, int io_bf16, hipStream_t s, hipEvent_t const* ev) {
  if (a.BH == 0 || a.T == 0) {
    // nothing to time: the stage events still mark the (empty) stages
    if (ev)
      for (int i = 0; i < 4; ++i)
        if (hipEventRecord(ev[i], s) != hipSuccess) return hipErrorInvalidValue;
  }
  if (a.BH == 0) return hipSuccess;
  if (a.T == 0) {
    const int64_t nS = a.BH * a.dk * a.dv, nA = a.BH * a.dk;
    const int64_t n = nS > nA ? nS : nA;
    hipLaunchKernelGGL(k0_copy_states, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s,
                       a, nS, nA);
    return hipGetLastError();
  }
  if (io_bf16) {
    return a.dk == 64 ? launch_all<bf16, 64>(a, s, ev) : launch_all<bf16, 128>(a, s, ev);
  }
  return a.dk == 64 ? launch_all<float, 64>(a, s, ev) : launch_all<float, 128>(a, s, ev);
}

}  // namespace pdn
