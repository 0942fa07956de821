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
#include <mutex>

#include "pdn_device.hpp"
#include "pdn_internal.hpp"

namespace pdn {


// ---------------------------------------------------------------- K1
// The chunk's affine summary: A_end = exp(sum gP) A_start + L with
// L = sum_r betaP_r exp(GP_end - GP_r) k_r^2, GP the in-chunk prefix of gP.
// Rows are weighted in parallel, then reduced per channel.
template <typename T, int DK, int C>
__global__ __launch_bounds__(256) void k1_precond_summary(FwdArgs a) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int VPR = DK / VEC;       // 16-byte vectors per row
  constexpr int RPP = 256 / VPR;      // rows per pass
  __shared__ float sW[C];
  __shared__ __attribute__((aligned(16))) float sRed[RPP * DK];
  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  // this thread's key vectors, issued first (rows past the sequence end
  // read the last valid row; their weight below is zero)
  const T* k = static_cast<const T*>(a.k);
  const int cg = tid % VPR, r0 = tid / VPR;
  static_assert(C % RPP == 0, "whole passes of rows");
  float4 raw[C / RPP];
#pragma unroll
  for (int j = 0; j < C / RPP; ++j) {
    const int r = min(r0 + j * RPP, n - 1);
    raw[j] = *reinterpret_cast<const float4*>(k + ((b * a.T + t0 + r) * a.H + h) * DK + cg * VEC);
  }
  if (tid < 64) {
    const int r = tid;
    const int64_t sidx = (b * a.T + t0 + min(r, n - 1)) * a.H + h;
    const float bp = a.beta_p[sidx];
    float gp = a.g_p ? a.g_p[sidx] : 0.f;
    if (r >= n) gp = 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(gp, off, 64);
      if (r >= off) gp += y;
    }
    const float gend = __shfl(gp, 63, 64);
    if (r < C) sW[r] = r < n ? bp * fast_exp(gend - gp) : 0.f;
    if (r == 0) a.sumD[bh * a.NT + i] = gend;
  }
  __syncthreads();
  float acc[VEC];
#pragma unroll
  for (int s = 0; s < VEC; ++s) acc[s] = 0.f;
#pragma unroll
  for (int j = 0; j < C / RPP; ++j) {
    const T* e = reinterpret_cast<const T*>(&raw[j]);
    const float wr = sW[r0 + j * RPP];
#pragma unroll
    for (int s = 0; s < VEC; ++s) {
      const float kv = to_f(e[s]);
      acc[s] += wr * kv * kv;
    }
  }
#pragma unroll
  for (int s = 0; s < VEC; ++s) sRed[r0 * DK + cg * VEC + s] = acc[s];
  __syncthreads();
  if (tid < DK) {
    float L = 0.f;
#pragma unroll
    for (int r = 0; r < RPP; ++r) L += sRed[r * DK + tid];
    a.sumL[(bh * a.NT + i) * DK + tid] = L;
  }
}

// The chunk summaries chained into the state before every chunk, A_{i+1} =
// exp(D_i) A_i + L_i per channel: 16 channels x 16 chunk segments a
// workgroup.  Each segment reduces to its affine map (prod exp D, partial
// sum from zero), a segment's start state chains the maps before it from
// A0, and each segment re-walks its chunks writing the states.
constexpr int kCarryCh = 16, kCarrySeg = 16;
template <int DK>
__global__ __launch_bounds__(256) void k1_precond_carry(FwdArgs a) {
  __shared__ float sE[kCarrySeg][kCarryCh], sP[kCarrySeg][kCarryCh];
  const int64_t bh = blockIdx.x / (DK / kCarryCh);
  const int ch = threadIdx.x % kCarryCh, sg = threadIdx.x / kCarryCh;
  const int c = static_cast<int>(blockIdx.x % (DK / kCarryCh)) * kCarryCh + ch;
  const int NT = a.NT, Ls = (NT + kCarrySeg - 1) / kCarrySeg;
  const int i0 = min(NT, sg * Ls), i1 = min(NT, i0 + Ls);
  float* out = a.Abound + bh * (NT + 1) * DK + c;
  const float* L = a.sumL + bh * NT * DK + c;
  const float* D = a.sumD + bh * NT;
  float E = 1.f, P = 0.f;
#pragma unroll 8
  for (int i = i0; i < i1; ++i) {
    const float e = fast_exp(D[i]);
    E *= e;
    P = e * P + L[(int64_t)i * DK];
  }
  sE[sg][ch] = E;
  sP[sg][ch] = P;
  __syncthreads();
  float A = a.A0 ? a.A0[bh * DK + c] : 0.f;
  if (sg == 0) out[0] = A;
  for (int q = 0; q < sg; ++q) A = sE[q][ch] * A + sP[q][ch];
#pragma unroll 8
  for (int i = i0; i < i1; ++i) {
    A = fast_exp(D[i]) * A + L[(int64_t)i * DK];
    out[(int64_t)(i + 1) * DK] = A;
  }
  if (a.A_T && i0 < i1 && i1 == NT) a.A_T[bh * DK + c] = A;
}

// ---------------------------------------------------------------- K2
// k2's tiles are read along rows (MFMA fragments, row staging) and down
// columns (the transposed outputs, the column-wise scans), with unpadded
// rows.  The column index is XOR-permuted in aligned groups (8 elements for
// the key / query tiles, 4 for the fp32 C x C tiles) by
// v(row) = (row mod G) ^ ((row / 8) mod 8), G the groups per row: the 16
// consecutive rows of an MFMA fragment read and the 8 rows 8 apart of a
// column read each land on distinct groups, while a group stays contiguous.
template <typename T>
__device__ __forceinline__ T* k2sw(T* base, int ld, int row, int col) {
  const int g = ld >> 3;
  return base + row * ld + (col ^ ((((row & (g - 1)) ^ ((row >> 3) & 7)) & (g - 1)) << 3));
}
__device__ __forceinline__ float* k2swc(float* base, int ld, int row, int col) {
  const int g = ld >> 2;
  return base + row * ld + (col ^ ((((row & (g - 1)) ^ ((row >> 3) & 7)) & (g - 1)) << 2));
}
// the per-channel gate tile (padded rows of d_k + 4 floats)
__device__ __forceinline__ float* k2swf(float* base, int ld, int row, int col) {
  return base + row * ld + (col ^ (((row >> 3) & 7) << 2));
}
// NOQ (per-channel gate, query not rewritten): the query tile is not staged
// (its rows are read from HBM where needed), and the solve's X uses the
// write-key tile's memory, which is dead once the write-key outputs are out.
// That keeps the block under 80 KB, two per CU.  (For the other gates the
// HBM reads of the transposed query cost more than a third block per CU
// gains.)
template <typename T, int DK, int GATE, int PREC, int C>
struct K2Smem {
  static constexpr int LDK = DK;              // row (elements; swizzled, unpadded)
  static constexpr int LDA = C;               // fp32 C x C rows (swizzled, unpadded)
  static constexpr size_t kRow = sizeof(T) * C * LDK;
  static constexpr size_t kFloatCC = sizeof(float) * C * LDA;
  static constexpr size_t kR1 = kRow > kFloatCC ? kRow : kFloatCC;  // sK, later sA
  static constexpr size_t kY = sizeof(float) * 4 * 16 * 17;
  static constexpr size_t kGc = GATE == kGateChannel ? sizeof(float) * C * (DK + 4) : 0;
  // (at d_k = 64 in bf16 the write-key tile is too small for X; that block is
  // small anyway)
  static constexpr bool NOQ = GATE == kGateChannel && PREC != kATQ && kRow >= kFloatCC;
  static constexpr size_t kR2 = NOQ ? 0 : kR1;                      // sQ, later sX
  static constexpr size_t kR3 = kRow;                               // sKt, later sX (NOQ)
  static constexpr size_t kScal = sizeof(float) * 8 * C;    // per-row scalars and the row norms
  static constexpr size_t kSeg = sizeof(float) * 2 * 256;   // preconditioner segment carries
  // the solve's partial products (sY) sit in the write-key tile, dead by the
  // solve, unless the per-channel gate needs them while that tile is live
  // (its gate prefix) or the tile is too small
  static constexpr bool YSEP = GATE == kGateChannel || kR3 < kY;
  static constexpr size_t kYs = YSEP ? kY : 0;
  static constexpr size_t kTotal = kR1 + kR2 + kR3 + kGc + kYs + kScal + kSeg;
};

// BWD: also write the operand layouts the backward kernels read (P^T, M^T,
// write-key rows, write-key rows decayed to the chunk end, (Lam o Q)^T and
// -(Lam o K)^T; Lam the scalar or per-channel in-chunk decay).
template <typename T, int DK, int GATE, int PREC, bool BWD, int C>
__global__ __launch_bounds__(256, 3) void k2_chunk_prep(FwdArgs a) {
  using SM = K2Smem<T, DK, GATE, PREC, C>;
  // row blocks of 16 tokens: wave w owns block w (C = 32: waves 2, 3 only
  // take part in the column-wise phases)
  constexpr int NB = C / 16;
  static_assert(NB == 2 || NB == 4, "chunk of 32 or 64 tokens");
  constexpr bool NOQ = SM::NOQ;
  constexpr int LDK = SM::LDK, LDA = SM::LDA;
  __shared__ __attribute__((aligned(16))) char smem[SM::kTotal];
  T* sK = reinterpret_cast<T*>(smem);
  float* sA = reinterpret_cast<float*>(smem);
  T* sQ = reinterpret_cast<T*>(smem + SM::kR1);   // (not used with NOQ)
  T* sKt = reinterpret_cast<T*>(smem + SM::kR1 + SM::kR2);
  float* sGc = reinterpret_cast<float*>(smem + SM::kR1 + SM::kR2 + SM::kR3);
  float* sX = reinterpret_cast<float*>(smem + SM::kR1);   // R2, or with NOQ the write-key tile
  float* sY = reinterpret_cast<float*>(smem + SM::kR1 + SM::kR2 + (SM::YSEP ? SM::kR3 + SM::kGc : 0));
  float* sBeta = reinterpret_cast<float*>(smem + SM::kR1 + SM::kR2 + SM::kR3 + SM::kGc + SM::kYs);
  float* sNrm = sBeta + 7 * C;   // row norms of the normalised write keys
  float* sBp = sBeta + C;
  float* sEgp = sBp + C;
  float* sG = sEgp + C;
  float* sGraw = sG + C;
  float* sLam = sGraw + C;   // scalar gate: exp(G_r)
  float* sWt = sLam + C;     // scalar gate: exp(G_{C-1} - G_r)
  float* sSegE = sNrm + C;
  float* sSegP = sSegE + 256;

  const int64_t blk = blockIdx.x;
  const int64_t bh = blk / a.NT;
  const int i = static_cast<int>(blk % a.NT);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int n = static_cast<int>(min<int64_t>(C, a.T - t0));
  constexpr int VEC = 16 / sizeof(T);
  constexpr int VPR = DK / VEC;  // vectors per row

  // ---- load key, query (and external write key) tiles, zero-padded.
  // Every global load of the phase is issued before the first is used (rows
  // past the sequence end read the last valid row and are zeroed after), so
  // the block waits for one memory round trip rather than one per vector.
  float Ab = 0.f;    // preconditioner state before this chunk, one channel per thread
  float lmu = 0.f;   // log of the squash scale
  {
    const T* kp = static_cast<const T*>(a.k);
    const T* qp = static_cast<const T*>(a.q);
    const T* xp = static_cast<const T*>(a.ktilde);
    static_assert((C * VPR) % 256 == 0, "whole rounds of 256 threads");
    constexpr int NJ = (C * VPR) / 256;
    constexpr int NG = GATE == kGateChannel ? (C * (DK / 4)) / 256 : 0;
    float4 kv[NJ], qv[NJ], xv[NJ], gv[NG > 0 ? NG : 1];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      const int idx = tid + 256 * jj;
      const int r = min(idx / VPR, n - 1), cv = idx % VPR;
      const int64_t off = ((b * a.T + t0 + r) * a.H + h) * DK + cv * VEC;
      kv[jj] = *reinterpret_cast<const float4*>(kp + off);
      if (!NOQ) qv[jj] = *reinterpret_cast<const float4*>(qp + off);
      if (PREC == kExternal) xv[jj] = *reinterpret_cast<const float4*>(xp + off);
    }
    if (GATE == kGateChannel) {
      static_assert((C * (DK / 4)) % 256 == 0, "whole rounds of 256 threads");
#pragma unroll
      for (int jj = 0; jj < NG; ++jj) {
        const int idx = tid + 256 * jj;
        const int r = min(idx / (DK / 4), n - 1), c4 = idx % (DK / 4);
        gv[jj] = *reinterpret_cast<const float4*>(a.g + ((b * a.T + t0 + r) * a.H + h) * DK + c4 * 4);
      }
    }
    // per-row scalars: every wave loads the chunk's rows (branch-free, so
    // the loads issue with the tiles'); the first C threads keep them
    const int64_t sidx = (b * a.T + t0 + min(tid % C, n - 1)) * a.H + h;
    const float vb = a.beta[sidx];
    float vbp = 0.f, vgp = 0.f, vg = 0.f;
    if (has_gram(PREC)) {
      vbp = a.beta_p[sidx];
      vgp = (a.g_p ? a.g_p : a.beta_p)[sidx];   // (unused without g_p)
      Ab = a.Abound[(bh * (a.NT + 1) + i) * DK + tid % DK];
      if (PREC == kSquash) lmu = a.log_a_scale[h];
    }
    if (GATE == kGateScalar) vg = a.g[sidx];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      const int idx = tid + 256 * jj;
      const int r = idx / VPR, cv = idx % VPR;
      const bool ok = r < n;
      *reinterpret_cast<float4*>(k2sw(sK, LDK, r, cv * VEC)) = keep_if(kv[jj], ok);
      if (!NOQ) *reinterpret_cast<float4*>(k2sw(sQ, LDK, r, cv * VEC)) = keep_if(qv[jj], ok);
      // identity write key: a copy of the key tile (the key tile's memory is
      // reused by the solve)
      if (PREC == kIdentity || PREC == kATQ) *reinterpret_cast<float4*>(k2sw(sKt, LDK, r, cv * VEC)) = keep_if(kv[jj], ok);
      if (PREC == kExternal) *reinterpret_cast<float4*>(k2sw(sKt, LDK, r, cv * VEC)) = keep_if(xv[jj], ok);
    }
    if (GATE == kGateChannel) {
#pragma unroll
      for (int jj = 0; jj < NG; ++jj) {
        const int idx = tid + 256 * jj;
        const int r = idx / (DK / 4), c4 = idx % (DK / 4);
        *reinterpret_cast<float4*>(k2swf(sGc, DK + 4, r, c4 * 4)) = keep_if(gv[jj], r < n);
      }
    }
    // every wave stores the same row scalars (identical values): no branch,
    // so the compiler keeps their loads with the tiles'
    {
      const int r = tid % C;
      const bool ok = r < n;
      sBeta[r] = ok ? vb : 0.f;
      if (has_gram(PREC)) {
        sBp[r] = ok ? vbp : 0.f;
        sEgp[r] = (ok && a.g_p) ? fast_exp(vgp) : 1.f;
      }
      if (GATE == kGateScalar) sGraw[r] = ok ? vg : 0.f;
    }
  }
  __syncthreads();

  // ---- gate prefix and preconditioner prefix
  if (GATE == kGateScalar && w == 0) {
    float x = l < C ? sGraw[l] : 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(x, off, 64);
      if (l >= off) x += y;
    }
    const float xC = __shfl(x, C - 1, 64);
    if (l < C) {
      sG[l] = x;
      a.G[bh * a.Tpad + t0 + l] = x;
      sLam[l] = fast_exp(x);
      sWt[l] = fast_exp(xC - x);
    }
  }
  if (GATE == kGateChannel) {
    // per-channel in-chunk prefix G of g (rows past the end hold g = 0) over
    // 8-row segments: each segment is summed, then re-walked from the total
    // of the segments before it (the backward rebuilds G from g with the
    // same sums in the same order).  Only the chunk-end row leaves the
    // kernel.
    constexpr int NS8 = C / 8, NSG = 256 / DK, SPT = NS8 / NSG;
    static_assert(NS8 % NSG == 0, "whole segments per thread");
    const int c = tid % DK, sg = tid / DK;
    float* sTot = sY;   // [NS8][DK] segment totals (sY is idle until the solve)
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      const int sgm = sg * SPT + u;
      float x = 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q) x += *k2swf(sGc, DK + 4, 8 * sgm + q, c);
      sTot[sgm * DK + c] = x;
    }
    __syncthreads();
    float x = 0.f;
#pragma unroll
    for (int u = 0; u < SPT; ++u) {
      const int sgm = sg * SPT + u;
      x = 0.f;
      for (int q = 0; q < sgm; ++q) x += sTot[q * DK + c];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        float* gp = k2swf(sGc, DK + 4, 8 * sgm + q, c);
        x += *gp;
        *gp = x;
      }
    }
    if (sg == NSG - 1) a.G[(bh * a.NT + i) * DK + c] = x;   // row C - 1
  }
  if (has_gram(PREC)) {
    // the in-chunk prefix A_r = a_r A_{r-1} + bP_r k_r^2 in NSEG row segments:
    // pass 1 reduces each segment to (prod a, partial sum), the segments are
    // chained from the chunk-start state, pass 2 re-walks its rows
    constexpr int NSEG = 256 / DK, SEG = C / NSEG;
    const int c = tid % DK, sg = tid / DK, r0 = sg * SEG;
    // this thread's key column over its segment and the rows' decay and
    // betaP: held in registers for every walk below, or (backward mode,
    // whose peak is elsewhere and tighter) read from LDS at each walk
    constexpr bool SEGREG = !BWD;
    static_assert(SEG % 4 == 0, "segment rows come in float4 groups");
    float kreg[SEGREG ? SEG : 1], egr[SEGREG ? SEG : 1], bpr[SEGREG ? SEG : 1];
    if constexpr (SEGREG) {
#pragma unroll
      for (int j = 0; j < SEG; ++j) kreg[j] = to_f(*k2sw(sK, LDK, r0 + j, c));
#pragma unroll
      for (int j = 0; j < SEG; j += 4) {
        const float4 e4 = *reinterpret_cast<const float4*>(sEgp + r0 + j);
        const float4 b4 = *reinterpret_cast<const float4*>(sBp + r0 + j);
        egr[j] = e4.x; egr[j + 1] = e4.y; egr[j + 2] = e4.z; egr[j + 3] = e4.w;
        bpr[j] = b4.x; bpr[j + 1] = b4.y; bpr[j + 2] = b4.z; bpr[j + 3] = b4.w;
      }
    }
    auto kv_at = [&](int j) { return SEGREG ? kreg[SEGREG ? j : 0] : to_f(*k2sw(sK, LDK, r0 + j, c)); };
    auto eg_at = [&](int j) { return SEGREG ? egr[SEGREG ? j : 0] : sEgp[r0 + j]; };
    auto bp_at = [&](int j) { return SEGREG ? bpr[SEGREG ? j : 0] : sBp[r0 + j]; };
    float E = 1.f, Pp = 0.f;
#pragma unroll
    for (int j = 0; j < SEG; ++j) {
      E *= eg_at(j);
      Pp = eg_at(j) * Pp + bp_at(j) * kv_at(j) * kv_at(j);
    }
    sSegE[sg * DK + c] = E;
    sSegP[sg * DK + c] = Pp;
    __syncthreads();
    float A = Ab;
    for (int q = 0; q < sg; ++q) A = sSegE[q * DK + c] * A + sSegP[q * DK + c];
    if (PREC == kSquash) {
      const float mu = fast_exp(lmu);
      const float A_seg = A;
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        const float kv = kv_at(j);
        A = eg_at(j) * A + bp_at(j) * kv * kv;
        *k2sw(sKt, LDK, r0 + j, c) = from_f<T>(squash_gain(A, mu, a.lnx) * kv);
      }
      if (a.knorm != kKnormNone) {
        // normalisation ablation: kt = B k * f(m), m = k . (B k) per row;
        // the rows' m from the stored keys, then the keys recomputed exactly
        // and scaled once
        __syncthreads();
        if ((tid >> 2) < C) {
          constexpr int PART = DK / 4;
          const int r = tid >> 2, part = tid & 3;
          float m = 0.f;
          for (int cc = part * PART; cc < (part + 1) * PART; ++cc)
            m += to_f(*k2sw(sK, LDK, r, cc)) * to_f(*k2sw(sKt, LDK, r, cc));
          m += __shfl_xor(m, 1, 64);
          m += __shfl_xor(m, 2, 64);
          if (part == 0) {
            float f = 0.f;   // rows past the sequence end: zero keys
            if (r < n) {
              if (a.knorm == kKnormM) f = 1.f / m;
              else if (a.knorm == kKnorm1pm) f = 1.f / (1.f + m);
              else {
                const float al = GATE == kGateScalar ? fast_exp(sGraw[r]) : 1.f;
                f = sBeta[r] / (al + sBeta[r] * m);
              }
            }
            sNrm[r] = f;
          }
        }
        __syncthreads();
        A = A_seg;
#pragma unroll
        for (int j = 0; j < SEG; ++j) {
          const float kv = kv_at(j);
          A = eg_at(j) * A + bp_at(j) * kv * kv;
          *k2sw(sKt, LDK, r0 + j, c) = from_f<T>(squash_gain(A, mu, a.lnx) * kv * sNrm[r0 + j]);
        }
      }
    }
    if (PREC == kATQ) {
      // preconditioned query q / (A_r + ridge), A_r including token r
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        const float kv = kv_at(j);
        A = eg_at(j) * A + bp_at(j) * kv * kv;
        *k2sw(sQ, LDK, r0 + j, c) = from_f<T>(to_f(*k2sw(sQ, LDK, r0 + j, c)) / (A + a.ridge));
      }
    }
    if (PREC == kDiagSM) {
      // Sherman-Morrison write key from the state before token r:
      //   p = k / (A_{r-1} + ridge),  kt = p / (1 + k . p)
      // the row sums k . p need every channel: the segment is walked once
      // for them and again for the exactly recomputed, normalised key
      const float A_seg = A;
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        const float kv = kv_at(j);
        *k2sw(sKt, LDK, r0 + j, c) = from_f<T>(kv / (A + a.ridge));
        A = eg_at(j) * A + bp_at(j) * kv * kv;
      }
      __syncthreads();
      if ((tid >> 2) < C) {
        constexpr int PART = DK / 4;
        const int r = tid >> 2, part = tid & 3;
        float sum = 0.f;
        for (int cc = part * PART; cc < (part + 1) * PART; ++cc)
          sum += to_f(*k2sw(sK, LDK, r, cc)) * to_f(*k2sw(sKt, LDK, r, cc));
        sum += __shfl_xor(sum, 1, 64);
        sum += __shfl_xor(sum, 2, 64);
        if (part == 0) sNrm[r] = 1.f + sum;
      }
      __syncthreads();
      A = A_seg;
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        const float kv = kv_at(j);
        *k2sw(sKt, LDK, r0 + j, c) = from_f<T>(kv / ((A + a.ridge) * sNrm[r0 + j]));
        A = eg_at(j) * A + bp_at(j) * kv * kv;
      }
    }
  }
  __syncthreads();
  if (PREC == kATQ) {
    // the preconditioned query rows for the scan's inter-chunk output
    T* qt = static_cast<T*>(a.Qt) + (bh * a.Tpad + t0) * DK;
    static_assert((C * VPR) % 256 == 0, "whole rounds of 256 threads");
#pragma unroll
    for (int jj = 0; jj < (C * VPR) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      const int r = idx / VPR, cv = idx % VPR;
      *reinterpret_cast<float4*>(qt + r * DK + cv * VEC) = *reinterpret_cast<const float4*>(k2sw(sQ, LDK, r, cv * VEC));
    }
  }
  // NOQ: the query fragments of this lane's A-operand row, straight from
  // HBM, issued here so they arrive during the decayed-row outputs
  Frag8<T> fqr[DK / 32];
  if (NOQ && (NB == 4 || w < NB)) {
    const int r = 16 * w + lr;
    const T* qrow = static_cast<const T*>(a.q) + ((b * a.T + t0 + min(r, n - 1)) * a.H + h) * DK;
#pragma unroll
    for (int kk = 0; kk < DK / 32; ++kk) fqr[kk] = ld8(qrow + kk * 32 + 8 * lg);
  }
  if (GATE == kGateChannel) {
    // Lam o Q and Lam o K (Lam_r = exp(G_r) per channel; Q the query the
    // scan reads: q, or for ATQ the preconditioned query): the rows the
    // scan reads, rounded to io as the scan would round them, and for the
    // backward their transposes (Lam o Q)^T and -(Lam o K)^T, [dk][C].  A
    // thread takes 8 rows x 4 channels, so each exponential serves all four
    // outputs.
    T* ql = static_cast<T*>(a.QL) + (bh * a.Tpad + t0) * DK;
    T* kl = static_cast<T*>(a.KL) + (bh * a.Tpad + t0) * DK;
    const T* qg = static_cast<const T*>(a.q) + ((b * a.T + t0) * a.H + h) * DK;
    using V4 = typename Vec4<T>::type;
    constexpr int RB = C / 8, NTILE = RB * (DK / 4);
#pragma unroll
    for (int jj = 0; jj < (NTILE + 255) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      if (NTILE % 256 != 0 && idx >= NTILE) break;
      const int r0 = (idx % RB) * 8, c0 = (idx / RB) * 4;
      V4 q4[8], k4[8];
      float4 g4[8];
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        const int r = r0 + s2;
        if (NOQ) q4[s2] = *reinterpret_cast<const V4*>(qg + static_cast<int64_t>(min(r, n - 1)) * a.H * DK + c0);
        else q4[s2] = *reinterpret_cast<const V4*>(k2sw(sQ, LDK, r, c0));
        k4[s2] = *reinterpret_cast<const V4*>(k2sw(sK, LDK, r, c0));
        g4[s2] = *reinterpret_cast<const float4*>(k2swf(sGc, DK + 4, r, c0));
      }
      Frag8<T> fq[4], fk[4];
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        const int r = r0 + s2;
        const float gv[4] = {g4[s2].x, g4[s2].y, g4[s2].z, g4[s2].w};
        float qo[4], ko[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lam = fast_exp(gv[e]);
          qo[e] = lam * ((NOQ && r >= n) ? 0.f : to_f(q4[s2][e]));
          ko[e] = lam * to_f(k4[s2][e]);
          fq[e].set(s2, qo[e]);
          fk[e].set(s2, -ko[e]);
        }
        st4<T>(ql + r * DK + c0, qo[0], qo[1], qo[2], qo[3]);
        st4<T>(kl + r * DK + c0, ko[0], ko[1], ko[2], ko[3]);
      }
      if (BWD) {
        T* QlT = static_cast<T*>(a.QlT) + (bh * a.NT + i) * (int64_t)(DK * C);
        T* KnT = static_cast<T*>(a.KnT) + (bh * a.NT + i) * (int64_t)(DK * C);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          st8(QlT + (c0 + e) * C + r0, fq[e]);
          st8(KnT + (c0 + e) * C + r0, fk[e]);
        }
      }
    }
  }

  // ---- interaction matrices on MFMA: wave w owns row block w
  floatx4 accA[NB], accP[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) { accA[j] = floatx4{0.f, 0.f, 0.f, 0.f}; accP[j] = accA[j]; }
  if (NB == 4 || w < NB) {
    const int r = 16 * w + lr;  // A-operand row of this lane
    if (NOQ && r >= n) {   // rows past the sequence end: zero queries
#pragma unroll
      for (int kk = 0; kk < DK / 32; ++kk) fqr[kk] = frag_zero<T>();
    }
    if (GATE == kGateChannel) {
      // the decay ratio e^{G_r - G_t} inside the contraction, split at a
      // reference row (the row block's first): the A operands take
      // e^{G_r - G_ref} (once per 32 channels, shared by every column
      // block), the B operands e^{G_ref - G_t}
      const int rref = 16 * w;
#pragma unroll
      for (int kk = 0; kk < DK / 32; ++kk) {
        const int c0 = kk * 32 + 8 * lg;
        Frag8<T> fk = ld8(k2sw(sK, LDK, r, c0));
        Frag8<T> fq = NOQ ? fqr[kk] : ld8(k2sw(sQ, LDK, r, c0));
        float gref[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          gref[s] = *k2swf(sGc, DK + 4, rref, c0 + s);
          const float fa = fast_exp(*k2swf(sGc, DK + 4, r, c0 + s) - gref[s]);
          fk.set(s, fk.get(s) * fa);
          fq.set(s, fq.get(s) * fa);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          if (j > w) break;
          const int t = 16 * j + lr;  // B-operand column of this lane
          Frag8<T> fb = ld8(k2sw(sKt, LDK, t, c0));
#pragma unroll
          for (int s = 0; s < 8; ++s)
            fb.set(s, fb.get(s) * fast_exp(gref[s] - *k2swf(sGc, DK + 4, t, c0 + s)));
          if (PREC != kATQ) mma(accA[j], fk, fb);
          mma(accP[j], fq, fb);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        if (j > w) break;
        const int t = 16 * j + lr;  // B-operand column of this lane
#pragma unroll
        for (int kk = 0; kk < DK / 32; ++kk) {
          const int c0 = kk * 32 + 8 * lg;
          const Frag8<T> fk = ld8(k2sw(sK, LDK, r, c0));
          const Frag8<T> fq = NOQ ? fqr[kk] : ld8(k2sw(sQ, LDK, r, c0));
          const Frag8<T> fb = ld8(k2sw(sKt, LDK, t, c0));
          // linear attention (ATQ): no delta-rule interaction, At = 0, T = Diag(beta)
          if (PREC != kATQ) mma(accA[j], fk, fb);
          mma(accP[j], fq, fb);
        }
      }
    }
  }
  // masks, beta and scalar decay; P goes straight to the workspace
  if (NB == 4 || w < NB) {
    T* P = static_cast<T*>(a.Pm) + (bh * a.NT + i) * (int64_t)(C * C);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int t = 16 * j + lr;
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int r = 16 * w + 4 * lg + ii;
        float fac = 1.f;
        if (GATE == kGateScalar) fac = fast_exp(sG[r] - sG[t]);
        accP[j][ii] = (j <= w && r >= t) ? accP[j][ii] * fac : 0.f;
        accA[j][ii] = (j <= w && r > t) ? sBeta[r] * accA[j][ii] * fac : 0.f;
        P[r * C + t] = from_f<T>(accP[j][ii]);
      }
      if (BWD) {
        T* PtT = static_cast<T*>(a.PtT) + (bh * a.NT + i) * (int64_t)(C * C);
        st_tile_t<T>(PtT + (16 * j) * C + 16 * w, C, accP[j], lr, lg);
      }
    }
  }
  if (BWD && GATE != kGateChannel) {
    // (Lam o Q)^T and -(Lam o K)^T per chunk, [dk][C] (per-channel gate:
    // written with the Lam o Q / Lam o K rows above)
    T* QlT = static_cast<T*>(a.QlT) + (bh * a.NT + i) * (int64_t)(DK * C);
    T* KnT = static_cast<T*>(a.KnT) + (bh * a.NT + i) * (int64_t)(DK * C);
    static_assert((DK * (C / 8)) % 256 == 0, "whole rounds of 256 threads");
#pragma unroll
    for (int jj = 0; jj < (DK * (C / 8)) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      const int c = idx / (C / 8), r0 = (idx % (C / 8)) * 8;
      Frag8<T> fq, fk;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        const int r = r0 + s2;
        const float lam = GATE == kGateScalar ? sLam[r] : 1.f;
        fq.set(s2, lam * to_f(*k2sw(sQ, LDK, r, c)));
        fk.set(s2, -lam * to_f(*k2sw(sK, LDK, r, c)));
      }
      st8(QlT + c * C + r0, fq);
      st8(KnT + c * C + r0, fk);
    }
  }
  // the write-key outputs (they need only sKt and the gate prefix), before
  // the solve
  if (BWD) {
    // write-key rows (the per-channel gate's decayed rows w_r o Kt go out
    // with the transposed decayed write keys below; with a scalar gate the
    // reverse scan applies w_r itself)
    T* Kr = static_cast<T*>(a.Ktr) + (bh * a.Tpad + t0) * DK;
    static_assert((C * (DK / 8)) % 256 == 0, "whole rounds of 256 threads");
#pragma unroll
    for (int jj = 0; jj < (C * (DK / 8)) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      const int r = idx / (DK / 8), c0 = (idx % (DK / 8)) * 8;
      st8(Kr + r * DK + c0, ld8(k2sw(sKt, LDK, r, c0)));
    }
  }
  // ---- decayed write keys, transposed per chunk: (Kt * Lam_C / Lam_t)^T
  if (GATE == kGateChannel) {
    // w_t = exp(G_{C-1} - G_t) per channel, 8 rows x 4 channels a thread:
    // each factor serves the transposed tile for the scan and, for the
    // backward, the row-major w o Kt
    T* Kout = static_cast<T*>(a.KtG) + (bh * a.NT + i) * (int64_t)(DK * C);
    T* Kw = static_cast<T*>(a.Kw) + (bh * a.Tpad + t0) * DK;
    using V4 = typename Vec4<T>::type;
    constexpr int RB = C / 8, NTILE = RB * (DK / 4);
#pragma unroll
    for (int jj = 0; jj < (NTILE + 255) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      if (NTILE % 256 != 0 && idx >= NTILE) break;
      const int r0 = (idx % RB) * 8, c0 = (idx / RB) * 4;
      const float4 ge = *reinterpret_cast<const float4*>(k2swf(sGc, DK + 4, C - 1, c0));
      const float gend[4] = {ge.x, ge.y, ge.z, ge.w};
      Frag8<T> f[4];
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        const int t = r0 + s2;
        const V4 kt4 = *reinterpret_cast<const V4*>(k2sw(sKt, LDK, t, c0));
        const float4 g4 = *reinterpret_cast<const float4*>(k2swf(sGc, DK + 4, t, c0));
        const float gv[4] = {g4.x, g4.y, g4.z, g4.w};
        float wv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wv[e] = fast_exp(gend[e] - gv[e]) * to_f(kt4[e]);
          f[e].set(s2, wv[e]);
        }
        if (BWD) st4<T>(Kw + t * DK + c0, wv[0], wv[1], wv[2], wv[3]);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) st8(Kout + (c0 + e) * C + r0, f[e]);
    }
  } else {
    T* Kout = static_cast<T*>(a.KtG) + (bh * a.NT + i) * (int64_t)(DK * C);
    static_assert((DK * C / 8) % 256 == 0, "whole rounds of 256 threads");
#pragma unroll
    for (int jj = 0; jj < (DK * C / 8) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      const int c = idx / (C / 8), tv = (idx % (C / 8)) * 8;
      Frag8<T> f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = tv + s;
        float val = to_f(*k2sw(sKt, LDK, t, c));
        if (GATE == kGateScalar) val *= sWt[t];
        f.set(s, val);
      }
      st8(Kout + c * C + tv, f);
    }
  }
  __syncthreads();  // sK / sQ are free from here on
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    if (j > w || !(NB == 4 || w < NB)) break;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) *k2swc(sA, LDA, 16 * w + 4 * lg + ii, 16 * j + lr) = accA[j][ii];
  }
  __syncthreads();

  // ---- X = (I + At)^{-1}: diagonal 16x16 blocks by forward substitution
  if ((NB == 4 || w < NB) && lg == 0) {
    const int col = lr;
    float x[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float s = (r == col) ? 1.f : 0.f;
#pragma unroll
      for (int t = 0; t < r; ++t) s -= *k2swc(sA, LDA, 16 * w + r, 16 * w + t) * x[t];
      x[r] = s;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) *k2swc(sX, LDA, 16 * w + r, 16 * w + col) = x[r];
  }
  __syncthreads();
  // off-diagonal blocks, by distance from the diagonal:
  //   X_ij = -X_ii * sum_{j <= m < i} At_im X_mj
  float* Yw = sY + w * 16 * 17;
  for (int d = 1; d < NB; ++d) {
    const int j = w, ib = w + d;
    const bool active = ib < NB;
    floatx4 y = {0.f, 0.f, 0.f, 0.f};
    if (active) {
      for (int kb = 0; kb < 4 * d; ++kb) {
        const float av = *k2swc(sA, LDA, 16 * ib + lr, 16 * j + 4 * kb + lg);
        const float bv = *k2swc(sX, LDA, 16 * j + 4 * kb + lg, 16 * j + lr);
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
        const float av = *k2swc(sX, LDA, 16 * ib + lr, 16 * ib + 4 * kb + lg);
        const float bv = Yw[(4 * kb + lg) * 17 + lr];
        mma4(z, av, bv);
      }
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) *k2swc(sX, LDA, 16 * ib + 4 * lg + ii, 16 * j + lr) = -z[ii];
    }
    __syncthreads();
  }

  // ---- T = X Diag(beta) (block-lower; upper blocks are zero)
  {
    T* Tout = static_cast<T*>(a.Tm) + (bh * a.NT + i) * (int64_t)(C * C);
    constexpr int NV = C * C / 8;
#pragma unroll
    for (int jj = 0; jj < (NV + 255) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      if (NV % 256 != 0 && idx >= NV) break;
      const int r = idx / (C / 8), t0v = (idx % (C / 8)) * 8;
      Frag8<T> f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int t = t0v + s;
        const bool lower = (t >> 4) < (r >> 4) || ((t >> 4) == (r >> 4) && t <= r);
        f.set(s, lower ? *k2swc(sX, LDA, r, t) * sBeta[t] : 0.f);
      }
      st8(Tout + r * C + t0v, f);
    }
  }
  if (BWD) {
    const int64_t cc = (bh * a.NT + i) * (int64_t)(C * C);
    T* MtT = static_cast<T*>(a.MtT) + cc;
    constexpr int NV = C * C / 8;
#pragma unroll
    for (int jj = 0; jj < (NV + 255) / 256; ++jj) {
      const int idx = tid + 256 * jj;
      if (NV % 256 != 0 && idx >= NV) break;
      const int r = idx / (C / 8), t0v = (idx % (C / 8)) * 8;
      Frag8<T> ft;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) {
        const int t = t0v + s2;
        // M^T[r][t] = M[t][r]; M is lower triangular (block-lower in sX)
        const bool upper = (r >> 4) < (t >> 4) || ((r >> 4) == (t >> 4) && r <= t);
        ft.set(s2, upper ? *k2swc(sX, LDA, t, r) : 0.f);
      }
      st8(MtT + r * C + t0v, ft);
    }
  }
}

// ---------------------------------------------------------------- K3
constexpr int BV = 32;  // value columns per workgroup

// One thread's share of a chunk's C x BV value (or output) slab, as 16-byte
// vectors: vector j of thread tid covers row idx / kSegs, elements
// [(idx % kSegs) * kVec, + kVec) with idx = tid + 256 j, for idx < kN (at
// C = 32 in bf16 only the first half of the threads have a vector).
template <typename T, int C>
struct SlabMap {
  static constexpr int kVec = 16 / static_cast<int>(sizeof(T));
  static constexpr int kSegs = BV / kVec;
  static constexpr int kN = C * kSegs;
  static constexpr int kPer = (kN + 255) / 256;
  static constexpr bool kWhole = kN % 256 == 0;
};

// sw() for the [v][t] slabs of C token columns: the XOR keeps the column
// inside the C columns of a row (C = 64: the same permutation as sw())
template <int COLS, typename T>
__device__ __forceinline__ T* swv(T* base, int ld, int row, int col) {
  return base + row * ld + (col ^ (((row >> 3) & (COLS / 16 - 1) & 3) << 4));
}

// Operands one wave needs for one chunk, loaded two chunks ahead of use.
// A-operand rows: token 16w + lr of the chunk; decayed write keys: rows
// c = 16*(w*CT + ct) + lr (per-channel gate: the read key and query rows
// arrive already decayed).  Gate values are kept raw (log-domain) and the
// value slab raw: nothing here is consumed at load time, so the loads stay
// in flight across the compute of the chunks before it.
//
// Rows past the end of the sequence (last chunk only) are loaded from the
// last valid row instead of being zeroed: their T columns and rows are zero
// (beta = 0 on padded rows), so they cannot reach any stored output.
template <typename T, int DK, int GATE, int C>
struct ScanFrags {
  static constexpr int KK = DK / 32, CT = DK / 64, KC = C / 32;
  Frag8<T> K[KK], Q[KK], Tm[KC], P[KC], G[CT][KC];
  float4 v[SlabMap<T, C>::kPer];                   // value slab share
  float g[GATE == kGateScalar ? 4 : 1];            // G of rows 16w + 4lg + ii
  float gC[GATE == kGateChannel ? CT : 1][GATE == kGateNone ? 1 : 4];  // G at the chunk end
};

struct ScanCtx {
  int64_t b, h, bh;
  int v0, w, lr, lg, tid;
  int c0;        // first chunk of this workgroup's run
  float vkeep;   // 1, or 0 for a transition workgroup (values zeroed)
};

// Each chunk's loads are a wave-uniform (scalar) base plus a 32-bit lane
// byte offset, so the loop does almost no per-lane address arithmetic.
// OUT = false (state-saving scan of the backward): the query and P tiles are
// not needed and not loaded.  LA (linear attention, ATQ): no read-key tile;
// the query tile is the preconditioned query the prep kernel left in the
// workspace.
//
// PARTS selects which loads to issue (bit mask, 7 = all): 1 the value slab and
// the read-key rows (for LA the query rows), 2 the query rows and T, 4 P, the
// decayed write keys and the gate values.  A step issues the loads of the
// chunk two ahead in these three parts, each right after one of its phases has
// issued its MFMAs: the per-CU vector memory path accepts one chunk's loads
// (about 90 KB per workgroup) only about as fast as the step's dependency
// chain runs, so loads issued as one block stall the wave in front of the
// chain instead of beside it.
template <int PARTS, bool OUT, bool LA, typename T, int DK, int GATE, int C>
__device__ __forceinline__ void scan_load(ScanFrags<T, DK, GATE, C>& f, const FwdArgs& a, int i,
                                          const ScanCtx& x) {
  constexpr int KK = DK / 32, CT = DK / 64, KC = C / 32, NB = C / 16;
  constexpr uint32_t E = sizeof(T);
  using SM = SlabMap<T, C>;
  // waves past the chunk's row blocks (C = 32: waves 2, 3) load no rows
  const bool rows = NB == 4 || x.w < NB;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int last = static_cast<int>(min<int64_t>(C, a.T - t0)) - 1;
  const int64_t HD = a.H * (int64_t)DK, HV = a.H * (int64_t)a.dv;
  // per-channel gate: the decayed rows Lam o K, Lam o Q the prep kernel left
  // in the workspace (row stride d_k)
  constexpr bool CH = GATE == kGateChannel;
  const int64_t ldk = CH ? DK : HD;
  const T* kb = CH ? static_cast<const T*>(a.KL) + (x.bh * a.Tpad + t0) * DK
                   : static_cast<const T*>(a.k) + (x.b * a.T + t0) * HD + x.h * DK;
  const T* qb = CH ? static_cast<const T*>(a.QL) + (x.bh * a.Tpad + t0) * DK
                   : static_cast<const T*>(a.q) + (x.b * a.T + t0) * HD + x.h * DK;
  const T* vb = static_cast<const T*>(a.v) + (x.b * a.T + t0) * HV + x.h * a.dv + x.v0;
  const T* tb = static_cast<const T*>(a.Tm) + (x.bh * a.NT + i) * (int64_t)(C * C);
  const T* pb = static_cast<const T*>(a.Pm) + (x.bh * a.NT + i) * (int64_t)(C * C);
  const T* gb = static_cast<const T*>(a.KtG) + (x.bh * a.NT + i) * (int64_t)(DK * C);
  // the value slab first: the step before this chunk's stages it into LDS
  // and so waits for it a step earlier than for the other operands; the
  // memory counter completes in issue order, so any load issued before it
  // would be waited for there too
  if (PARTS & 1) {
#pragma unroll
    for (int j = 0; j < SM::kPer; ++j) {
      const int idx = x.tid + 256 * j;
      if (!SM::kWhole && idx >= SM::kN) break;
      const uint32_t row = static_cast<uint32_t>(min(idx / SM::kSegs, last));
      const uint32_t off = (row * static_cast<uint32_t>(HV) + (idx % SM::kSegs) * SM::kVec) * E;
      f.v[j] = *reinterpret_cast<const float4*>(at_bytes(vb, off));
    }
  }
  const uint32_t rr = static_cast<uint32_t>(min(16 * x.w + x.lr, last));
  const uint32_t okq = (rr * static_cast<uint32_t>(ldk) + 8 * x.lg) * E;
  if (!rows) {
    // no rows of this chunk: only the decayed write keys and the chunk-end
    // gate values below
  } else if (LA) {
    if (PARTS & 1) {
      const T* qtb = CH ? qb : static_cast<const T*>(a.Qt) + (x.bh * a.Tpad + t0) * DK;
      const uint32_t oqt = (rr * static_cast<uint32_t>(DK) + 8 * x.lg) * E;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) f.Q[kk] = ld8(at_bytes(qtb, oqt + kk * 32 * E));
    }
  } else {
    if (PARTS & 1) {
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) f.K[kk] = ld8(at_bytes(kb, okq + kk * 32 * E));
    }
    if (OUT && (PARTS & 2)) {
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) f.Q[kk] = ld8(at_bytes(qb, okq + kk * 32 * E));
    }
  }
  const int ra = 16 * x.w + x.lr;
  const uint32_t otp = static_cast<uint32_t>(ra * C + 8 * x.lg) * E;
  if ((PARTS & 2) && rows) {
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) f.Tm[k2] = ld8(at_bytes(tb, otp + k2 * 32 * E));
  }
  if (!(PARTS & 4)) return;
  if (OUT && rows) {
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) f.P[k2] = ld8(at_bytes(pb, otp + k2 * 32 * E));
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2)
      f.G[ct][k2] = ld8(at_bytes(gb, static_cast<uint32_t>((16 * (x.w * CT + ct) + x.lr) * C + 8 * x.lg + k2 * 32) * E));
  if (GATE == kGateScalar) {
    const float* gs = a.G + x.bh * a.Tpad + t0;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii)
      f.g[ii] = rows ? *at_bytes(gs, static_cast<uint32_t>(16 * x.w + 4 * x.lg + ii) * 4u) : 0.f;
    f.gC[0][0] = gs[C - 1];
  }
  if (GATE == kGateChannel) {
    const float* ge = a.G + (x.bh * a.NT + i) * DK;   // G at the chunk end
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) f.gC[ct][ii] = ge[16 * (x.w * CT + ct) + 4 * x.lg + ii];
  }
}

// Workgroup barrier that only orders LDS: outstanding global loads (the
// next chunks' prefetch) stay in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// value slab share -> sVt[v][t] (transposed)
template <typename T, int C>
__device__ __forceinline__ void stage_values(const float4 (&v)[SlabMap<T, C>::kPer], T* sVt,
                                             int tid) {
  using SM = SlabMap<T, C>;
  constexpr int LDE = C + 8;
#pragma unroll
  for (int j = 0; j < SM::kPer; ++j) {
    const int idx = tid + 256 * j;
    if (!SM::kWhole && idx >= SM::kN) break;
    const int row = idx / SM::kSegs, c0 = (idx % SM::kSegs) * SM::kVec;
    const float4 raw = pin_here(v[j]);
    const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int s = 0; s < SM::kVec; ++s) *swv<C>(sVt, LDE, c0 + s, row) = e[s];
  }
}

// sO[v][t] -> o rows of chunk i (coalesced 16-byte stores); n valid rows
// (ALL: the whole chunk, no row check around the stores)
template <bool ALL, typename T, int C>
__device__ __forceinline__ void flush_output(const FwdArgs& a, int i, int n, const T* sO,
                                             const ScanCtx& x) {
  using SM = SlabMap<T, C>;
  constexpr int LDE = C + 8;
  if (!a.o) return;
  const int64_t t0 = static_cast<int64_t>(i) * C;
  const int64_t HV = a.H * (int64_t)a.dv;
  T* ob = static_cast<T*>(a.o) + (x.b * a.T + t0) * HV + x.h * a.dv + x.v0;
#pragma unroll
  for (int j = 0; j < SM::kPer; ++j) {
    const int idx = x.tid + 256 * j;
    if (!SM::kWhole && idx >= SM::kN) break;
    const int row = idx / SM::kSegs, c0 = (idx % SM::kSegs) * SM::kVec;
    float4 pk;
    T* e = reinterpret_cast<T*>(&pk);
#pragma unroll
    for (int s = 0; s < SM::kVec; ++s) e[s] = *swv<C>(sO, LDE, c0 + s, row);
    if (ALL || row < n)
      *reinterpret_cast<float4*>(at_bytes(ob, (static_cast<uint32_t>(row) * static_cast<uint32_t>(HV) + c0) *
                                                  static_cast<uint32_t>(sizeof(T)))) = pk;
  }
}

// One chunk step.  On entry sVt holds this chunk's values and sO the previous
// chunk's output (flushed first).  FULL: C valid tokens, so the step has no
// per-row branches (a conditional store would make the compiler wait for the
// prefetched loads); the ragged last chunk takes FULL = false.
// [v][t] (or [v][c]) LDS slab -> rows of a [rows][ld] global tensor: columns
// x.v0 .. x.v0 + BV of rows 0 .. NROWS-1, 16-byte stores (a fixed count per
// thread: no loop or branch around the stores inside the scan step)
template <int NROWS, typename T>
__device__ __forceinline__ void flush_slab_t(T* dst, int64_t ld, const T* src, int lds, int tid) {
  using SM = SlabMap<T, NROWS>;
#pragma unroll
  for (int j = 0; j < SM::kPer; ++j) {
    const int idx = tid + 256 * j;
    if (!SM::kWhole && idx >= SM::kN) break;
    const int row = idx / SM::kSegs, c0 = (idx % SM::kSegs) * SM::kVec;
    float4 pk;
    T* e = reinterpret_cast<T*>(&pk);
#pragma unroll
    for (int s2 = 0; s2 < SM::kVec; ++s2) e[s2] = *swv<NROWS>(src, lds, c0 + s2, row);
    *reinterpret_cast<float4*>(dst + row * ld + c0) = pk;
  }
}

// NEXT: also issue the loads of chunk `in` into `fn`, in three parts placed
// after the MFMAs of each phase (see scan_load).  Waves past the chunk's row
// blocks (C = 32: waves 2, 3) skip the row phases and take part in the state
// update only.
template <bool FULL, bool SAVE, bool OUT, bool LA, bool NEXT, typename T, int DK, int GATE, int C>
__device__ __forceinline__ void scan_step(ScanFrags<T, DK, GATE, C>& f, const float4* vnext,
                                          ScanFrags<T, DK, GATE, C>& fn, int in,
                                          floatx4 (&st)[DK / 64][2], const FwdArgs& a, int i,
                                          const ScanCtx& x, T* sH, T* sX, T* sE, T* sVt, T* sO) {
  constexpr int KK = DK / 32, CT = DK / 64, KC = C / 32, NB = C / 16;
  constexpr int LDH = DK + 8, LDE = C + 8;
  const int w = x.w, lr = x.lr, lg = x.lg;
  const bool rows = NB == 4 || w < NB;
  float lam[4];
#pragma unroll
  for (int ii = 0; ii < 4; ++ii) lam[ii] = GATE == kGateScalar ? fast_exp(f.g[ii]) : 1.f;
  // ---- (Lam K) S^T and (Lam Q) S^T;  X = V - (Lam K) S^T
  Frag8<T> bH[2][KK];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) bH[vt][kk] = ld8(sw(sH, LDH, 16 * vt + lr, kk * 32 + 8 * lg));
  typename Vec4<T>::type vv[2];
  if (rows) {
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      vv[vt] = *reinterpret_cast<const typename Vec4<T>::type*>(swv<C>(sVt, LDE, 16 * vt + lr, 16 * w + 4 * lg));
  }
  // the flushes' LDS reads go after this phase's operand reads (LDS reads
  // complete in issue order)
  if (OUT && i > x.c0) flush_output<true, T, C>(a, i - 1, C, sO, x);   // only full chunks precede this one
  if (SAVE)  // chunk-start state S^T of this chunk, rows c, columns of the slab
    flush_slab_t<DK>(static_cast<T*>(a.Hs) + (x.bh * a.NT + i) * (int64_t)DK * a.dv + x.v0, a.dv, sH,
                     LDH, x.tid);
  floatx4 accX[2], accO[2];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt) {
    accX[vt] = floatx4{0.f, 0.f, 0.f, 0.f};
    accO[vt] = accX[vt];
    if (!rows) continue;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (!LA) mma(accX[vt], f.K[kk], bH[vt][kk]);   // linear attention: X = V
      if (OUT) mma(accO[vt], f.Q[kk], bH[vt][kk]);
    }
  }
  if (NEXT) scan_load<1, OUT, LA>(fn, a, in, x);
  if (rows) {
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        accX[vt][ii] = x.vkeep * to_f(vv[vt][ii]) - lam[ii] * accX[vt][ii];
        if (OUT) accO[vt][ii] *= lam[ii];
      }
      st4<T>(swv<C>(sX, LDE, 16 * vt + lr, 16 * w + 4 * lg), accX[vt][0], accX[vt][1], accX[vt][2],
             accX[vt][3]);
    }
  }
  lds_barrier();
  // ---- E = T X
  floatx4 accE[2];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt) accE[vt] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (rows) {
    Frag8<T> bX[2][KC];
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) bX[vt][k2] = ld8(swv<C>(sX, LDE, 16 * vt + lr, k2 * 32 + 8 * lg));
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) mma(accE[vt], f.Tm[k2], bX[vt][k2]);
  }
  if (NEXT) scan_load<2, OUT, LA>(fn, a, in, x);
  if (rows) {
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      st4<T>(swv<C>(sE, LDE, 16 * vt + lr, 16 * w + 4 * lg), accE[vt][0], accE[vt][1], accE[vt][2],
             accE[vt][3]);
  }
  lds_barrier();
  // ---- O = scale [ (Lam Q) S^T + P E ];  S^T <- Diag(gamma_C) S^T + (Kt Gamma)^T E
  Frag8<T> fE[2][KC];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt)
#pragma unroll
    for (int k2 = 0; k2 < KC; ++k2) fE[vt][k2] = ld8(swv<C>(sE, LDE, 16 * vt + lr, k2 * 32 + 8 * lg));
  if (SAVE) {  // E rows of this chunk (whole chunk: padded rows included)
    const int64_t r0 = (x.bh * a.Tpad + static_cast<int64_t>(i) * C) * a.dv + x.v0;
    flush_slab_t<C>(static_cast<T*>(a.Er) + r0, a.dv, sE, LDE, x.tid);
  }
  if (OUT && rows) {
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) mma(accO[vt], f.P[k2], fE[vt][k2]);   // P is causal
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) {
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        float gam = 1.f;
        if (GATE == kGateScalar) gam = fast_exp(f.gC[0][0]);
        if (GATE == kGateChannel) gam = fast_exp(f.gC[ct][ii]);
        st[ct][vt][ii] *= gam;
      }
#pragma unroll
      for (int k2 = 0; k2 < KC; ++k2) mma(st[ct][vt], f.G[ct][k2], fE[vt][k2]);
    }
  if (NEXT) scan_load<4, OUT, LA>(fn, a, in, x);
  if (OUT && rows) {
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      st4<T>(swv<C>(sO, LDE, 16 * vt + lr, 16 * w + 4 * lg), a.scale * accO[vt][0], a.scale * accO[vt][1],
             a.scale * accO[vt][2], a.scale * accO[vt][3]);
  }
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
      st4<T>(sw(sH, LDH, 16 * vt + lr, 16 * (w * CT + ct) + 4 * lg), st[ct][vt][0], st[ct][vt][1],
             st[ct][vt][2], st[ct][vt][3]);
  if (vnext) stage_values<T, C>(*reinterpret_cast<const float4(*)[SlabMap<T, C>::kPer]>(vnext), sVt, x.tid);
  lds_barrier();
}

// SAVE: also write the chunk-start states and the E rows the backward
// reads.  OUT: compute and write the output (without it, queries and P are
// neither loaded nor used: the backward's recompute).
// One workgroup's run of the scan: chunks [x.c0, c1) of head x.bh, from the
// start state its role gives (S0, a composed segment start, zero, or for a
// transition slab the identity columns pv0 ..), ending with the end state
// written where its role sends it.
template <typename T, int DK, int GATE, bool SAVE, bool OUT, bool LA, int C>
__device__ __forceinline__ void k3_body(const FwdArgs& a, const ScanCtx& x, int seg, bool probe, int pv0,
                                        int c1, T* sH, T* sX, T* sE, T* sVt, T* sO) {
  constexpr int CT = DK / 64;
  constexpr int LDH = DK + 8;
  const int64_t bh = x.bh;
  const int c0 = x.c0;
  const int w = x.w, lr = x.lr, lg = x.lg;
  const int DV = a.dv;
  const int64_t BHDK = a.BH * static_cast<int64_t>(DK);

  // state slab: rows c = 16*(w*CT+ct) + 4*lg + ii, column v0 + 16*vt + lr
  floatx4 st[CT][2];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int vt = 0; vt < 2; ++vt)
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int c = 16 * (w * CT + ct) + 4 * lg + ii, v = 16 * vt + lr;
        float s0 = 0.f;   // middle segments' local runs start from zero
        if (a.seg_phase == 0 || (a.seg_phase == 1 && seg == 0))
          s0 = a.S0 ? a.S0[(bh * DK + c) * DV + x.v0 + v] : 0.f;
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
      st4<T>(sw(sH, LDH, 16 * vt + lr, 16 * (w * CT + ct) + 4 * lg), st[ct][vt][0],
             st[ct][vt][1], st[ct][vt][2], st[ct][vt][3]);

  // software pipeline, three deep: chunk i+2's operands load while chunk i
  // computes.  The loop covers the run's full chunks, three per trip, with
  // no exit in the middle and unconditional prefetches (past the end they
  // re-read the last chunk), so every path into the loop header has the same
  // loads in flight and the compiler's wait counts stay exact.  A ragged last
  // chunk (only the sequence's last) runs after it.
  ScanFrags<T, DK, GATE, C> f0, f1, f2;
  const int last = c1 - 1;
  const int NF = min(c1, static_cast<int>(a.T / C));   // end of the run's full chunks
  scan_load<7, OUT, LA>(f0, a, c0, x);
  scan_load<7, OUT, LA>(f1, a, min(c0 + 1, last), x);
  stage_values<T, C>(f0.v, sVt, x.tid);
  __syncthreads();
  int i = c0;
  for (; i + 2 < NF; i += 3) {
    scan_step<true, SAVE, OUT, LA, true>(f0, f1.v, f2, i + 2, st, a, i, x, sH, sX, sE, sVt, sO);
    scan_step<true, SAVE, OUT, LA, true>(f1, f2.v, f0, min(i + 3, last), st, a, i + 1, x, sH, sX, sE, sVt, sO);
    scan_step<true, SAVE, OUT, LA, true>(f2, f0.v, f1, min(i + 4, last), st, a, i + 2, x, sH, sX, sE, sVt, sO);
  }
  // f0, f1 hold chunks i, i + 1 (clamped to the last chunk)
  if (NF - i == 2) {
    scan_step<true, SAVE, OUT, LA, true>(f0, f1.v, f2, min(i + 2, last), st, a, i, x, sH, sX, sE, sVt, sO);
    scan_step<true, SAVE, OUT, LA, false>(f1, f2.v, f0, 0, st, a, i + 1, x, sH, sX, sE, sVt, sO);
    i += 2;
    if (i < c1) scan_step<false, SAVE, OUT, LA, false>(f2, nullptr, f0, 0, st, a, i, x, sH, sX, sE, sVt, sO);
  } else if (NF - i == 1) {
    scan_step<true, SAVE, OUT, LA, false>(f0, f1.v, f2, 0, st, a, i, x, sH, sX, sE, sVt, sO);
    i += 1;
    if (i < c1) scan_step<false, SAVE, OUT, LA, false>(f1, nullptr, f2, 0, st, a, i, x, sH, sX, sE, sVt, sO);
  } else if (i < c1) {
    scan_step<false, SAVE, OUT, LA, false>(f0, nullptr, f1, 0, st, a, i, x, sH, sX, sE, sVt, sO);
  }
  if (OUT) flush_output<false, T, C>(a, last, static_cast<int>(min<int64_t>(C, a.T - static_cast<int64_t>(last) * C)), sO, x);
  // the end state: S_T after the sequence's last chunk; phase 1: segment
  // 0's exact end, a middle segment's local end or its transition
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
  } else if (c1 == a.NT && a.S_T) {
    dst = a.S_T + bh * DK * DV;
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

template <typename T, int DK, int GATE, bool SAVE, bool OUT, bool LA, int C>
__global__ __launch_bounds__(256) void k3_chunk_scan(FwdArgs a) {
  constexpr int LDH = DK + 8, LDE = C + 8;
  // [v][.] slabs, addressed through sw() / swv() (bank-spread)
  __shared__ __attribute__((aligned(16))) T sH[BV * LDH];   // io copy of the S^T slab, [v][c]
  __shared__ __attribute__((aligned(16))) T sX[BV * LDE];   // X = V - Lam K S^T, [v][t]
  __shared__ __attribute__((aligned(16))) T sE[BV * LDE];   // E = T X, [v][t]
  __shared__ __attribute__((aligned(16))) T sVt[BV * LDE];  // this chunk's values, [v][t]
  __shared__ __attribute__((aligned(16))) T sO[BV * LDE];   // last chunk's output, [v][t]

  // workgroup -> (head, role, slab); the slabs of one head share an XCD
  // (and its L2).  Roles per head: phase 0, the value slabs of the whole
  // sequence; phase 1, segment 0's value slabs, then per middle segment its
  // value slabs (local, from zero) and d_k / BV transition slabs; phase 3,
  // the value slabs of segments 1 .. S - 1.
  const int nslab = a.dv / BV, npslab = DK / BV;
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
  int seg = 0, slab = role;
  bool probe = false;
  if (a.seg_phase == 1 && role >= nslab) {
    const int r = role - nslab;
    seg = 1 + r / (nslab + npslab);
    slab = r % (nslab + npslab);
    probe = slab >= nslab;
  } else if (a.seg_phase == 3) {
    seg = 1 + role / nslab;
    slab = role % nslab;
  }
  const int c0 = a.seg_phase == 0 ? 0 : seg * a.seg_len;
  const int c1 = a.seg_phase == 0 ? a.NT : min(a.NT, c0 + a.seg_len);
  ScanCtx x;
  x.bh = bh;
  x.b = bh / a.H;
  x.h = bh % a.H;
  x.tid = threadIdx.x;
  x.w = x.tid >> 6;
  x.lr = x.tid & 15;
  x.lg = (x.tid & 63) >> 4;
  // a transition slab reads (and zeroes) value slab 0; its own columns are
  // pv0 .. pv0 + BV of the d_k x d_k transition
  x.v0 = probe ? 0 : slab * BV;
  x.c0 = c0;
  x.vkeep = probe ? 0.f : 1.f;
  const int pv0 = probe ? (slab - nslab) * BV : 0;
  // middle segments of the first pass need only their end states: their
  // run skips the output and the saved rows (the third pass writes those)
  if constexpr (SAVE || OUT) {
    if (a.seg_phase == 1 && seg > 0) {
      k3_body<T, DK, GATE, false, false, LA, C>(a, x, seg, probe, pv0, c1, sH, sX, sE, sVt, sO);
      return;
    }
  }
  k3_body<T, DK, GATE, SAVE, OUT, LA, C>(a, x, seg, probe, pv0, c1, sH, sX, sE, sVt, sO);
}

// Exact start states of the segments from the first pass: forward (REV =
// false), start(1) = end(0) and start(s + 1) = Phi_s start(s) + end(s) up to
// s = S - 2; reverse (the state-adjoint scan, REV = true), start(S - 2) =
// end(S - 1) and start(s - 1) = Phi_s start(s) + end(s) down to s = 1 (end:
// the exact end of the first segment run, a local end otherwise).  The
// columns of a state are independent in these products, so each workgroup
// takes one head and 32 of its d_v columns; fp32 on MFMA (16x16x4): wave w
// owns rows [w DK/4, (w+1) DK/4) of every product.
template <int DK, int DV, bool REV>
__global__ __launch_bounds__(256) void seg_compose(FwdArgs a) {
  constexpr int NSL = DV / 32;              // column slabs per head
  constexpr int RW = DK / 4, RT = RW / 16, CV = 2;
  constexpr int LS = 48, LP = DK + 4;       // padded rows: conflict-free fragment reads
  __shared__ __attribute__((aligned(16))) float sS[DK * LS];
  __shared__ __attribute__((aligned(16))) float sP[DK * LP];
  const int64_t bh = blockIdx.x / NSL;
  const int col0 = static_cast<int>(blockIdx.x % NSL) * 32;
  const int tid = threadIdx.x, w = tid >> 6, lr = tid & 15, lg = (tid & 63) >> 4;
  const int64_t BHDK = a.BH * static_cast<int64_t>(DK);
  const int S = a.seg_cnt;
  auto state = [&](float* base, int sg) { return base + (sg * BHDK + bh * DK) * DV + col0; };
  const int first = REV ? S - 1 : 0, step = REV ? -1 : 1;
  // acc[rt][cv][ii]: row w RW + 16 rt + 4 lg + ii, column col0 + 16 cv + lr
  floatx4 acc[RT][CV];
  auto load_acc = [&](const float* src) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int cv = 0; cv < CV; ++cv)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
          acc[rt][cv][ii] = src[(w * RW + 16 * rt + 4 * lg + ii) * DV + 16 * cv + lr];
  };
  auto store_acc = [&](float* dst, int ld) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int cv = 0; cv < CV; ++cv)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii)
          dst[(w * RW + 16 * rt + 4 * lg + ii) * ld + 16 * cv + lr] = acc[rt][cv][ii];
  };
  load_acc(state(a.seg_end, first));
  store_acc(state(a.seg_start, first + step), DV);
  for (int k = 1; k + 1 < S; ++k) {
    const int sg = first + step * k;   // the middle segment crossed
    __syncthreads();   // the previous product is done with the LDS
    store_acc(sS, LS);
    // every global load of the step is issued before the first LDS store
    const float* phi = a.seg_phi + (sg * BHDK + bh * DK) * DK;
    constexpr int NPV = DK * DK / 1024;   // float4 per thread
    float4 pv[NPV];
#pragma unroll
    for (int u = 0; u < NPV; ++u) pv[u] = *reinterpret_cast<const float4*>(phi + tid * 4 + u * 1024);
    load_acc(state(a.seg_end, sg));
#pragma unroll
    for (int u = 0; u < NPV; ++u) {
      const int j = tid * 4 + u * 1024;
      *reinterpret_cast<float4*>(sP + (j / DK) * LP + j % DK) = pv[u];
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < DK; kk += 4) {
      float fa[RT], fb[CV];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) fa[rt] = sP[(w * RW + 16 * rt + lr) * LP + kk + lg];
#pragma unroll
      for (int cv = 0; cv < CV; ++cv) fb[cv] = sS[(kk + lg) * LS + 16 * cv + lr];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int cv = 0; cv < CV; ++cv) mma4(acc[rt][cv], fa[rt], fb[cv]);
    }
    store_acc(state(a.seg_start, sg + step), DV);
  }
}

template <bool REV>
static hipError_t launch_compose(const FwdArgs& a, hipStream_t s) {
  const unsigned n = static_cast<unsigned>(a.BH * (a.dv / 32));
  if (a.dk == 64 && a.dv == 64) hipLaunchKernelGGL((seg_compose<64, 64, REV>), dim3(n), dim3(256), 0, s, a);
  else if (a.dk == 64) hipLaunchKernelGGL((seg_compose<64, 128, REV>), dim3(n), dim3(256), 0, s, a);
  else if (a.dv == 64) hipLaunchKernelGGL((seg_compose<128, 64, REV>), dim3(n), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((seg_compose<128, 128, REV>), dim3(n), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_seg_compose(const FwdArgs& a, bool rev, hipStream_t s) {
  return rev ? launch_compose<true>(a, s) : launch_compose<false>(a, s);
}

// ---------------------------------------------------------------- T == 0
__global__ void k0_copy_states(FwdArgs a, int64_t nS, int64_t nA) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (a.S_T && idx < nS) a.S_T[idx] = a.S0 ? a.S0[idx] : 0.f;
  if (a.A_T && idx < nA) a.A_T[idx] = a.A0 ? a.A0[idx] : 0.f;
}

// ---------------------------------------------------------------- host side
static size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

WsLayout fwd_ws_layout(int64_t BH, int NT, int dk, int dv, int esz, int gate, int precond, int C) {
  WsLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256(off + bytes); return o; };
  const size_t bh = static_cast<size_t>(BH), nt = static_cast<size_t>(NT);
  if (has_gram(precond)) {
    L.sumL = take(bh * nt * dk * 4);
    L.sumD = take(bh * nt * 4);
    L.Abound = take(bh * (nt + 1) * dk * 4);
  }
  L.KtG = take(bh * nt * dk * C * esz);
  L.Tm = take(bh * nt * C * C * esz);
  L.Pm = take(bh * nt * C * C * esz);
  if (gate == kGateScalar) L.G = take(bh * nt * C * 4);
  if (gate == kGateChannel) L.G = take(bh * nt * dk * 4);   // chunk-end rows only
  if (precond == kATQ) L.Qt = take(bh * nt * C * dk * esz);
  if (gate == kGateChannel) {
    L.QL = take(bh * nt * C * dk * esz);
    L.KL = take(bh * nt * C * dk * esz);
  }
  L.split = scan_split(BH, NT, dk, dv);
  if (L.split.S > 1) {
    const size_t S = static_cast<size_t>(L.split.S);
    L.seg_end = take(S * bh * dk * dv * 4);
    L.seg_phi = take(S * bh * dk * dk * 4);
    L.seg_start = take(S * bh * dk * dv * 4);
  }
  L.total = off;
  return L;
}

template <typename T, int DK, int GATE, int PREC, bool BWD, int C>
static hipError_t launch_k2(const FwdArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k2_chunk_prep<T, DK, GATE, PREC, BWD, C>), dim3(static_cast<unsigned>(a.BH * a.NT)),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int DK, int GATE, bool BWD, int C>
static hipError_t launch_k2_prec(const FwdArgs& a, hipStream_t s) {
  switch (a.precond) {
    case kSquash: return launch_k2<T, DK, GATE, kSquash, BWD, C>(a, s);
    case kIdentity: return launch_k2<T, DK, GATE, kIdentity, BWD, C>(a, s);
    case kExternal: return launch_k2<T, DK, GATE, kExternal, BWD, C>(a, s);
    default:   // forward-only modes (the host rejects them for training)
      if constexpr (BWD) return hipErrorInvalidValue;
      else if (a.precond == kDiagSM) return launch_k2<T, DK, GATE, kDiagSM, false, C>(a, s);
      else return launch_k2<T, DK, GATE, kATQ, false, C>(a, s);
  }
}

// The state scan: one pass over the chunks, or with a sequence split
// (scan_split) the three passes: segment 0 next to the middle segments'
// local scans and transitions, the composition of the segment starts, and
// segments 1 .. S - 1 from their exact starts.  The first pass's middle
// segments also write outputs and saved rows for their chunks from the
// wrong start; the third pass overwrites every one of them.
template <typename T, int DK, int GATE, bool SAVE, bool OUT, bool LA, int C>
static hipError_t launch_k3(const FwdArgs& a0, hipStream_t s) {
  FwdArgs a = a0;
  const int nslab = a.dv / BV, npslab = DK / BV;
  auto grid = [&](int nrole) { return dim3(static_cast<unsigned>(((a.BH + 7) / 8) * 8 * nrole)); };
  if (a.seg_cnt < 3) {
    a.seg_phase = 0;
    hipLaunchKernelGGL((k3_chunk_scan<T, DK, GATE, SAVE, OUT, LA, C>), grid(nslab), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const int S = a.seg_cnt;
  a.seg_phase = 1;
  hipLaunchKernelGGL((k3_chunk_scan<T, DK, GATE, SAVE, OUT, LA, C>), grid(nslab + (S - 2) * (nslab + npslab)),
                     dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((e = launch_compose<false>(a, s)) != hipSuccess) return e;
  a.seg_phase = 3;
  hipLaunchKernelGGL((k3_chunk_scan<T, DK, GATE, SAVE, OUT, LA, C>), grid((S - 1) * nslab), dim3(256), 0, s, a);
  return hipGetLastError();
}

// SAVE: the training forward (k2 in backward mode, k3 also saving the
// chunk states and E rows)
template <typename T, int DK, bool SAVE, int C>
static hipError_t launch_all(const FwdArgs& a, hipStream_t s, hipEvent_t const* ev) {
  hipError_t e;
  auto mark = [&](int i) { return ev && ev[i] ? hipEventRecord(ev[i], s) : hipSuccess; };
  if ((e = mark(0)) != hipSuccess) return e;
  if (has_gram(a.precond)) {
    hipLaunchKernelGGL((k1_precond_summary<T, DK, C>), dim3(static_cast<unsigned>(a.BH * a.NT)), dim3(256),
                       0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((k1_precond_carry<DK>), dim3(static_cast<unsigned>(a.BH * (DK / kCarryCh))), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if ((e = mark(1)) != hipSuccess) return e;
  switch (a.gate) {
    case kGateNone: e = launch_k2_prec<T, DK, kGateNone, SAVE, C>(a, s); break;
    case kGateScalar: e = launch_k2_prec<T, DK, kGateScalar, SAVE, C>(a, s); break;
    default: e = launch_k2_prec<T, DK, kGateChannel, SAVE, C>(a, s); break;
  }
  if (e != hipSuccess) return e;
  if ((e = mark(2)) != hipSuccess) return e;
  if constexpr (!SAVE) {
    if (a.precond == kATQ) {   // linear attention with the preconditioned query
      switch (a.gate) {
        case kGateNone:
          e = launch_k3<T, DK, kGateNone, false, true, true, C>(a, s);
          break;
        case kGateScalar:
          e = launch_k3<T, DK, kGateScalar, false, true, true, C>(a, s);
          break;
        default:
          e = launch_k3<T, DK, kGateChannel, false, true, true, C>(a, s);
          break;
      }
      if (e != hipSuccess) return e;
      return mark(3);
    }
  }
  switch (a.gate) {
    case kGateNone:
      e = launch_k3<T, DK, kGateNone, SAVE, true, false, C>(a, s); break;
    case kGateScalar:
      e = launch_k3<T, DK, kGateScalar, SAVE, true, false, C>(a, s); break;
    default:
      e = launch_k3<T, DK, kGateChannel, SAVE, true, false, C>(a, s);
      break;
  }
  if (e != hipSuccess) return e;
  return mark(3);
}

// the backward's forward recompute: k1 (squash), k2 in backward mode and k3
// saving chunk states and E rows (no output)
template <typename T, int DK, int C>
static hipError_t launch_recompute(const FwdArgs& a, hipStream_t s, hipEvent_t const* ev) {
  hipError_t e;
  auto mark = [&](int i) { return ev && ev[i] ? hipEventRecord(ev[i], s) : hipSuccess; };
  if ((e = mark(0)) != hipSuccess) return e;
  if (has_gram(a.precond)) {
    hipLaunchKernelGGL((k1_precond_summary<T, DK, C>), dim3(static_cast<unsigned>(a.BH * a.NT)), dim3(256),
                       0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((k1_precond_carry<DK>), dim3(static_cast<unsigned>(a.BH * (DK / kCarryCh))), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if ((e = mark(1)) != hipSuccess) return e;
  switch (a.gate) {
    case kGateNone: e = launch_k2_prec<T, DK, kGateNone, true, C>(a, s); break;
    case kGateScalar: e = launch_k2_prec<T, DK, kGateScalar, true, C>(a, s); break;
    default: e = launch_k2_prec<T, DK, kGateChannel, true, C>(a, s); break;
  }
  if (e != hipSuccess) return e;
  if ((e = mark(2)) != hipSuccess) return e;
  switch (a.gate) {
    case kGateNone:
      e = launch_k3<T, DK, kGateNone, true, false, false, C>(a, s); break;
    case kGateScalar:
      e = launch_k3<T, DK, kGateScalar, true, false, false, C>(a, s); break;
    default:
      e = launch_k3<T, DK, kGateChannel, true, false, false, C>(a, s); break;
  }
  if (e != hipSuccess) return e;
  return mark(3);
}

template <int C>
static hipError_t launch_forward_parts_c(const FwdArgs& a, int io_bf16, hipStream_t s, hipEvent_t const* ev) {
  if (io_bf16) return a.dk == 64 ? launch_recompute<bf16, 64, C>(a, s, ev) : launch_recompute<bf16, 128, C>(a, s, ev);
  return launch_recompute<float, 64, C>(a, s, ev);
}

hipError_t launch_forward_parts(const FwdArgs& a, int io_bf16, hipStream_t s, hipEvent_t const* ev) {
  return a.chunk == 32 ? launch_forward_parts_c<32>(a, io_bf16, s, ev)
                       : launch_forward_parts_c<64>(a, io_bf16, s, ev);
}

// The workspace of pdn_chunk_fwd_noalloc.  Host code never uses this name
// as an address (on the host it is only a registration handle): kernels get
// the device address that noalloc_scratch looks up.
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

hipError_t noalloc_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[kNoallocMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kNoallocMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

template <int C>
static hipError_t launch_chunks(const FwdArgs& a, int io_bf16, hipStream_t s, hipEvent_t const* ev, bool train) {
  if (train) {   // the host admits fp32 io only with d_k = d_v = 64 here
    if (io_bf16) return a.dk == 64 ? launch_all<bf16, 64, true, C>(a, s, ev) : launch_all<bf16, 128, true, C>(a, s, ev);
    return launch_all<float, 64, true, C>(a, s, ev);
  }
  if (io_bf16) {
    return a.dk == 64 ? launch_all<bf16, 64, false, C>(a, s, ev) : launch_all<bf16, 128, false, C>(a, s, ev);
  }
  return a.dk == 64 ? launch_all<float, 64, false, C>(a, s, ev) : launch_all<float, 128, false, C>(a, s, ev);
}

hipError_t launch_forward(const FwdArgs& a, int io_bf16, hipStream_t s, hipEvent_t const* ev, bool train) {
  if (a.BH == 0 || a.T == 0) {
    // nothing to time: the stage events still mark the (empty) stages
    if (ev)
      for (int i = 0; i < 4; ++i)
        if (ev[i] && hipEventRecord(ev[i], s) != hipSuccess) return hipErrorInvalidValue;
  }
  if (a.BH == 0) return hipSuccess;
  if (a.T == 0) {
    const int64_t nS = a.BH * a.dk * a.dv, nA = a.BH * a.dk;
    const int64_t n = nS > nA ? nS : nA;
    hipLaunchKernelGGL(k0_copy_states, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s,
                       a, nS, nA);
    return hipGetLastError();
  }
  return a.chunk == 32 ? launch_chunks<32>(a, io_bf16, s, ev, train)
                       : launch_chunks<64>(a, io_bf16, s, ev, train);
}

}  // namespace pdn
