// Device-side building blocks for the gfx950 kernels: element types, 8-wide
// MFMA operand fragments, conversions and vector loads.
//
// MFMA tiles are 16x16 outputs with a 32-deep contraction slab.  A fragment
// is what one lane supplies for such a slab: 8 consecutive contraction
// elements.  With lane l, row/col index m = l % 16 and lane group g = l / 16:
//   A operand  A[m][8g + s],  B operand  B[8g + s][m],  s = 0..7
//   accumulator (floatx4) element i holds D[4g + i][m]
// For bf16 one v_mfma_f32_16x16x32_bf16 consumes the fragment; for fp32 the
// same fragment feeds eight v_mfma_f32_16x16x4_f32 (step s contracts the
// elements 8g + s of the four lane groups), so every kernel is written once
// for both element types.  (Layouts verified on gfx950.)
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pdn_internal.hpp"

namespace pdn {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16 x) { return static_cast<float>(x); }

template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float x) {
  return static_cast<bf16>(x);  // round to nearest even
}

template <typename T> struct Frag8;
template <> struct Frag8<bf16> {
  bf16x8 v;
  __device__ __forceinline__ float get(int s) const { return static_cast<float>(v[s]); }
  __device__ __forceinline__ void set(int s, float x) { v[s] = static_cast<bf16>(x); }
};
template <> struct Frag8<float> {
  floatx4 lo, hi;
  __device__ __forceinline__ float get(int s) const { return s < 4 ? lo[s] : hi[s - 4]; }
  __device__ __forceinline__ void set(int s, float x) {
    if (s < 4) lo[s] = x; else hi[s - 4] = x;
  }
};

template <typename T>
__device__ __forceinline__ Frag8<T> frag_zero() {
  Frag8<T> f;
#pragma unroll
  for (int s = 0; s < 8; ++s) f.set(s, 0.f);
  return f;
}

// 8 consecutive elements from a 16-byte (bf16) / 32-byte (fp32) aligned address
__device__ __forceinline__ Frag8<bf16> ld8(const bf16* p) {
  Frag8<bf16> f;
  f.v = *reinterpret_cast<const bf16x8*>(p);
  return f;
}
__device__ __forceinline__ Frag8<float> ld8(const float* p) {
  Frag8<float> f;
  f.lo = *reinterpret_cast<const floatx4*>(p);
  f.hi = *reinterpret_cast<const floatx4*>(p + 4);
  return f;
}
__device__ __forceinline__ void st8(bf16* p, const Frag8<bf16>& f) {
  *reinterpret_cast<bf16x8*>(p) = f.v;
}
__device__ __forceinline__ void st8(float* p, const Frag8<float>& f) {
  *reinterpret_cast<floatx4*>(p) = f.lo;
  *reinterpret_cast<floatx4*>(p + 4) = f.hi;
}

// base + a 32-bit byte offset: lets the backend use the scalar-base +
// vector-offset global addressing form (no 64-bit per-lane arithmetic)
template <typename T>
__device__ __forceinline__ const T* at_bytes(const T* base, uint32_t byte_off) {
  return reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + byte_off);
}
template <typename T>
__device__ __forceinline__ T* at_bytes(T* base, uint32_t byte_off) {
  return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + byte_off);
}

// acc += A_frag * B_frag over one 32-deep slab
__device__ __forceinline__ void mma(floatx4& acc, const Frag8<bf16>& a, const Frag8<bf16>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(floatx4& acc, const Frag8<float>& a, const Frag8<float>& b) {
#pragma unroll
  for (int s = 0; s < 8; ++s)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.get(s), b.get(s), acc, 0, 0, 0);
}

// fp32 16x16x4 step: acc += A[16 x 4] B[4 x 16]; lane supplies A[m][g], B[g][m]
__device__ __forceinline__ void mma4(floatx4& acc, float a, float b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
}

// Address of element (row, col) of an LDS slab [rows][ld] whose rows are
// also read across (a transposed column: one element from each of many
// rows).  With row strides of 72 or 136 elements, rows 8 apart fall on the
// same banks; XOR-ing the column by 16 * ((row >> 3) & 3) spreads them over
// distinct banks and keeps every aligned run of 16 elements contiguous, so
// 4- and 8-element vector accesses stay whole.
template <typename T>
__device__ __forceinline__ T* sw(T* base, int ld, int row, int col) {
  return base + row * ld + (col ^ (((row >> 3) & 3) << 4));
}
template <typename T>
__device__ __forceinline__ const T* sw(const T* base, int ld, int row, int col) {
  return base + row * ld + (col ^ (((row >> 3) & 3) << 4));
}

// Pins a prefetched 16-byte value to this point of the program: the empty
// volatile asm "redefines" it, so unpacking it cannot be hoisted up to its
// load (the wait for the load would then drain every later prefetch too).
__device__ __forceinline__ float4 pin_here(float4 v) {
  asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
  return v;
}

// 4 consecutive elements (8 / 16 bytes), used to stage accumulator columns
template <typename T> struct Vec4;
template <> struct Vec4<bf16> { typedef bf16x4 type; };
template <> struct Vec4<float> { typedef floatx4 type; };

template <typename T>
__device__ __forceinline__ void st4(T* p, float a, float b, float c, float d) {
  typename Vec4<T>::type v;
  v[0] = from_f<T>(a); v[1] = from_f<T>(b); v[2] = from_f<T>(c); v[3] = from_f<T>(d);
  *reinterpret_cast<typename Vec4<T>::type*>(p) = v;
}

// One 16x16 output tile of A Bt^T over a contraction of K (multiple of 32):
// A points at row 0 of the tile's rows (row-major, leading dim lda), Bt at
// row 0 of its columns stored as rows (row-major, leading dim ldb).  Every
// operand used this way is staged as [output index][contraction index], so
// each fragment is one contiguous 8-element read.
template <int K, typename T>
__device__ __forceinline__ void mma_tile(floatx4& acc, const T* A, int lda, const T* Bt, int ldb,
                                         int lr, int lg) {
#pragma unroll
  for (int kk = 0; kk < K / 32; ++kk)
    mma(acc, ld8(A + lr * lda + kk * 32 + 8 * lg), ld8(Bt + lr * ldb + kk * 32 + 8 * lg));
}

// accumulator tile -> memory, row-major (4 scalar stores) or transposed
// (one 4-vector store)
template <typename T>
__device__ __forceinline__ void st_tile(T* out, int ld, const floatx4& acc, int lr, int lg,
                                        float scale = 1.f) {
#pragma unroll
  for (int ii = 0; ii < 4; ++ii) out[(4 * lg + ii) * ld + lr] = from_f<T>(scale * acc[ii]);
}
template <typename T>
__device__ __forceinline__ void st_tile_t(T* out, int ld, const floatx4& acc, int lr, int lg,
                                          float scale = 1.f) {
  st4<T>(out + lr * ld + 4 * lg, scale * acc[0], scale * acc[1], scale * acc[2], scale * acc[3]);
}

// Word 3 of a raw (untyped, unswizzled) buffer resource on gfx9-family
// chips: a 32-bit data format, which untyped accesses need to be non-zero.
constexpr int kBufWord3 = 0x00020000;

constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLog2e = 1.4426950408889634f;
// v where ok, else zeros (per component, so the value stays in registers)
__device__ __forceinline__ float4 keep_if(float4 v, bool ok) {
  return make_float4(ok ? v.x : 0.f, ok ? v.y : 0.f, ok ? v.z : 0.f, ok ? v.w : 0.f);
}
__device__ __forceinline__ float fast_exp(float x) { return __expf(x); }
// 2^x on the hardware exponential (a result below the normal range flushes
// to zero)
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
// natural log on the hardware base-2 logarithm: ln x = ln 2 * log2 x.  x must
// be a positive normal number (callers clamp); denormal inputs are not
// rescaled.
__device__ __forceinline__ float fast_log(float x) { return kLn2 * __builtin_amdgcn_logf(x); }
// hardware reciprocal (1 ulp)
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Stable preconditioner gain B = exp(-log(x) * r / (1 + |r|)), r = log(A) - mu;
// A <= 0 (a key channel that has been zero so far) takes the r -> -inf limit,
// B = x.  Branch-free (a select), so unrolled callers keep one basic block.
__device__ __forceinline__ float squash_gain(float A, float mu, float lnx) {
  const float r = fast_log(fmaxf(A, 1e-30f)) - mu;
  const float s = A > 0.f ? r * fast_rcp(1.f + fabsf(r)) : -1.f;
  return exp2_hw((-lnx * kLog2e) * s);
}

}  // namespace pdn
