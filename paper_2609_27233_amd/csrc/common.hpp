// Device helpers shared by the span-merging kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spanmerge.h"

#define SM_API extern "C" __attribute__((visibility("default")))

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

namespace sm {

constexpr int kWave = 64;

// ---- bf16 <-> fp32 -------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Round to nearest even; NaN stays a quiet NaN.  gfx950 converts in one
// instruction (v_cvt_pk_bf16_f32, two values at a time).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// Two floats -> packed pair of bf16 (low half = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

// ---- element storage ------------------------------------------------------
template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float *p) { return *p; }
  static __device__ __forceinline__ float from_bits(float x) { return x; }
  static __device__ __forceinline__ float to_store(float x) { return x; }
};
template <> struct Elem<uint16_t> {
  static __device__ __forceinline__ float load(const uint16_t *p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ uint16_t to_store(float x) { return f32_to_bf16(x); }
};

// ---- wavefront / workgroup reductions ------------------------------------
// Butterfly over the 64 lanes without the LDS crossbar (ds_bpermute, one LDS
// round trip per step): four DPP steps inside each 16-lane row (swap
// neighbours, swap pairs, mirror within 8, mirror within 16), then the two
// gfx950 lane-swap instructions for row pairs and wave halves.  Every lane
// ends with the same value.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i <- 7 - i within 8
constexpr int kDppMirror = 0x140;      // lane i <- 15 - i within 16

// {a, b} = {v[lane], v[lane ^ 16]} (swap16) or {v[lane], v[lane ^ 32]} (swap32),
// in an order that depends on the lane; every caller combines them symmetrically.
// All 64 lanes must be active, as for the DPP steps.
__device__ __forceinline__ void swap16(float v, float &a, float &b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap32(float v, float &a, float &b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<kDppXor1>(v);
  v += dpp_f32<kDppXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  float a, b;
  swap16(v, a, b);
  v = a + b;
  swap32(v, a, b);
  return a + b;
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  float a, b;
  swap16(v, a, b);
  v = fmaxf(a, b);
  swap32(v, a, b);
  return fmaxf(a, b);
}

// Workgroup barrier that orders LDS only.  __syncthreads() also waits for
// every outstanding global load of the calling wave (vmcnt(0)); this one
// lets loads whose results are consumed later stay in flight across it.
// Use it only where no wave reads global data another wave wrote before
// the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Sum over the workgroup; `red` needs blockDim.x / 64 floats of LDS.
__device__ __forceinline__ float block_sum(float v, float *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}
__device__ __forceinline__ float block_max(float v, float *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = -INFINITY;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, red[i]);
  return t;
}

// Inclusive prefix sum over the workgroup (blockDim.x <= 1024);
// `red` needs 16 ints of LDS.  Returns the inclusive value, *total gets the
// workgroup total.
__device__ __forceinline__ int block_inclusive_scan(int v, int *red, int *total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int u = __shfl_up(v, off, kWave);
    if (lane >= off) v += u;
  }
  __syncthreads();
  if (lane == 63) red[w] = v;
  __syncthreads();
  int before = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) before += red[i];
    tot += red[i];
  }
  *total = tot;
  return v + before;
}

// GELU(x) = x Phi(x) with Phi(x) = erfc(-x / sqrt 2) / 2, written as
// max(x, 0) - |x| erfc(z) / 2 with z = |x| / sqrt 2 (for x >= 0,
// x Phi(x) = x - x erfc(z) / 2; for x < 0 it is x erfc(z) / 2).  erfc(z)
// comes from the Chebyshev-fitted formula of Numerical Recipes (2nd ed.,
// section 6.2, function erfcc: t = 1 / (1 + z / 2), erfc = t exp(-z^2 +
// P(t)) with a degree-9 polynomial P, fractional error below 1.2e-7 for
// every z); the factor 1 / 2 and the 1 / sqrt 2 of |x| = sqrt 2 z go into
// the exponent as -1/2 (log2 of sqrt 2 / 2).  One reciprocal, one
// exponential and twelve fused multiply-adds or multiplies; the form
// 0.5 x (1 + erf(x / sqrt 2)) costs about twice the instructions and loses
// all relative accuracy for x below about -4, where 1 + erf cancels.
// Measured against erfc in double: relative error below 1.3e-6 for
// |x| <= 3, absolute error below 4e-7 everywhere.
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.5f, z, 1.0f));
  float p = fmaf(t, 0.17087277f, -0.82215223f);
  p = fmaf(t, p, 1.48851587f);
  p = fmaf(t, p, -1.13520398f);
  p = fmaf(t, p, 0.27886807f);
  p = fmaf(t, p, -0.18628806f);
  p = fmaf(t, p, 0.09678418f);
  p = fmaf(t, p, 0.37409196f);
  p = fmaf(t, p, 1.00002368f);
  p = fmaf(t, p, -1.26551223f);
  // t 2^((P - z^2) log2 e - 1/2) = erfc(z) / (2 sqrt 2) = (erfc(z) / 2) / (|x| / z)
  const float te = t * __builtin_amdgcn_exp2f(fmaf(fmaf(-z, z, p), 1.4426950408889634f, -0.5f));
  return fmaf(-z, te, fmaxf(x, 0.f));
}

__device__ __forceinline__ void set_err(int32_t *err, int bit) {
  atomicOr(err, bit);
}


// Division by a runtime divisor d (1 <= d < 2^31) for 0 <= x < 2^31 as a
// multiply-high and shift (Granlund & Montgomery, "Division by invariant
// integers using multiplication", PLDI 1994): shift = ceil(log2 d),
// mul = floor(2^32 (2^shift - d) / d) + 1, q = (mulhi(x, mul) + x) >> shift.
struct FastDiv {
  uint32_t d, mul, shift;
};

static inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t sh = 0;
  while ((1ull << sh) < d) ++sh;
  const uint64_t m = ((1ull << 32) * ((1ull << sh) - d)) / d + 1;
  return FastDiv{d, (uint32_t)m, sh};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t x, const FastDiv &f) {
  return (__umulhi(x, f.mul) + x) >> f.shift;
}

}  // namespace sm
