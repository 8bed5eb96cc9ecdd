// Device-side helpers shared by the libxpipe HIP kernels (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define XP_DEV __device__ __forceinline__

typedef uint16_t bf16_t;  // bf16 bit pattern
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef double f64x4_t __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- bf16
// Workgroups are dispatched to the 8 XCDs (each with its own L2) round-robin
// by linear id.  Remap the linear id so that each XCD takes a contiguous run
// of the logical tile order: neighbouring tiles (shared input rows, shared
// pixel splits) then meet in one L2.  A bijection of [0, G).
constexpr int XP_XCDS = 8;
XP_DEV int xcd_tile(int l, int G) {
  const int x = l % XP_XCDS, q = l / XP_XCDS;
  const int per = G / XP_XCDS, rem = G % XP_XCDS;
  return x * per + (x < rem ? x : rem) + q;
}

XP_DEV float bf16_to_f32(bf16_t u) { return __uint_as_float((uint32_t)u << 16); }

// fp32 -> bf16, round to nearest, ties to even (the gfx950 conversion
// instruction); NaN stays a NaN.
XP_DEV bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// two fp32 -> two bf16 packed low, high (one conversion instruction)
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
XP_DEV uint32_t f32x2_to_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// ---------------------------------------------------------------- storage traits
// Activations are stored as float (XPIPE_F32) or bf16 (XPIPE_BF16); element-
// wise and reduction arithmetic is done in double and rounded once on store.
template <typename T> struct Store;
template <> struct Store<float> {
  static XP_DEV double ld(const float* p) { return (double)*p; }
  static XP_DEV void st(float* p, double v) { *p = (float)v; }
};
template <> struct Store<bf16_t> {
  static XP_DEV double ld(const bf16_t* p) { return (double)bf16_to_f32(*p); }
  // double -> fp32 (nearest) -> bf16 (nearest even), the storage model of the
  // bf16 variant
  static XP_DEV void st(bf16_t* p, double v) { *p = f32_to_bf16((float)v); }
};

template <typename T> XP_DEV double ldd(const T* p) { return Store<T>::ld(p); }
// v rounded to the storage type and widened back (what a store then a load gives)
template <typename T> XP_DEV double rnd(double v);
template <> XP_DEV double rnd<float>(double v) { return (double)(float)v; }
template <> XP_DEV double rnd<bf16_t>(double v) { return (double)bf16_to_f32(f32_to_bf16((float)v)); }
template <typename T> XP_DEV void std_(T* p, double v) { Store<T>::st(p, v); }

// ---------------------------------------------------------------- reductions
XP_DEV double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

XP_DEV double wave_max(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
  return v;
}

// ---------------------------------------------------------------- batch-norm statistics
// mean and 1/sqrt(biased variance + eps) from the column sum and sum of squares
XP_DEV void bn_stats_from_sums(double s0, double s1, int M, double eps, double* mean,
                               double* rstd) {
  const double mu = s0 / M;
  double var = s1 / M - mu * mu;
  if (var < 0.0) var = 0.0;
  *mean = mu;
  *rstd = 1.0 / sqrt(var + eps);
}
