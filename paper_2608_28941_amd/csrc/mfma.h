// MFMA 16x16x4 wrappers for gfx950 (CDNA4).
//
// v_mfma_f64_16x16x4_f64 and v_mfma_f32_16x16x4_f32 compute
// D (16x16) = A (16x4) * B (4x16) + C on one 64-lane wavefront.  With lane l,
// g = l / 16 and m = l % 16 (measured on gfx950):
//   A: lane l holds A[m][g]               (row m, k = g)     both types
//   B: lane l holds B[g][m]               (k = g, column m)  both types
//   C/D: lane l, item i = 0..3 holds D[drow(g, i)][m] with
//        drow = g + 4 i for f64 and 4 g + i for f32.
// The K index is a pure summation index, so kernels may assign any 4 source
// indices to the 4 lane groups as long as A and B agree.
#pragma once

#include <hip/hip_runtime.h>

namespace rrf {

typedef double d4_t __attribute__((ext_vector_type(4)));
typedef float f4_t __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;

template <> struct Mfma<double> {
  typedef d4_t acc_t;
  static __device__ __forceinline__ acc_t zero() { return acc_t{0.0, 0.0, 0.0, 0.0}; }
  static __device__ __forceinline__ acc_t op(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ int drow(int g, int i) { return g + 4 * i; }
};

template <> struct Mfma<float> {
  typedef f4_t acc_t;
  static __device__ __forceinline__ acc_t zero() { return acc_t{0.f, 0.f, 0.f, 0.f}; }
  static __device__ __forceinline__ acc_t op(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ int drow(int g, int i) { return 4 * g + i; }
};

}  // namespace rrf
