// Gaussian sketch Omega (Alg. 2, sketch step) as RRF-NORMAL-v1.
//
// Entry (row r, global column g) of the n x inf sketch is a pure function of
// (seed, g, r): Philox4x64-10 (Salmon et al., SC'11) with key (seed, 0) and
// counter (r / 4, g, 0, 0) gives four 64-bit words; each pair of words becomes
// two Gaussians by Box--Muller with a transcendental-free ln / sin / cos made
// of correctly rounded binary64 +, -, *, /, sqrt in a fixed order.  This file
// must be compiled with -ffp-contract=off (no fused multiply-add); the pragma
// below says the same for the functions that matter.
//
// Work: one thread per counter block (4 rows of one column).  The kernel is
// tiny next to the GEMM stages (n x b values per block of the method).

#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull;   // Philox4x64 multipliers
constexpr uint64_t kM1 = 0xCA5A826395121157ull;
constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull;   // Weyl key increments
constexpr uint64_t kW1 = 0xBB67AE8584CAA73Bull;

constexpr double kSqrtHalf = 0x1.6a09e667f3bcdp-1;  // nearest binary64 values
constexpr double kLn2 = 0x1.62e42fefa39efp-1;
constexpr double kPiO2 = 0x1.921fb54442d18p+0;
constexpr double kTwoM53 = 0x1p-53;

__device__ __forceinline__ void philox4x64_10(uint64_t c0, uint64_t c1,
                                              uint64_t c2, uint64_t c3,
                                              uint64_t k0, uint64_t k1,
                                              uint64_t out[4]) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += kW0;
      k1 += kW1;
    }
    const uint64_t lo0 = kM0 * c0, hi0 = __umul64hi(kM0, c0);
    const uint64_t lo1 = kM1 * c2, hi1 = __umul64hi(kM1, c2);
    const uint64_t n0 = hi1 ^ c1 ^ k0;
    const uint64_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

// ln u for u in (0, 1]: u = f 2^e, f in [sqrt(1/2), sqrt(2)); ln f by the
// series 2 atanh(s) = 2 s sum_{j<=10} s^(2j) / (2j+1), s = (f-1)/(f+1).
__device__ __forceinline__ double spec_ln(double u) {
#pragma clang fp contract(off)
  int e;
  double f = frexp(u, &e);
  if (f < kSqrtHalf) {
    f = f * 2.0;
    e = e - 1;
  }
  const double s = (f - 1.0) / (f + 1.0);
  const double z = s * s;
  double p = 1.0 / 21.0;
  p = p * z + 1.0 / 19.0;
  p = p * z + 1.0 / 17.0;
  p = p * z + 1.0 / 15.0;
  p = p * z + 1.0 / 13.0;
  p = p * z + 1.0 / 11.0;
  p = p * z + 1.0 / 9.0;
  p = p * z + 1.0 / 7.0;
  p = p * z + 1.0 / 5.0;
  p = p * z + 1.0 / 3.0;
  p = p * z + 1.0;
  return (double)e * kLn2 + (s + s) * p;
}

// cos and sin of 2 pi u for u in [0, 1): quadrant from 4u, then nested
// Taylor polynomials through phi^22 (cos) and phi^23 (sin) on [0, pi/2).
// The quadrant rotation is branch-free: the magnitude comes from the parity
// of q and the sign from its bits (q = 1, 2 negate cos; q = 2, 3 negate sin).
struct CosSin { double c, s; };

__device__ __forceinline__ CosSin spec_cos_sin_2pi(double u) {
#pragma clang fp contract(off)
  const double t = 4.0 * u;
  const double q = floor(t);
  const double phi = (t - q) * kPiO2;
  const double x = phi * phi;
  double ps = 1.0, pc = 1.0;
#pragma unroll
  for (int k = 11; k >= 1; --k) {
    const double sk = 1.0 / (double)((2 * k) * (2 * k + 1));
    const double ck = 1.0 / (double)((2 * k - 1) * (2 * k));
    ps = 1.0 - (x * ps) * sk;
    pc = 1.0 - (x * pc) * ck;
  }
  const double sn = phi * ps;
  const double cs = pc;
  const int qi = (int)q;
  const bool odd = (qi & 1) != 0;
  const double cmag = odd ? sn : cs;
  const double smag = odd ? cs : sn;
  CosSin r;
  r.c = (((qi + 1) & 2) != 0) ? -cmag : cmag;
  r.s = ((qi & 2) != 0) ? -smag : smag;
  return r;
}

__device__ __forceinline__ void box_muller(uint64_t wa, uint64_t wb,
                                           double* z0, double* z1) {
#pragma clang fp contract(off)
  const double u1 = (double)((wa >> 11) + 1ull) * kTwoM53;
  const double u2 = (double)(wb >> 11) * kTwoM53;
  const double r = sqrt(-2.0 * spec_ln(u1));
  const CosSin cs = spec_cos_sin_2pi(u2);
  *z0 = r * cs.c;
  *z1 = r * cs.s;
}

// Rows [n, n_pad) are written as zeros (the update stages whole chunks).
template <typename T>
__global__ __launch_bounds__(256) void sketch_kernel(
    uint64_t seed, int64_t n, int64_t n_pad, int64_t col0, int64_t ncols,
    T* out, int64_t row_stride, int64_t col_stride) {
  const int64_t nq = (n + 3) / 4;
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= nq) {
    const int64_t r0 = 4 * q;
    if (r0 < n_pad)
      for (int64_t j = blockIdx.y; j < ncols; j += gridDim.y)
        for (int t = 0; t < 4; ++t)
          if (r0 + t < n_pad) out[(r0 + t) * row_stride + j * col_stride] = T(0);
    return;
  }
  for (int64_t j = blockIdx.y; j < ncols; j += gridDim.y) {
    const uint64_t g = (uint64_t)(col0 + j);
    uint64_t w[4];
    philox4x64_10((uint64_t)q, g, 0ull, 0ull, seed, 0ull, w);
    double z[4];
    box_muller(w[0], w[1], &z[0], &z[1]);
    box_muller(w[2], w[3], &z[2], &z[3]);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t r = 4 * q + t;
      if (r < n) out[r * row_stride + j * col_stride] = (T)z[t];
      else if (r < n_pad) out[r * row_stride + j * col_stride] = T(0);
    }
  }
}

// Row-major output (col_stride 1): lanes along the columns, so that a
// wavefront store covers 64 consecutive columns of one row; each thread makes
// the four rows of one Philox block, as above (same blocks, same values).
// Wavefront w of a workgroup takes row quads blockIdx.x * 4 + w + 4 gridDim.x i.
template <typename T>
__global__ __launch_bounds__(256) void sketch_rows_kernel(
    uint64_t seed, int64_t n, int64_t n_pad, int64_t col0, int64_t ncols,
    T* out, int64_t row_stride) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t j = (int64_t)blockIdx.y * 64 + lane;
  if (j >= ncols) return;
  const int64_t nq = (n_pad + 3) / 4;
  for (int64_t q = (int64_t)blockIdx.x * 4 + wv; q < nq; q += (int64_t)gridDim.x * 4) {
    T v[4] = {T(0), T(0), T(0), T(0)};
    if (4 * q < n) {
      uint64_t w[4];
      philox4x64_10((uint64_t)q, (uint64_t)(col0 + j), 0ull, 0ull, seed, 0ull, w);
      double z[4];
      box_muller(w[0], w[1], &z[0], &z[1]);
      box_muller(w[2], w[3], &z[2], &z[3]);
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (4 * q + t < n) v[t] = (T)z[t];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (4 * q + t < n_pad) out[(4 * q + t) * row_stride + j] = v[t];
  }
}

}  // namespace

template <typename T>
hipError_t launch_sketch(uint64_t seed, int64_t n, int64_t n_pad, int64_t col0,
                         int64_t ncols, T* out, int64_t row_stride,
                         int64_t col_stride, hipStream_t s) {
  if (n <= 0 || ncols <= 0) return hipSuccess;
  if (n_pad < n) n_pad = n;
  const int64_t nq = (n_pad + 3) / 4;
  if (col_stride == 1 && ceil_div(ncols, 64) <= 65535) {
    const dim3 rgrid((unsigned)std::min<int64_t>(ceil_div(nq, 4), 4096),
                     (unsigned)ceil_div(ncols, 64));
    hipLaunchKernelGGL(sketch_rows_kernel<T>, rgrid, dim3(256), 0, s, seed, n, n_pad,
                       col0, ncols, out, row_stride);
    return hipGetLastError();
  }
  dim3 grid((unsigned)ceil_div(nq, 256), (unsigned)(ncols < 65535 ? ncols : 65535));
  hipLaunchKernelGGL(sketch_kernel<T>, grid, dim3(256), 0, s, seed, n, n_pad,
                     col0, ncols, out, row_stride, col_stride);
  return hipGetLastError();
}

template hipError_t launch_sketch<float>(uint64_t, int64_t, int64_t, int64_t,
                                         int64_t, float*, int64_t, int64_t,
                                         hipStream_t);
template hipError_t launch_sketch<double>(uint64_t, int64_t, int64_t, int64_t,
                                          int64_t, double*, int64_t, int64_t,
                                          hipStream_t);

}  // namespace rrf
