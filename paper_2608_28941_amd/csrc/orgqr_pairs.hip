// Compact WY of two adjacent blocks of reflectors for the explicit-Q pass
// (Q = H_0 ... H_{k-1} [I_k; 0], Sec. 4 storage scheme, Eq. (1)).
//
// For consecutive blocks with reflectors V_1 (b1 columns) and V_2 (b2
// columns, b1 + b2 <= 64) and their forward T factors (Eq. (4)):
//   (I - V_1 T_1 V_1^T)(I - V_2 T_2 V_2^T) = I - [V_1 V_2] T [V_1 V_2]^T,
//   T = [T_1  -T_1 (V_1^T V_2) T_2 ; 0  T_2]
// (the larft recursion one block at a time), so the backward pass applies
// the pair as one block of up to 64 reflectors: half the passes over Q when
// the blocks are 32 columns wide.
//
//   pair_gram_kernel  G_s = V_1^T V_2 over the rows of split s (rows above
//                     V_2's first row are zero in V_2), one workgroup per
//                     (pair, split);
//   pair_t_kernel     G = sum_s G_s in split order (deterministic), the
//                     merged T into its own 64 x 64 block, and explicit zeros
//                     in V_2's rows above its first row (the pass reads V_1
//                     and V_2 as one 64-column block).

#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr int kPairRows = 64;   // rows of V staged per chunk

__global__ __launch_bounds__(256) void pair_gram_kernel(PairArgs a) {
  __shared__ double v1[kPairRows][33];
  __shared__ double v2[kPairRows][33];
  const OrgqrPair pr = a.pairs[blockIdx.x];
  const int s = (int)blockIdx.y, t = (int)threadIdx.x;
  // Entries (i, j) = (t / 32 + 8 q, t % 32), q = 0..3, of the b1 x b2 block.
  const int i0 = t / 32, jj = t % 32;
  const int64_t r_first = pr.k0 + pr.b1;             // V_2's first row
  const int64_t rows = a.m - r_first;
  const int64_t per = ((rows + a.nsplit - 1) / a.nsplit + kPairRows - 1) / kPairRows * kPairRows;
  const int64_t r_begin = r_first + (int64_t)s * per;
  const int64_t r_end = min(a.m, r_begin + per);
  const double* V1 = a.V + pr.k0 * a.ldv;
  const double* V2 = a.V + (pr.k0 + pr.b1) * a.ldv;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int64_t r0 = r_begin; r0 < r_end; r0 += kPairRows) {
    __syncthreads();
    // Thread t stages row t % 64 of 8 columns of each block (coalesced rows).
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = t / 64 + 4 * u;
      const int64_t r = r0 + t % 64;
      const bool ok = r < r_end;
      v1[t % 64][c] = (ok && c < pr.b1) ? V1[r + (int64_t)c * a.ldv] : 0.0;
      v2[t % 64][c] = (ok && c < pr.b2) ? V2[r + (int64_t)c * a.ldv] : 0.0;
    }
    __syncthreads();
#pragma unroll 8
    for (int rr = 0; rr < kPairRows; ++rr) {
      const double y = v2[rr][jj];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[q] += v1[rr][i0 + 8 * q] * y;
    }
  }
  double* G = a.part + ((int64_t)blockIdx.x * a.nsplit + s) * 1024;
#pragma unroll
  for (int q = 0; q < 4; ++q) G[(i0 + 8 * q) * 32 + jj] = acc[q];
}

__global__ __launch_bounds__(256) void pair_t_kernel(PairArgs a) {
  __shared__ double T1[32][33], T2[32][33], G[32][33], M[32][33];
  const OrgqrPair pr = a.pairs[blockIdx.x];
  const int t = (int)threadIdx.x;
  const int b1 = pr.b1, b2 = pr.b2;
  // G = sum of the split partials in split order.
  for (int e = t; e < 1024; e += 256) {
    const double* src = a.part + (int64_t)blockIdx.x * a.nsplit * 1024 + e;
    double g = 0.0;
    for (int s = 0; s < a.nsplit; ++s) g += src[(int64_t)s * 1024];
    G[e / 32][e % 32] = g;
  }
  // T_1, T_2 (upper triangular, leading b x b blocks of their stored T).
  for (int e = t; e < 1024; e += 256) {
    const int i = e % 32, j = e / 32;
    T1[i][j] = (i <= j && j < b1) ? a.Tm[i + (pr.k0 + j) * a.ldt] : 0.0;
    T2[i][j] = (i <= j && j < b2) ? a.Tm[i + (pr.k0 + b1 + j) * a.ldt] : 0.0;
  }
  __syncthreads();
  // M = G T_2, then T_12 = -T_1 M.
  for (int e = t; e < 1024; e += 256) {
    const int i = e / 32, j = e % 32;
    double m = 0.0;
    for (int l = 0; l <= j; ++l) m += G[i][l] * T2[l][j];
    M[i][j] = m;
  }
  __syncthreads();
  // Only the pair's own b1 + b2 columns of Tp: a narrower pair's neighbour
  // starts right after them.
  double* To = a.Tp + pr.k0 * a.ldt;
  for (int e = t; e < 64 * (b1 + b2); e += 256) {
    const int i = e % 64, j = e / 64;
    double v = 0.0;
    if (i < b1 && j < b1) {
      v = T1[i][j];
    } else if (i < b1 && j >= b1 && j < b1 + b2) {
      double s = 0.0;
      for (int l = i; l < b1; ++l) s += T1[i][l] * M[l][j - b1];
      v = -s;
    } else if (i >= b1 && i < b1 + b2 && j >= b1 && j < b1 + b2) {
      v = T2[i - b1][j - b1];
    }
    To[i + (int64_t)j * a.ldt] = v;
  }
  // V_2 is zero above its first row.
  double* V2 = a.V + (pr.k0 + b1) * a.ldv + pr.k0;
  for (int e = t; e < b1 * b2; e += 256) V2[e % b1 + (int64_t)(e / b1) * a.ldv] = 0.0;
}

}  // namespace

hipError_t launch_orgqr_pairs(const PairArgs& a, int npairs, hipStream_t s) {
  if (npairs <= 0) return hipSuccess;
  if (a.nsplit < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pair_gram_kernel, dim3((unsigned)npairs, (unsigned)a.nsplit), dim3(256),
                     0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pair_t_kernel, dim3((unsigned)npairs), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rrf
