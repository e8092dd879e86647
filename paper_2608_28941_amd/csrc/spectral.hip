// Spectral-norm estimate of the rows not yet in B (the alternative stopping
// test of Sec. 3, proposed as future work in the conclusion), and the scaled
// identity that power iterations use as their W factor.
//
// With Bt the trailing rows after a block and Y = Bt Omega' the sample of
// the next sketch block (first min(b, 64) columns), Z = Bt^T Y, the estimate
// is the largest eigenvalue of the pencil (Z^T Z, Y^T Y):
//   max over x in span(Y) of ||Bt^T x||^2 / ||x||^2
// (one step of randomized subspace iteration; a lower bound of ||Bt||_2^2,
// exact when rank(Bt) <= the block width).  Y and Z arrive from the gather
// and the reduce kernel (Z as split partials); here:
//   spec_gram_kernel   partial Gram matrices G_Y = Y^T Y and G_Z = Z^T Z
//                      over row ranges, f64 MFMA, values scaled by ||A||_F
//                      (1/sqrt(E0) for Y, 1/E0 for Z) so nothing overflows;
//   spec_finish_kernel one workgroup: sums the partials in a fixed order,
//                      L = chol(G_Y + delta I), M = L^-1 G_Z L^-T, and the
//                      largest eigenvalue of M by repeated squaring, then a
//                      Rayleigh quotient; writes E_spec (times E0) to the run
//                      state and the trace.

#include "mfma.h"
#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr int kSpecRows = 64;   // rows per staged chunk

template <typename T>
__global__ __launch_bounds__(256) void spec_gram_kernel(SpecGramArgs<T> a) {
  __shared__ double X[kSpecRows][65];
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6, l16 = lane >> 4, m16 = lane & 15;
  const int w = (int)blockIdx.x;
  const bool isY = w < a.gy;
  const int64_t rows = isY ? a.my : a.nz;
  const int64_t rpw = isY ? a.rows_per_wg_y : a.rows_per_wg_z;
  const int64_t r_begin = (int64_t)(isY ? w : w - a.gy) * rpw;
  const int64_t r_end = min(rows, r_begin + rpw);
  const double E0 = a.st->E0;
  const double sc = E0 > 0.0 ? (isY ? 1.0 / sqrt(E0) : 1.0 / E0) : 0.0;

  d4_t acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = d4_t{0.0, 0.0, 0.0, 0.0};
  for (int64_t r0 = r_begin; r0 < r_end; r0 += kSpecRows) {
    __syncthreads();
    if (isY) {
      // Column-major Y: thread t loads row t % 64 of columns t / 64 + 4 i.
      const int rr = t % 64, c0 = t / 64;
      const int64_t r = r0 + rr;
      const bool ok = r < r_end;
      double v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int c = c0 + 4 * i;
        v[i] = (ok && c < a.bp) ? a.Y[r + (int64_t)c * a.ldy] : 0.0;
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) X[rr][c0 + 4 * i] = sc * v[i];
    } else {
      // Row-major Z partials Z_s[row * bp + c]: thread t loads column t % 64
      // of rows t / 64 + 4 i, summed over the splits in split order.
      const int cc = t % 64, q0 = t / 64;
#pragma unroll 4
      for (int i = 0; i < 16; ++i) {
        const int rr = q0 + 4 * i;
        const int64_t r = r0 + rr;
        double z = 0.0;
        if (r < r_end && cc < a.bp)
          for (int s = 0; s < a.nsplit; ++s)
            z += (double)a.Z[(int64_t)s * a.split_stride + r * a.bp + cc];
        X[rr][cc] = sc * z;
      }
    }
    __syncthreads();
    // G[16 pt + m][16 ct + n] += sum_r X[r][16 pt + m] X[r][16 ct + n],
    // pt = this wavefront, over the chunk's rows in K steps of 4.
#pragma unroll 4
    for (int s4 = 0; s4 < kSpecRows / 4; ++s4) {
      const double av = X[4 * s4 + l16][16 * wv + m16];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
        acc[ct] = Mfma<double>::op(av, X[4 * s4 + l16][16 * ct + m16], acc[ct]);
    }
  }
  // Lane holds G[16 wv + l16 + 4 i][16 ct + m16].
  double* out = a.part + (int64_t)w * 4096;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int i = 0; i < 4; ++i) out[(16 * wv + l16 + 4 * i) * 64 + 16 * ct + m16] = acc[ct][i];
}

// Packed lower triangle: row i, column j <= i.
__device__ __forceinline__ int tri(int i, int j) { return i * (i + 1) / 2 + j; }

__global__ __launch_bounds__(256) void spec_finish_kernel(SpecFinishArgs a) {
  __shared__ double G[64][65];     // G_Z, then G_Y / L work, then X, M powers
  __shared__ double Lp[64 * 65 / 2];
  __shared__ double red[256];
  __shared__ double scal[4];
  const int t = threadIdx.x;
  const int c = t;                 // the column threads c < 64 own

  // Sum the partials of one Gram matrix (gz or gy workgroups from w0) into G
  // in a fixed order.
  auto sum_into_G = [&](int w0, int nw) {
    for (int e = t; e < 4096; e += 256) {
      double s = 0.0;
      for (int w = 0; w < nw; ++w) s += a.part[(int64_t)(w0 + w) * 4096 + e];
      G[e / 64][e % 64] = s;
    }
    __syncthreads();
  };
  // G_Z column c into registers.
  sum_into_G(a.gy, a.gz);
  double x[64];
  if (c < 64) {
#pragma unroll
    for (int i = 0; i < 64; ++i) x[i] = G[i][c];
  }
  __syncthreads();
  sum_into_G(0, a.gy);
  // delta = 64 u max diag(G_Y); an all-zero G_Y means Y = 0: estimate 0.
  if (t == 0) {
    double dmax = 0.0;
    for (int i = 0; i < 64; ++i) dmax = fmax(dmax, G[i][i]);
    scal[0] = dmax;
  }
  __syncthreads();
  const double dmax = scal[0];
  if (!(dmax > 0.0)) {
    if (t == 0) {
      a.st->E_spec = 0.0;
      if (a.block >= 0) a.trace[a.block] = 0.0;
    }
    return;
  }
  const double delta = 64.0 * 1.1102230246251565e-16 * dmax;
  // Cholesky of G_Y + delta I by one wavefront (thread i owns row i):
  // column j: s_i = G[i][j] - sum_{k<j} L[i][k] L[j][k]; L[j][j] = sqrt(s_j);
  // L[i][j] = s_i / L[j][j] for i > j.  Results go to the packed Lp; the
  // wavefront's LDS accesses complete in order.
  if (t < 64) {
    const int i = t;
    for (int j = 0; j < 64; ++j) {
      double sj = 0.0;
      if (i >= j) {
        sj = G[i][j] + (i == j ? delta : 0.0);
        for (int k = 0; k < j; ++k) sj -= Lp[tri(i, k)] * Lp[tri(j, k)];
      }
      if (i == j) Lp[tri(j, j)] = sqrt(fmax(sj, delta));
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      if (i > j) Lp[tri(i, j)] = sj / Lp[tri(j, j)];
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
  }
  __syncthreads();
  // X = L^-1 G_Z, column c by forward substitution in registers.
  if (c < 64) {
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      double s = x[j];
#pragma unroll
      for (int k = 0; k < j; ++k) s -= Lp[tri(j, k)] * x[k];
      x[j] = s / Lp[tri(j, j)];
    }
#pragma unroll
    for (int i = 0; i < 64; ++i) G[i][c] = x[i];
  }
  __syncthreads();
  // M = X L^-T; M is symmetric, so its column c is L^-1 (row c of X)^T.
  if (c < 64) {
#pragma unroll
    for (int k = 0; k < 64; ++k) x[k] = G[c][k];
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      double s = x[j];
#pragma unroll
      for (int k = 0; k < j; ++k) s -= Lp[tri(j, k)] * x[k];
      x[j] = s / Lp[tri(j, j)];
    }
  }
  __syncthreads();
  if (c < 64) {
#pragma unroll
    for (int i = 0; i < 64; ++i) G[i][c] = x[i];   // M, kept in x for later
  }
  __syncthreads();
  // Repeated squaring P <- P^2 / trace(P^2) (P stays positive semidefinite),
  // 12 times: P ~ M^4096, whose columns lie along the top eigenvector.
  // Thread t computes the entries (i, j) with i = t / 4 and j = 16 (t % 4) + q.
  for (int it = 0; it < 12; ++it) {
    const int i = t / 4, j0 = 16 * (t % 4);
    double o[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) o[q] = 0.0;
    for (int k = 0; k < 64; ++k) {
      const double gik = G[i][k];
#pragma unroll
      for (int q = 0; q < 16; ++q) o[q] += gik * G[k][j0 + q];
    }
    double tr = 0.0;
    if (j0 <= i && i < j0 + 16) tr = o[i - j0];
    red[t] = tr;
    __syncthreads();
    if (t == 0) {
      double s = 0.0;
      for (int u = 0; u < 256; ++u) s += red[u];
      scal[1] = s;
    }
    __syncthreads();
    const double inv = scal[1] > 0.0 ? 1.0 / scal[1] : 0.0;
#pragma unroll
    for (int q = 0; q < 16; ++q) G[i][j0 + q] = o[q] * inv;
    __syncthreads();
  }
  // v = the column of P with the largest diagonal entry; estimate
  // v^T M v / v^T v with M's columns still in the registers x.
  if (t == 0) {
    int jb = 0;
    for (int j = 1; j < 64; ++j)
      if (G[j][j] > G[jb][jb]) jb = j;
    scal[2] = (double)jb;
  }
  __syncthreads();
  const int jb = (int)scal[2];
  double num = 0.0, den = 0.0;
  if (c < 64) {
    const double vc = G[c][jb];
    double mv = 0.0;
#pragma unroll
    for (int i = 0; i < 64; ++i) mv += x[i] * G[i][jb];
    num = vc * mv;
    den = vc * vc;
  }
  red[t] = num;
  __syncthreads();
  if (t == 0) {
    double s = 0.0;
    for (int u = 0; u < 64; ++u) s += red[u];
    scal[3] = s;
  }
  __syncthreads();
  red[t] = den;
  __syncthreads();
  if (t == 0) {
    double s = 0.0;
    for (int u = 0; u < 64; ++u) s += red[u];
    const double lam = s > 0.0 ? scal[3] / s : 0.0;
    const double E = fmax(lam, 0.0) * a.st->E0;
    a.st->E_spec = E;
    if (a.block >= 0) a.trace[a.block] = E;
  }
}

__global__ void scaled_identity_kernel(double* Tm, int64_t ldt, const DevState* st) {
  const int i = threadIdx.x % 64, j = threadIdx.x / 64;
  const double E0 = st->E0;
  const double d = E0 > 0.0 ? 1.0 / E0 : 0.0;
  for (int jj = j; jj < 64; jj += 4) Tm[i + jj * ldt] = (i == jj) ? d : 0.0;
}

}  // namespace

template <typename T>
hipError_t launch_spec_gram(SpecGramArgs<T>* ap, hipStream_t s) {
  SpecGramArgs<T>& a = *ap;
  if (a.bp < 1 || a.bp > 64) return hipErrorInvalidValue;
  a.gy = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxSpecWGs / 2, ceil_div(a.my, 256)));
  a.rows_per_wg_y = round_up(ceil_div(std::max<int64_t>(a.my, 1), a.gy), kSpecRows);
  a.gy = (int)std::max<int64_t>(1, ceil_div(std::max<int64_t>(a.my, 1), a.rows_per_wg_y));
  a.gz = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxSpecWGs / 2, ceil_div(a.nz, 256)));
  a.rows_per_wg_z = round_up(ceil_div(std::max<int64_t>(a.nz, 1), a.gz), kSpecRows);
  a.gz = (int)std::max<int64_t>(1, ceil_div(std::max<int64_t>(a.nz, 1), a.rows_per_wg_z));
  hipLaunchKernelGGL((spec_gram_kernel<T>), dim3((unsigned)(a.gy + a.gz)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_spec_finish(const SpecFinishArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(spec_finish_kernel, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_scaled_identity(double* Tm, int64_t ldt, const DevState* st, hipStream_t s) {
  hipLaunchKernelGGL(scaled_identity_kernel, dim3(1), dim3(256), 0, s, Tm, ldt, st);
  return hipGetLastError();
}

template hipError_t launch_spec_gram<float>(SpecGramArgs<float>*, hipStream_t);
template hipError_t launch_spec_gram<double>(SpecGramArgs<double>*, hipStream_t);

}  // namespace rrf
