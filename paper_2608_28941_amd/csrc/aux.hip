// Small kernels: residual-norm finalisation and stop test (Alg. 2 E update
// and loop condition), identity fill for the explicit Q, copies.

#include "rrf_internal.h"

namespace rrf {
namespace {

// Sums the per-workgroup norm partials in a fixed order (deterministic) and
// applies the stop test.  init: E0 = ||A||_F^2, sigma^2 = tol^2 E0.
// Otherwise: E_trail = ||B[k:m, :]||^2 directly, E_sub -= ||B_i||^2 (the
// paper's running difference, clamped at 0); in spectral mode (2) the
// estimate the spectral kernels left in the run state.  At the end of a block (block
// >= 0: the trace index) the stop test runs: stop iff E <= sigma^2 or the
// rank cap is reached (Sec. 4: the loop ends after at most min(m, n) / b
// blocks); inside a block (block < 0, the first 64 columns of a wider
// block) only errors stop.  A NaN norm fails "E > sigma^2" and would stop
// silently, so non-finite norms are flagged.
__global__ __launch_bounds__(256) void finalize_kernel(
    const double* np, int nparts, DevState* st, double* tt, double* ts,
    int block, int64_t k_after, int64_t k_cap, int mode, double tol, int init) {
  __shared__ double sb[256], stl[256];
  double a = 0.0, c = 0.0;
  for (int i = threadIdx.x; i < nparts; i += 256) {
    a += np[2 * i + 0];
    c += np[2 * i + 1];
  }
  sb[threadIdx.x] = a;
  stl[threadIdx.x] = c;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (threadIdx.x < h) {
      sb[threadIdx.x] += sb[threadIdx.x + h];
      stl[threadIdx.x] += stl[threadIdx.x + h];
    }
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  const double blk = sb[0], trail = stl[0];
  if (init) {
    const double E0 = blk + trail;
    st->E0 = E0;
    st->nonfinite = !isfinite(E0);
    st->sigma2 = (tol * tol) * E0;
    st->E_trail = E0;
    st->E_sub = E0;
    st->E_spec = E0;
    st->stop = st->nonfinite || !(E0 > st->sigma2) || k_cap == 0;
    st->barrier_err = 0;
  } else {
    double es = st->E_sub - blk;
    if (es < 0.0) es = 0.0;
    st->E_sub = es;
    st->E_trail = trail;
    if (!isfinite(trail)) st->nonfinite = 1;
    if (block >= 0) {
      tt[block] = trail;
      ts[block] = es;
      const double E = mode == 0 ? trail : (mode == 1 ? es : st->E_spec);
      st->stop = st->nonfinite || st->barrier_err || !(E > st->sigma2) ||
                 k_after >= k_cap;
    } else {
      st->stop = st->nonfinite || st->barrier_err;
    }
  }
}

template <typename T>
__global__ void fill_identity_kernel(T* Q, int64_t ldq, int64_t m, int64_t k) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= m) return;
  for (int64_t c = blockIdx.y; c < k; c += gridDim.y)
    Q[r + c * ldq] = (r == c) ? T(1) : T(0);
}

template <typename T>
__global__ void copy_kernel(const T* src, int64_t lds, T* dst, int64_t ldd,
                            int64_t rows, int64_t cols) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  for (int64_t c = blockIdx.y; c < cols; c += gridDim.y)
    dst[r + c * ldd] = src[r + c * lds];
}

template <typename Ts, typename Td>
__global__ void convert_kernel(const Ts* src, int64_t lds, Td* dst, int64_t ldd,
                               int64_t rows, int64_t cols) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  for (int64_t c = blockIdx.y; c < cols; c += gridDim.y)
    dst[r + c * ldd] = (Td)src[r + c * lds];
}

}  // namespace

hipError_t launch_finalize(const double* normpart, int nparts, DevState* st,
                           double* trace_trail, double* trace_sub, int block,
                           int64_t k_after, int64_t k_cap, int mode,
                           double tol, int init, hipStream_t s) {
  hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(256), 0, s, normpart,
                     nparts, st, trace_trail, trace_sub, block, k_after, k_cap,
                     mode, tol, init);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_fill_identity(T* Q, int64_t ldq, int64_t m, int64_t k,
                                hipStream_t s) {
  if (m <= 0 || k <= 0) return hipSuccess;
  dim3 grid((unsigned)ceil_div(m, 256), (unsigned)(k < 4096 ? k : 4096));
  hipLaunchKernelGGL(fill_identity_kernel<T>, grid, dim3(256), 0, s, Q, ldq, m, k);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_copy(const T* src, int64_t lds, T* dst, int64_t ldd,
                       int64_t rows, int64_t cols, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  dim3 grid((unsigned)ceil_div(rows, 256), (unsigned)(cols < 4096 ? cols : 4096));
  hipLaunchKernelGGL(copy_kernel<T>, grid, dim3(256), 0, s, src, lds, dst, ldd,
                     rows, cols);
  return hipGetLastError();
}

template <typename Ts, typename Td>
hipError_t launch_convert(const Ts* src, int64_t lds, Td* dst, int64_t ldd,
                          int64_t rows, int64_t cols, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  dim3 grid((unsigned)ceil_div(rows, 256), (unsigned)(cols < 4096 ? cols : 4096));
  hipLaunchKernelGGL((convert_kernel<Ts, Td>), grid, dim3(256), 0, s, src, lds,
                     dst, ldd, rows, cols);
  return hipGetLastError();
}

template hipError_t launch_fill_identity<float>(float*, int64_t, int64_t, int64_t, hipStream_t);
template hipError_t launch_fill_identity<double>(double*, int64_t, int64_t, int64_t, hipStream_t);
template hipError_t launch_copy<float>(const float*, int64_t, float*, int64_t, int64_t, int64_t, hipStream_t);
template hipError_t launch_copy<double>(const double*, int64_t, double*, int64_t, int64_t, int64_t, hipStream_t);
template hipError_t launch_convert<double, float>(const double*, int64_t, float*, int64_t, int64_t, int64_t, hipStream_t);
template hipError_t launch_convert<float, double>(const float*, int64_t, double*, int64_t, int64_t, int64_t, hipStream_t);

}  // namespace rrf
