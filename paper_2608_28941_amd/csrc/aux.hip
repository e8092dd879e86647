// Small kernels: residual-norm finalisation and stop test (Alg. 2 E update
// and loop condition), identity fill for the explicit Q, copies.

#include "finalize_body.h"
#include "rrf_internal.h"

namespace rrf {
namespace {

// The one-workgroup finalisation (finalize_body.h) from plain partials.
__global__ __launch_bounds__(256) void finalize_kernel(const double* np, FinalizeArgs f) {
  finalize_plain(np, f);
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
                           DevState* mirror, double* trace_trail, double* trace_sub, int block,
                           int64_t k_after, int64_t k_cap, int mode,
                           double tol, int init, hipStream_t s) {
  FinalizeArgs f{};
  f.nparts = nparts; f.st = st; f.mirror = mirror; f.tt = trace_trail; f.ts = trace_sub; f.block = block;
  f.k_after = k_after; f.k_cap = k_cap; f.mode = mode; f.tol = tol; f.init = init;
  hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(256), 0, s, normpart, f);
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
