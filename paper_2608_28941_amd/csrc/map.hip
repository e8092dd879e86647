// GaLore subspace-consistency map (Sec. 7): a low-rank optimizer state M
// (r_old x n) expressed in the basis Q_old is carried to the next basis as
// out = Q_new^T (Q_old M) = C M with C = Q_new^T Q_old (r_new x r_old).
//
// Three launches, MFMA 16x16x4 in the plan's dtype:
//   map_tn_kernel   C_s = Q_new[rows of split s]^T Q_old[rows of split s]
//                   (the reduction over the m rows is split so that the small
//                   r_new x r_old output fills the device);
//   map_sum_kernel  C = sum_s C_s in a fixed order (deterministic);
//   map_nn_kernel   out = C M.
// Each workgroup computes a 64 x 64 output tile from operands staged in LDS
// in chunks of 32 along the summation index.  Both GEMMs run in the
// transposed frame (the MFMA's output rows index the output's columns), so
// the 16 lanes of an output column write 16 consecutive rows of the
// column-major result.

#include <type_traits>

#include "mfma.h"
#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr int kMapTile = 64;
constexpr int kMapK = 32;

// Cpart_s[i + j ldc] = sum over rows r of split s of A[r + i lda] B[r + j ldb],
// i < M, j < N; grid (ceil(M / 64), ceil(N / 64), splits).
template <typename T>
__global__ __launch_bounds__(256) void map_tn_kernel(const T* A, int64_t lda, const T* B,
                                                     int64_t ldb, int64_t M, int64_t N,
                                                     int64_t K, int64_t rows_per_split,
                                                     T* Cpart, int64_t ldc,
                                                     int64_t split_stride) {
  typedef typename Mfma<T>::acc_t acc_t;
  __shared__ T As[kMapK][kMapTile + 1];   // As[kk][ii] = A[r0 + kk][i0 + ii]
  __shared__ T Bs[kMapK][kMapTile + 1];   // Bs[kk][jj] = B[r0 + kk][j0 + jj]
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6, g = lane >> 4, m16 = lane & 15;
  const int64_t i0 = (int64_t)blockIdx.x * kMapTile, j0 = (int64_t)blockIdx.y * kMapTile;
  const int64_t r_begin = (int64_t)blockIdx.z * rows_per_split;
  const int64_t r_end = min(K, r_begin + rows_per_split);
  // Staging: thread t loads row t % 32 of columns t / 32 + 8 q (q < 8).
  const int sr = t % kMapK, sc = t / kMapK;
  acc_t acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = Mfma<T>::zero();
  T av[8], bv[8];
  auto load = [&](int64_t r0) {
    const int64_t r = r0 + sr;
    const bool rok = r < r_end;
    const int64_t rc = rok ? r : r_begin;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t i = i0 + sc + 8 * q, j = j0 + sc + 8 * q;
      const T a = A[rc + (i < M ? i : 0) * lda];
      const T b = B[rc + (j < N ? j : 0) * ldb];
      av[q] = (rok && i < M) ? a : T(0);
      bv[q] = (rok && j < N) ? b : T(0);
    }
  };
  if (r_begin < r_end) load(r_begin);
  for (int64_t r0 = r_begin; r0 < r_end; r0 += kMapK) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      As[sr][sc + 8 * q] = av[q];
      Bs[sr][sc + 8 * q] = bv[q];
    }
    __syncthreads();
    if (r0 + kMapK < r_end) load(r0 + kMapK);
    // D[jj][ii] = sum_r B[r][j0 + jj] A[r][i0 + ii]: this wavefront's jj
    // strip (16 wv ..) against the four ii tiles.
#pragma unroll
    for (int s4 = 0; s4 < kMapK / 4; ++s4) {
      const T a_op = Bs[4 * s4 + g][16 * wv + m16];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
        acc[ct] = Mfma<T>::op(a_op, As[4 * s4 + g][16 * ct + m16], acc[ct]);
    }
    __syncthreads();
  }
  // Lane (g, m16) item q holds C[i0 + 16 ct + m16][j0 + 16 wv + drow(g, q)].
  T* Cs = Cpart + (int64_t)blockIdx.z * split_stride;
  const int64_t i_base = i0 + m16;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int64_t i = i_base + 16 * ct;
    if (i >= M) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t j = j0 + 16 * wv + Mfma<T>::drow(g, q);
      if (j < N) Cs[i + j * ldc] = acc[ct][q];
    }
  }
}

// C[e] = sum_s Cpart_s[e], e < count, in split order.
template <typename T>
__global__ void map_sum_kernel(const T* Cpart, int nsplit, int64_t split_stride, T* C,
                               int64_t count) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= count) return;
  double s = 0.0;
  for (int q = 0; q < nsplit; ++q) s += (double)Cpart[(int64_t)q * split_stride + e];
  C[e] = (T)s;
}

// out[i + j ldo] = sum_k C[i + k ldc] Mm[k + j ldm], i < M, j < N, k < K;
// grid (ceil(M / 64), ceil(N / 64)).
template <typename T>
__global__ __launch_bounds__(256) void map_nn_kernel(const T* C, int64_t ldc, const T* Mm,
                                                     int64_t ldm, int64_t M, int64_t N,
                                                     int64_t K, T* out, int64_t ldo) {
  typedef typename Mfma<T>::acc_t acc_t;
  __shared__ T Cs[kMapK][kMapTile + 1];   // Cs[kk][ii] = C[i0 + ii][k0 + kk]
  __shared__ T Ms[kMapK][kMapTile + 1];   // Ms[kk][jj] = M[k0 + kk][j0 + jj]
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6, g = lane >> 4, m16 = lane & 15;
  const int64_t i0 = (int64_t)blockIdx.x * kMapTile, j0 = (int64_t)blockIdx.y * kMapTile;
  // C staging: thread t loads row t % 64 of C columns t / 64 + 4 q (q < 8);
  // M staging: row t % 32 of M columns t / 32 + 8 q.
  const int cr = t % 64, cc = t / 64;
  const int mr = t % kMapK, mc = t / kMapK;
  acc_t acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = Mfma<T>::zero();
  T cv[8], mv[8];
  auto load = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t i = i0 + cr, k = k0 + cc + 4 * q;
      const bool ok = i < M && k < K;
      const T c = C[(i < M ? i : 0) + (k < K ? k : 0) * ldc];
      cv[q] = ok ? c : T(0);
      const int64_t kk = k0 + mr, j = j0 + mc + 8 * q;
      const bool ok2 = kk < K && j < N;
      const T v = Mm[(kk < K ? kk : 0) + (j < N ? j : 0) * ldm];
      mv[q] = ok2 ? v : T(0);
    }
  };
  load(0);
  for (int64_t k0 = 0; k0 < K; k0 += kMapK) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      Cs[cc + 4 * q][cr] = cv[q];
      Ms[mr][mc + 8 * q] = mv[q];
    }
    __syncthreads();
    if (k0 + kMapK < K) load(k0 + kMapK);
    // D[jj][ii] = sum_k M[k][j0 + jj] C[i0 + ii][k].
#pragma unroll
    for (int s4 = 0; s4 < kMapK / 4; ++s4) {
      const T a_op = Ms[4 * s4 + g][16 * wv + m16];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
        acc[ct] = Mfma<T>::op(a_op, Cs[4 * s4 + g][16 * ct + m16], acc[ct]);
    }
    __syncthreads();
  }
  const int64_t i_base = i0 + m16;
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int64_t i = i_base + 16 * ct;
    if (i >= M) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t j = j0 + 16 * wv + Mfma<T>::drow(g, q);
      if (j < N) out[i + j * ldo] = acc[ct][q];
    }
  }
}

}  // namespace

int map_splits(int64_t r_new, int64_t r_old, int64_t m, int num_cus) {
  const int64_t tiles = ceil_div(r_new, kMapTile) * ceil_div(r_old, kMapTile);
  int64_t s = ceil_div(2 * (int64_t)num_cus, std::max<int64_t>(tiles, 1));
  s = std::min<int64_t>({s, kMaxMapSplits, std::max<int64_t>(1, m / 256)});
  return (int)std::max<int64_t>(s, 1);
}

template <typename T>
hipError_t launch_subspace_map(const T* Qnew, int64_t ldqn, int64_t r_new, const T* Qold,
                               int64_t ldqo, int64_t r_old, const T* M, int64_t ldm,
                               int64_t m, int64_t n, T* out, int64_t ldo, T* Cpart,
                               T* C, int nsplit, hipStream_t s) {
  const int64_t rows = round_up(ceil_div(m, nsplit), kMapK);
  const int ns = (int)ceil_div(m, rows);
  const int64_t stride = r_new * r_old;
  hipLaunchKernelGGL((map_tn_kernel<T>),
                     dim3((unsigned)ceil_div(r_new, kMapTile), (unsigned)ceil_div(r_old, kMapTile),
                          (unsigned)ns),
                     dim3(256), 0, s, Qnew, ldqn, Qold, ldqo, r_new, r_old, m, rows, Cpart,
                     r_new, stride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((map_sum_kernel<T>), dim3((unsigned)ceil_div(stride, 256)), dim3(256), 0,
                     s, Cpart, ns, stride, C, stride);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((map_nn_kernel<T>),
                     dim3((unsigned)ceil_div(r_new, kMapTile), (unsigned)ceil_div(n, kMapTile)),
                     dim3(256), 0, s, C, r_new, M, ldm, r_new, n, r_old, out, ldo);
  return hipGetLastError();
}

template hipError_t launch_subspace_map<float>(const float*, int64_t, int64_t, const float*,
                                               int64_t, int64_t, const float*, int64_t,
                                               int64_t, int64_t, float*, int64_t, float*,
                                               float*, int, hipStream_t);
template hipError_t launch_subspace_map<double>(const double*, int64_t, int64_t,
                                                const double*, int64_t, int64_t,
                                                const double*, int64_t, int64_t, int64_t,
                                                double*, int64_t, double*, double*, int,
                                                hipStream_t);

}  // namespace rrf
