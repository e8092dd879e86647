// Panel Householder QR with T factor (Alg. 2, geqrt step).
//
// Factors the sampled panel Y (m x b, b <= 64) column by column with LAPACK
// dlarfg / geqr2 semantics and builds the compact WY factor T (Eq. (4)) on the
// fly by the forward columnwise recursion T[:j, j] = -tau_j T[:j, :j] V^T v_j.
//
// Layout: a cooperative grid of G workgroups of 256 threads.  Thread t owns
// column k = t % BP and row group g = t / BP; workgroup w owns rows
// [w RW, (w + 1) RW) with RW = (256 / BP) * RPT, and thread (k, g) keeps the
// RPT rows w RW + g + (256 / BP) q of column k in registers for the whole
// factorisation.  Column j is broadcast through LDS.
//
// One grid-wide reduction per column.  With x the current column j below the
// diagonal, every thread contributes the partial dot of its own column with x
// over rows > j; together with row j of every column (held by workgroup 0)
// this gives, in one reduction,
//   ||x||^2            (the dlarfg norm),
//   v_j^T y_k, k > j   (the rank-1 update of the trailing columns), and
//   v_k^T v_j, k < j   (the new column of T),
// because v_j = [1; x / (alpha - beta)].  Every workgroup sums the partials
// in the same order, so all derive identical scalars (deterministic, no
// floating-point atomics).
//
// The panel is gathered beforehand into a zero-padded binary64 buffer (the
// sum of the update's column-split partials); the factorisation runs in
// binary64 (registers, reductions, V, T, tau), so the reflectors are
// orthogonal to binary64 precision even for float data.
//
// Requires 256 / BP * RPT >= BP so that rows 0 .. b-1 sit in workgroup 0.

#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr unsigned kSpinLimit = 1u << 22;

// Sense-reversing grid barrier (all G workgroups are co-resident: the kernel
// is launched cooperatively).  Memory ordering: the partials are written by
// wave 0 of each workgroup before the barrier; thread 0's agent-scope
// acquire-release arrival publishes them (it writes back this XCD's L2 and
// waits for wave 0's stores); after the barrier every wave issues an
// agent-scope acquire fence before it reads other workgroups' partials.
// The wait is bounded: after kSpinLimit polls it records an error and every
// later barrier returns at once, so the kernel always drains.
__device__ void grid_barrier(unsigned* bar, int G, DevState* st) {
  __syncthreads();
  if (threadIdx.x == 0) {
    if (__hip_atomic_load(&st->barrier_err, __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_AGENT) == 0) {
      const unsigned gen = __hip_atomic_load(&bar[1], __ATOMIC_ACQUIRE,
                                             __HIP_MEMORY_SCOPE_AGENT);
      const unsigned arrived = __hip_atomic_fetch_add(
          &bar[0], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      if (arrived == (unsigned)G - 1u) {
        __hip_atomic_store(&bar[0], 0u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&bar[1], gen + 1u, __ATOMIC_RELEASE,
                           __HIP_MEMORY_SCOPE_AGENT);
      } else {
        unsigned spins = 0;
        while (__hip_atomic_load(&bar[1], __ATOMIC_ACQUIRE,
                                 __HIP_MEMORY_SCOPE_AGENT) == gen) {
          __builtin_amdgcn_s_sleep(1);
          if (++spins > kSpinLimit ||
              __hip_atomic_load(&st->barrier_err, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT) != 0) {
            __hip_atomic_store(&st->barrier_err, 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
      }
    }
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

template <int BP, int RPT>
__global__ __launch_bounds__(kPanelThreads) void panel_kernel(PanelArgs a) {
  constexpr int GR = kPanelThreads / BP;
  constexpr int RW = GR * RPT;
  static_assert(RW >= BP, "rows 0..b-1 must sit in workgroup 0");
  __shared__ double xs[RW];
  __shared__ double rowj_s[BP];
  __shared__ double red_l[GR][BP];
  __shared__ double tot[BP], rj[BP];
  __shared__ double Tl[BP][BP + 1];

  const int t = threadIdx.x;
  const int k = t % BP, g = t / BP;
  const int w = blockIdx.x;
  const int64_t base = (int64_t)w * RW;
  const int b = a.b;

  // The gathered panel has G * RW rows and BP columns, zero outside (m, b),
  // so the RPT loads are unconditional and all in flight together.
  double col[RPT];
  {
    const double* Yk = a.Y + base + g + (int64_t)k * a.ldy;
#pragma unroll
    for (int q = 0; q < RPT; ++q) col[q] = Yk[GR * q];
  }

  for (int j = 0; j < b; ++j) {
    const int par = j & 1;
    // 1. Broadcast column j (rows of this workgroup) and row j.
    if (k == j) {
#pragma unroll
      for (int q = 0; q < RPT; ++q) xs[g + GR * q] = col[q];
    }
#pragma unroll
    for (int q = 0; q < RPT; ++q)
      if (base + g + GR * q == j) rowj_s[k] = col[q];
    __syncthreads();
    // 2. Partial dot of this thread's column with x over rows > j.
    double d = 0.0;
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const int64_t r = base + g + GR * q;
      if (r > j && r < a.m) d += col[q] * xs[g + GR * q];
    }
    red_l[g][k] = d;
    __syncthreads();
    // 3. Workgroup partial to global memory.
    if (t < BP) {
      double s = 0.0;
      for (int gg = 0; gg < GR; ++gg) s += red_l[gg][t];
      a.red[((int64_t)par * a.G + w) * BP + t] = s;
      if (w == 0) a.rowj[par * BP + t] = rowj_s[t];
    }
    grid_barrier(a.bar, a.G, a.st);
    // 4. Every workgroup sums all partials in the same fixed order.
    {
      const int kk = t % BP, sub = t / BP;
      const double* rp = a.red + (int64_t)par * a.G * BP + kk;
      double s = 0.0;
      for (int w0 = sub; w0 < a.G; w0 += 8 * GR) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int ww = w0 + u * GR;
          v[u] = ww < a.G ? rp[(int64_t)ww * BP] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
      }
      red_l[sub][kk] = s;
    }
    __syncthreads();
    if (t < BP) {
      double s = 0.0;
      for (int gg = 0; gg < GR; ++gg) s += red_l[gg][t];
      tot[t] = s;
      rj[t] = a.rowj[par * BP + t];
    }
    __syncthreads();
    // 5. dlarfg scalars (identical in every workgroup).
    const double alpha = rj[j];
    const double xi2 = tot[j];
    double tau_j = 0.0, scale = 0.0;
    if (xi2 != 0.0) {
      const double nrm = sqrt(alpha * alpha + xi2);
      const double beta = (alpha >= 0.0) ? -nrm : nrm;
      tau_j = (beta - alpha) / beta;
      scale = 1.0 / (alpha - beta);
    }
    // 6. v_j = x * scale below the diagonal; trailing columns
    //    y_k -= tau_j (v_j^T y_k) v_j with v_j^T y_k = y_k[j] + scale * dot_k.
    if (k == j) {
#pragma unroll
      for (int q = 0; q < RPT; ++q) {
        const int64_t r = base + g + GR * q;
        if (r > j) col[q] = col[q] * scale;
      }
    } else if (k > j && k < b) {
      const double f = tau_j * (rj[k] + scale * tot[k]);
#pragma unroll
      for (int q = 0; q < RPT; ++q) {
        const int64_t r = base + g + GR * q;
        if (r > j) col[q] = col[q] - f * (xs[g + GR * q] * scale);
      }
    }
    // 7. Column j of T (workgroup 0): v_p^T v_j = V[j, p] + scale * dot_p.
    if (w == 0) {
      if (t < j) {
        double acc = 0.0;
        for (int p = t; p < j; ++p) acc += Tl[t][p] * (rj[p] + scale * tot[p]);
        Tl[t][j] = -tau_j * acc;
      } else if (t == j) {
        Tl[j][j] = tau_j;
      }
    }
    __syncthreads();
  }

  // Outputs: V with explicit unit diagonal and zeros above / beyond b.
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    const int64_t r = base + g + GR * q;
    if (r < a.m) {
      double v = 0.0;
      if (k < b) v = (r > k) ? col[q] : (r == k ? 1.0 : 0.0);
      a.V[r + k * a.ldv] = v;
    }
  }
  if (w == 0) {
    for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
      const int i = idx % BP, jj = idx / BP;
      a.Tm[i + (int64_t)jj * a.ldt] = (jj < b && i <= jj) ? Tl[i][jj] : 0.0;
    }
    if (t < b) a.tau[t] = Tl[t][t];
  }
}

template <typename T>
__global__ void gather_panel_kernel(const T* P, int64_t ldp, int64_t split_stride,
                                    int nsplit, int64_t m, int b, int bp,
                                    int64_t rows_pad, double* Y, int64_t ldy) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows_pad) return;
  for (int k = blockIdx.y; k < bp; k += gridDim.y) {
    double v = 0.0;
    if (r < m && k < b)
      for (int s = 0; s < nsplit; ++s) v += (double)P[s * split_stride + r + k * ldp];
    Y[r + k * ldy] = v;
  }
}

template <int BP, int RPT>
hipError_t panel_go(const PanelArgs& a, hipStream_t s) {
  auto fn = panel_kernel<BP, RPT>;
  int occ = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      &occ, reinterpret_cast<const void*>(fn), kPanelThreads, 0);
  if (e != hipSuccess) return e;
  int dev = 0, cus = 0;
  hipGetDevice(&dev);
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (occ < 1 || a.G > occ * cus) return hipErrorCooperativeLaunchTooLarge;
  PanelArgs arg = a;
  void* params[] = {&arg};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(fn),
                                    dim3(a.G), dim3(kPanelThreads), params, 0, s);
}

template <int BP>
hipError_t panel_rpt(const PanelArgs& a, int rpt, hipStream_t s) {
  switch (rpt) {
    case 4: if constexpr ((kPanelThreads / BP) * 4 >= BP) return panel_go<BP, 4>(a, s); break;
    case 8: if constexpr ((kPanelThreads / BP) * 8 >= BP) return panel_go<BP, 8>(a, s); break;
    case 16: return panel_go<BP, 16>(a, s);
    case 32: return panel_go<BP, 32>(a, s);
    case 64: return panel_go<BP, 64>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

bool panel_shape(int64_t m, int b, int num_cus, int target_wgs, PanelShape* out) {
  if (b < 1 || b > kMaxBlock || m < b) return false;
  const int bp = pad16(b);
  const int gr = kPanelThreads / bp;
  static const int rpts[] = {4, 8, 16, 32, 64};
  for (int rpt : rpts) {
    if (gr * rpt < bp) continue;
    const int64_t G = ceil_div(m, (int64_t)gr * rpt);
    if (G <= target_wgs || rpt == 64) {
      if (G > num_cus || G > kMaxPanelWGs) return false;
      out->bp = bp;
      out->rpt = rpt;
      out->G = (int)G;
      out->rows_pad = G * gr * rpt;
      return true;
    }
  }
  return false;
}

hipError_t launch_panel(const PanelArgs& a, const PanelShape& sh, hipStream_t s) {
  switch (sh.bp) {
    case 16: return panel_rpt<16>(a, sh.rpt, s);
    case 32: return panel_rpt<32>(a, sh.rpt, s);
    case 64: return panel_rpt<64>(a, sh.rpt, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_gather_panel(const T* P, int64_t ldp, int64_t split_stride,
                               int nsplit, int64_t m, int b, int bp,
                               int64_t rows_pad, double* Ysum, int64_t ldy,
                               hipStream_t s) {
  if (rows_pad <= 0) return hipSuccess;
  dim3 grid((unsigned)ceil_div(rows_pad, 256), (unsigned)bp);
  hipLaunchKernelGGL((gather_panel_kernel<T>), grid, dim3(256), 0, s, P, ldp,
                     split_stride, nsplit, m, b, bp, rows_pad, Ysum, ldy);
  return hipGetLastError();
}

template hipError_t launch_gather_panel<float>(const float*, int64_t, int64_t, int, int64_t, int, int, int64_t, double*, int64_t, hipStream_t);
template hipError_t launch_gather_panel<double>(const double*, int64_t, int64_t, int, int64_t, int, int, int64_t, double*, int64_t, hipStream_t);

}  // namespace rrf
