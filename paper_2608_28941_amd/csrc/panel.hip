// Panel Householder QR with T factor (Alg. 2, geqrt step): the panel kernel
// (a grid of mutually waiting workgroups; the workgroup body is in
// panel_body.h), the gather of the sampled panel and the launchers.

#include "gather_body.h"
#include "panel_body.h"

namespace rrf {
namespace {

template <int BP, int RPT>
__global__ __launch_bounds__(kPanelThreads) void panel_kernel(PanelArgs a) {
  panel_body<BP, RPT>(a, (int)blockIdx.x);
}

template <typename T>
__global__ void gather_panel_kernel(const T* P, int64_t ldp, int64_t split_stride,
                                    int nsplit, int64_t m, int b, int bp,
                                    int64_t rows_pad, double* Y, int64_t ldy) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows_pad) return;
  const GatherArgs<T> g{P, ldp, split_stride, nsplit, m, b, bp, rows_pad, Y, ldy};
  for (int k = blockIdx.y; k < bp; k += gridDim.y) gather_entry(g, r, k);
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
  return launch_resident(reinterpret_cast<const void*>(fn), dim3(a.G),
                         dim3(kPanelThreads), params, s);
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
