// Look-ahead kernel: the one-GPU form of the paper's two-queue overlap
// (Sec. 5, Fig. 2(b)).  While the update of block i streams over B, the panel
// of block i + 1 is factored on a few compute units: the first G workgroups
// of the launch run the panel (panel_body), the others the update tiles
// (update_body).  Workgroups are dispatched in order, so the panel's
// workgroups are resident from the start; the update's workgroups never wait
// on anything, so the panel's grid-wide waits always complete.
//
// The panel's input is the sample of block i + 1 taken one update earlier
// and brought up to date with Q_i^T before this launch (see rrf_run).

#include "panel_body.h"
#include "update_body.h"

namespace rrf {
namespace {

template <typename T, int BP, int RPT>
__global__ __launch_bounds__(256, 2) void update_panel_kernel(UpdateArgs<T> ua,
                                                              PanelArgs pa,
                                                              unsigned nrb) {
  if ((int)blockIdx.x < pa.G) {
    panel_body<BP, RPT>(pa, (int)blockIdx.x);
    return;
  }
  const unsigned t = blockIdx.x - (unsigned)pa.G;
  update_body<T, BP, BP, true>(ua, t % nrb, t / nrb, nrb);
}

template <typename T, int BP, int RPT>
hipError_t up_go(const UpdateArgs<T>& ua, int nsplit, const PanelArgs& pa,
                 hipStream_t s) {
  const unsigned nrb = (unsigned)ceil_div(ua.mr, kUpdRows);
  const dim3 grid((unsigned)pa.G + nrb * (unsigned)nsplit);
  hipLaunchKernelGGL((update_panel_kernel<T, BP, RPT>), grid, dim3(256), 0, s,
                     ua, pa, nrb);
  return hipGetLastError();
}

template <typename T, int BP>
hipError_t up_rpt(const UpdateArgs<T>& ua, int nsplit, const PanelArgs& pa,
                  int rpt, hipStream_t s) {
  switch (rpt) {
    case 4: if constexpr ((kPanelThreads / BP) * 4 >= BP) return up_go<T, BP, 4>(ua, nsplit, pa, s); break;
    case 8: if constexpr ((kPanelThreads / BP) * 8 >= BP) return up_go<T, BP, 8>(ua, nsplit, pa, s); break;
    case 16: return up_go<T, BP, 16>(ua, nsplit, pa, s);
    case 32: return up_go<T, BP, 32>(ua, nsplit, pa, s);
    case 64: return up_go<T, BP, 64>(ua, nsplit, pa, s);
  }
  return hipErrorNotSupported;
}

template <typename T, int BP, int RPT>
int up_occ() {
  static const int occ = [] {
    int o = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &o, reinterpret_cast<const void*>(update_panel_kernel<T, BP, RPT>), 256, 0) != hipSuccess)
      o = 0;
    return o;
  }();
  return occ;
}

template <typename T, int BP>
int up_occ_rpt(int rpt) {
  switch (rpt) {
    case 4: if constexpr ((kPanelThreads / BP) * 4 >= BP) return up_occ<T, BP, 4>(); break;
    case 8: if constexpr ((kPanelThreads / BP) * 8 >= BP) return up_occ<T, BP, 8>(); break;
    case 16: return up_occ<T, BP, 16>();
    case 32: return up_occ<T, BP, 32>();
    case 64: return up_occ<T, BP, 64>();
  }
  return 0;
}

}  // namespace

template <typename T>
int update_panel_occupancy(const PanelShape& sh) {
  switch (sh.bp) {
    case 16: return up_occ_rpt<T, 16>(sh.rpt);
    case 32: return up_occ_rpt<T, 32>(sh.rpt);
    case 64: return up_occ_rpt<T, 64>(sh.rpt);
  }
  return 0;
}

template int update_panel_occupancy<float>(const PanelShape&);
template int update_panel_occupancy<double>(const PanelShape&);

bool update_panel_supported(int bp, int qp, const PanelShape& sh) {
  return bp > 0 && bp == qp && bp == sh.bp;
}

template <typename T>
hipError_t launch_update_panel(const UpdateArgs<T>& ua, int nsplit,
                               const PanelArgs& pa, const PanelShape& sh,
                               hipStream_t s) {
  if (!update_panel_supported(ua.bp, ua.qp, sh) || !ua.dst || ua.mr <= 0 || ua.n <= 0)
    return hipErrorNotSupported;
  // 32-bit buffer offsets, as in launch_update.
  const int64_t ld = std::max(ua.lds, ua.ldd);
  if (ld < ua.mr || (int64_t)kUpdChunk * ld * (int64_t)sizeof(T) > ((int64_t)1 << 30))
    return hipErrorInvalidValue;
  switch (sh.bp) {
    case 16: return up_rpt<T, 16>(ua, nsplit, pa, sh.rpt, s);
    case 32: return up_rpt<T, 32>(ua, nsplit, pa, sh.rpt, s);
    case 64: return up_rpt<T, 64>(ua, nsplit, pa, sh.rpt, s);
  }
  return hipErrorNotSupported;
}

template hipError_t launch_update_panel<float>(const UpdateArgs<float>&, int, const PanelArgs&, const PanelShape&, hipStream_t);
template hipError_t launch_update_panel<double>(const UpdateArgs<double>&, int, const PanelArgs&, const PanelShape&, hipStream_t);

}  // namespace rrf
