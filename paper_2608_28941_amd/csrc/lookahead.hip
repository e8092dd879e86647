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
//
// Block 0 has no update to hide its panel in, but its panel and the first
// look-ahead sample S_1 = A Omega_1 are independent: the same launch shape
// runs them together (SAMPLE_ONLY: the non-panel workgroups only sample,
// update_body with no reflectors and no store).

#include "panel_body.h"
#include "update_body.h"

namespace rrf {
namespace {

template <typename T, int BP, int RPT, bool SAMPLE_ONLY>
__global__ __launch_bounds__(256, 2) void update_panel_kernel(UpdateArgs<T> ua,
                                                              PanelArgs pa,
                                                              unsigned nrb) {
  if ((int)blockIdx.x < pa.G) {
    panel_body<BP, RPT>(pa, (int)blockIdx.x);
    return;
  }
  const unsigned t = blockIdx.x - (unsigned)pa.G;
  if constexpr (SAMPLE_ONLY)
    update_body<T, 0, BP, false>(ua, t % nrb, t / nrb, nrb);
  else
    update_body<T, BP, BP, true>(ua, t % nrb, t / nrb, nrb);
}

// The sample-only form is built for 64-column panels, the width that takes
// the look-ahead.
template <int BP, bool SAMPLE_ONLY>
constexpr bool up_built() { return !SAMPLE_ONLY || BP == 64; }

template <typename T, int BP, int RPT, bool SO>
hipError_t up_go(const UpdateArgs<T>& ua, int nsplit, const PanelArgs& pa,
                 hipStream_t s) {
  const unsigned nrb = (unsigned)ceil_div(ua.mr, kUpdRows);
  const dim3 grid((unsigned)pa.G + nrb * (unsigned)nsplit);
  hipLaunchKernelGGL((update_panel_kernel<T, BP, RPT, SO>), grid, dim3(256), 0, s,
                     ua, pa, nrb);
  return hipGetLastError();
}

template <typename T, int BP, bool SO>
hipError_t up_rpt(const UpdateArgs<T>& ua, int nsplit, const PanelArgs& pa,
                  int rpt, hipStream_t s) {
  if constexpr (up_built<BP, SO>()) {
    switch (rpt) {
      case 4: if constexpr ((kPanelThreads / BP) * 4 >= BP) return up_go<T, BP, 4, SO>(ua, nsplit, pa, s); break;
      case 8: if constexpr ((kPanelThreads / BP) * 8 >= BP) return up_go<T, BP, 8, SO>(ua, nsplit, pa, s); break;
      case 16: return up_go<T, BP, 16, SO>(ua, nsplit, pa, s);
      case 32: return up_go<T, BP, 32, SO>(ua, nsplit, pa, s);
      case 64: return up_go<T, BP, 64, SO>(ua, nsplit, pa, s);
    }
  }
  return hipErrorNotSupported;
}

template <typename T, int BP, int RPT, bool SO>
int up_occ() {
  static const int occ = [] {
    int o = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &o, reinterpret_cast<const void*>(update_panel_kernel<T, BP, RPT, SO>), 256, 0) != hipSuccess)
      o = 0;
    return o;
  }();
  return occ;
}

template <typename T, int BP, bool SO>
int up_occ_rpt(int rpt) {
  if constexpr (up_built<BP, SO>()) {
    switch (rpt) {
      case 4: if constexpr ((kPanelThreads / BP) * 4 >= BP) return up_occ<T, BP, 4, SO>(); break;
      case 8: if constexpr ((kPanelThreads / BP) * 8 >= BP) return up_occ<T, BP, 8, SO>(); break;
      case 16: return up_occ<T, BP, 16, SO>();
      case 32: return up_occ<T, BP, 32, SO>();
      case 64: return up_occ<T, BP, 64, SO>();
    }
  }
  return 0;
}

}  // namespace

template <typename T>
int update_panel_occupancy(const PanelShape& sh) {
  switch (sh.bp) {
    case 16: return up_occ_rpt<T, 16, false>(sh.rpt);
    case 32: return up_occ_rpt<T, 32, false>(sh.rpt);
    case 64: return up_occ_rpt<T, 64, false>(sh.rpt);
  }
  return 0;
}

template <typename T>
int sample_panel_occupancy(const PanelShape& sh) {
  return sh.bp == 64 ? up_occ_rpt<T, 64, true>(sh.rpt) : 0;
}

template int sample_panel_occupancy<float>(const PanelShape&);
template int sample_panel_occupancy<double>(const PanelShape&);

bool sample_panel_supported(int qp, const PanelShape& sh) {
  return qp == 64 && sh.bp == 64;
}

template <typename T>
hipError_t launch_sample_panel(const UpdateArgs<T>& ua, int nsplit,
                               const PanelArgs& pa, const PanelShape& sh,
                               hipStream_t s) {
  if (!sample_panel_supported(ua.qp, sh) || ua.bp != 0 || ua.dst || ua.mr <= 0 ||
      ua.n <= 0)
    return hipErrorNotSupported;
  // 32-bit buffer offsets, as in launch_update.
  if (ua.lds < ua.mr || (int64_t)kUpdChunk * ua.lds * (int64_t)sizeof(T) > ((int64_t)1 << 30))
    return hipErrorInvalidValue;
  return up_rpt<T, 64, true>(ua, nsplit, pa, sh.rpt, s);
}

template hipError_t launch_sample_panel<float>(const UpdateArgs<float>&, int, const PanelArgs&, const PanelShape&, hipStream_t);
template hipError_t launch_sample_panel<double>(const UpdateArgs<double>&, int, const PanelArgs&, const PanelShape&, hipStream_t);

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
    case 16: return up_rpt<T, 16, false>(ua, nsplit, pa, sh.rpt, s);
    case 32: return up_rpt<T, 32, false>(ua, nsplit, pa, sh.rpt, s);
    case 64: return up_rpt<T, 64, false>(ua, nsplit, pa, sh.rpt, s);
  }
  return hipErrorNotSupported;
}

template hipError_t launch_update_panel<float>(const UpdateArgs<float>&, int, const PanelArgs&, const PanelShape&, hipStream_t);
template hipError_t launch_update_panel<double>(const UpdateArgs<double>&, int, const PanelArgs&, const PanelShape&, hipStream_t);

}  // namespace rrf
