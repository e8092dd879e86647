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
//
// Blocks of at most 32 columns take the panel from its Gram matrix (one
// exchange per sweep of columns instead of one per column) in the same
// arrangement: update_gram_kernel's first G workgroups run panel_gram_body.

#include "panel_body.h"
#include "panel_gram_body.h"
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

template <typename T, int BP, int RPT>
__global__ __launch_bounds__(256, 2) void update_gram_kernel(UpdateArgs<T> ua,
                                                             GramPanelArgs ga,
                                                             unsigned nrb) {
  if ((int)blockIdx.x < ga.p.G) {
    panel_gram_body<BP, RPT, 256>(ga, (int)blockIdx.x);
    return;
  }
  const unsigned t = blockIdx.x - (unsigned)ga.p.G;
  update_body<T, BP, BP, true>(ua, t % nrb, t / nrb, nrb);
}

// Rows per thread the Gram body accepts at 256 threads: whole staged chunks
// of BP rows (BP^2 / 256 register slots each) and at least BP rows per
// workgroup; at most 16, beyond which the body no longer fits the update's
// register budget (two workgroups per compute unit) without spilling.
constexpr int kUgMaxRpt = 16;
template <int BP, int RPT>
constexpr bool ug_built() {
  return (BP == 16 || BP == 32) && RPT <= kUgMaxRpt && RPT % (BP * BP / 256) == 0 &&
         (256 / BP) * RPT >= BP;
}

template <typename T, int BP, int RPT>
hipError_t ug_go(const UpdateArgs<T>& ua, int nsplit, const GramPanelArgs& ga,
                 hipStream_t s) {
  const unsigned nrb = (unsigned)ceil_div(ua.mr, kUpdRows);
  const dim3 grid((unsigned)ga.p.G + nrb * (unsigned)nsplit);
  hipLaunchKernelGGL((update_gram_kernel<T, BP, RPT>), grid, dim3(256), 0, s, ua, ga, nrb);
  return hipGetLastError();
}

template <typename T, int BP, int RPT>
int ug_occ() {
  static const int occ = [] {
    int o = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &o, reinterpret_cast<const void*>(update_gram_kernel<T, BP, RPT>), 256, 0) != hipSuccess)
      o = 0;
    return o;
  }();
  return occ;
}

// Dispatch over rows per thread: go(integral_constant<RPT>) for a built
// shape, else fallback.
template <int BP, typename F, typename R>
R ug_rpt(int rpt, F&& go, R fallback) {
  switch (rpt) {
    case 4: if constexpr (ug_built<BP, 4>()) return go(std::integral_constant<int, 4>{}); break;
    case 8: if constexpr (ug_built<BP, 8>()) return go(std::integral_constant<int, 8>{}); break;
    case 16: if constexpr (ug_built<BP, 16>()) return go(std::integral_constant<int, 16>{}); break;
    case 32: if constexpr (ug_built<BP, 32>()) return go(std::integral_constant<int, 32>{}); break;
    case 64: if constexpr (ug_built<BP, 64>()) return go(std::integral_constant<int, 64>{}); break;
  }
  return fallback;
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

bool update_gram_supported(int bp, int qp, const PanelShape& sh) {
  if (bp <= 0 || bp != qp || bp != sh.bp || sh.G < 1 || sh.G > kMaxGramWGs) return false;
  if (sh.bp == 16) return ug_rpt<16>(sh.rpt, [](auto) { return true; }, false);
  if (sh.bp == 32) return ug_rpt<32>(sh.rpt, [](auto) { return true; }, false);
  return false;
}

template <typename T>
int update_gram_occupancy(const PanelShape& sh) {
  if (sh.bp == 16)
    return ug_rpt<16>(sh.rpt, [](auto r) { return ug_occ<T, 16, decltype(r)::value>(); }, 0);
  if (sh.bp == 32)
    return ug_rpt<32>(sh.rpt, [](auto r) { return ug_occ<T, 32, decltype(r)::value>(); }, 0);
  return 0;
}

template int update_gram_occupancy<float>(const PanelShape&);
template int update_gram_occupancy<double>(const PanelShape&);

template <typename T>
hipError_t launch_update_gram(const UpdateArgs<T>& ua, int nsplit, const GramPanelArgs& ga,
                              const PanelShape& sh, hipStream_t s) {
  if (!update_gram_supported(ua.bp, ua.qp, sh) || !ua.dst || ua.mr <= 0 || ua.n <= 0 ||
      ga.p.G != sh.G || ga.p.b < 1 || ga.p.b > sh.bp)
    return hipErrorNotSupported;
  // 32-bit buffer offsets, as in launch_update.
  const int64_t ld = std::max(ua.lds, ua.ldd);
  if (ld < ua.mr || (int64_t)kUpdChunk * ld * (int64_t)sizeof(T) > ((int64_t)1 << 30))
    return hipErrorInvalidValue;
  if (sh.bp == 16)
    return ug_rpt<16>(sh.rpt, [&](auto r) { return ug_go<T, 16, decltype(r)::value>(ua, nsplit, ga, s); },
                      hipErrorNotSupported);
  return ug_rpt<32>(sh.rpt, [&](auto r) { return ug_go<T, 32, decltype(r)::value>(ua, nsplit, ga, s); },
                    hipErrorNotSupported);
}

template hipError_t launch_update_gram<float>(const UpdateArgs<float>&, int, const GramPanelArgs&, const PanelShape&, hipStream_t);
template hipError_t launch_update_gram<double>(const UpdateArgs<double>&, int, const GramPanelArgs&, const PanelShape&, hipStream_t);

template hipError_t launch_update_panel<float>(const UpdateArgs<float>&, int, const PanelArgs&, const PanelShape&, hipStream_t);
template hipError_t launch_update_panel<double>(const UpdateArgs<double>&, int, const PanelArgs&, const PanelShape&, hipStream_t);

}  // namespace rrf
