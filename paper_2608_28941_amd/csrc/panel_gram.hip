// Panel Householder QR with T factor from the panel's Gram matrix, as a
// kernel of its own (the body and its description are in panel_gram_body.h).

#include "panel_gram_body.h"

namespace rrf {
namespace {

template <int BP, int RPT, int NT>
__global__ __launch_bounds__(NT) void panel_gram_kernel(GramPanelArgs ga) {
  panel_gram_body<BP, RPT, NT>(ga, (int)blockIdx.x);
}

// Threads per workgroup: 512 at 64 columns (2 x 4 F entries per thread, two
// wavefronts per SIMD), 256 otherwise.
template <int BP>
constexpr int gram_threads() { return BP == 64 ? 512 : 256; }

template <int BP, int RPT>
hipError_t gram_go(const GramPanelArgs& a, hipStream_t s) {
  constexpr int NT = gram_threads<BP>();
  auto fn = panel_gram_kernel<BP, RPT, NT>;
  int occ = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
      &occ, reinterpret_cast<const void*>(fn), NT, 0);
  if (e != hipSuccess) return e;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return hipErrorInvalidDevice;
  if (occ < 1 || a.p.G > occ * cus) return hipErrorCooperativeLaunchTooLarge;
  GramPanelArgs arg = a;
  void* params[] = {&arg};
  return launch_resident(reinterpret_cast<const void*>(fn), dim3(a.p.G), dim3(NT),
                         params, s);
}

template <int BP>
hipError_t gram_rpt(const GramPanelArgs& a, int rpt, hipStream_t s) {
  constexpr int NT = gram_threads<BP>();
  constexpr int QC = BP * BP / NT;
  switch (rpt) {
    case 4: if constexpr (4 % QC == 0 && (NT / BP) * 4 >= BP) return gram_go<BP, 4>(a, s); break;
    case 8: if constexpr (8 % QC == 0 && (NT / BP) * 8 >= BP) return gram_go<BP, 8>(a, s); break;
    case 16: if constexpr (16 % QC == 0) return gram_go<BP, 16>(a, s); break;
    case 32: return gram_go<BP, 32>(a, s);
    case 64: return gram_go<BP, 64>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

bool gram_panel_shape(int64_t m, int b, int num_cus, PanelShape* out) {
  if (b < 1 || b > kMaxBlock || m < b) return false;
  const int bp = pad16(b);
  const int nt = bp == 64 ? gram_threads<64>() : gram_threads<32>();
  const int gr = nt / bp;
  const int qc = bp * bp / nt;
  static const int rpts[] = {4, 8, 16, 32, 64};
  // The smallest rows-per-thread (short Gram sums, short bulk updates) whose
  // grid stays within half the compute units (a smaller grid exchanges
  // less); failing that, within one workgroup per compute unit.
  for (int pass = 0; pass < 2; ++pass) {
    const int64_t cap = pass == 0 ? std::max(1, num_cus / 2) : num_cus;
    for (int rpt : rpts) {
      if (rpt % qc != 0 || gr * rpt < bp) continue;
      const int64_t G = ceil_div(m, (int64_t)gr * rpt);
      if (G <= cap && G <= kMaxGramWGs) {
        out->bp = bp;
        out->rpt = rpt;
        out->G = (int)G;
        out->rows_pad = G * gr * rpt;
        return true;
      }
    }
  }
  return false;
}

bool gram_fused_shape(int64_t m, int b, int max_wgs, PanelShape* out) {
  if (b < 1 || b > 32 || m < b) return false;
  const int bp = pad16(b);
  const int gr = 256 / bp;
  const int qc = bp * bp / 256;
  // At most 16 rows per thread (the update's register budget; lookahead.hip).
  static const int rpts[] = {4, 8, 16};
  for (int rpt : rpts) {
    if (rpt % qc != 0 || gr * rpt < bp) continue;
    const int64_t G = ceil_div(m, (int64_t)gr * rpt);
    if (G <= max_wgs && G <= kMaxGramWGs) {
      out->bp = bp;
      out->rpt = rpt;
      out->G = (int)G;
      out->rows_pad = G * gr * rpt;
      return true;
    }
  }
  return false;
}

hipError_t launch_panel_gram(const GramPanelArgs& a, const PanelShape& sh, hipStream_t s) {
  if (a.p.G != sh.G || a.p.b < 1 || a.p.b > sh.bp) return hipErrorInvalidValue;
  switch (sh.bp) {
    case 16: return gram_rpt<16>(a, sh.rpt, s);
    case 32: return gram_rpt<32>(a, sh.rpt, s);
    case 64: return gram_rpt<64>(a, sh.rpt, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace rrf
