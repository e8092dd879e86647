// Panel Householder QR with T factor (Alg. 2, geqrt step) for callers that
// cannot allocate device memory: rrf_panel_qr_noalloc.
//
// The same kernels as rrf_panel_qr's column-by-column route (gather, the
// register-resident panel grid, copies out), with every buffer beyond the
// caller's inputs and outputs in one file-scope device array per GPU
// (`scratch`).  Host code reaches the array only through the address
// hipGetSymbolAddress returns for the current device; the array's name on
// the host is a stand-in, not a device address.
//
// Each call first clears the exchange words and the wait flag with a fill
// kernel (no memset node, so the sequence may sit in a captured graph), so
// the fixed epoch base never meets a word left by an earlier call.  Calls on
// one GPU share the array: calls that overlap on one GPU (several streams)
// race.

#include <mutex>
#include <type_traits>

#include <cstring>

#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr int64_t kNaMaxRows = 16384;            // largest panel height
constexpr int64_t kNaLdy = kNaMaxRows + 1024;    // gathered panel rows (>= any rows_pad)
constexpr int kNaMaxG = 64;                       // panel workgroups at most
// Scratch layout (byte offsets, each a multiple of 256).
constexpr size_t kNaYsum = 0;                                            // kNaLdy x 64 doubles
constexpr size_t kNaV = kNaYsum + (size_t)kNaLdy * 64 * 8;               // kNaMaxRows x 64 doubles
constexpr size_t kNaT = kNaV + (size_t)kNaMaxRows * 64 * 8;              // 64 x 64 doubles
constexpr size_t kNaTau = kNaT + 64 * 64 * 8;                            // 64 doubles
constexpr size_t kNaWords = kNaTau + 64 * 8;                             // exchange words
constexpr size_t kNaRedWords = (size_t)2 * kNaMaxG * 64 * 2;             // 2 x G x 64 values
constexpr size_t kNaRowWords = (size_t)2 * 64 * 2;                       // 2 x 64 values
constexpr size_t kNaState = kNaWords + (kNaRedWords + kNaRowWords) * 8;  // DevState
constexpr size_t kNaBytes = kNaState + 256;
static_assert(kNaV % 256 == 0 && kNaT % 256 == 0 && kNaTau % 256 == 0 &&
                  kNaWords % 256 == 0 && kNaState % 256 == 0,
              "scratch segments stay 256-byte aligned");
static_assert(sizeof(DevState) <= 256, "run state fits its segment");

__device__ __align__(256) unsigned char scratch[kNaBytes];

// Zero the exchange words and the run state, then set the spin limit.
__global__ void na_clear_kernel(unsigned long long* words, int64_t nwords, DevState* st,
                                unsigned spin_limit) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nwords) words[i] = 0ull;
  if (i == 0) {
    st->E0 = st->sigma2 = st->E_trail = st->E_sub = st->E_spec = 0.0;
    st->stop = st->nonfinite = st->barrier_err = 0;
    st->spin_limit = spin_limit;
  }
}

struct NaDevice {
  unsigned char* ptr = nullptr;   // device address of `scratch` on this GPU
  int num_cus = 0;
  bool ready = false;
};
constexpr int kNaMaxDevices = 64;
NaDevice g_na[kNaMaxDevices];
std::mutex g_na_mu;

// Per-device set-up, once, with that device current.
hipError_t na_device(NaDevice** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kNaMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_na_mu);
  NaDevice& d = g_na[dev];
  if (!d.ready) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    e = hipDeviceGetAttribute(&d.num_cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    d.ptr = static_cast<unsigned char*>(p);
    d.ready = true;
  }
  *out = &d;
  return hipSuccess;
}

template <typename T>
hipError_t na_out(const double* src, int64_t lds, T* dst, int64_t ldd, int64_t rows,
                  int64_t cols, hipStream_t s) {
  if constexpr (std::is_same<T, double>::value)
    return launch_copy<double>(src, lds, dst, ldd, rows, cols, s);
  else
    return launch_convert<double, float>(src, lds, dst, ldd, rows, cols, s);
}

// The panel grid for an m x b panel within the scratch's limits.
bool na_shape(int64_t m, int b, int num_cus, PanelShape* sh) {
  return m <= kNaMaxRows && panel_shape(m, b, num_cus, kNaMaxG, sh) && sh->G <= kNaMaxG &&
         sh->rows_pad <= kNaLdy;
}

template <typename T>
hipError_t na_panel(const NaDevice* d, const PanelShape& sh, const T* Y, int64_t m, int b,
                    int64_t ldy, T* Vout, int64_t ldv, T* Tout, int64_t ldt, T* tauout,
                    int* wait_status, hipStream_t s) {
  hipError_t e;
  double* Ysum = reinterpret_cast<double*>(d->ptr + kNaYsum);
  double* Vs = reinterpret_cast<double*>(d->ptr + kNaV);
  double* Ts = reinterpret_cast<double*>(d->ptr + kNaT);
  double* taus = reinterpret_cast<double*>(d->ptr + kNaTau);
  unsigned long long* words = reinterpret_cast<unsigned long long*>(d->ptr + kNaWords);
  DevState* st = reinterpret_cast<DevState*>(d->ptr + kNaState);
  const int64_t nwords = (int64_t)(kNaRedWords + kNaRowWords);
  hipLaunchKernelGGL(na_clear_kernel, dim3((unsigned)ceil_div(nwords, 256)), dim3(256), 0, s,
                     words, nwords, st, kSpinLimit);
  e = hipGetLastError();
  if (e == hipSuccess)
    e = launch_gather_panel<T>(Y, ldy, 0, 1, m, b, sh.bp, sh.rows_pad, Ysum, kNaLdy, s);
  if (e != hipSuccess) return e;
  PanelArgs pa{};
  pa.Y = Ysum; pa.ldy = kNaLdy;
  pa.m = m; pa.b = b;
  pa.V = Vs; pa.ldv = kNaMaxRows;
  pa.Tm = Ts; pa.ldt = 64; pa.tau = taus;
  pa.red = words; pa.rowj = words + kNaRedWords;
  pa.epoch_base = 128;      // the words were zeroed above
  pa.st = st; pa.G = sh.G;
  e = launch_panel(pa, sh, s);
  if (e == hipSuccess) e = na_out<T>(Vs, kNaMaxRows, Vout, ldv, m, b, s);
  if (e == hipSuccess) e = na_out<T>(Ts, 64, Tout, ldt, b, b, s);
  if (e == hipSuccess) e = na_out<T>(taus, 1, tauout, 1, b, 1, s);
  if (e == hipSuccess && wait_status)
    e = hipMemcpyAsync(wait_status, &st->barrier_err, sizeof(int), hipMemcpyDeviceToDevice, s);
  return e;
}

}  // namespace
}  // namespace rrf

using namespace rrf;

extern "C" rrf_status rrf_panel_qr_noalloc(rrf_dtype dtype, const void* Y, int64_t m,
                                           int64_t b, int64_t ldy, void* V, int64_t ldv,
                                           void* T, int64_t ldt, void* tau, int* wait_status,
                                           void* hip_stream) {
  // dtype validated on its bits (a C caller may pass any int).
  int dt;
  static_assert(sizeof(dtype) == sizeof(int), "int-sized enum");
  std::memcpy(&dt, &dtype, sizeof dt);
  if ((dt != RRF_F32 && dt != RRF_F64) || !Y || !V || !T || !tau)
    return RRF_ERR_INVALID_ARG;
  if (b < 1 || b > kMaxBlock || m < b || ldy < m || ldv < m || ldt < b)
    return RRF_ERR_INVALID_ARG;
  if (m > kNaMaxRows) return RRF_ERR_SHAPE;
  NaDevice* d = nullptr;
  if (na_device(&d) != hipSuccess) return RRF_ERR_HIP;
  PanelShape sh;
  if (!na_shape(m, (int)b, d->num_cus, &sh)) return RRF_ERR_SHAPE;
  const hipStream_t s = (hipStream_t)hip_stream;
  hipError_t e;
  if (dtype == RRF_F64)
    e = na_panel<double>(d, sh, (const double*)Y, m, (int)b, ldy, (double*)V, ldv,
                         (double*)T, ldt, (double*)tau, wait_status, s);
  else
    e = na_panel<float>(d, sh, (const float*)Y, m, (int)b, ldy, (float*)V, ldv,
                        (float*)T, ldt, (float*)tau, wait_status, s);
  return e == hipSuccess ? RRF_OK : RRF_ERR_HIP;
}
