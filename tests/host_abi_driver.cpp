// Host-side checks of the C ABI (include/rrf.h) for a sanitizer build of the
// host driver: every entry point's argument validation, on a machine with or
// without a GPU.  Calls that pass validation but need a device end in
// RRF_ERR_HIP when there is none, which runs the plan's clean-up path too.
// Prints one line per failed expectation and exits with their count.

#include <cstdint>
#include <cstdio>
#include <cstring>

#include "../include/rrf.h"

static int failures = 0;

static void expect(bool ok, const char* what) {
  if (!ok) {
    std::printf("FAILED: %s\n", what);
    ++failures;
  }
}

int main() {
  const int kInvalid = RRF_ERR_INVALID_ARG;
  for (int c = -7; c <= 2; ++c) {
    const char* s = rrf_status_string((rrf_status)c);
    expect(s && std::strncmp(s, "RRF", 3) == 0, "status string");
  }
  expect(rrf_status_string((rrf_status)42) != nullptr, "unknown status string");

  size_t ws = 0;
  expect(rrf_workspace_size(RRF_F64, 16384, 16384, 64, 0, &ws) == RRF_OK && ws > 0,
         "workspace size");
  expect(rrf_workspace_size(RRF_F64, 0, 10, 8, 0, &ws) == kInvalid, "workspace m_max");
  expect(rrf_workspace_size(RRF_F64, 10, 10, 129, 0, &ws) == kInvalid, "workspace b");
  expect(rrf_workspace_size((rrf_dtype)7, 10, 10, 8, 0, &ws) == kInvalid, "workspace dtype");
  expect(rrf_workspace_size(RRF_F32, 10, 10, 8, 0, nullptr) == kInvalid, "workspace out");

  rrf_plan_t plan = nullptr;
  expect(rrf_plan_create(nullptr, RRF_F64, 10, 10, 8, 0, nullptr) == kInvalid, "create null");
  expect(rrf_plan_create(&plan, (rrf_dtype)3, 10, 10, 8, 0, nullptr) == kInvalid,
         "create dtype");
  expect(rrf_plan_create(&plan, RRF_F64, -1, 10, 8, 0, nullptr) == kInvalid, "create m");
  expect(rrf_plan_create(&plan, RRF_F64, 10, 10, 0, 0, nullptr) == kInvalid, "create b");
  expect(rrf_plan_create(&plan, RRF_F64, 10, 10, 8, -2, nullptr) == kInvalid, "create k");
  expect(plan == nullptr, "no plan after failures");
  size_t need = 0;
  expect(rrf_workspace_size(RRF_F64, 300, 200, 16, 0, &need) == RRF_OK, "need");
  expect(rrf_plan_create_in(&plan, RRF_F64, 300, 200, 16, 0, nullptr,
                            reinterpret_cast<void*>(0x10008), need) == kInvalid,
         "workspace alignment");
  expect(rrf_plan_create_in(&plan, RRF_F64, 300, 200, 16, 0, nullptr,
                            reinterpret_cast<void*>(0x100000), need - 1) == kInvalid,
         "workspace size");
  // Valid arguments: a plan on a GPU, RRF_ERR_HIP without one.
  rrf_status st = rrf_plan_create(&plan, RRF_F64, 300, 200, 16, 0, nullptr);
  expect(st == RRF_OK || st == RRF_ERR_HIP, "create valid");
  if (st == RRF_OK) {
    expect(rrf_run(plan, nullptr, 300, 200, 300, 1e-3, 16, 1, nullptr, nullptr, nullptr,
                   nullptr, nullptr) == kInvalid, "run null A");
    expect(rrf_destroy(plan) == RRF_OK, "destroy");
  }

  void* q = nullptr;
  void* b = nullptr;
  int64_t ldq = 0, k = 0, ldb = 0;
  double x = 0.0;
  expect(rrf_run(nullptr, &x, 10, 10, 10, 1e-3, 8, 1, &q, &ldq, &k, &b, &ldb) == kInvalid,
         "run null plan");
  expect(rrf_destroy(nullptr) == RRF_OK, "destroy null");
  expect(rrf_set_stop_mode(nullptr, RRF_STOP_TRAILING) == kInvalid, "stop mode null");
  expect(rrf_set_power_iterations(nullptr, 1) == kInvalid, "power null");
  expect(rrf_set_timing(nullptr, 1) == kInvalid, "timing null");
  int64_t nb = 0;
  double e0 = 0, s2 = 0, et[4], es[4];
  expect(rrf_get_trace(nullptr, 4, &nb, et, es, nullptr, &e0, &s2) == kInvalid, "trace null");
  double ms[8], fl[8], by[8];
  int64_t la[8];
  expect(rrf_get_stage_stats(nullptr, ms, la, fl, by) == kInvalid, "stats null");
  const void* v = nullptr;
  const void* t = nullptr;
  const void* tau = nullptr;
  int64_t ldv = 0, ldt = 0;
  expect(rrf_get_reflectors(nullptr, &v, &ldv, &t, &ldt, &tau) == kInvalid,
         "reflectors null");
  expect(rrf_sketch(RRF_F64, 1, 10, 0, 4, nullptr, 10, nullptr) == kInvalid, "sketch out");
  expect(rrf_sketch(RRF_F64, 1, 10, 0, 4, &x, 5, nullptr) == kInvalid, "sketch ldo");
  expect(rrf_sketch(RRF_F64, 1, 0, 0, 4, &x, 1, nullptr) == RRF_OK, "sketch empty");
  expect(rrf_panel_qr(nullptr, &x, 10, 4, 10, &x, 10, &x, 4, &x) == kInvalid, "panel null");
  expect(rrf_apply_block_reflector(nullptr, 1, &x, 10, &x, 4, 4, &x, 10, 4, 10) == kInvalid,
         "larfb null");
  expect(rrf_subspace_map(nullptr, &x, 10, 2, &x, 10, 2, &x, 2, 10, 3, &x, 2) == kInvalid,
         "map null");
  expect(rrf_panel_qr_noalloc(RRF_F64, &x, 10, 0, 10, &x, 10, &x, 4, &x, nullptr, nullptr) ==
             kInvalid, "noalloc b");
  expect(rrf_panel_qr_noalloc(RRF_F64, &x, 1 << 20, 64, 1 << 20, &x, 1 << 20, &x, 64, &x,
                              nullptr, nullptr) == RRF_ERR_SHAPE, "noalloc rows");
  expect(rrf_copy_matrix(RRF_F64, nullptr, 10, &x, 10, 10, 1, nullptr) == kInvalid,
         "copy null");
  std::printf("%d failures\n", failures);
  return failures;
}
