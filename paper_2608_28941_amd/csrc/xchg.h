// Cross-workgroup exchange of epoch-tagged binary64 values (the panel
// kernels' grid-wide reductions).

#pragma once

#include "rrf_internal.h"

namespace rrf {
namespace {

// Cross-workgroup traffic uses agent-scope atomic accesses only (coherent
// across the XCDs without L2 write-back or invalidation, which an
// agent-scope fence would cost on every step).
//
// Publication without flags: a workgroup publishes each double of its step
// partials as two 64-bit words, each holding one 32-bit half of the value in
// its upper half and the step's epoch in its lower half.  A 64-bit atomic
// access is single-copy atomic, so a reader that sees the step's epoch in
// both words of a value has that step's value; it re-reads until every word
// it needs carries the epoch.  One trip through the coherent memory path per
// step instead of three (partials, completion wait, flag, flag poll, partial
// read).  Epochs are unique per launch and step (the buffer is zeroed at
// plan creation and epoch 0 is never used), so words left by earlier steps
// or launches never match.  A slot is rewritten two steps later only by a
// workgroup that has seen every workgroup's next-step partials, so no reader
// is still reading it.  The wait is bounded: after the run state's spin limit
// (kSpinLimit polls, each a sleep of about 128 cycles plus a trip to the
// coherent memory path: tens of seconds) it records an error and every later
// wait returns at once, so the kernel always drains (the host then reports
// RRF_ERR_INTERNAL and discards the results).
typedef unsigned long long u64;

__device__ __forceinline__ void put_tagged(u64* p, double v, unsigned epoch) {
  const u64 u = (u64)__double_as_longlong(v);
  __hip_atomic_store(p, (u & 0xFFFFFFFF00000000ull) | epoch, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(p + 1, (u << 32) | epoch, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ u64 get_word(const u64* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double untag(u64 hi, u64 lo) {
  return __longlong_as_double((long long)((hi & 0xFFFFFFFF00000000ull) | (lo >> 32)));
}
__device__ __forceinline__ bool tagged(u64 w, unsigned epoch) {
  return (unsigned)w == epoch;
}

// One poll round failed: back off, count, and give up (recording the error)
// after the run state's spin limit or once another thread has given up.  A
// spin limit of 0 makes every wait give up at its first poll, complete or
// not (the host sets it only to test this path); the kernel still drains.
__device__ __forceinline__ bool keep_waiting(unsigned* spins, DevState* st) {
  const unsigned lim = st->spin_limit;
  __builtin_amdgcn_s_sleep(2);
  ++*spins;
  if (*spins > lim ||
      ((*spins & 255u) == 0u &&
       __hip_atomic_load(&st->barrier_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
    __hip_atomic_store(&st->barrier_err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return false;
  }
  return true;
}

// Whether this launch's waits are forced to give up (read once per kernel).
__device__ __forceinline__ bool waits_forced(const DevState* st) {
  return st->spin_limit == 0u;
}

}  // namespace
}  // namespace rrf
