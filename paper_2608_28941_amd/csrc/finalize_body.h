// Residual-norm finalisation and stop test (Alg. 2 E update and loop
// condition), shared by the one-workgroup finalize kernel and by the last
// workgroup of an update launch (which takes the step over when the update
// publishes its norm partials as epoch-tagged words).
//
// Sums the per-workgroup norm partials in a fixed order (deterministic) and
// applies the stop test.  init: E0 = ||A||_F^2, sigma^2 = tol^2 E0.
// Otherwise: E_trail = ||B[k:m, :]||^2 directly, E_sub -= ||B_i||^2 (the
// paper's running difference, clamped at 0); in spectral mode (2) the
// estimate the spectral kernels left in the run state.  At the end of a
// block (block >= 0: the trace index) the stop test runs: stop iff E <=
// sigma^2 or the rank cap is reached (Sec. 4: the loop ends after at most
// min(m, n) / b blocks); inside a block (block < 0, the first 64 columns of
// a wider block) only errors stop.  A NaN norm fails "E > sigma^2" and would
// stop silently, so non-finite norms are flagged.

#pragma once

#include "rrf_internal.h"
#include "xchg.h"

namespace rrf {
namespace {

// Both sums over a 256-thread workgroup: thread t adds parts t, t + 256, ...
// in order, each wavefront folds its 64 values by a butterfly, and the four
// wavefront sums are added as (w0 + w1) + (w2 + w3).  get(i, &a, &c) yields
// part i.  Returns the totals in every thread.
template <typename Get>
__device__ __forceinline__ void finalize_sums(int nparts, Get&& get, double& blk,
                                              double& trail) {
  __shared__ double fred[2][4];
  double a = 0.0, c = 0.0;
  for (int i = (int)threadIdx.x; i < nparts; i += 256) {
    double x, y;
    get(i, x, y);
    a += x;
    c += y;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off);
    c += __shfl_xor(c, off);
  }
  const int wv = (int)threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    fred[0][wv] = a;
    fred[1][wv] = c;
  }
  __syncthreads();
  blk = (fred[0][0] + fred[0][1]) + (fred[0][2] + fred[0][3]);
  trail = (fred[1][0] + fred[1][1]) + (fred[1][2] + fred[1][3]);
}

// The run-state update (one thread).  The wait error is read through the
// coherent path: another thread of this workgroup may have just set it.
__device__ __forceinline__ void finalize_state(const FinalizeArgs& f, double blk,
                                               double trail) {
  DevState* st = f.st;
  const int werr =
      __hip_atomic_load(&st->barrier_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (f.init) {
    const double E0 = blk + trail;
    st->E0 = E0;
    st->nonfinite = !isfinite(E0);
    st->sigma2 = (f.tol * f.tol) * E0;
    st->E_trail = E0;
    st->E_sub = E0;
    st->E_spec = E0;
    // The wait error is cleared by the host before the run (this step may
    // itself have waited).
    st->stop = st->nonfinite || werr || !(E0 > st->sigma2) || f.k_cap == 0;
  } else {
    double es = st->E_sub - blk;
    if (es < 0.0) es = 0.0;
    st->E_sub = es;
    st->E_trail = trail;
    if (!isfinite(trail)) st->nonfinite = 1;
    if (f.block >= 0) {
      f.tt[f.block] = trail;
      f.ts[f.block] = es;
      const double E = f.mode == 0 ? trail : (f.mode == 1 ? es : st->E_spec);
      st->stop = st->nonfinite || werr || !(E > st->sigma2) || f.k_after >= f.k_cap;
    } else {
      st->stop = st->nonfinite || werr;
    }
  }
  // The host reads the decision from its pinned copy once the launch has
  // completed (no copy in the stream).  A wait error recorded later in the
  // same launch stays in *st and reaches the host with a later decision or
  // an explicit state read.
  if (DevState* h = f.mirror) {
    h->E0 = st->E0;
    h->sigma2 = st->sigma2;
    h->E_trail = st->E_trail;
    h->E_sub = st->E_sub;
    h->stop = st->stop;
    h->nonfinite = st->nonfinite;
    h->barrier_err = werr;
    h->spin_limit = st->spin_limit;
    h->E_spec = st->E_spec;
  }
}

// Finalize from plain partials (2 doubles per part).
__device__ __forceinline__ void finalize_plain(const double* np, const FinalizeArgs& f) {
  double blk, trail;
  finalize_sums(f.nparts, [&](int i, double& x, double& y) {
    x = np[2 * i + 0];
    y = np[2 * i + 1];
  }, blk, trail);
  if (threadIdx.x == 0) finalize_state(f, blk, trail);
}

// Finalize from epoch-tagged partials (4 words per part), waiting until every
// part of this launch is there (bounded wait: a give-up is recorded in the
// run state and the host reports it).
__device__ __forceinline__ void finalize_tagged(const u64* nt, unsigned epoch,
                                                const FinalizeArgs& f) {
  const bool forced = waits_forced(f.st);
  double blk, trail;
  finalize_sums(f.nparts, [&](int i, double& x, double& y) {
    const u64* q = nt + 4 * (int64_t)i;
    u64 w[4];
    unsigned spins = 0;
    bool ok;
    do {
#pragma unroll
      for (int u = 0; u < 4; ++u) w[u] = get_word(q + u);
      ok = tagged(w[0], epoch) && tagged(w[1], epoch) && tagged(w[2], epoch) &&
           tagged(w[3], epoch);
    } while ((!ok || forced) && keep_waiting(&spins, f.st));
    x = untag(w[0], w[1]);
    y = untag(w[2], w[3]);
  }, blk, trail);
  if (threadIdx.x == 0) finalize_state(f, blk, trail);
}

}  // namespace
}  // namespace rrf
