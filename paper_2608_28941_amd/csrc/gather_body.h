// The gather of a sample taken in column splits (Alg. 2 sample step): every
// update workgroup adds its column range's share of B Omega to a partial, and
// the gathered sample is their sum.  One entry per call, summed in split
// order in binary64 (every launch that gathers gives the same bits).

#pragma once

#include "rrf_internal.h"

namespace rrf {
namespace {

template <typename T>
__device__ __forceinline__ void gather_entry(const GatherArgs<T>& g, int64_t r, int k) {
  double v = 0.0;
  if (r < g.m && k < g.b)
    for (int s = 0; s < g.nsplit; ++s) v += (double)g.P[s * g.split_stride + r + k * g.ldp];
  g.Y[r + k * g.ldy] = v;
}

}  // namespace
}  // namespace rrf
