// Blocked WY update (Alg. 2, update step, Theorem 3.1) of one workgroup:
// B <- B - V W on a 128-row block and one column split, fused with the next
// sample P = B_new Omega and the residual norms.  Used by update_kernel and
// by the update part of the look-ahead kernel.

#pragma once

#include <type_traits>

#include "finalize_body.h"
#include "mfma.h"
#include "rrf_internal.h"

namespace rrf {
namespace {

// ---------------------------------------------------------------------------
// Buffer access to the B tiles.  A raw buffer resource (base, byte count)
// makes the hardware bounds-check every access: an out-of-range load returns
// zero and an out-of-range store is dropped.  Rows past mr get a lane offset
// beyond any record count and columns past n fall beyond the record count of
// their chunk, so the update needs no per-lane branches, its stores are
// unconditional instructions, and the waits on the next chunk's loads never
// have to cover the previous chunk's stores.  Offsets are 32-bit bytes: the
// host keeps kUpdChunk * ld * sizeof(T) <= 2^30.
// ---------------------------------------------------------------------------
constexpr unsigned kOOB = 1u << 30;   // lane offset of a masked row
// s_waitcnt operand (gfx9 encoding) that waits for vmcnt 0 and leaves
// expcnt (7) and lgkmcnt (15) at their maximum.
constexpr int kVmcntZero = 0x0F70;

typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, int64_t bytes) {
  // Third word 0x00020000: the gfx9-family raw-buffer format (32-bit data).
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                           (int)bytes, 0x00020000);
}

template <typename T> struct Buf;
template <> struct Buf<double> {
  static __device__ __forceinline__ double ld(__amdgpu_buffer_rsrc_t r, unsigned vo) {
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, (int)vo, 0, 0));
  }
  // so: uniform byte offset (not part of the bounds check; in range here).
  static __device__ __forceinline__ double ld_s(__amdgpu_buffer_rsrc_t r, unsigned vo, int so) {
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, (int)vo, so, 0));
  }
  static __device__ __forceinline__ void st(double v, __amdgpu_buffer_rsrc_t r, unsigned vo) {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, v), r, (int)vo, 0, 0);
  }
};
template <> struct Buf<float> {
  static __device__ __forceinline__ float ld(__amdgpu_buffer_rsrc_t r, unsigned vo) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)vo, 0, 0));
  }
  static __device__ __forceinline__ float ld_s(__amdgpu_buffer_rsrc_t r, unsigned vo, int so) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)vo, so, 0));
  }
  static __device__ __forceinline__ void st(float v, __amdgpu_buffer_rsrc_t r, unsigned vo) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, (int)vo, 0, 0);
  }
};

// ---------------------------------------------------------------------------
// update: X <- X - V W (BP > 0), store (STORE), norms, and P = X_new Omega,
// for the workgroup of row block rb (of nrb) and column split `split`;
// 256 threads; wavefront w owns RT adjacent 16-row tiles, so every staged W
// and Omega value read from LDS feeds RT MFMAs.
// ---------------------------------------------------------------------------
template <typename T, int BP, int QP, bool STORE>
__device__ __forceinline__ void update_body(const UpdateArgs<T>& a, const unsigned rb,
                                            const unsigned split, const unsigned nrb) {
  typedef typename Mfma<T>::acc_t acc_t;
  constexpr int RT = kUpdRowTiles;
  constexpr int NP4 = BP / 4;        // K-steps of the rank-b update
  constexpr int NQT = QP / 16;       // 16-wide tiles of the sample
  constexpr int LDW = BP + 1;        // odd: conflict-free column reads
  constexpr int LDO = QP + 1;
  constexpr int NCT = kUpdChunk / 16;
  constexpr int E = (int)sizeof(T);
  static_assert(kUpdRows == 64 * RT, "workgroup height");
  // Staged W and Omega chunks, double buffered: chunk c is read from buffer
  // c % 2 while chunk c + 1 is written to the other one, so one barrier per
  // chunk separates both the reads from the next overwrite and the writes
  // from the next reads.
  __shared__ T wl[2][kUpdChunk * (BP > 0 ? LDW : 1)];
  __shared__ T ol[2][kUpdChunk * (QP > 0 ? LDO : 1)];
  __shared__ double nred[2][4];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t cs = (int64_t)split * a.cols_per_split;
  const int64_t ce = min(a.n, cs + a.cols_per_split);
  // This workgroup's norm partials (thread 0's values): plain, or tagged with
  // the finalisation in the last update workgroup.
  auto publish = [&](const double nbv, const double ntv) {
    const int64_t wg = (int64_t)split * nrb + rb;
    if (a.normtag) {
      if (threadIdx.x == 0) {
        put_tagged(&a.normtag[4 * wg], nbv, a.fin_epoch);
        put_tagged(&a.normtag[4 * wg + 2], ntv, a.fin_epoch);
      }
      if (wg == a.fin_nwg - 1) finalize_tagged(a.normtag, a.fin_epoch, a.fin);   // uniform
    } else if (threadIdx.x == 0) {
      a.normpart[2 * wg + 0] = nbv;
      a.normpart[2 * wg + 1] = ntv;
    }
  };
  if (cs >= ce) {          // empty split (uniform per workgroup, before any barrier)
    if (a.normpart) publish(0.0, 0.0);
    return;
  }
  int64_t r[RT];
  bool rowok[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    r[rt] = (int64_t)rb * kUpdRows + 16 * (RT * wave + rt) + m16;
    rowok[rt] = r[rt] < a.mr;
  }

  // This wavefront's slices of -V^T as MFMA B operands:
  // B[g][m] = -V[r[rt]][4 p4 + g].
  T vreg[RT][NP4 > 0 ? NP4 : 1];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const double vmask = rowok[rt] ? -1.0 : 0.0;   // mask multiply keeps loads batched
    const int64_t rr = rowok[rt] ? r[rt] : 0;
#pragma unroll
    for (int p4 = 0; p4 < NP4; ++p4)
      vreg[rt][p4] = (T)(vmask * a.V[rr + (4 * p4 + g) * a.ldv]);
  }

  acc_t pacc[RT][NQT > 0 ? NQT : 1];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) pacc[rt][qt] = Mfma<T>::zero();
  // Squared norms per row tile (one FMA per element: f64 VALU work takes
  // issue slots from the MFMA); a lane's rows of one tile fall either in the
  // block rows (< s0) or in the trailing rows, split after the sweep.
  double nq[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) nq[rt] = 0.0;

  // Byte offsets.  Item i of a tile holds column drow(g, i) = drow(g, 0) +
  // i * dstep; the lane part covers the row and drow(g, 0), the uniform part
  // (ct * 16 + i * dstep) * ld.
  const int d0 = Mfma<T>::drow(g, 0);
  const int dstep = Mfma<T>::drow(0, 1) - Mfma<T>::drow(0, 0);
  unsigned vs[RT], vd[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    vs[rt] = rowok[rt] ? (unsigned)((r[rt] + (int64_t)d0 * a.lds) * E) : kOOB;
    vd[rt] = rowok[rt] ? (unsigned)((r[rt] + (int64_t)d0 * a.ldd) * E) : kOOB;
  }
  const unsigned cstep_s = (unsigned)(dstep * a.lds * E);
  const unsigned cstep_d = (unsigned)(dstep * a.ldd * E);
  const unsigned tstep_s = (unsigned)(16 * a.lds * E);
  const unsigned tstep_d = (unsigned)(16 * a.ldd * E);

  // Staging values (W, Omega) and the B tiles of the next chunk are loaded
  // while the current chunk computes.  Chunks start at multiples of kUpdChunk
  // and split boundaries are multiples of kUpdChunk, so a chunk that starts
  // before ce only runs past it at the end of the matrix, where W and Omega
  // carry zero rows up to the next multiple and the B loads return zero.  A
  // chunk that starts at or past ce (the prefetch after the last chunk, and
  // the second chunk of the last pair when the count is odd) gets buffer
  // resources of zero bytes: its loads return zero without touching memory
  // and its stores are dropped, so it adds nothing to P or the norms.  The
  // chunk loop therefore always runs whole pairs, with no branch between the
  // two chunks of a pair: a conditional second chunk gave the loop header two
  // predecessors, and the waits merged there covered the stores of the
  // previous chunk.
  //
  // Schedule per chunk: issue the next chunk's loads, compute and store this
  // chunk, then move the next chunk's staging values into the other LDS
  // buffer and its B tiles into the accumulators, and meet at the barrier.
  // The waits for those loads sit in straight-line code after the stores, so
  // they never wait for stores (the vector-memory counter retires in issue
  // order).
  constexpr int NW = BP > 0 ? (kUpdChunk * BP) / 256 : 0;
  constexpr int NO = (kUpdChunk * QP) / 256;
  static_assert((kUpdChunk * BP) % 256 == 0 && (kUpdChunk * QP) % 256 == 0,
                "chunk staging assumes whole passes of 256 threads");
  // W and Omega staging offsets: thread t, pass it reads row t / BP + it *
  // (256 / BP), entry t % BP of the chunk; the pass part is uniform.
  const unsigned wo_lane = BP > 0 ? (unsigned)(((threadIdx.x / (BP > 0 ? BP : 1)) * a.ldw +
                                                threadIdx.x % (BP > 0 ? BP : 1)) * E) : 0u;
  const unsigned oo_lane = QP > 0 ? (unsigned)(((threadIdx.x / (QP > 0 ? QP : 1)) * a.ldo +
                                                threadIdx.x % (QP > 0 ? QP : 1)) * E) : 0u;
  const int wo_pass = BP > 0 ? (256 / (BP > 0 ? BP : 1)) * a.ldw * E : 0;
  const int oo_pass = QP > 0 ? (256 / (QP > 0 ? QP : 1)) * a.ldo * E : 0;
  T tw[NW > 0 ? NW : 1], to[NO > 0 ? NO : 1];
  acc_t bx[RT][NCT];
  auto load_chunk = [&](int64_t cc0) {
    const bool live = cc0 < ce;
    if (NW > 0) {
      const __amdgpu_buffer_rsrc_t rw =
          buf_rsrc(a.W + cc0 * a.ldw, live ? (int64_t)kUpdChunk * a.ldw * E : 0);
#pragma unroll
      for (int it = 0; it < NW; ++it) tw[it] = Buf<T>::ld_s(rw, wo_lane, it * wo_pass);
    }
    if (NO > 0) {
      const __amdgpu_buffer_rsrc_t ro =
          buf_rsrc(a.Om + cc0 * a.ldo, live ? (int64_t)kUpdChunk * a.ldo * E : 0);
#pragma unroll
      for (int it = 0; it < NO; ++it) to[it] = Buf<T>::ld_s(ro, oo_lane, it * oo_pass);
    }
    const int64_t cn = min((int64_t)kUpdChunk, ce - cc0);
    const __amdgpu_buffer_rsrc_t rs =
        buf_rsrc(a.src + cc0 * a.lds, cn > 0 ? ((cn - 1) * a.lds + a.mr) * E : 0);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          bx[rt][ct][i] = Buf<T>::ld(rs, vs[rt] + ct * tstep_s + i * cstep_s);
  };
  auto stage_chunk = [&](T* wb, T* ob) {
#pragma unroll
    for (int it = 0; it < NW; ++it) {
      const int idx = threadIdx.x + 256 * it;
      wb[(idx / BP) * LDW + idx % BP] = tw[it];
    }
#pragma unroll
    for (int it = 0; it < NO; ++it) {
      const int idx = threadIdx.x + 256 * it;
      ob[(idx / QP) * LDO + idx % QP] = to[it];
    }
  };

  acc_t t[RT][NCT];
  load_chunk(cs);
  stage_chunk(wl[0], ol[0]);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) t[rt][ct] = bx[rt][ct];
  __syncthreads();
  // Every load of the first chunk has arrived before the loop (vmcnt(0)).
  // In steady state a chunk starts with the B tiles in flight ahead of the
  // previous chunk's stores; if the loop were entered with them in flight
  // too but no stores after them, the waits merged at the loop entry would
  // count the stores and hold the first MFMAs of every chunk until they
  // complete.
  __builtin_amdgcn_s_waitcnt(kVmcntZero);

  // One chunk from buffer CUR (a compile-time constant: the loop below is
  // unrolled by two so that both buffers have fixed LDS offsets).
  auto chunk = [&](const int64_t c0, auto cur_tag) {
    constexpr int CUR = decltype(cur_tag)::value;
    const T* wlc = wl[CUR];
    const T* olc = ol[CUR];
    load_chunk(c0 + kUpdChunk);
    // Keep the prefetch at the top of the chunk: under full register use the
    // scheduler otherwise sinks the B loads into the middle of the chunk.
    __builtin_amdgcn_sched_barrier(0);

    // Rank-b update of all tiles first, so that the samples do not wait on
    // the result of the MFMA chain that just produced their operand.
    // D[M = column drow(g, i)][N = row m16] of each 16 x 16 tile.
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int p4 = 0; p4 < NP4; ++p4) {
        const T wa = wlc[(ct * 16 + m16) * LDW + 4 * p4 + g];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          t[rt][ct] = Mfma<T>::op(wa, vreg[rt][p4], t[rt][ct]);
      }
    if (STORE) {
      const int64_t cn = min((int64_t)kUpdChunk, ce - c0);
      const __amdgpu_buffer_rsrc_t rd =
          buf_rsrc(a.dst + c0 * a.ldd, cn > 0 ? ((cn - 1) * a.ldd + a.mr) * E : 0);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            Buf<T>::st(t[rt][ct][i], rd, vd[rt] + ct * tstep_d + i * cstep_d);
    }
    // Invalid rows and columns hold zeros here (zero loads, zero V and W).
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const double v = (double)t[rt][ct][i];
          nq[rt] = fma(v, v, nq[rt]);
        }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
          const T oa = olc[(ct * 16 + Mfma<T>::drow(g, s)) * LDO + qt * 16 + m16];
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
            pacc[rt][qt] = Mfma<T>::op(oa, t[rt][ct][s], pacc[rt][qt]);
        }
    stage_chunk(wl[CUR ^ 1], ol[CUR ^ 1]);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) t[rt][ct] = bx[rt][ct];
    __syncthreads();
  };
  for (int64_t c0 = cs; c0 < ce; c0 += 2 * kUpdChunk) {
    chunk(c0, std::integral_constant<int, 0>());
    chunk(c0 + kUpdChunk, std::integral_constant<int, 1>());
  }

  if (QP > 0) {
    T* P = a.P + (int64_t)split * a.split_stride;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      if (rowok[rt]) {
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            P[r[rt] + (qt * 16 + Mfma<T>::drow(g, i)) * a.ldp] = pacc[rt][qt][i];
      }
  }
  if (a.normpart) {
    double nb = 0.0, nt = 0.0;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (r[rt] < a.s0) nb += nq[rt];
      else nt += nq[rt];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      nb += __shfl_xor(nb, off);
      nt += __shfl_xor(nt, off);
    }
    if (lane == 0) {
      nred[0][wave] = nb;
      nred[1][wave] = nt;
    }
    __syncthreads();
    publish(((nred[0][0] + nred[0][1]) + nred[0][2]) + nred[0][3],
            ((nred[1][0] + nred[1][1]) + nred[1][2]) + nred[1][3]);
  }
}

}  // namespace
}  // namespace rrf
