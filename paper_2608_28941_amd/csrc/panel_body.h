// Panel Householder QR with T factor (Alg. 2, geqrt step): the body of one
// workgroup w of the panel grid (panel_kernel, and the panel part
// of the look-ahead kernel).
//
// Factors the sampled panel Y (m x b, b <= 64) column by column with LAPACK
// dlarfg / geqr2 semantics and builds the compact WY factor T (Eq. (4)) on the
// fly by the forward columnwise recursion T[:j, j] = -tau_j T[:j, :j] V^T v_j.
//
// Layout: a grid of G workgroups of 256 threads, all resident at once.  Thread t owns
// column k = t % BP and row group g = t / BP; workgroup w owns rows
// [w RW, (w + 1) RW) with RW = (256 / BP) * RPT, and thread (k, g) keeps the
// RPT rows w RW + g + (256 / BP) q of column k in registers for the whole
// factorisation.  Column j is broadcast through LDS.
//
// One grid-wide reduction per column.  With x the current column j below the
// diagonal, every thread contributes the partial dot of its own column with x
// over rows > j; together with row j of every column (held by workgroup 0)
// this gives, in one reduction,
//   ||x||^2            (the dlarfg norm),
//   v_j^T y_k, k > j   (the rank-1 update of the trailing columns), and
//   v_k^T v_j, k < j   (the new column of T),
// because v_j = [1; x / (alpha - beta)].  Every workgroup sums the partials
// in the same order, so all derive identical scalars (deterministic, no
// floating-point atomics).
//
// The panel is gathered beforehand into a zero-padded binary64 buffer (the
// sum of the update's column-split partials); the factorisation runs in
// binary64 (registers, reductions, V, T, tau), so the reflectors are
// orthogonal to binary64 precision even for float data.
//
// Requires 256 / BP * RPT >= BP so that rows 0 .. b-1 sit in workgroup 0.

#pragma once

#include "xchg.h"

namespace rrf {
namespace {

template <int BP, int RPT>
__device__ __forceinline__ void panel_body(const PanelArgs& a, const int w) {
  constexpr int GR = kPanelThreads / BP;
  constexpr int RW = GR * RPT;
  static_assert(RW >= BP, "rows 0..b-1 must sit in workgroup 0");
  static_assert(64 % BP == 0, "a wavefront holds whole row groups");
  __shared__ double xs[RW];           // column j below the diagonal, by row
  __shared__ double red_l[2][GR][BP]; // step partials of this workgroup, by parity
  __shared__ double red_r[GR][BP];    // sums of the gathered partials
  __shared__ double rj[BP];           // row j of every column
  __shared__ double Gm[BP][BP + 1];   // Gm[p][c] = v_p^T v_c, p < c (T workgroup)
  __shared__ double tau_s[BP];

  const int t = threadIdx.x;
  const int k = t % BP, g = t / BP;
  const int64_t base = (int64_t)w * RW;
  const int b = a.b;
  // The last workgroup collects V^T V and builds T at the end; workgroup 0
  // (which publishes row j every step) has no extra work.
  const bool tw = (w == a.G - 1);
  const bool forced = waits_forced(a.st);

  // The gathered panel has G * RW rows and BP columns, zero outside (m, b),
  // so the RPT loads are unconditional and all in flight together.
  double col[RPT];
  {
    const double* Yk = a.Y + base + g + (int64_t)k * a.ldy;
#pragma unroll
    for (int q = 0; q < RPT; ++q) col[q] = Yk[GR * q];
  }
  if (tw) {
    for (int idx = t; idx < BP * (BP + 1); idx += kPanelThreads) (&Gm[0][0])[idx] = 0.0;
    if (t < BP) tau_s[t] = 0.0;
  }

  constexpr int QJ = (BP + GR - 1) / GR;   // registers that can hold rows < BP
  for (int j = 0; j < b; ++j) {
    const int par = j & 1;
    const unsigned epoch = a.epoch_base + (unsigned)j + 1u;
    // 1. Row j of every column (final after step j - 1) sits in workgroup 0,
    //    row group j % GR, register j / GR: publish it at once.
    if (w == 0 && g == j % GR) {
      const int qj = j / GR;
      double v = 0.0;
#pragma unroll
      for (int q = 0; q < QJ; ++q) v = (q == qj) ? col[q] : v;
      put_tagged(&a.rowj[(par * BP + k) * 2], v, epoch);
    }
    // 2. Broadcast column j with its rows <= j zeroed (then every dot below
    //    is over rows > j and the rank-1 update leaves rows <= j untouched,
    //    with no per-row conditions).  Each row group lies inside one
    //    wavefront, whose lane k == j writes the group's rows and whose
    //    lanes read them: LDS operations of a wavefront complete in order,
    //    so no workgroup barrier is needed, and the next step's write comes
    //    after this step's last read in the same order.
    if (k == j) {
      if (w == 0) {
#pragma unroll
        for (int q = 0; q < RPT; ++q)
          xs[g + GR * q] = (q < QJ && g + GR * q <= j) ? 0.0 : col[q];
      } else {
#pragma unroll
        for (int q = 0; q < RPT; ++q) xs[g + GR * q] = col[q];
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // 3. Partial dot of this thread's column with x (rows > j).
    {
      double d0 = 0.0, d1 = 0.0;
#pragma unroll
      for (int q = 0; q < RPT; q += 2) {
        d0 += col[q] * xs[g + GR * q];
        if (q + 1 < RPT) d1 += col[q + 1] * xs[g + GR * (q + 1)];
      }
      red_l[par][g][k] = d0 + d1;
    }
    __syncthreads();
    // 4. Workgroup partial to global memory as epoch-tagged words.
    if (t < BP) {
      double s = 0.0;
#pragma unroll
      for (int gg = 0; gg < GR; ++gg) s += red_l[par][gg][t];
      put_tagged(&a.red[(((int64_t)par * a.G + w) * BP + t) * 2], s, epoch);
    }
    // 5. Every workgroup sums all partials in the same fixed order, polling
    //    each batch until it is complete; threads t < BP read row j in the
    //    first batch.
    {
      const int kk = t % BP, sub = t / BP;
      const u64* rp = a.red + ((int64_t)par * a.G * BP + kk) * 2;
      const u64* rq = &a.rowj[(par * BP + kk) * 2];
      unsigned spins = 0;
      double s = 0.0;
      for (int w0 = sub; w0 < a.G; w0 += 16 * GR) {
        const bool row = (w0 == 0);   // only sub == 0 starts at 0
        u64 hi[16], lo[16], rh = 0, rl = 0;
        bool ok;
        do {
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const int ww = w0 + u * GR;
            const u64* q = &rp[(int64_t)(ww < a.G ? ww : 0) * BP * 2];
            hi[u] = get_word(q);
            lo[u] = get_word(q + 1);
          }
          if (row) {
            rh = get_word(rq);
            rl = get_word(rq + 1);
          }
          ok = !row || (tagged(rh, epoch) && tagged(rl, epoch));
#pragma unroll
          for (int u = 0; u < 16; ++u)
            ok = ok && tagged(hi[u], epoch) && tagged(lo[u], epoch);
        } while ((!ok || forced) && keep_waiting(&spins, a.st));
#pragma unroll
        for (int u = 0; u < 16; ++u)
          if (w0 + u * GR < a.G) s += untag(hi[u], lo[u]);
        if (row) rj[kk] = untag(rh, rl);
      }
      red_r[sub][kk] = s;
    }
    __syncthreads();
    // 6. Totals and dlarfg scalars (identical in every thread of every
    //    workgroup: the same sums in the same order).
    double tk = 0.0, tj = 0.0;
#pragma unroll
    for (int gg = 0; gg < GR; ++gg) {
      tk += red_r[gg][k];
      tj += red_r[gg][j];
    }
    const double alpha = rj[j], rk = rj[k];
    double tau_j = 0.0, scale = 0.0;
    if (tj != 0.0) {
      const double nrm = sqrt(alpha * alpha + tj);
      const double beta = (alpha >= 0.0) ? -nrm : nrm;
      tau_j = (beta - alpha) / beta;
      scale = 1.0 / (alpha - beta);
    }
    // 7. v_j = x * scale below the diagonal (rows <= j of column j are never
    //    read again); trailing columns y_k -= tau_j (v_j^T y_k) v_j with
    //    v_j^T y_k = y_k[j] + scale * dot_k (xs is zero on rows <= j; row j
    //    of y_k, an entry of R, is not needed again).
    const double wk = rk + scale * tk;
    if (k == j) {
#pragma unroll
      for (int q = 0; q < RPT; ++q) col[q] = col[q] * scale;
    } else if (k > j && k < b) {
      const double fs = tau_j * wk * scale;
#pragma unroll
      for (int q = 0; q < RPT; ++q) col[q] = col[q] - fs * xs[g + GR * q];
    }
    // 8. v_p^T v_j = V[j, p] + scale * dot_p (p < j), for T.
    if (tw && g == 0) {
      if (k < j) Gm[k][j] = wk;
      else if (k == j) tau_s[j] = tau_j;
    }
  }
  __syncthreads();

  // Outputs: V with explicit unit diagonal and zeros above / beyond b.
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    const int64_t r = base + g + GR * q;
    if (r < a.m) {
      double v = 0.0;
      if (k < b) v = (r > k) ? col[q] : (r == k ? 1.0 : 0.0);
      a.V[r + k * a.ldv] = v;
    }
  }
  // T (Eq. (4)) from V^T V and tau: with U = striu(V^T V), T is the inverse
  // of diag(1/tau) + U, i.e. T[c][c] = tau_c and, for i < c,
  // T[i][c] = -tau_i sum_{i < p <= c} U[i][p] T[p][c] (written with tau as
  // a factor, so tau_i = 0 gives a zero row: H_i = I).  Thread c solves
  // column c by back substitution in registers.  U is zero outside the
  // written entries, and T[p][c] = 0 for p > c, so the full sums are exact.
  if (tw && t < BP) {
    const int c = t;
    double tc[BP];
#pragma unroll
    for (int i = BP - 1; i >= 0; --i) {
      double s0 = 0.0, s1 = 0.0;
#pragma unroll
      for (int p = i + 1; p < BP; p += 2) {
        s0 += Gm[i][p] * tc[p];
        if (p + 1 < BP) s1 += Gm[i][p + 1] * tc[p + 1];
      }
      const double ti = tau_s[i];
      tc[i] = (c < b && i < c) ? -ti * (s0 + s1) : ((c < b && i == c) ? ti : 0.0);
    }
#pragma unroll
    for (int i = 0; i < BP; ++i) a.Tm[i + (int64_t)c * a.ldt] = tc[i];
    if (c < b) a.tau[c] = tau_s[c];
  }
}

}  // namespace
}  // namespace rrf
