// Panel Householder QR with T factor (Alg. 2, geqrt step) computed from the
// panel's Gram matrix: one grid-wide exchange per sweep of columns instead of
// one per column.
//
// The reflectors are those of LAPACK dlarfg / geqr2 (same signs, tau, V with
// unit diagonal); only the inner products they need come from a different
// place.  Householder steps are orthogonal, so the Gram matrix of the columns
// over the rows a step touches is invariant under it, and every quantity of
// the column recurrence (the norm below the diagonal, v_j^T y_k, v_p^T v_j)
// follows from
//
//   F = X^T X over rows > j,  X = [v_0 .. v_{j-1}  y_j .. y_{b-1}]
//
// (finished reflector vectors and the not yet factored columns) together
// with rows 0 .. b-1 of X (the "top" block).  Each step updates F and the top
// block with O(b^2) work; the bulk rows are updated by the same rank-1
// recurrence without any inner product.  So after one exchange (F's partial
// sums over each workgroup's rows, reduced in two phases) every workgroup
// runs the column recurrence on its own copy of F and the top block, all of
// them bit for bit alike, and applies it to its rows.
//
// Downdating a norm loses relative accuracy when the column has shrunk: the
// rounding error of F[j][j] after s steps is about s u nu_j, nu_j being the
// column's norm^2 (rows >= sweep start) when F was last formed.  When
// F[j][j] < theta nu_j the sweep ends and F is formed again from the current
// rows (the safeguard LAPACK's dgeqp3 applies to its downdated column norms),
// so the norm behind each reflector has relative error <= ~64 u / theta and
// the reflector is orthogonal to that accuracy; a well-conditioned panel
// needs one exchange.  T (Eq. (4)) comes from the recorded v_p^T v_j and tau
// by back substitution.
//
// Layout: as the column-by-column panel (thread (k, g) keeps rows
// w RW + g + (256 / BP) q of column k in registers); F and the top block live
// in LDS.  Workgroup 0's register copy of rows 0 .. b-1 is not used: those
// rows are taken from the top block.
//
// The body runs as a kernel of its own (panel_gram.hip) or on the first
// workgroups of the look-ahead launch (lookahead.hip); w is the panel
// workgroup's index, NT the launch's threads per workgroup.

#pragma once

#include "mfma.h"
#include "xchg.h"

namespace rrf {
namespace {

constexpr double kGramTheta = 0.125;

// Exchanged Gram values: the upper-triangle 16 x 16 tiles of F in the MFMA
// output layout (tile x, item i, lane l holds F[16 ti + l/16 + 4 i][16 tj +
// l%16]), so that each lane's tagged stores are coalesced.
template <int BP>
struct GramGeom {
  static constexpr int N16 = BP / 16;
  static constexpr int NTL = N16 * (N16 + 1) / 2;
  static constexpr int NSLOT = NTL * 256;
  static constexpr int NEX = NSLOT + BP * BP;   // then the top block
  static __device__ __forceinline__ int tile(int ti, int tj) {
    return ti * N16 - ti * (ti - 1) / 2 + (tj - ti);
  }
  // Slot of F[r][c] (either orientation).
  static __device__ __forceinline__ int slot(int r, int c) {
    int a = r, b = c;
    if ((a >> 4) > (b >> 4) || ((a >> 4) == (b >> 4) && a > b)) {
      a = c;
      b = r;
    }
    const int ra = a & 15, cb = b & 15;
    return tile(a >> 4, b >> 4) * 256 + (ra >> 2) * 64 + (ra & 3) * 16 + cb;
  }
};

template <int BP, int RPT, int NT>
struct GramLds {
  static constexpr int GR = NT / BP;
  double S[BP][BP + 2];         // staged rows for the Gram sums
  double top[BP][BP + 2];       // rows 0..b-1 of X; above the diagonal of finished
                                // rows p: v_p^T v_c (c > p), for T
  double xs[GR][RPT + 2];       // column j at each row group's rows
  double ujv[2][BP];            // column j of F, by step parity
  double fdiag[2];              // F[j+1][j+1] before step j, by parity
  double cw[BP], zv[BP], xt[BP], nu[BP], tau[BP];
  double colscale[BP];          // 1 / (alpha - beta) of finished columns, else 1
  double red2[NT];
};

template <int BP, int RPT, int NT>
__device__ __forceinline__ void panel_gram_body(const GramPanelArgs& ga, const int w) {
  typedef GramGeom<BP> Geo;
  constexpr int GR = NT / BP;
  constexpr int RW = GR * RPT;
  constexpr int QC = BP / GR;        // register slots per staged chunk of BP rows
  constexpr int BC = BP / 16;        // F block per thread: BR rows x BC columns,
  constexpr int BR = BP * BP / NT / BC;   // 16 blocks across, NT / 16 down
  constexpr int QJ = (BP + GR - 1) / GR;
  constexpr int NW = NT / 64;        // wavefronts
  constexpr int NTW = (Geo::NTL + NW - 1) / NW;   // Gram tiles per wavefront
  static_assert(RPT % QC == 0 && RW >= BP, "panel shape");
  static_assert(BR >= 1 && BR * BC * NT == BP * BP, "F blocks");
  __shared__ GramLds<BP, RPT, NT> L;

  const PanelArgs& a = ga.p;
  const int t = threadIdx.x;
  const int k = t % BP, g = t / BP;           // register layout (column k, row group g)
  const int bi = t / 16, bj = t % 16;         // F / top block (rows BR bi.., cols BC bj..)
  const int wv = t / 64, l16 = (t % 64) / 16, m16 = t % 16;   // MFMA lane roles
  const int64_t base = (int64_t)w * RW;
  const int b = a.b, G = a.G;
  const bool forced = waits_forced(a.st);

  double col[RPT];
  {
    const double* Yk = a.Y + base + g + (int64_t)k * a.ldy;
#pragma unroll
    for (int q = 0; q < RPT; ++q) col[q] = Yk[GR * q];
  }
  if (t < BP) L.colscale[t] = 1.0;
  double Fr[BR][BC];
  int tti[NTW], ttj[NTW];
#pragma unroll
  for (int x = 0; x < NTW; ++x) {
    int r = wv + NW * x;
    tti[x] = -1;
    ttj[x] = -1;
    for (int i = 0; i < Geo::N16; ++i) {
      if (r < Geo::N16 - i) {
        tti[x] = i;
        ttj[x] = i + r;
        break;
      }
      r -= Geo::N16 - i;
    }
  }

  unsigned exch = 0;
  // F (rows > j0) from the current rows: MFMA partial sums over this
  // workgroup's rows (workgroup 0's rows j0+1 .. b-1 went through the same
  // updates as the top block), reduced in two phases (workgroup w sums its
  // slice of slots over all workgroups, then every workgroup reads the slots
  // of its F entries).  The first call also distributes workgroup 0's rows
  // 0 .. b-1 as the top block.
  auto form_gram = [&](const int j0, const bool first) __attribute__((always_inline)) {
    const unsigned epoch = a.epoch_base + 1u + exch;
    const int par = (int)(exch & 1u);
    ++exch;
    d4_t acc[NTW];
#pragma unroll
    for (int x = 0; x < NTW; ++x) acc[x] = d4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int c = 0; c < RPT / QC; ++c) {
      __syncthreads();
#pragma unroll
      for (int qq = 0; qq < QC; ++qq) {
        const int q = c * QC + qq;
        const int64_t r = base + g + GR * q;
        L.S[g + GR * qq][k] = (r <= j0) ? 0.0 : col[q] * L.colscale[k];
      }
      __syncthreads();
#pragma unroll
      for (int x = 0; x < NTW; ++x) {
        if (tti[x] >= 0) {
#pragma unroll 4
          for (int s4 = 0; s4 < BP / 4; ++s4) {
            const double av = L.S[4 * s4 + l16][16 * tti[x] + m16];
            const double bv = L.S[4 * s4 + l16][16 * ttj[x] + m16];
            acc[x] = Mfma<double>::op(av, bv, acc[x]);
          }
        }
      }
    }
    {
      u64* dst = ga.part + ((int64_t)par * G + w) * Geo::NSLOT * 2;
#pragma unroll
      for (int x = 0; x < NTW; ++x) {
        if (tti[x] >= 0) {
          const int tl = Geo::tile(tti[x], ttj[x]);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            put_tagged(&dst[(tl * 256 + i * 64 + (t % 64)) * 2], acc[x][i], epoch);
        }
      }
    }
    if (first && w == 0) {
#pragma unroll
      for (int q = 0; q < QJ; ++q) {
        const int r = g + GR * q;
        if (r < b)
          put_tagged(&ga.sums[((int64_t)par * Geo::NEX + Geo::NSLOT + r * BP + k) * 2], col[q], epoch);
      }
    }
    // Phase 2: this workgroup's slice of slots, summed over all workgroups
    // in a fixed order (nsub threads per slot, then in LDS).
    {
      constexpr int NS = Geo::NSLOT;
      const int se = (NS + G - 1) / G;
      const int e0 = w * se;
      const int ne = max(0, min(NS, e0 + se) - e0);
      const int nsub = max(1, min(16, NT / max(ne, 1)));
      const int per = NT / nsub;
      for (int p0 = 0; p0 < ne; p0 += per) {
        const int el = p0 + t % per, sub = t / per;
        double s = 0.0;
        if (el < ne && sub < nsub) {
          const u64* src = ga.part + ((int64_t)par * G * NS + e0 + el) * 2;
          unsigned spins = 0;
          for (int w0 = sub; w0 < G; w0 += 8 * nsub) {
            u64 hi[8], lo[8];
            bool ok;
            do {
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                const int ww = w0 + u * nsub;
                const u64* q = src + (int64_t)(ww < G ? ww : 0) * NS * 2;
                hi[u] = get_word(q);
                lo[u] = get_word(q + 1);
              }
              ok = true;
#pragma unroll
              for (int u = 0; u < 8; ++u) ok = ok && tagged(hi[u], epoch) && tagged(lo[u], epoch);
            } while ((!ok || forced) && keep_waiting(&spins, a.st));
#pragma unroll
            for (int u = 0; u < 8; ++u)
              if (w0 + u * nsub < G) s += untag(hi[u], lo[u]);
          }
        }
        L.red2[t] = s;
        __syncthreads();
        if (t < per && p0 + t < ne) {
          double tot = 0.0;
          for (int sb = 0; sb < nsub; ++sb) tot += L.red2[sb * per + t];
          put_tagged(&ga.sums[((int64_t)par * Geo::NEX + e0 + p0 + t) * 2], tot, epoch);
        }
        __syncthreads();
      }
    }
    // Phase 3: every thread reads the sums of its F entries (and, the first
    // time, its entries of the top block).
    {
      constexpr int NQ = BR * BC;
      unsigned spins = 0;
      auto fetch = [&](const bool topblk) __attribute__((always_inline)) {
        u64 hi[NQ], lo[NQ];
        bool ok;
        do {
#pragma unroll
          for (int i = 0; i < BR; ++i)
#pragma unroll
            for (int jj = 0; jj < BC; ++jj) {
              const int r = BR * bi + i, c = BC * bj + jj;
              const int idx = (topblk && r < b) ? Geo::NSLOT + r * BP + c : Geo::slot(r, c);
              const u64* q = ga.sums + ((int64_t)par * Geo::NEX + idx) * 2;
              hi[i * BC + jj] = get_word(q);
              lo[i * BC + jj] = get_word(q + 1);
            }
          ok = true;
#pragma unroll
          for (int i = 0; i < NQ; ++i) ok = ok && tagged(hi[i], epoch) && tagged(lo[i], epoch);
        } while ((!ok || forced) && keep_waiting(&spins, a.st));
#pragma unroll
        for (int i = 0; i < BR; ++i)
#pragma unroll
          for (int jj = 0; jj < BC; ++jj) {
            const double v = untag(hi[i * BC + jj], lo[i * BC + jj]);
            if (!topblk) Fr[i][jj] = v;
            else L.top[BR * bi + i][BC * bj + jj] = (BR * bi + i < b) ? v : 0.0;
          }
      };
      fetch(false);
      if (first) fetch(true);
    }
  };

  // Exports for step jn (parity pn) by the owners of the entries: column jn
  // of F, and F[jn+1][jn+1] (the next pivot's norm before step jn).
  auto export_step = [&](const int jn, const int pn) __attribute__((always_inline)) {
    const int jb = jn / BC, jo = jn % BC;
    const int j1r = (jn + 1) / BR, j1i = (jn + 1) % BR;
    const int j1c = (jn + 1) / BC, j1o = (jn + 1) % BC;
    // jo, j1i, j1o are the same in every thread: the branches below are
    // uniform, and every register index is a constant (no dynamically
    // indexed array).
    if (bj == jb) {
#pragma unroll
      for (int jj = 0; jj < BC; ++jj)
        if (jj == jo)
#pragma unroll
          for (int i = 0; i < BR; ++i) L.ujv[pn][BR * bi + i] = Fr[i][jj];
    }
    if (bi == j1r && bj == j1c) {
#pragma unroll
      for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int jj = 0; jj < BC; ++jj)
          if (i == j1i && jj == j1o) L.fdiag[pn] = Fr[i][jj];
    }
  };
  // dlarfg scalars of a step from alpha = top[j][j] and ||x||^2 = F[j][j]
  // (every thread computes them from the same values); flag: the downdated
  // norm has cancelled and F must be formed again first.
  auto scalars = [&](const double alpha, const double xn2, const double nuj, const bool fresh,
                     double& flag, double& tau_j, double& scale) __attribute__((always_inline)) {
    flag = 0.0;
    tau_j = 0.0;
    scale = 0.0;
    if (!fresh && nuj > 0.0 && !(xn2 >= kGramTheta * nuj)) {
      flag = 1.0;
    } else if (xn2 > 0.0) {
      const double nrm = sqrt(alpha * alpha + xn2);
      const double beta = (alpha >= 0.0) ? -nrm : nrm;
      tau_j = (beta - alpha) / beta;
      scale = 1.0 / (alpha - beta);
    }
  };
  // After a Gram formation at j0: exports, then the reference norms
  // nu_c = F[c][c] + top[j0][c]^2 (the column's norm^2 over rows >= j0).
  double s_flag = 0.0, s_tau = 0.0, s_scale = 0.0;   // scalars of the next step
  auto after_form = [&](const int j0) __attribute__((always_inline)) {
    export_step(j0, j0 & 1);
    __syncthreads();
    scalars(L.top[j0][j0], L.ujv[j0 & 1][j0], 0.0, true, s_flag, s_tau, s_scale);
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
      for (int jj = 0; jj < BC; ++jj) {
        const int r = BR * bi + i, c = BC * bj + jj;
        if (r == c) L.nu[c] = Fr[i][jj] + L.top[j0][c] * L.top[j0][c];
      }
    __syncthreads();
  };

  form_gram(0, true);
  after_form(0);
  int j = 0;
  // Column steps in an inner loop of their own; a cancelled pivot norm leaves
  // it to form F again (the formation code stays out of the step loop).
  for (;;) {
  while (j < b && s_flag == 0.0) {
    const int p = j & 1;
    const double tau_j = s_tau, scale = s_scale;
    // The next pivot before this step: F[j+1][j+1] and top[j+1][j+1] (row
    // j + 1 is not written before the barrier below).
    const double fd1 = L.fdiag[p];
    const double td1 = (j + 1 < b) ? L.top[j + 1][j + 1] : 0.0;
    // Per column: c_k = tau w_k scale with w_k = v_j^T y_k (k > j), v_p^T v_j
    // (p < j) for T, column j at the top rows below the diagonal, and row
    // j + 1 after this step (removed from F).
    if (t < BP) {
      const int kk = t;
      // Every read first: the only top entry written here, (kk, j) for
      // kk < j, is none of the entries read (rows j and j + 1, and (kk, j)
      // for kk > j), so no read waits for a write.
      const int j1 = (j + 1 < BP) ? j + 1 : j;
      const double tjk = L.top[j][kk], ujk = L.ujv[p][kk], tkj = L.top[kk][j];
      const double xj1 = L.top[j1][j], yk = L.top[j1][kk];
      const double wv2 = tjk + scale * ujk;
      const double cwk = (kk > j && kk < b) ? tau_j * wv2 * scale : 0.0;
      L.cw[kk] = cwk;
      if (kk < j) L.top[kk][j] = wv2;   // v_kk^T v_j, for T
      L.xt[kk] = (kk > j && kk < b) ? tkj : 0.0;
      double zk = 0.0;
      if (j + 1 < b && kk < b)
        zk = (kk > j) ? yk - cwk * xj1 : ((kk == j) ? scale * xj1 : yk);
      L.zv[kk] = zk;
      if (kk == j) {
        L.tau[j] = tau_j;
        L.colscale[j] = scale;
      }
    }
    if (k == j) {
#pragma unroll
      for (int q = 0; q < RPT; ++q) L.xs[g][q] = col[q];
    }
    __syncthreads();
    // Scalars of step j + 1: its pivot after this step, by the formulas of
    // the F and top updates below (every thread, from the same values).
    if (j + 1 < b) {
      const double fjj0 = L.ujv[p][j];
      const double c1 = L.cw[j + 1], u1 = L.ujv[p][j + 1], z1 = L.zv[j + 1];
      double f = fd1 - c1 * u1;
      f = f - c1 * u1;
      f = f + (c1 * c1) * fjj0;
      const double xn2n = f - z1 * z1;
      const double alphan = td1 - c1 * L.xt[j + 1];
      scalars(alphan, xn2n, L.nu[j + 1], false, s_flag, s_tau, s_scale);
    }
    // Apply the step: registers (this workgroup's rows), F and top blocks.
    {
      // Columns k > j lose c_k x_j (c_k = 0 elsewhere).  Column j keeps its
      // unscaled values: v_j = colscale_j x_j is formed where it is read
      // (Gram sums, output).
      const double ck = L.cw[k];
#pragma unroll
      for (int q = 0; q < RPT; ++q) col[q] = col[q] - ck * L.xs[g][q];
    }
    {
      const double fjj = L.ujv[p][j];
      double cwc[BC], ujc[BC], zc[BC];
#pragma unroll
      for (int jj = 0; jj < BC; ++jj) {
        const int c = BC * bj + jj;
        cwc[jj] = L.cw[c];
        ujc[jj] = L.ujv[p][c];
        zc[jj] = L.zv[c];
      }
      const bool top_rows = (BR * bi + BR - 1 > j) && (BR * bi < b);
#pragma unroll
      for (int i = 0; i < BR; ++i) {
        const int r = BR * bi + i;
        const double cwr = L.cw[r], ujr = L.ujv[p][r], zr = L.zv[r];
        const double sr = (r == j) ? scale : 1.0;
#pragma unroll
        for (int jj = 0; jj < BC; ++jj) {
          const int c = BC * bj + jj;
          const double sc = (c == j) ? scale : 1.0;
          double f = Fr[i][jj] - cwc[jj] * ujr;
          f = f - cwr * ujc[jj];
          f = f + (cwr * cwc[jj]) * fjj;
          Fr[i][jj] = (sr * sc) * f - zr * zc[jj];
        }
      }
      if (top_rows) {
#pragma unroll
        for (int i = 0; i < BR; ++i) {
          const int r = BR * bi + i;
          if (r > j && r < b) {
            // The row's entries are read together, then written (each entry
            // belongs to one thread).
            const double xr = L.xt[r];
            double tv[BC];
#pragma unroll
            for (int jj = 0; jj < BC; ++jj) tv[jj] = L.top[r][BC * bj + jj];
#pragma unroll
            for (int jj = 0; jj < BC; ++jj) {
              const int c = BC * bj + jj;
              L.top[r][c] = (c == j) ? scale * xr : tv[jj] - cwc[jj] * xr;
            }
          }
        }
      }
    }
    if (j + 1 < b) export_step(j + 1, p ^ 1);
    __syncthreads();
    ++j;
  }
  if (j >= b) break;
  form_gram(j, false);
  after_form(j);
  }

  // The top block holds rows 0 .. b-1 of V below the diagonal and v_p^T v_c
  // above it.
  // V with explicit unit diagonal and zeros above / beyond b.
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    const int64_t r = base + g + GR * q;
    if (r < a.m) {
      double v = 0.0;
      if (k < b) {
        if (r < b) v = (r > k) ? L.top[r][k] : (r == k ? 1.0 : 0.0);
        else v = col[q] * L.colscale[k];
      }
      a.V[r + k * a.ldv] = v;
    }
  }
  // T (Eq. (4)) from v_p^T v_c and tau: T[c][c] = tau_c, T[i][c] =
  // -tau_i sum_{i < p <= c} (v_i^T v_p) T[p][c] (tau_i = 0 gives a zero row).
  if (w == G - 1 && t < BP) {
    const int c = t;
    double tc[BP];
#pragma unroll
    for (int i = BP - 1; i >= 0; --i) {
      double s0 = 0.0, s1 = 0.0;
#pragma unroll
      for (int pp = i + 1; pp < BP; pp += 2) {
        s0 += ((pp <= c) ? L.top[i][pp] : 0.0) * tc[pp];
        if (pp + 1 < BP) s1 += ((pp + 1 <= c) ? L.top[i][pp + 1] : 0.0) * tc[pp + 1];
      }
      const double ti2 = L.tau[i];
      tc[i] = (c < b && i < c) ? -ti2 * (s0 + s1) : ((c < b && i == c) ? ti2 : 0.0);
    }
#pragma unroll
    for (int i = 0; i < BP; ++i) a.Tm[i + (int64_t)c * a.ldt] = tc[i];
    if (c < b) a.tau[c] = L.tau[c];
  }
}

}  // namespace
}  // namespace rrf
