// Panel Householder QR by tall-skinny QR and Householder reconstruction
// (Alg. 2, geqrt step; same V, tau, T as geqr2 + larft up to rounding).
//
// The column-by-column panel needs one grid-wide reduction per column.  Here
// the panel rows are split into blocks that workgroups factor on their own
// (workgroup-local reductions only); their R factors are stacked and
// factored again, level by level, up to one root (a reduction tree of
// Householder QRs: TSQR).  The explicit orthonormal factor Q (m x b) is
// then formed top-down, and the compact-WY Householder form of the panel is
// recovered from it (Householder reconstruction: an LU factorisation without
// pivoting of Q - S, with S = diag(+-1) chosen on the fly as -sign of the
// current diagonal, gives V = L, U, and T = -U S L_1^{-T}).  The sign choice
// makes the reflectors those of Householder QR with LAPACK's dlarfg
// convention, so V, tau and T agree with the column-by-column panel (and the
// oracle's geqr2 / larft) up to rounding; every factorisation in the tree is
// Householder, so the panel stays unconditionally stable.  Launches: the
// leaves, one per tree level, the top-down pass, the LU, and V = Q U^{-1}.
//
// Thread layout of a block factorisation (as in the column-by-column panel):
// thread t owns column k = t % BP and row group g = t / BP and keeps rows
// g + (256 / BP) q, q < RPT, of its column in registers.

#include "rrf_internal.h"

namespace rrf {
namespace {

template <int BP, int RPT>
struct LocalQR {
  static constexpr int GR = kPanelThreads / BP;
  static constexpr int RW = GR * RPT;
  double xs[RW];
  double rowj[BP];
  double red[GR][BP];
  double tot[BP];
  double Tl[BP][BP + 1];
  double Rl[BP][BP + 1];
  double Ej[BP];
};

// Householder QR (geqr2 semantics, dlarfg convention) of the RW x BP block in
// `col`, columns < b, with workgroup-local reductions.  Afterwards col holds V
// (unit lower trapezoidal with explicit ones and zeros; columns >= b zero),
// s.Rl the R factor and s.Tl the forward columnwise T factor (zero outside
// b x b).  One reduction per column gives ||x||^2, v_j^T y_k and v_p^T v_j at
// once (v_j = [1; x / (alpha - beta)]), as in the column-by-column panel.
template <int BP, int RPT>
__device__ __forceinline__ void local_qr(double (&col)[RPT], const int b,
                                         LocalQR<BP, RPT>& s) {
  constexpr int GR = LocalQR<BP, RPT>::GR;
  constexpr int QJ = (BP + GR - 1) / GR;   // registers that can hold rows < BP
  const int t = threadIdx.x, k = t % BP, g = t / BP;
  for (int idx = t; idx < BP * (BP + 1); idx += kPanelThreads) {
    (&s.Rl[0][0])[idx] = 0.0;
    (&s.Tl[0][0])[idx] = 0.0;
  }
  for (int j = 0; j < b; ++j) {
    // Column j with rows <= j zeroed, and row j of every column.
    if (k == j) {
#pragma unroll
      for (int q = 0; q < RPT; ++q)
        s.xs[g + GR * q] = (q < QJ && g + GR * q <= j) ? 0.0 : col[q];
    }
    if (g == j % GR) {
      const int qj = j / GR;
      double v = 0.0;
#pragma unroll
      for (int q = 0; q < QJ; ++q) v = (q == qj) ? col[q] : v;
      s.rowj[k] = v;
    }
    __syncthreads();
    double d0 = 0.0, d1 = 0.0, d2 = 0.0, d3 = 0.0;
#pragma unroll
    for (int q = 0; q < RPT; q += 4) {
      d0 += col[q] * s.xs[g + GR * q];
      if (q + 1 < RPT) d1 += col[q + 1] * s.xs[g + GR * (q + 1)];
      if (q + 2 < RPT) d2 += col[q + 2] * s.xs[g + GR * (q + 2)];
      if (q + 3 < RPT) d3 += col[q + 3] * s.xs[g + GR * (q + 3)];
    }
    s.red[g][k] = (d0 + d1) + (d2 + d3);
    __syncthreads();
    if (t < BP) {
      double sum = 0.0;
#pragma unroll
      for (int gg = 0; gg < GR; ++gg) sum += s.red[gg][t];
      s.tot[t] = sum;
    }
    __syncthreads();
    // dlarfg scalars (identical in every thread).
    const double alpha = s.rowj[j];
    const double xi2 = s.tot[j];
    double tau_j = 0.0, scale = 0.0, beta = alpha;
    if (xi2 != 0.0) {
      const double nrm = sqrt(alpha * alpha + xi2);
      beta = (alpha >= 0.0) ? -nrm : nrm;
      tau_j = (beta - alpha) / beta;
      scale = 1.0 / (alpha - beta);
    }
    // Row j of R: R[j][j] = beta, R[j][k] = y_k[j] - tau_j (v_j^T y_k).
    // v_p^T v_j = V[j][p] + scale * dot_p for the new column of T.
    if (t < BP) {
      if (t == j) s.Rl[j][j] = beta;
      else if (t > j && t < b) s.Rl[j][t] = s.rowj[t] - tau_j * (s.rowj[t] + scale * s.tot[t]);
      if (t < j) s.Ej[t] = s.rowj[t] + scale * s.tot[t];
    }
    if (k == j) {
#pragma unroll
      for (int q = 0; q < RPT; ++q) col[q] = col[q] * scale;
    } else if (k > j && k < b) {
      const double fs = tau_j * (s.rowj[k] + scale * s.tot[k]) * scale;
#pragma unroll
      for (int q = 0; q < RPT; ++q) col[q] = col[q] - fs * s.xs[g + GR * q];
    }
    __syncthreads();
    // Column j of T: T[:j, j] = -tau_j T[:j, :j] (V^T v_j), T[j][j] = tau_j.
    if (t < j) {
      double acc = 0.0;
      for (int p = t; p < j; ++p) acc += s.Tl[t][p] * s.Ej[p];
      s.Tl[t][j] = -tau_j * acc;
    } else if (t == j) {
      s.Tl[j][j] = tau_j;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    const int r = g + GR * q;
    double v = 0.0;
    if (k < b) v = (r > k) ? col[q] : (r == k ? 1.0 : 0.0);
    col[q] = v;
  }
}

// One tree level: node w factors rows [w RW, (w + 1) RW) of `in` (rows at or
// past in_rows read as zero) and writes its V block, M = T V_top^T (BP x BP,
// column-major) and its R factor (rows [w BP, (w + 1) BP) of the next stack).
template <int BP, int RPT>
__global__ __launch_bounds__(kPanelThreads) void tsqr_qr_kernel(TsqrLevelArgs a) {
  constexpr int GR = LocalQR<BP, RPT>::GR;
  constexpr int RW = LocalQR<BP, RPT>::RW;
  constexpr int QJ = (BP + GR - 1) / GR;
  static_assert(RW >= BP, "a block holds at least BP rows");
  __shared__ LocalQR<BP, RPT> s;
  __shared__ double Vt[BP][BP + 1];
  const int t = threadIdx.x, k = t % BP, g = t / BP;
  const int64_t base = (int64_t)blockIdx.x * RW;

  // Clamped addresses and a mask multiply keep the loads unconditional.
  double col[RPT];
  {
    const int64_t last = a.in_rows - 1;
    const double* ink = a.in + (int64_t)k * a.ldin;
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      const int64_t r = base + g + GR * q;
      const double msk = (r < a.in_rows && k < a.b) ? 1.0 : 0.0;
      col[q] = msk * ink[r < a.in_rows ? r : last];
    }
  }
  __syncthreads();   // every thread has read its rows (V may overwrite `in`)
  local_qr<BP, RPT>(col, a.b, s);

#pragma unroll
  for (int q = 0; q < RPT; ++q)
    a.V[base + g + GR * q + (int64_t)k * a.ldv] = col[q];
#pragma unroll
  for (int q = 0; q < QJ; ++q) {
    const int r = g + GR * q;
    if (r < BP) Vt[r][k] = col[q];
  }
  __syncthreads();
  // M[p][c] = sum_q T[p][q] V_top[c][q]; T upper (q >= p), V_top unit lower
  // (q <= c), so q runs over [p, c].
  double* M = a.M + (int64_t)blockIdx.x * BP * BP;
  for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
    const int p = idx % BP, c = idx / BP;
    double acc = 0.0;
    for (int q = p; q <= c; ++q) acc += s.Tl[p][q] * Vt[c][q];
    M[p + c * BP] = acc;
  }
  for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
    const int i = idx % BP, j = idx / BP;
    a.R[(int64_t)blockIdx.x * BP + i + (int64_t)j * a.ldr] = s.Rl[i][j];
  }
}

// Top-down pass: leaf w forms its rows of the explicit Q.  With X_root = I,
// a node's explicit factor restricted to child c's rows is
// (E_c - V[c rows] M) X_node (E_c: rows c BP.. of [I; 0]), which is the
// child's X; the leaf's rows of Q are (E - V_leaf M_leaf) X_leaf.
template <int BP, int RPTL>
__global__ __launch_bounds__(kPanelThreads) void tsqr_back_kernel(TsqrBackArgs a) {
  constexpr int GR = kPanelThreads / BP;
  constexpr int RWL = GR * RPTL;
  constexpr int CH = 32;   // leaf rows staged per pass
  static_assert(RWL % CH == 0 && CH % GR == 0, "leaf staging");
  __shared__ double X[BP][BP + 1];
  __shared__ double Y2[BP][BP + 1];
  __shared__ double Ml[BP][BP + 1];
  __shared__ double Vr[CH > BP ? CH : BP][BP + 1];
  const int t = threadIdx.x;
  const int w = blockIdx.x;
  for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
    const int i = idx % BP, j = idx / BP;
    X[i][j] = (i == j) ? 1.0 : 0.0;
  }
  int64_t div = 1;   // leaves per node one level below the current one
  for (int l = 1; l < a.nlev; ++l) div *= a.F;
  for (int l = a.nlev; l >= 1; --l) {
    const int64_t node = w / (div * a.F);
    const int c = (int)((w / div) % a.F);
    const double* Vn = a.Vlev[l - 1] + node * a.rwi + (int64_t)c * BP;
    const double* Mn = a.Mlev[l - 1] + node * BP * BP;
    __syncthreads();
    for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
      const int i = idx % BP, p = idx / BP;
      Vr[i][p] = Vn[i + (int64_t)p * a.ldvlev[l - 1]];
      Ml[i][p] = Mn[i + p * BP];
    }
    __syncthreads();
    for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
      const int p = idx % BP, q = idx / BP;
      double acc = 0.0;
      for (int r = 0; r < BP; ++r) acc += Ml[p][r] * X[r][q];
      Y2[p][q] = acc;
    }
    __syncthreads();
    // X <- E_c X - Vr Y2, through Ml (free once Y2 is formed).
    for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
      const int i = idx % BP, q = idx / BP;
      double v = (c == 0) ? X[i][q] : 0.0;
      for (int p = 0; p < BP; ++p) v -= Vr[i][p] * Y2[p][q];
      Ml[i][q] = v;
    }
    __syncthreads();
    for (int idx = t; idx < BP * BP; idx += kPanelThreads) X[idx % BP][idx / BP] = Ml[idx % BP][idx / BP];
    div /= a.F;
  }
  // Leaf: Y2 = M_leaf X, then Q rows = E X - V_leaf Y2.
  __syncthreads();
  {
    const double* Mn = a.Mleaf + (int64_t)w * BP * BP;
    for (int idx = t; idx < BP * BP; idx += kPanelThreads) Ml[idx % BP][idx / BP] = Mn[idx];
  }
  __syncthreads();
  for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
    const int p = idx % BP, q = idx / BP;
    double acc = 0.0;
    for (int r = 0; r < BP; ++r) acc += Ml[p][r] * X[r][q];
    Y2[p][q] = acc;
  }
  const int q = t % BP, g = t / BP;
  const int64_t base = (int64_t)w * RWL;
  for (int r0 = 0; r0 < RWL; r0 += CH) {
    __syncthreads();
    for (int idx = t; idx < CH * BP; idx += kPanelThreads) {
      const int i = idx % CH, p = idx / CH;
      Vr[i][p] = a.Vleaf[base + r0 + i + (int64_t)p * a.ldvl];
    }
    __syncthreads();
    for (int i = g; i < CH; i += GR) {
      const int64_t r = base + r0 + i;
      double v = (r0 + i < BP) ? X[r0 + i][q] : 0.0;
      for (int p = 0; p < BP; ++p) v -= Vr[i][p] * Y2[p][q];
      if (r < a.m) a.Q[r + (int64_t)q * a.ldq] = v;
    }
  }
}

// Householder reconstruction, part 1 (one workgroup): LU without pivoting of
// the top b x b block of Q - S, S_ii = -sign of the current diagonal
// (counting +0 as positive, like dlarfg's beta); then V's top rows
// (the unit lower L_1), U^{-1} for part 2, and T = -U S L_1^{-T}, tau = diag T.
template <int BP>
__global__ __launch_bounds__(kPanelThreads) void hr_lu_kernel(HrArgs a) {
  __shared__ double A[BP][BP + 1];
  __shared__ double Ui[BP][BP + 1];
  __shared__ double Z[BP][BP + 1];
  __shared__ double S[BP];
  const int t = threadIdx.x;
  const int b = a.b;
  for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
    const int r = idx % BP, c = idx / BP;
    A[r][c] = (r < b && c < b) ? a.Q[r + (int64_t)c * a.ldq] : 0.0;
  }
  __syncthreads();
  for (int i = 0; i < b; ++i) {
    if (t == i) {
      const double d = A[i][i];
      const double s = (d >= 0.0) ? -1.0 : 1.0;
      S[i] = s;
      A[i][i] = d - s;
    }
    __syncthreads();
    if (t > i && t < b) {
      const double l = A[t][i] / A[i][i];
      A[t][i] = l;
      for (int c = i + 1; c < b; ++c) A[t][c] -= l * A[i][c];
    }
    __syncthreads();
  }
  // Thread c: column c of U^{-1} (U X = I) and of Z = L_1^{-T} (L_1^T Z = I),
  // by back substitution.
  if (t < BP) {
    const int c = t;
    for (int i = BP - 1; i >= 0; --i) {
      double x = 0.0, z = 0.0;
      if (c < b && i <= c) {
        x = (i == c) ? 1.0 : 0.0;
        z = x;
        for (int p = i + 1; p <= c; ++p) {
          x -= A[i][p] * Ui[p][c];
          z -= A[p][i] * Z[p][c];
        }
        x /= A[i][i];
      }
      Ui[i][c] = x;
      Z[i][c] = z;
    }
  }
  __syncthreads();
  // Outputs.  T[i][c] = -sum_{p in [i, c]} U[i][p] S[p] Z[p][c].  A square
  // panel's last column has no rows below its diagonal: geqr2 leaves it
  // alone (tau = 0, H = I) where the reconstruction would reflect it, and the
  // other reflectors do not depend on that choice, so its column of T is 0.
  const int last_free = (a.m == b) ? b - 1 : -1;
  for (int idx = t; idx < BP * BP; idx += kPanelThreads) {
    const int i = idx % BP, c = idx / BP;
    double tv = 0.0;
    if (c < b && i <= c && c != last_free) {
      for (int p = i; p <= c; ++p) tv -= A[i][p] * S[p] * Z[p][c];
    }
    a.Tm[i + (int64_t)c * a.ldt] = tv;
    if (i == c && c < b) a.tau[c] = tv;
    a.Uinv[i + c * BP] = Ui[i][c];
    if (i < b) {
      double v = 0.0;
      if (c < b) v = (i > c) ? A[i][c] : (i == c ? 1.0 : 0.0);
      a.Q[i + (int64_t)c * a.ldq] = v;   // V's top rows, in place
    }
  }
}

// Householder reconstruction, part 2: rows r >= b of V = Q U^{-1} (in place),
// zero in columns >= b.  One thread per row.
template <int BP>
__global__ __launch_bounds__(256) void hr_v2_kernel(HrArgs a) {
  __shared__ double Ui[BP][BP];
  for (int idx = threadIdx.x; idx < BP * BP; idx += 256) Ui[idx % BP][idx / BP] = a.Uinv[idx];
  __syncthreads();
  const int64_t r = a.b + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r >= a.m) return;
  double qv[BP];
#pragma unroll
  for (int p = 0; p < BP; ++p) qv[p] = (p < a.b) ? a.Q[r + (int64_t)p * a.ldq] : 0.0;
#pragma unroll
  for (int c = 0; c < BP; ++c) {
    double v = 0.0;
#pragma unroll
    for (int p = 0; p <= c; ++p) v += qv[p] * Ui[p][c];
    a.Q[r + (int64_t)c * a.ldq] = (c < a.b) ? v : 0.0;
  }
}

template <int BP>
hipError_t tsqr_go(const PanelArgs& pa, const TsqrShape& sh, double* scratch,
                   hipStream_t s) {
  constexpr int GR = kPanelThreads / BP;
  constexpr int RPTL = kTsqrLeafRpt;
  constexpr int RPTI = kTsqrNodeRows / GR;
  // Scratch: M and R of the leaves, then per level V, M, R; finally U^{-1}.
  double* p = scratch;
  double* Mleaf = p; p += (int64_t)sh.G[0] * BP * BP;
  double* Rcur = p; p += (int64_t)sh.G[0] * BP * BP;
  TsqrLevelArgs la{};
  la.in = pa.Y; la.ldin = pa.ldy; la.in_rows = pa.m;
  la.V = const_cast<double*>(pa.Y); la.ldv = pa.ldy;   // leaf V in place
  la.M = Mleaf; la.R = Rcur; la.ldr = (int64_t)sh.G[0] * BP; la.b = pa.b;
  hipLaunchKernelGGL((tsqr_qr_kernel<BP, RPTL>), dim3(sh.G[0]), dim3(kPanelThreads), 0, s, la);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  TsqrBackArgs ba{};
  for (int l = 1; l <= sh.nlev; ++l) {
    TsqrLevelArgs li{};
    li.in = Rcur; li.ldin = (int64_t)sh.G[l - 1] * BP; li.in_rows = (int64_t)sh.G[l - 1] * BP;
    double* Vl = p; p += (int64_t)sh.G[l] * kTsqrNodeRows * BP;
    double* Ml = p; p += (int64_t)sh.G[l] * BP * BP;
    double* Rl = p; p += (int64_t)sh.G[l] * BP * BP;
    li.V = Vl; li.ldv = (int64_t)sh.G[l] * kTsqrNodeRows;
    li.M = Ml; li.R = Rl; li.ldr = (int64_t)sh.G[l] * BP; li.b = pa.b;
    hipLaunchKernelGGL((tsqr_qr_kernel<BP, RPTI>), dim3(sh.G[l]), dim3(kPanelThreads), 0, s, li);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    ba.Vlev[l - 1] = Vl; ba.ldvlev[l - 1] = li.ldv; ba.Mlev[l - 1] = Ml;
    Rcur = Rl;
  }
  ba.Vleaf = pa.Y; ba.ldvl = pa.ldy; ba.Mleaf = Mleaf;
  ba.nlev = sh.nlev; ba.F = sh.F; ba.rwi = kTsqrNodeRows;
  ba.Q = pa.V; ba.ldq = pa.ldv; ba.m = pa.m;
  hipLaunchKernelGGL((tsqr_back_kernel<BP, RPTL>), dim3(sh.G[0]), dim3(kPanelThreads), 0, s, ba);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  HrArgs ha{};
  ha.Q = pa.V; ha.ldq = pa.ldv; ha.m = pa.m; ha.b = pa.b;
  ha.Tm = pa.Tm; ha.ldt = pa.ldt; ha.tau = pa.tau; ha.Uinv = p;
  hipLaunchKernelGGL((hr_lu_kernel<BP>), dim3(1), dim3(kPanelThreads), 0, s, ha);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (pa.m > pa.b) {
    const unsigned nb = (unsigned)ceil_div(pa.m - pa.b, 256);
    hipLaunchKernelGGL((hr_v2_kernel<BP>), dim3(nb), dim3(256), 0, s, ha);
    e = hipGetLastError();
  }
  (void)RPTI;
  return e;
}

}  // namespace

bool tsqr_shape(int64_t m, int b, TsqrShape* out) {
  if (b < 1 || b > kMaxBlock || m < b) return false;
  const int bp = pad16(b);
  const int gr = kPanelThreads / bp;
  TsqrShape sh{};
  sh.bp = bp;
  sh.F = kTsqrNodeRows / bp;
  sh.G[0] = (int)ceil_div(m, (int64_t)gr * kTsqrLeafRpt);
  sh.nlev = 0;
  while (sh.G[sh.nlev] > 1) {
    if (sh.nlev + 1 >= kTsqrMaxLev) return false;
    sh.G[sh.nlev + 1] = (int)ceil_div(sh.G[sh.nlev], sh.F);
    ++sh.nlev;
  }
  int64_t elems = 2 * (int64_t)sh.G[0] * bp * bp;
  for (int l = 1; l <= sh.nlev; ++l)
    elems += (int64_t)sh.G[l] * kTsqrNodeRows * bp + 2 * (int64_t)sh.G[l] * bp * bp;
  elems += (int64_t)bp * bp;
  sh.scratch_elems = elems;
  sh.rows_pad = (int64_t)sh.G[0] * gr * kTsqrLeafRpt;
  *out = sh;
  return true;
}

hipError_t launch_panel_tsqr(const PanelArgs& a, const TsqrShape& sh, double* scratch,
                             hipStream_t s) {
  switch (sh.bp) {
    case 16: return tsqr_go<16>(a, sh, scratch, s);
    case 32: return tsqr_go<32>(a, sh, scratch, s);
    case 64: return tsqr_go<64>(a, sh, scratch, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace rrf
