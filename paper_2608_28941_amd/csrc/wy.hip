// Blocked WY reflector application (Alg. 2, update step) and the fused sample
// of the next sketch block.
//
// The block update B <- Q_i^T B = B - V_i T_i^T (V_i^T B) (Theorem 3.1:
// A~ = Q_1^T A; compact WY form Eq. (4)) runs as three kernels:
//   reduce  Z_s = V_i^T B[rows of split s, :]      (b x n per split)
//   formW   W   = T_i^T sum_s Z_s                  (b x n)
//   update  B  -= V_i W, and in the same pass over B
//           P   = B_new Omega_{i+1}  (next sample, Alg. 2 sketch/qr steps)
//           ||B_new[rows < s0]||^2, ||B_new[rows >= s0]||^2  (Alg. 2 E step,
//           fused as the paper's outlook suggests)
// With trans = 0 the same kernels apply Q_i = I - V_i T_i V_i^T (explicit Q).
//
// Both GEMM-shaped kernels run on MFMA 16x16x4 (f64 or f32).  V and T are
// kept in binary64 for both dtypes; the f32 kernels round V on load.  They are
// written in the transposed frame so that the 16 lanes of an MFMA column index
// consecutive rows of the column-major B: each wavefront load or store then
// touches 16 contiguous rows (128 B of f64) of 4 columns.
//   update: a wavefront owns 16 rows; its slice of V (16 x b) stays in
//           registers for the whole sweep over the columns; W and Omega
//           chunks are staged in LDS and shared by the 4 wavefronts.
//   reduce: a wavefront owns 16 columns and all b reflectors; V rows are
//           staged in LDS and shared; B is read straight into registers.

#include <type_traits>

#include "gather_body.h"
#include "mfma.h"
#include "rrf_internal.h"
#include "update_body.h"

namespace rrf {
namespace {

// ---------------------------------------------------------------------------
// reduce: Z_s[c * BP + p] = sum_{r in split s} V[r, p] X[r, c]
// grid (ceil(n / (64 CT)), nsplit), 256 threads; V is staged in chunks of
// RC rows.
//
// An MFMA operand puts the summation index (rows of X) on the 4 lane groups
// and 16 columns on the lanes of a group, so a scalar load of X touches 16
// columns with 4 rows (32 B for f64) each.  With VEC > 1 every lane loads VEC
// consecutive rows in one 16-byte load (64 B per column per instruction) and
// feeds them to VEC MFMA steps; the K order is permuted accordingly (row
// offset 4 VEC u + VEC g + h for load u, lane group g, element h), and the
// staged V rows are read in the same order.  VEC > 1 needs X, ldx and mr
// aligned to VEC elements (the host checks).
// ---------------------------------------------------------------------------
template <typename T, int VEC>
struct alignas(sizeof(T) * VEC) XPack {
  T v[VEC];
};

template <typename T, int BP, int VEC, int CT, int RC>
__global__ __launch_bounds__(256, 2) void reduce_kernel(ReduceArgs<T> a) {
  typedef typename Mfma<T>::acc_t acc_t;
  typedef XPack<T, VEC> pack_t;
  constexpr int NPT = BP / 16;
  constexpr int LDV = RC + 1;
  constexpr int GR = 4 * VEC;              // rows of one load per column
  constexpr int NX = RC / GR;              // loads per lane per chunk and tile
  constexpr int PSTEP = 256 / RC;          // reflectors staged per pass
  constexpr int NIT = (BP * RC) / 256;     // V values per thread per chunk
  static_assert(RC % GR == 0 && kRedChunk % RC == 0 && 256 % RC == 0 &&
                (BP * RC) % 256 == 0, "chunk shape");
  constexpr int COLS = 64 * CT;            // columns per workgroup
  // Staged V rows, double buffered (chunk c in buffer c % 2): one barrier per
  // chunk orders the reads of a buffer before its next overwrite and the
  // writes before the next reads.
  __shared__ T vl[2][BP * LDV];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  // Wavefront w owns CT adjacent 16-column tiles; every staged V value read
  // from LDS feeds CT MFMAs.
  const int64_t cb = (int64_t)blockIdx.x * COLS + 16 * CT * wave;
  const int64_t r_begin = (int64_t)blockIdx.y * a.rows_per_split;
  const int64_t r_end = min(a.mr, r_begin + a.rows_per_split);
  const T* Xc[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) {
    const int64_t col = cb + 16 * ct + m16;
    Xc[ct] = a.X + (col < a.n ? col : a.n - 1) * a.ldx;
  }

  acc_t acc[CT][NPT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int pt = 0; pt < NPT; ++pt) acc[ct][pt] = Mfma<T>::zero();

  // Loads are unconditional from clamped in-bounds addresses (the last whole
  // pack of the column); rows past r_end are cancelled by zero V rows (mask
  // multiply, so the compiler cannot turn the loads into branches), columns
  // past n are not stored.  The next chunk's X packs and V rows are loaded
  // into registers while the current chunk computes; after a barrier the V
  // rows go to LDS.  Those waits sit after the compute in straight-line code.
  // The last chunk prefetches itself again (harmless, keeps loads
  // unconditional).
  const int64_t xlast = a.mr - VEC;
  const int64_t rlast = a.mr - 1;
  const int64_t R_last = r_begin + (r_end - r_begin - 1) / RC * RC;
  const int rr = threadIdx.x % RC;
  const int p0 = threadIdx.x / RC;
  pack_t xcur[CT][NX], xnxt[CT][NX];
  double vt[NIT];
  auto load_x = [&](int64_t R, pack_t (*xd)[NX]) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int u = 0; u < NX; ++u) {
        const int64_t r = R + GR * u + VEC * g;
        xd[ct][u] = *reinterpret_cast<const pack_t*>(Xc[ct] + (r < xlast ? r : xlast));
      }
  };
  auto load_v = [&](int64_t R) {
    const int64_t r = R + rr;
    const double* Vr = a.V + (r < r_end ? r : rlast);
#pragma unroll
    for (int it = 0; it < NIT; ++it) vt[it] = Vr[(int64_t)(p0 + PSTEP * it) * a.ldv];
  };
  auto stage_v = [&](int64_t R, T* vb) {
    const double mask = R + rr < r_end ? 1.0 : 0.0;
#pragma unroll
    for (int it = 0; it < NIT; ++it) vb[(p0 + PSTEP * it) * LDV + rr] = (T)(mask * vt[it]);
  };

  load_x(r_begin, xcur);
  load_v(r_begin);
  stage_v(r_begin, vl[0]);
  __syncthreads();
  // One chunk from buffer CUR (a compile-time constant: the loop is unrolled
  // by two so that both buffers have fixed LDS offsets).
  auto chunk = [&](const int64_t R, auto cur_tag) {
    constexpr int CUR = decltype(cur_tag)::value;
    const T* vc = vl[CUR];
    const int64_t Rn = min(R + RC, R_last);
    load_x(Rn, xnxt);
    load_v(Rn);
#pragma unroll
    for (int u = 0; u < NX; ++u) {
#pragma unroll
      for (int h = 0; h < VEC; ++h) {
        const int k = GR * u + VEC * g + h;
#pragma unroll
        for (int pt = 0; pt < NPT; ++pt) {
          const T bv = vc[(pt * 16 + m16) * LDV + k];
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
            acc[ct][pt] = Mfma<T>::op(xcur[ct][u].v[h], bv, acc[ct][pt]);
        }
      }
    }
    stage_v(Rn, vl[CUR ^ 1]);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int u = 0; u < NX; ++u) xcur[ct][u] = xnxt[ct][u];
    __syncthreads();
  };
  for (int64_t R = r_begin; R < r_end; R += 2 * RC) {
    chunk(R, std::integral_constant<int, 0>());
    if (R + RC < r_end) chunk(R + RC, std::integral_constant<int, 1>());
  }
  // Lane holds Z^T[c = cb + 16 ct + drow(g, i)][p = pt * 16 + m16].
  T* Z = a.Z + (int64_t)blockIdx.y * a.split_stride;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int pt = 0; pt < NPT; ++pt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t c = cb + 16 * ct + Mfma<T>::drow(g, i);
        if (c < a.n) Z[c * BP + pt * 16 + m16] = acc[ct][pt][i];
      }
    }
}

// ---------------------------------------------------------------------------
// formW: W[c * BP + p] = (T^T z_c)_p (trans) or (T z_c)_p, z_c = sum_s Z_s[c]
// Only the leading b x b block of T is used (the padding columns of a stored
// block may already hold the next block's T), so W rows >= b are zero.
// Workgroups past the first a.nfw gather the look-ahead sample instead (one
// per 256 rows of one column, as the gather kernel).
// ---------------------------------------------------------------------------
template <typename T, int BP>
__global__ __launch_bounds__(256) void formw_kernel(FormWArgs<T> a) {
  if ((int)blockIdx.x >= a.nfw) {   // uniform
    const int64_t gi = (int64_t)blockIdx.x - a.nfw;
    const int64_t nrb = (a.g.rows_pad + 255) / 256;
    const int k = (int)(gi / nrb);
    const int64_t r = (gi % nrb) * 256 + threadIdx.x;
    if (r < a.g.rows_pad && k < a.g.bp) gather_entry(a.g, r, k);
    return;
  }
  constexpr int CPB = 256 / BP;
  constexpr int NT = (BP * BP) / 256;
  constexpr int ZB = 8;                // split partials loaded together
  __shared__ double Tl[BP][BP + 1];
  __shared__ double zs[CPB][BP + 1];
  // T to LDS: all loads issued before the first use (in-bounds addresses:
  // columns past b read column 0), entries outside the upper b x b triangle
  // replaced by zero.
  {
    double tv[NT];
#pragma unroll
    for (int it = 0; it < NT; ++it) {
      const int idx = threadIdx.x + 256 * it;
      const int i = idx % BP, j = idx / BP;
      tv[it] = a.Tm[i + (int64_t)(j < a.b ? j : 0) * a.ldt];
    }
#pragma unroll
    for (int it = 0; it < NT; ++it) {
      const int idx = threadIdx.x + 256 * it;
      const int i = idx % BP, j = idx / BP;
      Tl[i][j] = (i <= j && j < a.b) ? tv[it] : 0.0;
    }
  }
  const int p = threadIdx.x % BP, cl = threadIdx.x / BP;
  // Rows [n, round_up(n, kUpdChunk)) of W are written as zeros so the update
  // can stage whole chunks without predicates.
  const int64_t n_pad = (a.n + kUpdChunk - 1) / kUpdChunk * kUpdChunk;
  for (int64_t c0 = (int64_t)blockIdx.x * CPB; c0 < n_pad;
       c0 += (int64_t)a.nfw * CPB) {
    __syncthreads();
    const int64_t c = c0 + cl;
    // z_c = sum over the splits in split order, ZB loads in flight at a time
    // (clamped split index, surplus loads not added).
    const T* zp = a.Z + (c < a.n ? c : 0) * BP + p;
    double z = 0.0;
    for (int s0 = 0; s0 < a.nsplit; s0 += ZB) {
      T v[ZB];
#pragma unroll
      for (int u = 0; u < ZB; ++u)
        v[u] = zp[(int64_t)min(s0 + u, a.nsplit - 1) * a.split_stride];
#pragma unroll
      for (int u = 0; u < ZB; ++u)
        if (s0 + u < a.nsplit) z += (double)v[u];
    }
    zs[cl][p] = c < a.n ? z : 0.0;
    __syncthreads();
    // Four independent partial sums (the terms past the triangle are zero in
    // Tl), added in a fixed order.
    double w4[4] = {0.0, 0.0, 0.0, 0.0};
    if (a.trans) {
      for (int l = 0; l <= p; l += 4)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (l + u < BP) w4[u] += Tl[l + u][p] * zs[cl][l + u];
    } else {
      for (int l = p & ~3; l < BP; l += 4)
#pragma unroll
        for (int u = 0; u < 4; ++u) w4[u] += Tl[p][l + u] * zs[cl][l + u];
    }
    const double w = (w4[0] + w4[1]) + (w4[2] + w4[3]);
    if (c < n_pad) a.W[c * BP + p] = (T)w;
  }
}

// formW at 128 reflectors, W = T z_c (the explicit-Q pass of a block group):
// one workgroup per tile of CW columns (CW = 4, 8 or 16, chosen so that
// narrow passes still spread over many compute units).
// * The tile's split partials are summed in split order, as in formw_kernel,
//   16 loads of 16 bytes in flight per thread, and z goes to LDS.
// * The product with the upper b x b triangle of T runs on MFMA 16x16x4:
//   D rows are the tile's columns c (rows >= CW zero), D columns 16 values
//   of p, K the index l.  Wave w takes the p-tiles w and 7 - w, 36 K-steps
//   of 4 between them (l >= p, so tile pt needs l >= 16 pt only).
// * Its T operand, T[p][l] with p <= l < b, is loaded at the start, beside
//   the partials.
template <int CW>
__global__ __launch_bounds__(256) void formw128_kernel(FormWArgs<double> a) {
  constexpr int BP = 128;
  constexpr int PK = CW * BP / 2 / 256;  // 16-byte packs per thread per split
  constexpr int SB = 16 / PK;            // splits in flight
  constexpr int NS = 36;                 // K-steps per wave
  __shared__ double zs[16][BP + 1];
  const int t = threadIdx.x, w = t >> 6, lane = t & 63, g = lane >> 4, m = lane & 15;
  const int64_t c0 = (int64_t)blockIdx.x * CW;
  // T operand: steps [0, nA) belong to p-tile w, the rest to p-tile 7 - w.
  const int nA = 32 - 4 * w;
  double bv[NS];
#pragma unroll
  for (int st = 0; st < NS; ++st) {
    const bool inA = st < nA;
    const int pt = inA ? w : 7 - w;
    const int l = 16 * pt + 4 * (inA ? st : st - nA) + g;
    const int p = 16 * pt + m;
    bv[st] = (p <= l && l < a.b) ? a.Tm[p + (int64_t)l * a.ldt] : 0.0;
  }
  // Split sums: pack q = t + 256 j covers z[c0 + q / 64][2 (q % 64) + {0, 1}].
  double2 z[PK];
  const double2* zp[PK];
  bool ok[PK];
#pragma unroll
  for (int j = 0; j < PK; ++j) {
    const int q = t + 256 * j;
    const int64_t c = c0 + q / 64;
    ok[j] = c < a.n;
    zp[j] = reinterpret_cast<const double2*>(a.Z + (ok[j] ? c : 0) * BP + 2 * (q % 64));
    z[j] = make_double2(0.0, 0.0);
  }
  const int64_t ss = a.split_stride / 2;  // in packs
  for (int s0 = 0; s0 < a.nsplit; s0 += SB) {
    double2 v[SB][PK];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int64_t su = min(s0 + u, a.nsplit - 1);
#pragma unroll
      for (int j = 0; j < PK; ++j) v[u][j] = zp[j][su * ss];
    }
#pragma unroll
    for (int u = 0; u < SB; ++u)
      if (s0 + u < a.nsplit)
#pragma unroll
        for (int j = 0; j < PK; ++j) {
          z[j].x += v[u][j].x;
          z[j].y += v[u][j].y;
        }
  }
#pragma unroll
  for (int j = 0; j < PK; ++j) {
    const int q = t + 256 * j;
    zs[q / 64][2 * (q % 64) + 0] = ok[j] ? z[j].x : 0.0;
    zs[q / 64][2 * (q % 64) + 1] = ok[j] ? z[j].y : 0.0;
  }
  __syncthreads();
  d4_t accA = Mfma<double>::zero(), accB = Mfma<double>::zero();
#pragma unroll
  for (int st = 0; st < NS; ++st) {
    const bool inA = st < nA;
    const int pt = inA ? w : 7 - w;
    const int l = 16 * pt + 4 * (inA ? st : st - nA) + g;
    const double av = m < CW ? zs[m][l] : 0.0;
    if (inA)
      accA = Mfma<double>::op(av, bv[st], accA);
    else
      accB = Mfma<double>::op(av, bv[st], accB);
  }
  // Lane (g, m), item i: W[c0 + g + 4 i][16 pt + m]; rows [n, n_pad) get the
  // zeros of their zero z.
  const int64_t n_pad = (a.n + kUpdChunk - 1) / kUpdChunk * kUpdChunk;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = Mfma<double>::drow(g, i);
    const int64_t c = c0 + r;
    if (r < CW && c < n_pad) {
      a.W[c * BP + 16 * w + m] = accA[i];
      a.W[c * BP + 16 * (7 - w) + m] = accB[i];
    }
  }
}

template <typename T, int BP, int QP, bool STORE>
__global__ __launch_bounds__(256, 2) void update_kernel(UpdateArgs<T> a) {
  update_body<T, BP, QP, STORE>(a, blockIdx.x, blockIdx.y, gridDim.x);
}

template <typename T, int BP, int QP>
hipError_t upd_go(const UpdateArgs<T>& a, dim3 grid, hipStream_t s) {
  if (a.dst)
    hipLaunchKernelGGL((update_kernel<T, BP, QP, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((update_kernel<T, BP, QP, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename T, int BP>
hipError_t upd_q(const UpdateArgs<T>& a, dim3 grid, hipStream_t s) {
  if constexpr (BP == 128) {
    // 128 reflectors: the explicit-Q pass only (binary64, no sample).
    if constexpr (std::is_same<T, double>::value) {
      if (a.qp == 0) return upd_go<T, 128, 0>(a, grid, s);
    }
    return hipErrorInvalidValue;
  } else {
    switch (a.qp) {
      case 0: return upd_go<T, BP, 0>(a, grid, s);
      case 16: return upd_go<T, BP, 16>(a, grid, s);
      case 32: return upd_go<T, BP, 32>(a, grid, s);
      case 64: return upd_go<T, BP, 64>(a, grid, s);
    }
    return hipErrorInvalidValue;
  }
}

template <typename T, int BP>
hipError_t red_go(const ReduceArgs<T>& a, int nsplit, hipStream_t s) {
  // 16-byte packs of X when the region is aligned to them.
  constexpr int VEC = 16 / (int)sizeof(T);
  const bool vec_ok = (reinterpret_cast<uintptr_t>(a.X) % 16) == 0 &&
                      a.ldx % VEC == 0 && a.mr % VEC == 0 &&
                      a.rows_per_split % VEC == 0;
  constexpr int CT = red_col_tiles(BP);
  const dim3 grid((unsigned)ceil_div(a.n, 64 * CT), (unsigned)nsplit);
  if (vec_ok)
    hipLaunchKernelGGL((reduce_kernel<T, BP, VEC, CT, kRedRows>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((reduce_kernel<T, BP, 1, CT, kRedRows>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

template <typename T>
hipError_t launch_update(const UpdateArgs<T>& a, int nsplit, hipStream_t s) {
  if (a.mr <= 0 || a.n <= 0) return hipSuccess;
  // 32-bit buffer offsets: a chunk of columns must span at most 2^30 bytes.
  const int64_t ld = a.dst ? std::max(a.lds, a.ldd) : a.lds;
  if (ld < a.mr || (int64_t)kUpdChunk * ld * (int64_t)sizeof(T) > ((int64_t)1 << 30))
    return hipErrorInvalidValue;
  dim3 grid((unsigned)ceil_div(a.mr, kUpdRows), (unsigned)nsplit);
  switch (a.bp) {
    case 0: return upd_q<T, 0>(a, grid, s);
    case 16: return upd_q<T, 16>(a, grid, s);
    case 32: return upd_q<T, 32>(a, grid, s);
    case 64: return upd_q<T, 64>(a, grid, s);
    case 128: return upd_q<T, 128>(a, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_reduce(const ReduceArgs<T>& a, int nsplit, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  switch (a.bp) {
    case 16: return red_go<T, 16>(a, nsplit, s);
    case 32: return red_go<T, 32>(a, nsplit, s);
    case 64: return red_go<T, 64>(a, nsplit, s);
    case 128:
      if constexpr (std::is_same<T, double>::value) return red_go<T, 128>(a, nsplit, s);
      break;
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_formw(const FormWArgs<T>& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  const int cpb = 256 / a.bp;
  int64_t blocks = ceil_div(a.n, cpb);
  // Every workgroup stages all of T (bp^2 values): at 128 reflectors fewer
  // workgroups, each over more columns, keep that re-read small.
  const int64_t cap = a.bp == 128 ? 256 : 2048;
  if (blocks > cap) blocks = cap;
  // The gather's workgroups follow formW's.
  FormWArgs<T> a2 = a;
  a2.nfw = (int)blocks;
  int64_t gblocks = 0;
  if (a.g.nsplit > 0 && a.g.rows_pad > 0) {
    if (a.bp > 64 || a.g.bp < 1) return hipErrorInvalidValue;
    gblocks = ceil_div(a.g.rows_pad, 256) * a.g.bp;
  } else {
    a2.g.nsplit = 0;
  }
  dim3 grid((unsigned)(blocks + gblocks));
  switch (a.bp) {
    case 16: hipLaunchKernelGGL((formw_kernel<T, 16>), grid, dim3(256), 0, s, a2); break;
    case 32: hipLaunchKernelGGL((formw_kernel<T, 32>), grid, dim3(256), 0, s, a2); break;
    case 64: hipLaunchKernelGGL((formw_kernel<T, 64>), grid, dim3(256), 0, s, a2); break;
    case 128:
      if constexpr (std::is_same<T, double>::value) {
        if (!a.trans) {
          // The widest tile that still gives half the compute units a
          // workgroup; the partials are 16-byte packs.
          if (reinterpret_cast<uintptr_t>(a.Z) % 16 != 0 || a.split_stride % 2 != 0)
            return hipErrorInvalidValue;
          const int64_t n_pad = ceil_div(a.n, kUpdChunk) * kUpdChunk;
          if (ceil_div(n_pad, 16) >= 128)
            hipLaunchKernelGGL((formw128_kernel<16>), dim3((unsigned)ceil_div(n_pad, 16)),
                               dim3(256), 0, s, a);
          else if (ceil_div(n_pad, 8) >= 128)
            hipLaunchKernelGGL((formw128_kernel<8>), dim3((unsigned)ceil_div(n_pad, 8)),
                               dim3(256), 0, s, a);
          else
            hipLaunchKernelGGL((formw128_kernel<4>), dim3((unsigned)ceil_div(n_pad, 4)),
                               dim3(256), 0, s, a);
          break;
        }
        hipLaunchKernelGGL((formw_kernel<T, 128>), grid, dim3(256), 0, s, a2);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t launch_update<float>(const UpdateArgs<float>&, int, hipStream_t);
template hipError_t launch_update<double>(const UpdateArgs<double>&, int, hipStream_t);
template hipError_t launch_reduce<float>(const ReduceArgs<float>&, int, hipStream_t);
template hipError_t launch_reduce<double>(const ReduceArgs<double>&, int, hipStream_t);
template hipError_t launch_formw<float>(const FormWArgs<float>&, hipStream_t);
template hipError_t launch_formw<double>(const FormWArgs<double>&, hipStream_t);

}  // namespace rrf
