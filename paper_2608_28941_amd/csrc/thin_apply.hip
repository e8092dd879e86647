// Block reflector applied to a thin matrix in one launch (all workgroups
// resident, launch_resident):
// Y <- Q^T Y = Y - V T^T (V^T Y) (Alg. 2, update step, Eq. (4)) for Y of at
// most 64 columns, the look-ahead's redundant panel update Q_i^T S_{i+1}
// (Sec. 5), or Y <- Q Y = Y - V T (V^T Y), the last block of the explicit-Q
// pass.  Three phases instead of three launches (reduce, formW, update):
//   1. every workgroup forms the partial Z_w = V_w^T Y_w of its rows with f64
//      MFMA (16 x 16 tiles, the output layout kept so that the tagged words
//      are coalesced);
//   2. the partials are summed across the grid in two phases (workgroup w
//      sums its slice of Z over all workgroups in a fixed order, then every
//      workgroup reads all of Z): deterministic, no floating-point atomics;
//   3. every workgroup forms W = T^T Z (the same values everywhere) and
//      updates its rows, Y_w -= V_w W, in the transposed MFMA frame (16
//      consecutive rows per lane group: coalesced loads and stores).
// The exchange uses the epoch-tagged words of the panel kernels (xchg.h),
// and carries only the 16 x 16 tiles of Z that the block has: ceil(b / 16)
// x ceil(ncols / 16) of the 4 x 4 (4 of 16 at b = ncols = 32).

#include "mfma.h"
#include "xchg.h"

namespace rrf {
namespace {

constexpr int kThinSlots = 16 * 256;   // 64 x 64 values in MFMA tile order (at most)

// Rows of a chunk staged in LDS (V and Y, 64 columns each).
constexpr int kThinChunk = 64;

// TM: 16 x 16 tiles per side that the MFMA loops cover (2: b and ncols at
// most 32; 4: up to 64); the tiles past it are zero and are not computed.
template <int TM>
__global__ __launch_bounds__(256) void thin_apply_kernel(ThinApplyArgs a) {
  __shared__ double Vs[kThinChunk][65];
  __shared__ double Ys[kThinChunk][65];
  __shared__ double Tl[64][65];
  __shared__ double ZW[64][65];      // Z, then W = T^T Z in place
  __shared__ double red2[256];
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6, l16 = lane >> 4, m16 = lane & 15;
  const int w = (int)blockIdx.x, G = (int)gridDim.x;
  const int64_t r_begin = (int64_t)w * a.rows_per_wg;
  const int64_t r_end = min(a.mr, r_begin + a.rows_per_wg);
  const unsigned epoch = a.epoch_base + 1u;
  const bool forced = waits_forced(a.st);
  // Exchanged tiles: PT row tiles (reflectors) x CT column tiles, slot
  // ((pt CT + ct) 4 + i) 64 + lane; NS slots in all (uniform).
  const int PT = (min(a.b, 64) + 15) / 16, CT = (min(a.ncols, 64) + 15) / 16;
  const int NS = PT * CT * 256;

  // The loops below read rows and columns of Tl, Vs and Ys below TD only.
  constexpr int TD = 16 * TM;
  // T (leading b x b block, upper triangular) to LDS: all loads issued
  // before the first use (columns past b read column 0), entries outside the
  // triangle replaced by zero (a select: whatever the padding holds, even a
  // NaN, does not reach W).
  {
    constexpr int NTT = TD * TD / 256;
    double tv[NTT];
#pragma unroll
    for (int it = 0; it < NTT; ++it) {
      const int idx = t + 256 * it;
      const int i = idx % TD, j = idx / TD;
      tv[it] = a.Tm[i + (int64_t)(j < a.b ? j : 0) * a.ldt];
    }
#pragma unroll
    for (int it = 0; it < NTT; ++it) {
      const int idx = t + 256 * it;
      const int i = idx % TD, j = idx / TD;
      Tl[i][j] = (i <= j && j < a.b) ? tv[it] : 0.0;
    }
  }
  // Rows [r0, r0 + 64) of V (reflectors < b) and Y (columns < ncols) to LDS,
  // zero elsewhere up to column TD: thread t loads row t % 64 of TD / 4
  // columns, so every wavefront load reads 64 consecutive rows of one column.
  auto stage = [&](int64_t r0) {
    const int rr = t % 64, c0 = t / 64;
    const int64_t r = r0 + rr;
    const bool ok = r < r_end;
    const int64_t rc = ok ? r : r_begin;   // in range; masked below
    double vv[TD / 4], yy[TD / 4];
#pragma unroll
    for (int i = 0; i < TD / 4; ++i) {
      const int c = c0 + 4 * i;
      vv[i] = a.V[rc + (int64_t)(c < a.b ? c : 0) * a.ldv];
      yy[i] = a.Y[rc + (int64_t)(c < a.ncols ? c : 0) * a.ldy];
    }
#pragma unroll
    for (int i = 0; i < TD / 4; ++i) {
      const int c = c0 + 4 * i;
      Vs[rr][c] = (ok && c < a.b) ? vv[i] : 0.0;
      Ys[rr][c] = (ok && c < a.ncols) ? yy[i] : 0.0;
    }
  };

  // 1. Z_w tile (pt = wv, ct) = sum over rows of V[r][16 pt + m] Y[r][16 ct + n].
  d4_t acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = d4_t{0.0, 0.0, 0.0, 0.0};
  for (int64_t r0 = r_begin; r0 < r_end; r0 += kThinChunk) {
    __syncthreads();
    stage(r0);
    __syncthreads();
    if (wv < TM) {
#pragma unroll 4
      for (int s4 = 0; s4 < kThinChunk / 4; ++s4) {
        const double av = Vs[4 * s4 + l16][16 * wv + m16];
#pragma unroll
        for (int ct = 0; ct < TM; ++ct)
          acc[ct] = Mfma<double>::op(av, Ys[4 * s4 + l16][16 * ct + m16], acc[ct]);
      }
    }
  }
  if (wv < PT) {
    u64* dst = a.part + (int64_t)w * NS * 2;
#pragma unroll
    for (int ct = 0; ct < TM; ++ct)
      if (ct < CT) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          put_tagged(&dst[(((wv * CT + ct) * 4 + i) * 64 + lane) * 2], acc[ct][i], epoch);
      }
  }
  // 2. This workgroup's slice of Z, summed over all workgroups in a fixed
  //    order (nsub threads per entry, then in LDS).
  {
    const int se = (NS + G - 1) / G;
    const int e0 = w * se;
    const int ne = max(0, min(NS, e0 + se) - e0);
    const int nsub = max(1, min(16, 256 / max(ne, 1)));
    const int per = 256 / nsub;
    for (int p0 = 0; p0 < ne; p0 += per) {
      const int el = p0 + t % per, sub = t / per;
      double s = 0.0;
      if (el < ne && sub < nsub) {
        const u64* src = a.part + (int64_t)(e0 + el) * 2;
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
      red2[t] = s;
      __syncthreads();
      if (t < per && p0 + t < ne) {
        double tot = 0.0;
        for (int sb = 0; sb < nsub; ++sb) tot += red2[sb * per + t];
        put_tagged(&a.sums[(int64_t)(e0 + p0 + t) * 2], tot, epoch);
      }
      __syncthreads();
    }
  }
  // 3. Every workgroup reads all of Z: slot ((pt CT + ct) 4 + i) 64 + lane
  //    holds Z[16 pt + lane/16 + 4 i][16 ct + lane%16]; tiles not exchanged
  //    are zero (reflectors >= b and columns >= ncols contribute nothing).
  {
    constexpr int NPT = TM * TM;
    const int nq = NS / 256;
    u64 hi[NPT], lo[NPT];
    unsigned spins = 0;
    bool ok;
    do {
#pragma unroll
      for (int i = 0; i < NPT; ++i) {
        const u64* q = a.sums + (int64_t)(t + 256 * (i < nq ? i : 0)) * 2;
        hi[i] = get_word(q);
        lo[i] = get_word(q + 1);
      }
      ok = true;
#pragma unroll
      for (int i = 0; i < NPT; ++i) ok = ok && tagged(hi[i], epoch) && tagged(lo[i], epoch);
    } while ((!ok || forced) && keep_waiting(&spins, a.st));
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      const int e = t + 256 * i;
      const int ln = e % 64, it = (e / 64) % 4, tile = e / 256;
      if (i < nq) {
        const int pt = tile / CT, ct = tile % CT;
        ZW[16 * pt + ln / 16 + 4 * it][16 * ct + ln % 16] = untag(hi[i], lo[i]);
      }
    }
    // Tiles outside PT x CT.
    for (int e = t; e < 4096; e += 256) {
      const int r = e / 64, c = e % 64;
      if (r >= 16 * PT || c >= 16 * CT) ZW[r][c] = 0.0;
    }
  }
  __syncthreads();
  // W = T^T Z or T Z (T is zero outside its upper b x b triangle) with MFMA:
  // tile (pt = wave, ct), A[m][k] = T[k][16 pt + m] (or T[16 pt + m][k]),
  // B[k][n] = Z[k][16 ct + n], into registers, then over Z.
  {
    // Rows of W past 16 TM are zero (T is), as are the terms k >= 16 TM.
    d4_t wacc[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) wacc[ct] = d4_t{0.0, 0.0, 0.0, 0.0};
    if (wv < TM) {
#pragma unroll
      for (int s4 = 0; s4 < 4 * TM; ++s4) {
        const double av = a.trans ? Tl[4 * s4 + l16][16 * wv + m16]
                                  : Tl[16 * wv + m16][4 * s4 + l16];
#pragma unroll
        for (int ct = 0; ct < TM; ++ct)
          wacc[ct] = Mfma<double>::op(av, ZW[4 * s4 + l16][16 * ct + m16], wacc[ct]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) ZW[16 * wv + l16 + 4 * i][16 * ct + m16] = wacc[ct][i];
  }
  // 4. Y_w -= V_w W in the transposed frame, chunk by chunk: tile (row tile
  //    rt = wv, ct) with D[m = column 16 ct + m][n = row 16 rt + n] =
  //    Y^T - W^T V^T; lane l item i holds column 16 ct + l/16 + 4 i of row
  //    16 rt + l%16 (16 consecutive rows per lane group: coalesced stores).
  for (int64_t r0 = r_begin; r0 < r_end; r0 += kThinChunk) {
    __syncthreads();
    if (r0 != r_begin || a.rows_per_wg > kThinChunk) stage(r0);
    __syncthreads();
    const int rrow = 16 * wv + m16;
    const int64_t r = r0 + rrow;
#pragma unroll
    for (int ct = 0; ct < TM; ++ct) {
      if (16 * ct >= a.ncols) continue;   // uniform
      d4_t d;
#pragma unroll
      for (int i = 0; i < 4; ++i) d[i] = Ys[rrow][16 * ct + l16 + 4 * i];
#pragma unroll
      for (int s4 = 0; s4 < 4 * TM; ++s4)
        d = Mfma<double>::op(-ZW[4 * s4 + l16][16 * ct + m16], Vs[rrow][4 * s4 + l16], d);
      if (r < r_end) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = 16 * ct + l16 + 4 * i;
          if (c < a.ncols) a.Y[r + (int64_t)c * a.ldy] = d[i];
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_thin_apply(ThinApplyArgs a, int num_cus, hipStream_t s) {
  if (a.mr <= 0 || a.ncols <= 0) return hipSuccess;
  if (a.b < 1 || a.b > 64 || a.ncols > 64) return hipErrorInvalidValue;
  // Blocks and widths of at most 32 need the 2 x 2 corner of the tiles.
  const void* fn = a.b <= 32 && a.ncols <= 32
                       ? reinterpret_cast<const void*>(thin_apply_kernel<2>)
                       : reinterpret_cast<const void*>(thin_apply_kernel<4>);
  int occ = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, 256, 0);
  if (e != hipSuccess) return e;
  // About 64 rows per workgroup, at most one workgroup per compute unit that
  // can be resident (the workgroups wait on each other).
  int64_t G = std::min<int64_t>((int64_t)num_cus * std::max(occ, 1), kMaxThinWGs);
  G = std::max<int64_t>(1, std::min<int64_t>(G, ceil_div(a.mr, 64)));
  a.rows_per_wg = round_up(ceil_div(a.mr, G), 16);
  G = ceil_div(a.mr, a.rows_per_wg);
  if (occ < 1 || G > (int64_t)occ * num_cus) return hipErrorCooperativeLaunchTooLarge;
  void* params[] = {&a};
  return launch_resident(fn,
                         dim3((unsigned)G), dim3(256), params, s);
}

}  // namespace rrf
