// Compact WY of a group of adjacent blocks of reflectors for the explicit-Q
// pass (Q = H_0 ... H_{k-1} [I_k; 0], Sec. 4 storage scheme, Eq. (1)).
//
// For consecutive blocks V_1, ..., V_q (widths b_c, total w <= 128) and their
// own forward T factors T_c (Eq. (4)),
//   (I - V_1 T_1 V_1^T) ... (I - V_q T_q V_q^T) = I - V T V^T,
//   V = [V_1 ... V_q],
// where the upper triangular T is built one block at a time (the larft
// recursion taken by blocks): with S = [V_1 ... V_{c-1}] and T_S its T,
//   T_{[S V_c]} = [T_S  -T_S (S^T V_c) T_c ; 0  T_c].
// The explicit-Q pass then applies the whole group as one block of up to 128
// reflectors: a quarter of the passes over Q for 32-column blocks, half for
// 64-column blocks.
//
//   group_gram_kernel  the tiles of G_s = V^T V that the recursion reads
//                      (S^T V_c for each block c), over the rows of split s,
//                      one workgroup per (group, split), f64 MFMA 16x16x4
//                      from LDS-staged rows; rows of block c above its own
//                      first row read as zero (V_c is zero there by
//                      definition);
//   group_sum_kernel   G = sum_s G_s in split order (deterministic), the
//                      strictly upper entries only;
//   group_t_kernel     the recursion above in LDS, the merged T into the
//                      group's columns of Tg, and explicit zeros in the rows
//                      of each block c > 1 above its first row (the pass
//                      reads the group as one column block of V).

#include "mfma.h"
#include "rrf_internal.h"

namespace rrf {
namespace {

constexpr int kGR = 32;      // rows of V staged per chunk
constexpr int kGLd = 144;    // LDS row stride in doubles (128 + 16: the four
                             // lane groups of an operand read fall on
                             // alternate bank halves)
constexpr int kGEnt = kGroupMax * kGroupMax;   // entries of one G

__device__ __forceinline__ int block_of(const OrgqrGroup& gr, int col) {
  int c = 0;
#pragma unroll
  for (int i = 1; i < kMaxGroupBlocks; ++i) c += (i < gr.nb && col >= gr.off[i]) ? 1 : 0;
  return c;
}

__global__ __launch_bounds__(256, 2) void group_gram_kernel(GroupArgs a) {
  typedef Mfma<double>::acc_t acc_t;
  __shared__ double vs[2][kGR * kGLd];
  const OrgqrGroup& gr = a.groups[blockIdx.x];     // read in place (uniform)
  const int sp = (int)blockIdx.y, t = (int)threadIdx.x;
  const int lane = t & 63, wave = t >> 6, m16 = lane & 15, g = lane >> 4;
  const int64_t mr = a.m - gr.k0;
  const int64_t per = ((mr + a.nsplit - 1) / a.nsplit + kGR - 1) / kGR * kGR;
  const int64_t r_begin = gr.k0 + (int64_t)sp * per;          // absolute rows
  const int64_t r_end = min(a.m, r_begin + per);
  const double* Vg = a.V + gr.k0 * a.ldv;                      // column k0

  // Staging: thread t loads row t % 32 of columns t / 32 + 8 u (coalesced
  // along the rows of each column).  Column col of block c is zero above
  // row k0 + off[c] and past w.
  const int sr = t % kGR, sc0 = t / kGR;
  // First row of each staged column relative to k0 (columns past w: never).
  int first[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int col = sc0 + 8 * u;
    first[u] = col < gr.w ? gr.off[block_of(gr, col)] : 0x7fffffff;
  }
  // The 16 loads of a chunk are issued together from clamped in-bounds
  // addresses; the masks are applied when the values go to LDS (a mask
  // applied at the load made each load wait for the one before).
  double st[16];
  int64_t r_st = 0;                          // row of this thread's staged values
  auto load = [&](int64_t R) {
    const int64_t r = min(R + sr, a.m - 1);
    r_st = R + sr;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int col = sc0 + 8 * u;
      st[u] = Vg[r + (int64_t)(col < gr.w ? col : 0) * a.ldv];
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto stage = [&](double* buf) {
    const int rl = (int)(r_st - gr.k0);
    const bool in = r_st < r_end;
#pragma unroll
    for (int u = 0; u < 16; ++u)
      buf[sr * kGLd + sc0 + 8 * u] = (in && rl >= first[u]) ? st[u] : 0.0;
  };

  // The listed tiles (ti, tj) of the 128 x 128 Gram matrix,
  // D[i][j] = sum_r V[r][16 ti + i] V[r][16 tj + j], go round-robin to the
  // wavefronts: tile n to wavefront n % 4, accumulator n / 4.  A operand
  // V[r0 + g][16 ti + m], B operand V[r0 + g][16 tj + m].
  // Tile offsets in registers before the loop: the group is read through a
  // generic pointer, which the compiler would otherwise reload after every
  // LDS store.  Values are uniform per wavefront.
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int ntiles = __builtin_amdgcn_readfirstlane(gr.ntiles);
  int ta[16], tb[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int n = 4 * q + wv;
    const int tl = __builtin_amdgcn_readfirstlane(n < ntiles ? (int)gr.tile[n] : 0);
    ta[q] = (tl >> 3) * 16;
    tb[q] = (tl & 7) * 16;
  }
  acc_t acc[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) acc[q] = Mfma<double>::zero();

  if (r_begin < r_end) {
    load(r_begin);
    stage(vs[0]);
    __syncthreads();
    int cur = 0;
    for (int64_t R = r_begin; R < r_end; R += kGR) {
      const bool more = R + kGR < r_end;     // uniform
      if (more) load(R + kGR);
      const double* vb = vs[cur];
      // One uniform branch per tile, its K steps inside.
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (4 * q + wv < ntiles) {
#pragma unroll
          for (int kk = 0; kk < kGR / 4; ++kk) {
            const double* row = vb + (4 * kk + g) * kGLd;
            acc[q] = Mfma<double>::op(row[ta[q] + m16], row[tb[q] + m16], acc[q]);
          }
        }
      if (more) stage(vs[cur ^ 1]);
      __syncthreads();
      cur ^= 1;
    }
  }
  // Lane (g, m), item i holds G[16 ti + g + 4 i][16 tj + m].
  double* P = a.part + ((int64_t)blockIdx.x * a.nsplit + sp) * kGEnt;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    if (4 * q + wv < ntiles) {
#pragma unroll
      for (int i = 0; i < 4; ++i) P[(ta[q] + g + 4 * i) * kGroupMax + tb[q] + m16] = acc[q][i];
    }
  }
}

// grid (ngroups, kGEnt / 256): entry e of group blockIdx.x.
__global__ __launch_bounds__(256) void group_sum_kernel(GroupArgs a) {
  constexpr int ZB = 8;
  const int e = (int)blockIdx.y * 256 + (int)threadIdx.x;
  const int i = e / kGroupMax, j = e % kGroupMax;
  double* sums = a.part + (int64_t)a.ngroups * a.nsplit * kGEnt;
  if (i >= j) {      // the recursion reads strictly upper entries of listed tiles
    sums[(int64_t)blockIdx.x * kGEnt + e] = 0.0;
    return;
  }
  const double* src = a.part + (int64_t)blockIdx.x * a.nsplit * kGEnt + e;
  double s = 0.0;
  for (int s0 = 0; s0 < a.nsplit; s0 += ZB) {
    double v[ZB];
#pragma unroll
    for (int u = 0; u < ZB; ++u) v[u] = src[(int64_t)min(s0 + u, a.nsplit - 1) * kGEnt];
#pragma unroll
    for (int u = 0; u < ZB; ++u)
      if (s0 + u < a.nsplit) s += v[u];
  }
  sums[(int64_t)blockIdx.x * kGEnt + e] = s;
}

// One workgroup per group.  Tl holds the merged T (column-major, stride
// kTS); while block c is merged at offset s (width bc):
//   rows [s, s + bc) x cols [s, s + bc)   T_c (its final place),
//   rows [s, s + bc) x cols [0, s)        G[0:s, s:s+bc], then M = G T_c,
//                                         both transposed (entries below the
//                                         diagonal of T, unused until the end),
//   rows [0, s) x cols [s, s + bc)        the new block -T_S M.
__global__ __launch_bounds__(256) void group_t_kernel(GroupArgs a) {
  constexpr int kTS = kGroupMax + 1;
  __shared__ double Tl[kGroupMax * kTS];
  const OrgqrGroup& gr = a.groups[blockIdx.x];     // read in place (uniform)
  const int t = (int)threadIdx.x;
  const double* G = a.part + (int64_t)a.ngroups * a.nsplit * kGEnt + (int64_t)blockIdx.x * kGEnt;
  const double* Tm = a.Tm + gr.k0 * a.ldt;
  {
    const int b0 = gr.off[1];
    for (int e = t; e < b0 * b0; e += 256) {
      const int i = e % b0, j = e / b0;
      Tl[i + j * kTS] = i <= j ? Tm[i + (int64_t)j * a.ldt] : 0.0;
    }
  }
  const int nb = __builtin_amdgcn_readfirstlane(gr.nb);
  for (int c = 1; c < nb; ++c) {
    const int s = __builtin_amdgcn_readfirstlane(gr.off[c]);
    const int bc = __builtin_amdgcn_readfirstlane(gr.off[c + 1]) - s;
    for (int e = t; e < bc * bc; e += 256) {
      const int i = e % bc, j = e / bc;
      Tl[(s + i) + (s + j) * kTS] = i <= j ? Tm[i + (int64_t)(s + j) * a.ldt] : 0.0;
    }
    for (int e = t; e < s * bc; e += 256) {
      const int i = e % s, j = e / s;
      Tl[(s + j) + i * kTS] = G[i * kGroupMax + s + j];
    }
    __syncthreads();
    // M = G[0:s, s:s+bc] T_c, then -T_S M, each in 4 x 4 register blocks
    // (rows 4 ra.., columns 4 rb..; at most two blocks a thread): the T_c and
    // T_S staged above are zero below their diagonals.  Entries past s or bc
    // read clamped indices and are not stored.
    const int nra = (s + 3) / 4, nrb = (bc + 3) / 4, nblk = nra * nrb;
    double blk[2][4][4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int bi = t + 256 * h;
      const int ra = 4 * (bi % nra), rb = 4 * (bi / nra);
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) blk[h][x][y] = 0.0;
      if (bi < nblk) {
        int ri[4], cj[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          ri[x] = min(ra + x, s - 1);
          cj[x] = min(rb + x, bc - 1);
        }
        for (int l = 0; l < bc; ++l) {
          double gv[4], tv[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            gv[x] = Tl[(s + l) + ri[x] * kTS];
            tv[x] = Tl[(s + l) + (s + cj[x]) * kTS];
          }
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) blk[h][x][y] += gv[x] * tv[y];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int bi = t + 256 * h;
      if (bi < nblk) {
        const int ra = 4 * (bi % nra), rb = 4 * (bi / nra);
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y)
            if (ra + x < s && rb + y < bc) Tl[(s + rb + y) + (ra + x) * kTS] = blk[h][x][y];
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int bi = t + 256 * h;
      const int ra = 4 * (bi % nra), rb = 4 * (bi / nra);
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) blk[h][x][y] = 0.0;
      if (bi < nblk) {
        int ri[4], cj[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          ri[x] = min(ra + x, s - 1);
          cj[x] = min(rb + x, bc - 1);
        }
        for (int l = 0; l < s; ++l) {
          double sv[4], mv[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            sv[x] = Tl[ri[x] + l * kTS];
            mv[x] = Tl[(s + cj[x]) + l * kTS];
          }
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) blk[h][x][y] -= sv[x] * mv[y];
        }
      }
    }
    __syncthreads();
    // The new columns, and zeros over M (below the diagonal of the next T_S).
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int bi = t + 256 * h;
      if (bi < nblk) {
        const int ra = 4 * (bi % nra), rb = 4 * (bi / nra);
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y)
            if (ra + x < s && rb + y < bc) {
              Tl[(ra + x) + (s + rb + y) * kTS] = blk[h][x][y];
              Tl[(s + rb + y) + (ra + x) * kTS] = 0.0;
            }
      }
    }
    __syncthreads();
  }
  double* To = a.Tg + gr.k0 * a.ldg;
  for (int e = t; e < gr.w * gr.w; e += 256) {
    const int i = e % gr.w, j = e / gr.w;
    To[i + (int64_t)j * a.ldg] = i <= j ? Tl[i + j * kTS] : 0.0;
  }
  // Block c >= 1 is zero above its first row (rows k0 .. k0 + off[c] - 1).
  for (int c = 1; c < gr.nb; ++c) {
    const int s = gr.off[c], bc = gr.off[c + 1] - gr.off[c];
    double* Vc = a.V + (gr.k0 + s) * a.ldv + gr.k0;
    for (int e = t; e < s * bc; e += 256) Vc[e % s + (int64_t)(e / s) * a.ldv] = 0.0;
  }
}

}  // namespace

hipError_t launch_orgqr_groups(const GroupArgs& a, hipStream_t s) {
  if (a.ngroups <= 0) return hipSuccess;
  if (a.nsplit < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(group_gram_kernel, dim3((unsigned)a.ngroups, (unsigned)a.nsplit),
                     dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_sum_kernel, dim3((unsigned)a.ngroups, (unsigned)(kGEnt / 256)),
                     dim3(256), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_t_kernel, dim3((unsigned)a.ngroups), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rrf
