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

#include "mfma.h"
#include "rrf_internal.h"

namespace rrf {
namespace {

// ---------------------------------------------------------------------------
// reduce: Z_s[c * BP + p] = sum_{r in split s} V[r, p] X[r, c]
// grid (ceil(n / kRedCols), nsplit), 256 threads; V is staged in chunks of
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
  static_assert(kRedCols == 64 * CT, "workgroup width");
  __shared__ T vl[BP * LDV];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  // Wavefront w owns CT adjacent 16-column tiles; every staged V value read
  // from LDS feeds CT MFMAs.
  const int64_t cb = (int64_t)blockIdx.x * kRedCols + 16 * CT * wave;
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
  auto stage_v = [&](int64_t R) {
    const double mask = R + rr < r_end ? 1.0 : 0.0;
#pragma unroll
    for (int it = 0; it < NIT; ++it) vl[(p0 + PSTEP * it) * LDV + rr] = (T)(mask * vt[it]);
  };

  load_x(r_begin, xcur);
  load_v(r_begin);
  stage_v(r_begin);
  __syncthreads();
  for (int64_t R = r_begin; R < r_end; R += RC) {
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
          const T bv = vl[(pt * 16 + m16) * LDV + k];
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
            acc[ct][pt] = Mfma<T>::op(xcur[ct][u].v[h], bv, acc[ct][pt]);
        }
      }
    }
    __syncthreads();
    stage_v(Rn);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int u = 0; u < NX; ++u) xcur[ct][u] = xnxt[ct][u];
    __syncthreads();
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
// ---------------------------------------------------------------------------
template <typename T, int BP>
__global__ __launch_bounds__(256) void formw_kernel(FormWArgs<T> a) {
  constexpr int CPB = 256 / BP;
  __shared__ double Tl[BP][BP + 1];
  __shared__ double zs[CPB][BP + 1];
  for (int idx = threadIdx.x; idx < BP * BP; idx += 256) {
    const int i = idx % BP, j = idx / BP;
    Tl[i][j] = (i <= j && j < a.b) ? a.Tm[i + j * a.ldt] : 0.0;
  }
  const int p = threadIdx.x % BP, cl = threadIdx.x / BP;
  // Rows [n, round_up(n, kUpdChunk)) of W are written as zeros so the update
  // can stage whole chunks without predicates.
  const int64_t n_pad = (a.n + kUpdChunk - 1) / kUpdChunk * kUpdChunk;
  for (int64_t c0 = (int64_t)blockIdx.x * CPB; c0 < n_pad;
       c0 += (int64_t)gridDim.x * CPB) {
    __syncthreads();
    const int64_t c = c0 + cl;
    double z = 0.0;
    if (c < a.n)
      for (int s = 0; s < a.nsplit; ++s)
        z += (double)a.Z[s * a.split_stride + c * BP + p];
    zs[cl][p] = z;
    __syncthreads();
    double w = 0.0;
    if (a.trans) {
      for (int l = 0; l <= p; ++l) w += Tl[l][p] * zs[cl][l];
    } else {
      for (int l = p; l < BP; ++l) w += Tl[p][l] * zs[cl][l];
    }
    if (c < n_pad) a.W[c * BP + p] = (T)w;
  }
}

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
// update: X <- X - V W (BP > 0), store (STORE), norms, and P = X_new Omega.
// grid (ceil(mr / kUpdRows), nsplit), 256 threads; wavefront w owns RT
// adjacent 16-row tiles, so every staged W and Omega value read from LDS
// feeds RT MFMAs.
// ---------------------------------------------------------------------------
template <typename T, int BP, int QP, bool STORE>
__global__ __launch_bounds__(256, 2) void update_kernel(UpdateArgs<T> a) {
  typedef typename Mfma<T>::acc_t acc_t;
  constexpr int RT = kUpdRowTiles;
  constexpr int NP4 = BP / 4;        // K-steps of the rank-b update
  constexpr int NQT = QP / 16;       // 16-wide tiles of the sample
  constexpr int LDW = BP + 1;        // odd: conflict-free column reads
  constexpr int LDO = QP + 1;
  constexpr int NCT = kUpdChunk / 16;
  constexpr int E = (int)sizeof(T);
  static_assert(kUpdRows == 64 * RT, "workgroup height");
  __shared__ T wl[kUpdChunk * (BP > 0 ? LDW : 1)];
  __shared__ T ol[kUpdChunk * (QP > 0 ? LDO : 1)];
  __shared__ double nred[2][4];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const unsigned nrb = gridDim.x, rb = blockIdx.x, split = blockIdx.y;
  const int64_t cs = (int64_t)split * a.cols_per_split;
  const int64_t ce = min(a.n, cs + a.cols_per_split);
  if (cs >= ce) {          // empty split (uniform per workgroup, before any barrier)
    if (a.normpart && threadIdx.x == 0) {
      a.normpart[2 * ((int64_t)split * nrb + rb) + 0] = 0.0;
      a.normpart[2 * ((int64_t)split * nrb + rb) + 1] = 0.0;
    }
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
  double nb = 0.0, nt = 0.0;
  double wb[RT], wt[RT];   // block-row or trailing norm
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    wb[rt] = r[rt] < a.s0 ? 1.0 : 0.0;
    wt[rt] = 1.0 - wb[rt];
  }

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
  // while the current chunk computes; the last chunk prefetches itself again
  // (harmless, and it keeps the loads unconditional).  Chunks start at
  // multiples of kUpdChunk and split boundaries are multiples of kUpdChunk, so
  // a chunk only runs past ce at the end of the matrix, where W and Omega
  // carry zero rows up to the next multiple and the B loads return zero.
  //
  // Schedule per chunk: issue the next chunk's loads, compute and store this
  // chunk, then (after a barrier) move the next chunk's staging values into
  // LDS and its B tiles into the accumulators.  The waits for those loads sit
  // in straight-line code after the stores, so they never wait for stores
  // (the vector-memory counter retires in issue order).
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
  const int64_t c_last = cs + (ce - cs - 1) / kUpdChunk * kUpdChunk;
  auto load_chunk = [&](int64_t cc0) {
    if (NW > 0) {
      const __amdgpu_buffer_rsrc_t rw =
          buf_rsrc(a.W + cc0 * a.ldw, (int64_t)kUpdChunk * a.ldw * E);
#pragma unroll
      for (int it = 0; it < NW; ++it) tw[it] = Buf<T>::ld_s(rw, wo_lane, it * wo_pass);
    }
    if (NO > 0) {
      const __amdgpu_buffer_rsrc_t ro =
          buf_rsrc(a.Om + cc0 * a.ldo, (int64_t)kUpdChunk * a.ldo * E);
#pragma unroll
      for (int it = 0; it < NO; ++it) to[it] = Buf<T>::ld_s(ro, oo_lane, it * oo_pass);
    }
    const int64_t cn = min((int64_t)kUpdChunk, a.n - cc0);
    const __amdgpu_buffer_rsrc_t rs =
        buf_rsrc(a.src + cc0 * a.lds, ((cn - 1) * a.lds + a.mr) * E);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          bx[rt][ct][i] = Buf<T>::ld(rs, vs[rt] + ct * tstep_s + i * cstep_s);
  };
  auto stage_chunk = [&]() {
#pragma unroll
    for (int it = 0; it < NW; ++it) {
      const int idx = threadIdx.x + 256 * it;
      wl[(idx / BP) * LDW + idx % BP] = tw[it];
    }
#pragma unroll
    for (int it = 0; it < NO; ++it) {
      const int idx = threadIdx.x + 256 * it;
      ol[(idx / QP) * LDO + idx % QP] = to[it];
    }
  };

  acc_t t[RT][NCT];
  load_chunk(cs);
  stage_chunk();
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) t[rt][ct] = bx[rt][ct];
  __syncthreads();

  for (int64_t c0 = cs; c0 < ce; c0 += kUpdChunk) {
    load_chunk(min(c0 + kUpdChunk, c_last));

    // Rank-b update of all tiles first, so that the samples do not wait on
    // the result of the MFMA chain that just produced their operand.
    // D[M = column drow(g, i)][N = row m16] of each 16 x 16 tile.
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int p4 = 0; p4 < NP4; ++p4) {
        const T wa = wl[(ct * 16 + m16) * LDW + 4 * p4 + g];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          t[rt][ct] = Mfma<T>::op(wa, vreg[rt][p4], t[rt][ct]);
      }
    if (STORE) {
      const int64_t cn = min((int64_t)kUpdChunk, a.n - c0);
      const __amdgpu_buffer_rsrc_t rd =
          buf_rsrc(a.dst + c0 * a.ldd, ((cn - 1) * a.ldd + a.mr) * E);
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
          nb = fma(v * wb[rt], v, nb);
          nt = fma(v * wt[rt], v, nt);
        }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
          const T oa = ol[(ct * 16 + Mfma<T>::drow(g, s)) * LDO + qt * 16 + m16];
#pragma unroll
          for (int rt = 0; rt < RT; ++rt)
            pacc[rt][qt] = Mfma<T>::op(oa, t[rt][ct][s], pacc[rt][qt]);
        }
    __syncthreads();
    stage_chunk();
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) t[rt][ct] = bx[rt][ct];
    __syncthreads();
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
    if (threadIdx.x == 0) {
      const int64_t wg = (int64_t)split * nrb + rb;
      a.normpart[2 * wg + 0] = ((nred[0][0] + nred[0][1]) + nred[0][2]) + nred[0][3];
      a.normpart[2 * wg + 1] = ((nred[1][0] + nred[1][1]) + nred[1][2]) + nred[1][3];
    }
  }
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
  switch (a.qp) {
    case 0: return upd_go<T, BP, 0>(a, grid, s);
    case 16: return upd_go<T, BP, 16>(a, grid, s);
    case 32: return upd_go<T, BP, 32>(a, grid, s);
    case 64: return upd_go<T, BP, 64>(a, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T, int BP>
hipError_t red_go(const ReduceArgs<T>& a, dim3 grid, hipStream_t s) {
  // 16-byte packs of X when the region is aligned to them.
  constexpr int VEC = 16 / (int)sizeof(T);
  const bool vec_ok = (reinterpret_cast<uintptr_t>(a.X) % 16) == 0 &&
                      a.ldx % VEC == 0 && a.mr % VEC == 0 &&
                      a.rows_per_split % VEC == 0;
  constexpr int CT = kRedCols / 64;
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
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_reduce(const ReduceArgs<T>& a, int nsplit, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  dim3 grid((unsigned)ceil_div(a.n, kRedCols), (unsigned)nsplit);
  switch (a.bp) {
    case 16: return red_go<T, 16>(a, grid, s);
    case 32: return red_go<T, 32>(a, grid, s);
    case 64: return red_go<T, 64>(a, grid, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_formw(const FormWArgs<T>& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  const int cpb = 256 / a.bp;
  int64_t blocks = ceil_div(a.n, cpb);
  if (blocks > 2048) blocks = 2048;
  dim3 grid((unsigned)blocks);
  switch (a.bp) {
    case 16: hipLaunchKernelGGL((formw_kernel<T, 16>), grid, dim3(256), 0, s, a); break;
    case 32: hipLaunchKernelGGL((formw_kernel<T, 32>), grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL((formw_kernel<T, 64>), grid, dim3(256), 0, s, a); break;
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
