// Internal declarations shared by the HIP sources of librrf.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/rrf.h"

namespace rrf {

// Tiling constants (see each kernel for its use).
constexpr int kMaxBlock = 64;      // widest sub-block / panel (MFMA tiles of 16)
constexpr int kMaxBlockB = 128;    // largest block size b of a run (sub-blocks of <= 64)
constexpr int kMaxPower = 8;       // largest number of power iterations per sample
constexpr int kUpdRowTiles = 2;    // 16-row tiles per update wavefront
constexpr int kUpdRows = 128;      // rows per update workgroup (4 waves x 2 x 16)
constexpr int kUpdChunk = 16;      // columns per staged chunk in the update
constexpr int kRedCols = 128;      // columns per reduce workgroup (4 waves x 2 x 16)
// 16-column tiles per reduce wavefront: two, or one at 128 reflectors (whose
// accumulators take twice the registers); a workgroup spans 64 of them.
constexpr int red_col_tiles(int bp) { return bp == 128 ? 1 : kRedCols / 64; }
inline int64_t red_cols(int bp) { return 64 * red_col_tiles(bp); }
constexpr int kRedRows = 32;       // rows per staged V chunk in the reduce
constexpr int kRedChunk = 64;      // granularity of the reduce's row splits
constexpr int kPanelThreads = 256;
constexpr int kMaxPanelWGs = 1024;

// Poll rounds before a grid-wide wait gives up (each a short sleep plus a
// trip to the coherent memory path: tens of seconds in all).
constexpr unsigned kSpinLimit = 1u << 24;

inline int pad16(int64_t b) { return b <= 16 ? 16 : (b <= 32 ? 32 : 64); }
// Padded width of a block of up to 128 reflectors (the explicit-Q pass).
inline int pad_group(int64_t b) { return b <= 64 ? pad16(b) : 128; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Device-side run state (one per plan).
struct DevState {
  double E0;        // ||A||_F^2
  double sigma2;    // (tol ||A||_F)^2
  double E_trail;   // ||B[k:m, :]||_F^2 after the last block
  double E_sub;     // running difference (paper's rule), clamped at 0
  int stop;         // 1: stop after this block
  int nonfinite;    // 1: a norm was NaN / Inf
  int barrier_err;  // 1: a grid-wide wait gave up (sticky until cleared)
  unsigned spin_limit;  // poll rounds before a grid-wide wait gives up; 0:
                        // every wait gives up at its first poll (tests)
  double E_spec;    // spectral-norm estimate of ||B[k:m, :]||_2^2 (spectral mode)
};

// Launch descriptors -------------------------------------------------------

// Residual-norm finalisation and stop test of one launch's norm partials
// (finalize_body.h): nparts parts; traces tt, ts at index block (< 0: inside
// a block, no trace and no stop test but on errors); init: the first sample.
struct FinalizeArgs {
  int nparts;
  DevState* st;
  DevState* mirror;   // pinned host copy of *st, written with the decision
                      // (device address; nullable)
  double* tt; double* ts;
  int block;
  int64_t k_after, k_cap;
  int mode;
  double tol;
  int init;
};

template <typename T>
struct UpdateArgs {
  const T* src; int64_t lds;   // region rows start at the pointer
  T* dst; int64_t ldd;         // nullptr: do not store
  int64_t mr, n;               // region rows / columns
  const double* V; int64_t ldv;  // mr x bp, zero padded (binary64 for both
  int bp;                        // dtypes; 0: no reflector update)
  const T* W; int ldw;         // W[c * ldw + p], n x bp
  const T* Om; int ldo;        // Omega[c * ldo + q], n x qp
  int qp;                      // 0: no sample
  T* P; int64_t ldp; int64_t split_stride;  // P_s[r + q * ldp], per column split
  int64_t s0;                  // rows < s0: block-row norm; >= s0: trailing norm
  double* normpart;            // 2 doubles per workgroup, or nullptr
  int64_t cols_per_split;
  // Optional (normtag != nullptr, with normpart): the norm partials are
  // published as epoch-tagged words (4 per workgroup, epoch fin_epoch)
  // instead, and the last of the fin_nwg update workgroups (the last one
  // dispatched) waits for them and runs the finalisation fin.
  unsigned long long* normtag;
  unsigned fin_epoch;
  int fin_nwg;
  FinalizeArgs fin;
};

template <typename T>
struct ReduceArgs {
  const T* X; int64_t ldx;     // mr x n region
  int64_t mr, n;
  const double* V; int64_t ldv; int bp;
  T* Z; int64_t split_stride;  // Z_s[c * bp + p]
  int64_t rows_per_split;
};

// The gathered sample: Y[r + k ldy] = sum over the split partials
// P[s split_stride + r + k ldp] in split order (binary64), for rows < m and
// columns < b, zero elsewhere up to rows_pad x bp (gather_body.h).
template <typename T>
struct GatherArgs {
  const T* P; int64_t ldp, split_stride; int nsplit;
  int64_t m; int b, bp; int64_t rows_pad;
  double* Y; int64_t ldy;
};

template <typename T>
struct FormWArgs {
  const T* Z; int nsplit; int64_t split_stride;
  const double* Tm; int64_t ldt;  // bp x bp upper triangular (binary64)
  T* W;                        // W[c * bp + p]
  int64_t n; int bp;
  int b;                       // block width: T rows / columns >= b are ignored
  int trans;                   // 1: W = T^T Z,  0: W = T Z
  // Optional (g.nsplit > 0, bp <= 64): extra workgroups of the same launch
  // gather the look-ahead sample (the inputs of both come from the last
  // update); nfw, the formW workgroups, is set by the launcher.
  GatherArgs<T> g;
  int nfw;
};

struct PanelArgs {
  const double* Y; int64_t ldy;  // gathered panel, zero beyond (m, b), at
                                 // least G * RW rows and BP columns
  int64_t m; int b;            // panel rows, columns (b <= BP)
  double* V; int64_t ldv;      // m x BP output (binary64 for both dtypes)
  double* Tm; int64_t ldt;     // BP x BP output
  double* tau;                 // b outputs
  unsigned long long* red;     // 2 x G x BP epoch-tagged values (2 words each)
  unsigned long long* rowj;    // 2 x BP epoch-tagged values
  unsigned epoch_base;         // unique per launch, multiple of 128, > 0
  DevState* st;
  int G;
};

// Launchers (return hipError_t of the launch) ------------------------------

// Rows [n, n_pad) of the output are written as zeros.
template <typename T>
hipError_t launch_sketch(uint64_t seed, int64_t n, int64_t n_pad, int64_t col0,
                         int64_t ncols, T* out, int64_t row_stride,
                         int64_t col_stride, hipStream_t s);
template <typename T>
hipError_t launch_update(const UpdateArgs<T>& a, int nsplit, hipStream_t s);
template <typename T>
hipError_t launch_reduce(const ReduceArgs<T>& a, int nsplit, hipStream_t s);
template <typename T>
hipError_t launch_formw(const FormWArgs<T>& a, hipStream_t s);

// Panel: picks rows-per-thread and grid size; returns hipErrorInvalidValue
// if the panel does not fit the register-resident capacity.
struct PanelShape { int bp, rpt, G; int64_t rows_pad; };

// Launch of a grid whose workgroups wait on each other through the tagged
// exchange (xchg.h), so all of them must be resident at once.  The launchers
// check that the grid fits the kernel's occupancy on every compute unit; an
// ordinary launch then dispatches the whole grid at once (the stream runs
// one kernel at a time, as the look-ahead kernel's panel part also relies
// on).  The cooperative-launch API, which also guarantees it beside other
// streams' work, cost about 10 us of idle device before and after every
// launch here.  If other work holds compute units, late workgroups start
// when it drains; the bounded waits (many seconds) absorb that and report
// an error beyond it, so a wait never hangs.
inline hipError_t launch_resident(const void* fn, dim3 grid, dim3 block, void** params,
                                  hipStream_t s) {
  return hipLaunchKernel(fn, grid, block, params, 0, s);
}
bool panel_shape(int64_t m, int b, int num_cus, int target_wgs, PanelShape* out);
hipError_t launch_panel(const PanelArgs& a, const PanelShape& sh, hipStream_t s);
// Panel by tall-skinny QR + Householder reconstruction (tsqr.hip).  Leaves
// factor kTsqrLeafRpt * (256 / bp) rows each; tree nodes factor
// kTsqrNodeRows stacked rows (kTsqrNodeRows / bp children).
constexpr int kTsqrLeafRpt = 64;
constexpr int kTsqrNodeRows = 256;
constexpr int kTsqrMaxLev = 8;
struct TsqrShape {
  int bp, F, nlev;
  int G[kTsqrMaxLev];          // nodes per level (G[0]: leaves)
  int64_t scratch_elems;       // binary64 scratch the launch needs
  int64_t rows_pad;            // rows of Y the leaves cover (V is written there)
};
struct TsqrLevelArgs {
  const double* in; int64_t ldin; int64_t in_rows;  // rows >= in_rows read as 0
  double* V; int64_t ldv;      // node V blocks (RW rows each)
  double* M;                   // T V_top^T per node (BP x BP, column-major)
  double* R; int64_t ldr;      // R of node w at rows [w BP, (w + 1) BP)
  int b;
};
struct TsqrBackArgs {
  const double* Vleaf; int64_t ldvl;
  const double* Mleaf;
  int nlev, F; int64_t rwi;
  const double* Vlev[kTsqrMaxLev]; int64_t ldvlev[kTsqrMaxLev];
  const double* Mlev[kTsqrMaxLev];
  double* Q; int64_t ldq; int64_t m;
};
struct HrArgs {
  double* Q; int64_t ldq; int64_t m; int b;   // explicit Q in, V out (in place)
  double* Tm; int64_t ldt; double* tau;
  double* Uinv;                                // BP x BP scratch
};
bool tsqr_shape(int64_t m, int b, TsqrShape* out);
// Y (a.Y, read and overwritten: the leaves keep their reflectors there),
// outputs a.V, a.Tm, a.tau as launch_panel; a.m, a.b.
hipError_t launch_panel_tsqr(const PanelArgs& a, const TsqrShape& sh, double* scratch,
                             hipStream_t s);

// Panel from the Gram matrix (one grid exchange per sweep of columns); the
// scratch holds 2 x G x NS tagged partial sums (part) and 2 x (NS + bp^2)
// tagged sums (sums), NS = 256 x the upper-triangle 16 x 16 tiles of a
// bp x bp matrix (2560 for bp = 64), zeroed once.
constexpr int kMaxGramWGs = 256;
constexpr int64_t kGramSlots = 10 * 256;
constexpr int64_t kGramPartWords = 2LL * kMaxGramWGs * kGramSlots * 2;
constexpr int64_t kGramSumWords = 2LL * (kGramSlots + 64 * 64) * 2;
struct GramPanelArgs {
  PanelArgs p;                 // Y, ldy, m, b, V, Tm, tau, st, G, epoch_base
  unsigned long long* part;
  unsigned long long* sums;
};
bool gram_panel_shape(int64_t m, int b, int num_cus, PanelShape* out);
hipError_t launch_panel_gram(const GramPanelArgs& a, const PanelShape& sh, hipStream_t s);

// Explicit-Q pass: adjacent blocks of reflectors applied as one block of up
// to kGroupMax (orgqr_groups.hip).  Per group: k0, the first column; nb
// blocks at column offsets off[0] = 0 < off[1] < ... < off[nb] = w; the
// 16 x 16 tiles (ti, tj) of the Gram matrix V^T V that the merge reads
// (tile[n] = 8 ti + tj, those holding an entry (i, j) with block(i) <
// block(j)).  part holds ngroups x nsplit partial Gram matrices, then
// ngroups sums (each kGroupMax^2 doubles, only the listed tiles written);
// the merged T of the group at column k0 goes to Tg + k0 ldg (w x w,
// ldg >= kGroupMax).  Tm, ldt: the blocks' own T.
constexpr int kGroupMax = 128;
constexpr int kMaxGroupBlocks = 8;
constexpr int kGroupTiles = (kGroupMax / 16) * (kGroupMax / 16);
struct OrgqrGroup {
  int64_t k0;
  int nb, w, ntiles;
  int off[kMaxGroupBlocks + 1];
  unsigned char tile[kGroupTiles];
};
struct GroupArgs {
  const OrgqrGroup* groups; int ngroups;
  double* V; int64_t ldv; int64_t m;
  const double* Tm; int64_t ldt;
  double* Tg; int64_t ldg;
  double* part; int nsplit;
};
hipError_t launch_orgqr_groups(const GroupArgs& a, hipStream_t s);

// Y <- Y - V T^T (V^T Y) for a thin Y (mr x ncols, ncols <= 64), binary64,
// one launch (reflectors p >= b and columns >= ncols are
// treated as zero).  part: kMaxThinWGs x 4096 tagged values, sums: 4096;
// both zeroed once, epoch unique per launch.
constexpr int kMaxThinWGs = 256;
constexpr int64_t kThinPartWords = (int64_t)kMaxThinWGs * 4096 * 2;
constexpr int64_t kThinSumWords = 4096 * 2;
struct ThinApplyArgs {
  const double* V; int64_t ldv;
  const double* Tm; int64_t ldt; int b;
  int trans;                    // 1: Y <- Q^T Y (W = T^T Z),  0: Y <- Q Y (W = T Z)
  double* Y; int64_t ldy;
  int64_t mr; int ncols;
  int64_t rows_per_wg;          // set by the launcher
  unsigned long long* part;
  unsigned long long* sums;
  unsigned epoch_base;
  DevState* st;
};
hipError_t launch_thin_apply(ThinApplyArgs a, int num_cus, hipStream_t s);

// Look-ahead: the update (store, sample width qp) and the panel of the next
// block in one launch; supported when bp == qp == the panel's padded width.
bool update_panel_supported(int bp, int qp, const PanelShape& sh);
template <typename T>
hipError_t launch_update_panel(const UpdateArgs<T>& ua, int nsplit,
                               const PanelArgs& pa, const PanelShape& sh,
                               hipStream_t s);
// Workgroups of that launch resident per compute unit (0 if unknown).
template <typename T>
int update_panel_occupancy(const PanelShape& sh);
// Block 0: the first look-ahead sample (ua.bp = 0, no store, qp = 64) and the
// panel of block 0 in one launch; supported for 64-column panels.
bool sample_panel_supported(int qp, const PanelShape& sh);
template <typename T>
hipError_t launch_sample_panel(const UpdateArgs<T>& ua, int nsplit,
                               const PanelArgs& pa, const PanelShape& sh,
                               hipStream_t s);
template <typename T>
int sample_panel_occupancy(const PanelShape& sh);
// Look-ahead for blocks of at most 32 columns: the update and the next
// block's Gram panel (256 threads per workgroup) in one launch; supported
// when bp == qp == the panel's padded width (16 or 32).
bool update_gram_supported(int bp, int qp, const PanelShape& sh);
template <typename T>
hipError_t launch_update_gram(const UpdateArgs<T>& ua, int nsplit, const GramPanelArgs& ga,
                              const PanelShape& sh, hipStream_t s);
template <typename T>
int update_gram_occupancy(const PanelShape& sh);
// Shape of a Gram panel inside that launch: the fewest rows per thread whose
// grid has at most max_wgs workgroups.
bool gram_fused_shape(int64_t m, int b, int max_wgs, PanelShape* out);
// Ysum[r + k * ldy] = sum_s P_s[r + k * ldp] for r < m, k < b; 0 elsewhere
// for r < rows_pad, k < bp (binary64).
template <typename T>
hipError_t launch_gather_panel(const T* P, int64_t ldp, int64_t split_stride,
                               int nsplit, int64_t m, int b, int bp,
                               int64_t rows_pad, double* Ysum, int64_t ldy,
                               hipStream_t s);

// Spectral-norm estimate (spectral.hip).  Y: my x bp binary64 (ldy, zero
// columns up to bp); Z: split partials Z_s[row * bp + c] of nz rows (T).
// The launcher sets gy, gz (workgroups per matrix) and the row ranges; part
// holds (gy + gz) x 64 x 64 doubles.
constexpr int kMaxSpecWGs = 128;
template <typename T>
struct SpecGramArgs {
  const double* Y; int64_t ldy; int64_t my;
  const T* Z; int nsplit; int64_t split_stride; int64_t nz;
  int bp;
  double* part;
  const DevState* st;          // E0 scales the values
  int gy, gz;
  int64_t rows_per_wg_y, rows_per_wg_z;
};
struct SpecFinishArgs {
  const double* part; int gy, gz;
  DevState* st;
  double* trace; int block;    // trace[block] = estimate (block >= 0)
};
template <typename T>
hipError_t launch_spec_gram(SpecGramArgs<T>* a, hipStream_t s);
hipError_t launch_spec_finish(const SpecFinishArgs& a, hipStream_t s);
// Tm (64 x 64, ldt) = I / ||A||_F^2, the W factor of a power step.
hipError_t launch_scaled_identity(double* Tm, int64_t ldt, const DevState* st, hipStream_t s);

// GaLore subspace map (map.hip): out = (Q_new^T Q_old) M with split-K
// partials Cpart (nsplit x r_new x r_old) and C (r_new x r_old).
constexpr int kMaxMapSplits = 16;
int map_splits(int64_t r_new, int64_t r_old, int64_t m, int num_cus);
template <typename T>
hipError_t launch_subspace_map(const T* Qnew, int64_t ldqn, int64_t r_new, const T* Qold,
                               int64_t ldqo, int64_t r_old, const T* M, int64_t ldm,
                               int64_t m, int64_t n, T* out, int64_t ldo, T* Cpart,
                               T* C, int nsplit, hipStream_t s);

hipError_t launch_finalize(const double* normpart, int nparts, DevState* st,
                           DevState* mirror, double* trace_trail, double* trace_sub, int block,
                           int64_t k_after, int64_t k_cap, int mode,
                           double tol, int init, hipStream_t s);
template <typename T>
hipError_t launch_fill_identity(T* Q, int64_t ldq, int64_t m, int64_t k,
                                hipStream_t s);
template <typename T>
hipError_t launch_copy(const T* src, int64_t lds, T* dst, int64_t ldd,
                       int64_t rows, int64_t cols, hipStream_t s);
template <typename Ts, typename Td>
hipError_t launch_convert(const Ts* src, int64_t lds, Td* dst, int64_t ldd,
                          int64_t rows, int64_t cols, hipStream_t s);

}  // namespace rrf
