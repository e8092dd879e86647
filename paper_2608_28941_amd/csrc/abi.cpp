// C ABI and host driver of the range finder (Alg. 2, then explicit Q).
//
// Per block i (all on the plan's stream):
//   panel   (V_i, T_i, tau_i) <- Householder QR of Y_i       (geqrt step)
//   reduce  Z = V_i^T B[ib:m, :]                              (update step)
//   formW   W = T_i^T Z
//   sketch  Omega_{i+1}                                       (sketch step)
//   update  B[ib:m, :] -= V_i W; Y_{i+1} = B[(i+1)b:m, :] Omega_{i+1};
//           ||B_i||^2 and ||B[(i+1)b:m, :]||^2                (E step)
//   final   E, stop flag; the host reads the flag (8 bytes) once per block.
// Block 0 reads A and writes the workspace, so A itself is never modified.
// Q = H_0 ... H_{k-1} [I_k; 0] is then formed backward block by block with
// the same reduce / formW / update kernels (trans = 0).  V, T and tau are
// binary64 for both dtypes; for float plans Q is accumulated in binary64 and
// rounded once at the end, because rounding Q to float after each of the s
// block applications costs about 2 sqrt(s) u sqrt(k) in ||Q^T Q - I||_F.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "rrf_internal.h"

using namespace rrf;

namespace {

constexpr int kMaxUpdSplits = 8;
constexpr int kMaxRedSplits = 32;
constexpr int kOmLd = 256;        // Omega stored [c][q]: a batch of 256 sketch columns
constexpr int kPanelGrid = 0;      // column-by-column panel, one grid reduction per column
constexpr int kPanelTsqr = 1;      // tall-skinny QR + Householder reconstruction
constexpr int kPanelGram = 2;      // column recurrence from the Gram matrix, one exchange per sweep
constexpr int kPanelAuto = 3;      // kPanelGram for blocks of <= 32 columns, else kPanelGrid
constexpr int kTLd = 64;          // T stored like geqrt's T: 64 rows

struct Sizes {
  int64_t ldb, kcap, kcols;
  int64_t ldysum;
  size_t Bws, V, Tm, tau, Ypart, Ysum, Om, Zpart, W, Q, Q64, normpart, normtag, red,
      rowj, st, trace, tsqr, gx, tx, Yest, spec, Tpow, Tp, groups;
  // Every buffer at a 256-byte boundary (a caller-provided workspace is
  // carved in this order).
  size_t total() const {
    const size_t parts[] = {Bws, V, Tm, tau, Ypart, Ysum, Om, Zpart, W, Q, Q64,
                            normpart, normtag, tsqr, red, rowj, gx, tx, st, trace / 3,
                            trace / 3, trace / 3, Yest, spec, Tpow, Tp, groups};
    size_t t = 0;
    for (size_t x : parts)
      if (x) t += (std::max<size_t>(x, 256) + 255) / 256 * 256;
    return t;
  }
};

Sizes compute_sizes(rrf_dtype dt, int64_t m_max, int64_t n_max, int64_t b_max,
                    int64_t k_max) {
  Sizes z;
  const size_t e = dt == RRF_F32 ? 4 : 8;
  // 64 rows of slack: the reduce reads whole 64-row chunks of V.
  z.ldb = round_up(std::max<int64_t>(m_max, 1), 64) + 64;
  z.kcap = std::min(m_max, n_max);
  if (k_max > 0) z.kcap = std::min(z.kcap, k_max);
  z.kcols = z.kcap + 64;
  z.Bws = (size_t)z.ldb * n_max * e;
  z.V = (size_t)z.ldb * z.kcols * 8;
  z.Tm = (size_t)kTLd * z.kcols * 8;
  z.tau = (size_t)z.kcols * 8;
  z.Ypart = (size_t)kMaxUpdSplits * z.ldb * 64 * e;
  z.ldysum = z.ldb + 1024;   // >= the panel grid's padded row count
  z.Ysum = (size_t)z.ldysum * 64 * 8;
  // Omega and W carry zero rows up to the next multiple of the update chunk.
  z.Om = (size_t)(n_max + kUpdChunk) * kOmLd * e;
  z.Zpart = (size_t)kMaxRedSplits * n_max * 64 * 8;
  // W rows of up to 128 reflectors (the explicit-Q pass applies groups of
  // blocks as one); the bulk update uses 64.
  z.W = (size_t)(n_max + kUpdChunk) * kGroupMax * 8;
  z.Q = (size_t)z.ldb * std::max<int64_t>(z.kcap, 1) * e;
  z.Q64 = dt == RRF_F32 ? (size_t)z.ldb * std::max<int64_t>(z.kcap, 1) * 8 : 0;
  z.normpart = (size_t)(ceil_div(m_max, kUpdRows) * kMaxUpdSplits + 1) * 2 * 8;
  // The same partials as epoch-tagged words (two per value), when the
  // update's last workgroup finalizes.
  z.normtag = z.normpart * 2;
  // Panel partials: two epoch-tagged 64-bit words per value.
  z.red = (size_t)2 * kMaxPanelWGs * 64 * 2 * 8;
  z.rowj = (size_t)2 * 64 * 2 * 8;
  z.gx = (size_t)(kGramPartWords + kGramSumWords) * 8;
  z.tx = (size_t)(kThinPartWords + kThinSumWords) * 8;
  z.st = sizeof(DevState);
  z.trace = (size_t)3 * std::max<int64_t>(z.kcap, 1) * 8;
  // Spectral-norm estimate: the gathered next sample, the Gram partials;
  // power iterations: their scaled identity.
  z.Yest = (size_t)z.ldysum * 64 * 8;
  z.spec = (size_t)kMaxSpecWGs * 4096 * 8;
  z.Tpow = (size_t)64 * 64 * 8;
  // Explicit-Q pass: merged T of block groups (kGroupMax rows per column)
  // and the group list (blocks of at least one column each).
  z.Tp = (size_t)kGroupMax * z.kcols * 8;
  z.groups = (size_t)(z.kcols + 2) * sizeof(OrgqrGroup);
  // Tall-skinny QR panel: the largest tree over the block widths the plan
  // allows (the tree shrinks with the panel's rows).
  z.tsqr = 8;
  for (int bb = 16; bb <= pad16(std::max<int64_t>(b_max, 1)); bb *= 2) {
    TsqrShape ts;
    if (tsqr_shape(std::max<int64_t>(m_max, bb), bb, &ts))
      z.tsqr = std::max(z.tsqr, (size_t)ts.scratch_elems * 8);
  }
  return z;
}

}  // namespace

// Work credited to a stage for the sub-block that starts at column col.
struct SpecWork {
  int stage;
  int64_t col;
  double flops, bytes;
};

struct rrf_plan {
  rrf_dtype dtype;
  size_t elem;
  int64_t m_max, n_max, b_max, k_max;
  hipStream_t stream;
  int lookahead;             // factor the next panel during the update
  int device, num_cus;
  Sizes sz;
  std::vector<void*> dev_allocs;
  void *Bws, *Ypart, *Om, *Zpart, *W, *Q, *Q64;
  char* ws_base = nullptr;   // caller-provided device workspace, or null
  size_t ws_bytes = 0, ws_used = 0;
  double* tsqr;              // scratch of the tall-skinny QR panel
  double* Tp;                // merged T of block groups (explicit-Q pass)
  OrgqrGroup* groups_d;      // group list, device
  OrgqrGroup* groups_h;      // group list, pinned host staging
  int panel_mode;            // kPanelGrid, kPanelTsqr, kPanelGram or kPanelAuto
  double *V, *Tm, *tau, *Ysum;
  double *normpart, *trace_trail_d, *trace_sub_d, *trace_spec_d;
  unsigned long long* normtag;   // tagged norm partials (finalisation in the update)
  double *Yest, *spec_part, *Tpow;
  int power;                 // power iterations per block sample
  unsigned long long *red, *rowj, *gx, *tx;
  DevState* st;
  DevState* st_host;
  DevState* st_mirror;   // st_host's device address (the finalisation's copy)
  int stop_mode, timing, panel_target;
  int log;                   // RRF_LOG=1: one stderr line per run, one per block
  int gram_fused_max;         // most workgroups of a Gram panel inside the update's launch
  int sub_max;                // widest sub-block (16, 32 or 64 columns; 0: by size)
  unsigned spin_limit;       // poll rounds of a grid-wide wait (run state)
  unsigned panel_launches;   // epochs of the panel's tagged partials
  // last run
  int64_t last_m, last_n, last_k, last_b, nblocks;
  double E0, sigma2;
  std::vector<double> trace_trail, trace_sub, trace_spec;
  std::vector<int64_t> sub_start;   // first column of each sub-block of the last run
  std::vector<SpecWork> spec;       // speculative credits of the last run
  double ms[RRF_NUM_STAGES], flops[RRF_NUM_STAGES], bytes[RRF_NUM_STAGES];
  int64_t launches[RRF_NUM_STAGES];
  std::vector<hipEvent_t> events;
  hipEvent_t state_ev = nullptr;   // the launch holding a stop test has completed
  void* map_c = nullptr;           // subspace map: split partials and C
  size_t map_c_bytes = 0;
  std::vector<int> event_stage;
  size_t events_used;
};

namespace {

rrf_status hip_fail(hipError_t e) {
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) return RRF_ERR_NOMEM;
  return RRF_ERR_HIP;
}

// RRF_FAULT_ALLOC=N makes the N-th device allocation of a plan fail (tests).
// With a caller-provided workspace the buffers are carved from it instead
// (256-byte boundaries, in the order of Sizes::total).
hipError_t dev_alloc(rrf_plan* p, void** out, size_t bytes, int* counter) {
  if (p->ws_base) {
    const size_t b = (std::max<size_t>(bytes, 256) + 255) / 256 * 256;
    if (p->ws_used + b > p->ws_bytes) return hipErrorOutOfMemory;
    *out = p->ws_base + p->ws_used;
    p->ws_used += b;
    return hipSuccess;
  }
  ++*counter;
  const char* f = std::getenv("RRF_FAULT_ALLOC");
  if (f && std::atoi(f) == *counter) return hipErrorOutOfMemory;
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(out, bytes);
  if (e == hipSuccess) p->dev_allocs.push_back(*out);
  return e;
}

void free_plan(rrf_plan* p) {
  for (void* q : p->dev_allocs) (void)hipFree(q);
  p->dev_allocs.clear();
  if (p->st_host) (void)hipHostFree(p->st_host);
  if (p->groups_h) (void)hipHostFree(p->groups_h);
  for (hipEvent_t e : p->events) (void)hipEventDestroy(e);
  if (p->state_ev) (void)hipEventDestroy(p->state_ev);
  if (p->map_c) (void)hipFree(p->map_c);
  delete p;
}

int upd_splits(int64_t mr, int64_t n, int num_cus) {
  const int64_t row_wgs = ceil_div(mr, kUpdRows);
  int64_t s = ceil_div(4 * (int64_t)num_cus, std::max<int64_t>(row_wgs, 1));
  s = std::min<int64_t>(s, kMaxUpdSplits);
  s = std::min<int64_t>(s, std::max<int64_t>(1, n / 256));
  return (int)std::max<int64_t>(s, 1);
}

// Column splits of the fused update + panel launch.  The panel holds G
// workgroup slots for most of the launch, and the update's workgroups run in
// rounds over the free slots; the split count that minimises rounds x
// columns per split avoids a nearly empty last round (fewest splits on ties:
// less partial-sample traffic).
int upd_splits_fused(int64_t mr, int64_t n, int64_t free_slots) {
  const int64_t row_wgs = std::max<int64_t>(ceil_div(mr, kUpdRows), 1);
  const int64_t smax = std::max<int64_t>(1, std::min<int64_t>(kMaxUpdSplits, n / 256));
  const int64_t slots = std::max<int64_t>(free_slots, 1);
  int best = 1;
  double best_cost = 1e300;
  for (int64_t sp = 1; sp <= smax; ++sp) {
    const double cost = (double)ceil_div(row_wgs * sp, slots) / (double)sp;
    if (cost < best_cost * (1.0 - 1e-9)) {
      best_cost = cost;
      best = (int)sp;
    }
  }
  return best;
}

int red_splits(int64_t mr, int64_t n, int num_cus) {
  const int64_t col_wgs = ceil_div(n, kRedCols);
  int64_t s = ceil_div(4 * (int64_t)num_cus, std::max<int64_t>(col_wgs, 1));
  s = std::min<int64_t>(s, kMaxRedSplits);
  s = std::min<int64_t>(s, std::max<int64_t>(1, mr / kRedChunk));
  return (int)std::max<int64_t>(s, 1);
}

// Row splits of a reduce over few columns (the explicit-Q pass, a general
// block reflector), where 32 splits leave each workgroup streaming hundreds
// of rows on its own: up to 128 splits of at least kNarrowRows rows, two
// workgroups per compute unit, within the partial buffer (max_splits); never
// fewer than the wide-matrix choice.  Each split's rows are a chain of
// dependent chunks, so short splits keep a narrow reduce off the latency of
// that chain.
constexpr int kNarrowRows = 32;

// Splits of a length len (in multiples of gran) into s parts, each part
// `other` workgroups wide, on `slots` resident workgroups: the s in [1, smax]
// that minimises rounds x (part length + one granule of per-workgroup
// set-up), fewest splits on ties (a nearly empty last round costs as much as
// a full one).
int64_t splits_by_rounds(int64_t other, int64_t len, int64_t gran, int64_t slots,
                         int64_t smax) {
  other = std::max<int64_t>(other, 1);
  slots = std::max<int64_t>(slots, 1);
  int64_t best = 1, best_cost = INT64_MAX;
  for (int64_t s = 1; s <= std::max<int64_t>(smax, 1); ++s) {
    const int64_t cost =
        ceil_div(other * s, slots) * (round_up(ceil_div(len, s), gran) + gran);
    if (cost < best_cost) {
      best_cost = cost;
      best = s;
    }
  }
  return best;
}

// Both 128-reflector kernels of the explicit-Q pass (reduce and update) hold
// two workgroups per compute unit: their LDS and VGPR use allow no more.
constexpr int kWide128PerCu = 2;

int red_splits_narrow(int64_t mr, int64_t n, int bp, int num_cus, int64_t max_splits) {
  const int64_t col_wgs = ceil_div(n, red_cols(bp));
  if (bp == 128) {
    // Never more than one round's worth: each split adds a partial for
    // formW to read.
    const int64_t slots = (int64_t)kWide128PerCu * num_cus;
    return (int)splits_by_rounds(col_wgs, mr, kNarrowRows, slots,
                                 std::min<int64_t>({ceil_div(slots, col_wgs), 128, max_splits,
                                                    std::max<int64_t>(1, mr / kNarrowRows)}));
  }
  int64_t s = ceil_div(2 * (int64_t)num_cus, std::max<int64_t>(col_wgs, 1));
  s = std::min<int64_t>({s, 128, max_splits, std::max<int64_t>(1, mr / kNarrowRows)});
  // At 128 reflectors two workgroups per compute unit are the whole target:
  // more splits only add partial sums for formW to read.
  if (bp < 128) s = std::max<int64_t>(s, red_splits(mr, n, num_cus));
  // The wide-matrix choice assumes 64 reflectors; the buffer bound holds for
  // any width.
  return (int)std::max<int64_t>(1, std::min<int64_t>(s, max_splits));
}

// ---- timing / statistics --------------------------------------------------

void stats_reset(rrf_plan* p) {
  for (int i = 0; i < RRF_NUM_STAGES; ++i) {
    p->ms[i] = p->flops[i] = p->bytes[i] = 0.0;
    p->launches[i] = 0;
  }
  p->events_used = 0;
  p->event_stage.clear();
}

hipError_t ev_mark(rrf_plan* p, int stage, hipStream_t s) {
  if (!p->timing) return hipSuccess;
  if (p->events_used == p->events.size()) {
    hipEvent_t e;
    hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) return r;
    p->events.push_back(e);
  }
  if (p->event_stage.size() < p->events_used + 1) p->event_stage.resize(p->events_used + 1);
  p->event_stage[p->events_used] = stage;
  return hipEventRecord(p->events[p->events_used++], s);
}

// Pairs of events (begin, end) were recorded per launch.
void stats_collect(rrf_plan* p) {
  if (!p->timing) return;
  for (size_t i = 0; i + 1 < p->events_used; i += 2) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p->events[i], p->events[i + 1]) == hipSuccess)
      p->ms[p->event_stage[i]] += ms;
  }
}

// Launch on stream s_ with per-launch statistics (and HIP-event timing when
// enabled: a begin/end pair on the launch's own stream).
#define RRF_LAUNCH_ON(p, s_, stage, fl, by, expr)          \
  do {                                                     \
    hipError_t e_ = ev_mark((p), (stage), (s_));           \
    if (e_ == hipSuccess) e_ = (expr);                     \
    if (e_ == hipSuccess) e_ = ev_mark((p), (stage), (s_)); \
    if (e_ != hipSuccess) return hip_fail(e_);             \
    (p)->launches[stage] += 1;                             \
    (p)->flops[stage] += (fl);                             \
    (p)->bytes[stage] += (by);                             \
  } while (0)
#define RRF_LAUNCH(p, stage, fl, by, expr) RRF_LAUNCH_ON(p, (p)->stream, stage, fl, by, expr)

// Epoch base of the next panel launch: a nonzero multiple of 128 (the
// tagged partials are zeroed at plan creation and a step adds j + 1 <= 64).
unsigned next_epoch(rrf_plan* p) {
  p->panel_launches = (p->panel_launches + 1u) & 0x1FFFFFFu;
  if (p->panel_launches == 0u) p->panel_launches = 1u;
  return p->panel_launches << 7;
}

hipError_t read_state(rrf_plan* p) {
  hipError_t e = hipMemcpyAsync(p->st_host, p->st, sizeof(DevState),
                                hipMemcpyDeviceToHost, p->stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(p->stream);
}

// The panel algorithm for a block of b columns.  Narrow panels take the Gram
// form (its column steps are cheap at 32 columns and it exchanges once per
// sweep); 64-column panels take the column-by-column grid.  The look-ahead
// hides either inside the update.
int panel_alg(const rrf_plan* p, int64_t b) {
  if (p->panel_mode != kPanelAuto) return p->panel_mode;
  return pad16(b) <= 32 ? kPanelGram : kPanelGrid;
}

// The route an m x b panel takes: the plan's algorithm when its
// register-resident grid fits on the device, else the tall-skinny QR, whose
// tree has no register-capacity bound (Alg. 2 puts no limit on m).  -1 if
// no route fits (beyond the tree's depth).  sh->rows_pad is the row count
// the gathered panel must cover.
int panel_route(const rrf_plan* p, int64_t m, int b, PanelShape* sh) {
  const int alg = panel_alg(p, b);
  if (alg == kPanelGram && gram_panel_shape(m, b, p->num_cus, sh)) return kPanelGram;
  if (alg == kPanelGrid && panel_shape(m, b, p->num_cus, p->panel_target, sh)) return kPanelGrid;
  TsqrShape ts;
  if (!tsqr_shape(m, b, &ts)) return -1;
  sh->bp = ts.bp;
  sh->rpt = 0;
  sh->G = 0;
  sh->rows_pad = ts.rows_pad;
  return kPanelTsqr;
}
bool panel_fits(const rrf_plan* p, int64_t m, int b, PanelShape* sh) {
  return panel_route(p, m, b, sh) >= 0;
}

// Panel QR of the gathered panel pa.Y (m x b) into pa.V, pa.Tm, pa.tau by
// route alg (from panel_route, with sh its shape; pa.Y is overwritten by the
// tall-skinny QR).
hipError_t run_panel(rrf_plan* p, PanelArgs& pa, int alg, const PanelShape& sh,
                     hipStream_t s) {
  if (alg == kPanelGram) {
    GramPanelArgs ga{};
    ga.p = pa;
    ga.p.epoch_base = next_epoch(p);
    ga.part = p->gx;
    ga.sums = p->gx + kGramPartWords;
    return launch_panel_gram(ga, sh, s);
  }
  if (alg == kPanelTsqr) {
    TsqrShape ts;
    if (!tsqr_shape(pa.m, pa.b, &ts)) return hipErrorInvalidValue;
    return launch_panel_tsqr(pa, ts, p->tsqr, s);
  }
  if (alg != kPanelGrid) return hipErrorInvalidValue;
  pa.epoch_base = next_epoch(p);
  return launch_panel(pa, sh, s);
}

// A grid-wide wait that gave up stays recorded in the run state until
// cleared; entry points clear it before their own launches.
hipError_t clear_wait_error(rrf_plan* p) {
  return hipMemsetAsync(&p->st->barrier_err, 0, sizeof(int), p->stream);
}

// X (mr x ncols) <- (I - V T V^T)^T X (trans) or (I - V T V^T) X, with V, T
// already zero padded to bp columns in plan-compatible layout.
template <typename T>
rrf_status apply_wy(rrf_plan* p, int trans, const double* V, int64_t ldv,
                    const double* Tm, int64_t ldt, int b, int bp, T* X,
                    int64_t ldx, int64_t mr, int64_t ncols, int stage,
                    T* Zs = nullptr, T* Ws = nullptr) {
  if (mr <= 0 || ncols <= 0) return RRF_OK;
  if (!Zs) Zs = (T*)p->Zpart;
  if (!Ws) Ws = (T*)p->W;
  const double e = (double)sizeof(T);
  const int sr0 = red_splits_narrow(mr, ncols, bp, p->num_cus,
                                    (int64_t)(p->sz.Zpart / 8) / (ncols * bp));
  ReduceArgs<T> ra{};
  ra.X = X; ra.ldx = ldx; ra.mr = mr; ra.n = ncols;
  ra.V = V; ra.ldv = ldv; ra.bp = bp;
  ra.Z = Zs; ra.split_stride = ncols * bp;
  ra.rows_per_split = round_up(ceil_div(mr, sr0), kNarrowRows);
  const int sr = (int)ceil_div(mr, ra.rows_per_split);
  // The split partials (sr x ncols x bp) and W (ncols rows of bp, padded to
  // the update chunk) must fit their buffers.
  if ((size_t)sr * ncols * bp * sizeof(T) > p->sz.Zpart ||
      (size_t)round_up(ncols, kUpdChunk) * bp * sizeof(T) > p->sz.W)
    return RRF_ERR_INTERNAL;
  const double fl = 2.0 * mr * ncols * b;
  RRF_LAUNCH(p, stage == RRF_STAGE_UPDATE ? RRF_STAGE_REDUCE : stage, fl,
             e * mr * ncols, launch_reduce<T>(ra, sr, p->stream));
  FormWArgs<T> fa{};
  fa.Z = Zs; fa.nsplit = sr; fa.split_stride = ra.split_stride;
  fa.Tm = Tm; fa.ldt = ldt; fa.W = Ws; fa.n = ncols; fa.bp = bp;
  fa.trans = trans;
  fa.b = b;
  RRF_LAUNCH(p, stage == RRF_STAGE_UPDATE ? RRF_STAGE_FORMW : stage,
             (double)ncols * b * b, e * ncols * b * (sr + 1),
             launch_formw<T>(fa, p->stream));
  UpdateArgs<T> ua{};
  ua.src = X; ua.lds = ldx; ua.dst = X; ua.ldd = ldx; ua.mr = mr; ua.n = ncols;
  ua.V = V; ua.ldv = ldv; ua.bp = bp; ua.W = Ws; ua.ldw = bp;
  ua.Om = nullptr; ua.ldo = kOmLd; ua.qp = 0; ua.P = nullptr; ua.ldp = 0;
  ua.split_stride = 0; ua.s0 = 0; ua.normpart = nullptr;
  // No sample here, so column splits cost nothing but a reload of the V
  // rows: about four workgroups per compute unit, 32 columns or more each.
  {
    const int64_t row_wgs = std::max<int64_t>(ceil_div(mr, kUpdRows), 1);
    int64_t su0 = ceil_div(4 * (int64_t)p->num_cus, row_wgs);
    su0 = std::max<int64_t>(1, std::min<int64_t>({su0, ncols / 32, 64}));
    // At 128 reflectors, whole rounds over the two resident workgroups per
    // compute unit.
    if (bp == 128)
      su0 = splits_by_rounds(row_wgs, ncols, 2 * kUpdChunk,
                             (int64_t)kWide128PerCu * p->num_cus,
                             std::max<int64_t>(1, std::min<int64_t>(ncols / 32, 64)));
    ua.cols_per_split = round_up(ceil_div(ncols, su0), 2 * kUpdChunk);
  }
  const int su = (int)ceil_div(ncols, ua.cols_per_split);
  RRF_LAUNCH(p, stage, fl, 2.0 * e * mr * ncols, launch_update<T>(ua, su, p->stream));
  return RRF_OK;
}

// The update launch u finalizes its own norm partials (the stop test of
// the finalize kernel, in its last workgroup): nparts update workgroups,
// trace index block (< 0: none), init for the first sample.
template <typename T>
void set_finalize(rrf_plan* p, UpdateArgs<T>& u, int nparts, int block, int64_t k_after,
                  int64_t k_cap, int mode, double tol, int init) {
  u.normtag = p->normtag;
  u.fin_epoch = next_epoch(p) + 1u;
  u.fin_nwg = nparts;
  FinalizeArgs& f = u.fin;
  f.nparts = nparts; f.st = p->st; f.mirror = p->st_mirror; f.tt = p->trace_trail_d; f.ts = p->trace_sub_d;
  f.block = block; f.k_after = k_after; f.k_cap = k_cap; f.mode = mode; f.tol = tol;
  f.init = init;
}

template <typename T>
rrf_status run_impl(rrf_plan* p, const T* A, int64_t m, int64_t n, int64_t lda,
                    double tol, int64_t b, uint64_t seed, int64_t* k_out,
                    bool* warn_kmax) {
  hipStream_t s = p->stream;
  const int64_t ldb = p->sz.ldb;
  T* Bws = (T*)p->Bws;
  double* V = p->V;
  double* Tm = p->Tm;
  double* tau = p->tau;
  T* Yp = (T*)p->Ypart;
  T* Om = (T*)p->Om;
  T* Q = (T*)p->Q;
  const double e = (double)p->elem;
  int64_t kcap = std::min(m, n);
  if (p->k_max > 0) kcap = std::min(kcap, p->k_max);
  const int mode = p->stop_mode;
  p->trace_trail.clear();
  p->trace_sub.clear();
  p->sub_start.clear();
  p->spec.clear();
  p->nblocks = 0;

  // Blocks of b columns (the last one ragged at k_cap) run as sub-blocks of
  // at most 64 columns: Householder QR is column by column, so factoring a
  // block's first 64 columns, updating, and sampling the rest from the
  // updated B gives the block's reflectors (Q_1^T (B Omega_2) =
  // (Q_1^T B) Omega_2).  The stop test runs at the end of each block only.
  //
  // The sub-block width: 64 columns, or 32 when the matrix is small (at most
  // 512 MiB).  There a 64-column update is short beside the 64-column panel
  // factored inside its launch (4096 x 11008 fp32: about 100 us against
  // 300 us), while 32-column sub-blocks put a Gram panel of about the
  // update's length beside each update (15.1 -> 12.7 ms per run there; at
  // 16384 x 16384 fp64 64 columns stay faster, 33.5 against 45.6 ms).
  // The spectral stop test estimates from the next block's first min(b, 64)
  // sketch columns, the sample of a 64-column sub-block.
  int sub_max = mode == RRF_STOP_SPECTRAL ? kMaxBlock : p->sub_max;
  if (sub_max == 0) {
    sub_max = kMaxBlock;
    PanelShape sh32;
    if (p->lookahead != 0 && p->power == 0 && p->panel_mode == kPanelAuto &&
        std::min(b, kcap) > 32 && (double)m * (double)n * e <= 512.0 * (1 << 20) &&
        gram_fused_shape(m, 32, p->gram_fused_max, &sh32))
      sub_max = 32;
  }
  auto sub_width = [&](int64_t kk) -> int64_t {
    if (kk >= kcap) return 0;
    const int64_t be = std::min((kk / b) * b + b, kcap);
    return std::min<int64_t>(sub_max, be - kk);
  };
  // Work credited to a stage for the sub-block that starts at column col,
  // taken back after the run if the run stopped before that sub-block (a
  // sample, panel or W queued ahead of the stop test that the method never
  // used).
  auto spec = [&](int stage, int64_t col, double fl, double by) {
    p->spec.push_back(SpecWork{stage, col, fl, by});
  };

  // Sketch columns are generated kOmLd at a time: Om holds the global
  // columns [om_k0, om_k0 + kOmLd) (row-major, rows padded with zeros to the
  // update's chunk), and a batch is generated when a sample needs a column
  // window beyond the one held (one launch per batch of sub-blocks instead
  // of one per sub-block).  Columns of a window past the sample's width are
  // other sketch columns; the sample's unused columns are never read.
  int64_t om_k0 = -1;
  auto sketch_window = [&](int64_t col, int qp, T** win) -> rrf_status {
    if (om_k0 < 0 || col < om_k0 || col + qp > om_k0 + kOmLd) {
      const int64_t nc = std::min<int64_t>(kOmLd, kcap - col);
      RRF_LAUNCH(p, RRF_STAGE_SKETCH, 0.0, e * n * nc,
                 launch_sketch<T>(seed, n, round_up(n, kUpdChunk), col, nc, Om, kOmLd, 1, s));
      spec(RRF_STAGE_SKETCH, col, 0.0, e * n * nc);
      om_k0 = col;
    }
    *win = Om + (col - om_k0);
    return RRF_OK;
  };

  // Initial sample Y_0 = A Omega_0 and ||A||_F^2 in one read of A.
  const int64_t b0 = sub_width(0);
  const int q0 = b0 > 0 ? pad16(b0) : 0;
  T* om_win = Om;
  if (b0 > 0) {
    rrf_status rs = sketch_window(0, q0, &om_win);
    if (rs != RRF_OK) return rs;
  }
  // A wait error left by an earlier call is cleared before the first launch
  // (the first sample's finalisation waits on the tagged norm partials).
  {
    hipError_t he0 = clear_wait_error(p);
    if (he0 != hipSuccess) return hip_fail(he0);
  }
  UpdateArgs<T> u{};
  u.src = A; u.lds = lda; u.dst = nullptr; u.ldd = 0; u.mr = m; u.n = n;
  u.V = nullptr; u.ldv = 0; u.bp = 0; u.W = nullptr; u.ldw = 0;
  u.Om = om_win; u.ldo = kOmLd; u.qp = q0; u.P = Yp; u.ldp = ldb;
  u.split_stride = ldb * 64; u.s0 = 0; u.normpart = p->normpart;
  {
    const int su0 = upd_splits(m, n, p->num_cus);
    u.cols_per_split = round_up(ceil_div(n, su0), 2 * kUpdChunk);
  }
  int ysplits = (int)ceil_div(n, u.cols_per_split);
  int nparts = (int)(ceil_div(m, kUpdRows) * ysplits);
  // E0 and sigma^2 from the sample's own launch (its last workgroup).
  set_finalize(p, u, nparts, -1, 0, kcap, mode, tol, 1);
  RRF_LAUNCH(p, RRF_STAGE_SAMPLE, 2.0 * m * n * b0, e * (m * n + m * b0),
             launch_update<T>(u, ysplits, s));
  hipError_t he = read_state(p);
  if (he != hipSuccess) return hip_fail(he);
  if (p->st_host->barrier_err) return RRF_ERR_INTERNAL;
  if (p->st_host->nonfinite) return RRF_ERR_NONFINITE;
  const int power = p->power;
  if (power > 0)
    RRF_LAUNCH(p, RRF_STAGE_SAMPLE, 0.0, 0.0, launch_scaled_identity(p->Tpow, 64, p->st, s));

  // Look-ahead (the paper's two-queue overlap, Sec. 5, on one GPU): the
  // update of sub-block i samples Omega_{i+2} instead of Omega_{i+1}; the
  // sample for sub-block i + 1 is the one the previous update took,
  // S_{i+1} = B^(i) Omega_{i+1}, brought up to date with the redundant panel
  // update Y_{i+1} = Q_i^T S_{i+1} as soon as W_i exists (Q_i^T (B Omega) =
  // (Q_i^T B) Omega).  The panel of sub-block i + 1 is then factored by a
  // few workgroups of the update's own launch while the rest update B.
  // It pays when the panel grid is small: a panel of more than a quarter of
  // the compute units takes too many slots from the update it runs beside.
  // Power iterations need the whole updated trailing matrix before the
  // sample, so they run without it.
  // Blocks of at most 32 columns take their panels from the Gram matrix
  // (la_gram); wider ones column by column.
  const int alg0 = panel_alg(p, b0);
  const bool la_gram = alg0 == kPanelGram && pad16(b0) <= 32;
  bool la = p->lookahead != 0 && power == 0 && kcap > b0 && (alg0 == kPanelGrid || la_gram);
  // The shape of the look-ahead panel of a sub-block (mr rows, width bb).
  auto la_shape = [&](int64_t mr, int64_t bb, PanelShape* sh) -> bool {
    if (la_gram) return gram_fused_shape(mr, (int)bb, p->gram_fused_max, sh);
    return panel_shape(mr, (int)bb, p->num_cus, p->panel_target, sh) && sh->G <= p->num_cus / 4;
  };
  if (la) {
    PanelShape sh1;
    la = la_shape(m - b0, sub_width(b0), &sh1);
  }
  int64_t k = 0;
  int64_t yoff = 0;          // row offset of the next sample in the slabs
  int blk = 0;               // blocks finished (stop tests run)
  int sub = 0;               // sub-blocks started
  bool panel_ready = false;  // the panel of this sub-block was factored by the last update
  bool stop = p->st_host->stop != 0;
  bool w_ready = false;      // W of this sub-block was formed at the end of the last one
  bool w_gathered = false;   // ... together with its look-ahead gather
  double E_prev2 = 0.0;      // the stopping quantity one state read earlier

  // The look-ahead gather of the sample S that the panel of sub-block
  // kk + bb is factored from (sums of the split partials, slab rows from yo,
  // ys splits, rows kk..m), as the look-ahead branch below issues it.  It
  // needs only the update before sub-block kk, so it rides in the formW
  // launch of sub-block kk.  False: no look-ahead panel follows.
  auto la_gather = [&](int64_t kk, int64_t bb, int64_t yo, int ys, GatherArgs<T>* g,
                       double* gby) -> bool {
    const int64_t bn = sub_width(kk + bb);
    if (!la || bn <= 0) return false;
    const int64_t mpp = m - kk;
    PanelShape shn;
    if (!la_shape(mpp - bb, bn, &shn)) return false;
    g->P = Yp + yo; g->ldp = ldb; g->split_stride = ldb * 64; g->nsplit = ys;
    g->m = mpp; g->b = (int)bn; g->bp = pad16(bn); g->rows_pad = bb + shn.rows_pad;
    g->Y = p->Ysum; g->ldy = p->sz.ldysum;
    *gby = e * mpp * bn * ys + 8.0 * mpp * bn;
    return true;
  };
  // Z = V^T B[kk:m, :] and W = T^T Z of the sub-block at kk (width bb),
  // from the rows kk..m of sx; speculative when queued ahead of a stop test.
  // ga (nullable): the look-ahead gather for sub-block kk + bb, in the same
  // launch as formW (gby: its bytes).
  auto issue_w = [&](int64_t kk, int64_t bb, const T* sx, int64_t ldsx,
                     bool speculative, const GatherArgs<T>* ga = nullptr,
                     double gby = 0.0) -> rrf_status {
    const int64_t mpp = m - kk;
    const int bpp = pad16(bb);
    const int sr0 = red_splits(mpp, n, p->num_cus);
    ReduceArgs<T> ra{};
    ra.X = sx + kk; ra.ldx = ldsx; ra.mr = mpp; ra.n = n;
    ra.V = V + kk + kk * ldb; ra.ldv = ldb; ra.bp = bpp;
    ra.Z = (T*)p->Zpart; ra.split_stride = n * bpp;
    ra.rows_per_split = round_up(ceil_div(mpp, sr0), kRedChunk);
    const int sr = (int)ceil_div(mpp, ra.rows_per_split);
    const double rfl = 2.0 * mpp * n * bb, rby = e * mpp * n;
    RRF_LAUNCH(p, RRF_STAGE_REDUCE, rfl, rby, launch_reduce<T>(ra, sr, s));
    FormWArgs<T> fa{};
    fa.Z = (T*)p->Zpart; fa.nsplit = sr; fa.split_stride = ra.split_stride;
    fa.Tm = Tm + kk * kTLd; fa.ldt = kTLd; fa.W = (T*)p->W; fa.n = n; fa.bp = bpp;
    fa.trans = 1;
    fa.b = (int)bb;
    if (ga) fa.g = *ga;
    const double wfl = 1.0 * n * bb * bb, wby = e * n * bb * (sr + 1);
    RRF_LAUNCH(p, RRF_STAGE_FORMW, wfl, wby + (ga ? gby : 0.0), launch_formw<T>(fa, s));
    if (speculative) {
      spec(RRF_STAGE_REDUCE, kk, rfl, rby);
      spec(RRF_STAGE_FORMW, kk, wfl, wby);
    }
    if (ga) spec(RRF_STAGE_FORMW, kk + bb, 0.0, gby);
    return RRF_OK;
  };
  auto panel_flops = [](double mr, double bb) {
    return 2.0 * mr * bb * bb - 2.0 / 3.0 * bb * bb * bb + 1.0 * mr * bb * bb;
  };
  // Power iterations (the conclusion's proposal for slowly decaying
  // spectra): the gathered sample Y in Ysum (rows kk..m, width bb) becomes
  // (B B^T)^q Y on the rows kk..m of sx.  Each step is a reduce (Z = B^T Y as
  // split partials), a formW with T = I / ||A||_F^2 (the scale keeps the
  // products bounded and leaves the reflectors unchanged: QR of Y D has the
  // reflectors of Y for positive diagonal D), a sample-only pass P = B Z and
  // a gather back into Ysum.
  auto power_steps = [&](int64_t kk, int64_t bb, const T* sx, int64_t ldsx, int64_t rows_pad,
                         bool speculative) -> rrf_status {
    const int64_t mpp = m - kk;
    const int bpp = pad16(bb);
    for (int it = 0; it < power; ++it) {
      const int sr0 = red_splits(mpp, n, p->num_cus);
      ReduceArgs<T> ra{};
      ra.X = sx + kk; ra.ldx = ldsx; ra.mr = mpp; ra.n = n;
      ra.V = p->Ysum; ra.ldv = p->sz.ldysum; ra.bp = bpp;
      ra.Z = (T*)p->Zpart; ra.split_stride = n * bpp;
      ra.rows_per_split = round_up(ceil_div(mpp, sr0), kRedChunk);
      const int sr = (int)ceil_div(mpp, ra.rows_per_split);
      const double fl = 2.0 * mpp * n * bb;
      const double rby = e * mpp * n, wby = e * n * bb * (sr + 1);
      RRF_LAUNCH(p, RRF_STAGE_SAMPLE, fl, rby, launch_reduce<T>(ra, sr, s));
      FormWArgs<T> fa{};
      fa.Z = (T*)p->Zpart; fa.nsplit = sr; fa.split_stride = ra.split_stride;
      fa.Tm = p->Tpow; fa.ldt = 64; fa.W = (T*)p->W; fa.n = n; fa.bp = bpp;
      fa.trans = 1; fa.b = (int)bb;
      RRF_LAUNCH(p, RRF_STAGE_SAMPLE, 1.0 * n * bb, wby, launch_formw<T>(fa, s));
      UpdateArgs<T> us{};
      us.src = sx + kk; us.lds = ldsx; us.dst = nullptr; us.ldd = 0; us.mr = mpp; us.n = n;
      us.V = nullptr; us.ldv = 0; us.bp = 0; us.W = nullptr; us.ldw = 0;
      us.Om = (T*)p->W; us.ldo = bpp; us.qp = bpp; us.P = Yp; us.ldp = ldb;
      us.split_stride = ldb * 64; us.s0 = 0; us.normpart = nullptr;
      us.cols_per_split = round_up(ceil_div(n, upd_splits(mpp, n, p->num_cus)), 2 * kUpdChunk);
      const int sus = (int)ceil_div(n, us.cols_per_split);
      const double uby = e * (mpp * n + mpp * bb);
      RRF_LAUNCH(p, RRF_STAGE_SAMPLE, fl, uby, launch_update<T>(us, sus, s));
      const double gby = e * mpp * bb * sus + 8.0 * mpp * bb;
      RRF_LAUNCH(p, RRF_STAGE_SAMPLE, 0.0, gby,
                 launch_gather_panel<T>(Yp, ldb, ldb * 64, sus, mpp, (int)bb, bpp, rows_pad,
                                        p->Ysum, p->sz.ldysum, s));
      if (speculative)
        spec(RRF_STAGE_SAMPLE, kk, 2.0 * fl + 1.0 * n * bb, rby + wby + uby + gby);
    }
    return RRF_OK;
  };
  // Spectral-norm estimate of B[kk:m, :] (spectral stop mode) from its
  // sample Y = B[kk:m, :] Omega' (binary64, rows kk..m at Y, width bb, zero
  // columns up to pad16(bb)): Z = B^T Y, the Gram matrices of Y and Z, and
  // the largest eigenvalue of their pencil into the run state and trace.
  auto spectral = [&](int64_t kk, int64_t bb, const double* Yy, int64_t ldyy,
                      int trace_block) -> rrf_status {
    const int64_t mpp = m - kk;
    const int bpp = pad16(bb);
    const int sr0 = red_splits(mpp, n, p->num_cus);
    ReduceArgs<T> ra{};
    ra.X = Bws + kk; ra.ldx = ldb; ra.mr = mpp; ra.n = n;
    ra.V = Yy; ra.ldv = ldyy; ra.bp = bpp;
    ra.Z = (T*)p->Zpart; ra.split_stride = n * bpp;
    ra.rows_per_split = round_up(ceil_div(mpp, sr0), kRedChunk);
    const int sr = (int)ceil_div(mpp, ra.rows_per_split);
    RRF_LAUNCH(p, RRF_STAGE_FINALIZE, 2.0 * mpp * n * bb, e * mpp * n,
               launch_reduce<T>(ra, sr, s));
    SpecGramArgs<T> ga{};
    ga.Y = Yy; ga.ldy = ldyy; ga.my = mpp;
    ga.Z = (T*)p->Zpart; ga.nsplit = sr; ga.split_stride = n * bpp; ga.nz = n;
    ga.bp = bpp; ga.part = p->spec_part; ga.st = p->st;
    RRF_LAUNCH(p, RRF_STAGE_FINALIZE, 2.0 * (mpp + n) * bpp * bpp,
               8.0 * mpp * bpp + e * n * bpp * sr, launch_spec_gram<T>(&ga, s));
    SpecFinishArgs fa{};
    fa.part = p->spec_part; fa.gy = ga.gy; fa.gz = ga.gz; fa.st = p->st;
    fa.trace = p->trace_spec_d; fa.block = trace_block;
    RRF_LAUNCH(p, RRF_STAGE_FINALIZE, 0.0, 8.0 * 4096 * (ga.gy + ga.gz),
               launch_spec_finish(fa, s));
    return RRF_OK;
  };
  while (!stop) {
    const int64_t bi = sub_width(k);
    const int bp = pad16(bi);
    const int64_t mp = m - k;
    p->sub_start.push_back(k);
    const int64_t k_next = k + bi;
    const bool at_end = k_next == kcap || k_next % b == 0;   // a stop test follows
    const int64_t b_next = sub_width(k_next);
    bool s1_done = false;      // sub-block 0: S_1 = A Omega_1 taken with the panel
    if (panel_ready) {
      panel_ready = false;
    } else {
      PanelShape sh;
      const int route = panel_route(p, mp, (int)bi, &sh);
      if (route < 0) return RRF_ERR_SHAPE;
      RRF_LAUNCH(p, RRF_STAGE_PANEL, 0.0, e * mp * bi * ysplits + 8.0 * mp * bi,
                 launch_gather_panel<T>(Yp + yoff, ldb, ldb * 64, ysplits, mp,
                                        (int)bi, bp, sh.rows_pad, p->Ysum,
                                        p->sz.ldysum, s));
      PanelArgs pa{};
      pa.Y = p->Ysum; pa.ldy = p->sz.ldysum;
      pa.m = mp; pa.b = (int)bi;
      pa.V = V + k + k * ldb; pa.ldv = ldb;
      pa.Tm = Tm + k * kTLd; pa.ldt = kTLd; pa.tau = tau + k;
      pa.red = p->red; pa.rowj = p->rowj; pa.st = p->st; pa.G = sh.G;
      const double pflops = panel_flops((double)mp, (double)bi);
      const int occ0 = la && sub == 0 && b_next > 0 && pad16(b_next) == 64 &&
                               route == kPanelGrid && sample_panel_supported(64, sh)
                           ? sample_panel_occupancy<T>(sh) : 0;
      if (occ0 > 0 && (int64_t)occ0 * p->num_cus > sh.G) {
        // Look-ahead, sub-block 0: the panel of sub-block 0 and the first
        // look-ahead sample S_1 = A Omega_1 (independent of it) in one
        // launch.  The gather above has already read the partials of Y_0
        // that S_1 replaces.
        rrf_status rs = sketch_window(k_next, 64, &om_win);
        if (rs != RRF_OK) return rs;
        UpdateArgs<T> u1 = u;
        u1.Om = om_win;
        u1.qp = 64;
        u1.normpart = nullptr;
        const int su1 = upd_splits_fused(m, n, (int64_t)occ0 * p->num_cus - sh.G);
        u1.cols_per_split = round_up(ceil_div(n, su1), 2 * kUpdChunk);
        const int ys1 = (int)ceil_div(n, u1.cols_per_split);
        pa.epoch_base = next_epoch(p);
        const double sfl = 2.0 * m * n * b_next, sby = e * (m * n + m * b_next);
        RRF_LAUNCH(p, RRF_STAGE_SAMPLE, sfl + pflops, sby + 16.0 * mp * bi,
                   launch_sample_panel<T>(u1, ys1, pa, sh, s));
        spec(RRF_STAGE_SAMPLE, k_next, sfl, sby);
        ysplits = ys1;
        yoff = 0;
        s1_done = true;
      } else {
        if (power > 0) {
          rrf_status rs = power_steps(k, bi, sub == 0 ? A : Bws, sub == 0 ? lda : ldb,
                                      sh.rows_pad, false);
          if (rs != RRF_OK) return rs;
        }
        RRF_LAUNCH(p, RRF_STAGE_PANEL, pflops, 16.0 * mp * bi,
                   run_panel(p, pa, route, sh, s));
      }
    }

    const T* src = sub == 0 ? A : Bws;
    const int64_t lsrc = sub == 0 ? lda : ldb;

    // Look-ahead, sub-block 0: S_1 = A Omega_1 if it was not taken with the
    // panel above (later sub-blocks get their look-ahead sample from the
    // previous update).
    if (la && sub == 0 && b_next > 0 && !s1_done) {
      rrf_status rs = sketch_window(k_next, pad16(b_next), &om_win);
      if (rs != RRF_OK) return rs;
      UpdateArgs<T> u1 = u;
      u1.Om = om_win;
      u1.qp = pad16(b_next);
      u1.normpart = nullptr;
      const double sfl = 2.0 * m * n * b_next, sby = e * (m * n + m * b_next);
      RRF_LAUNCH(p, RRF_STAGE_SAMPLE, sfl, sby, launch_update<T>(u1, ysplits, s));
      spec(RRF_STAGE_SAMPLE, k_next, sfl, sby);
      yoff = 0;
    }

    // Z = V_i^T B[k:m, :], W = T_i^T Z (unless queued at the end of the last
    // block).
    bool gathered = false;     // the look-ahead gather rode in formW's launch
    if (w_ready) {
      w_ready = false;
      gathered = w_gathered;
    } else {
      GatherArgs<T> ga{};
      double gby = 0.0;
      gathered = la_gather(k, bi, yoff, ysplits, &ga, &gby);
      rrf_status rs = issue_w(k, bi, src, lsrc, false, gathered ? &ga : nullptr, gby);
      if (rs != RRF_OK) return rs;
    }

    PanelArgs pan{};          // look-ahead panel of sub-block i + 1
    PanelShape pan_shape{};
    double pan_flops = 0.0, pan_bytes = 0.0;
    if (la && b_next > 0) {
      // Y_{i+1} = Q_i^T S_{i+1}[rows k..m), in binary64; its panel (rows
      // k_next..m) is factored with the update below.
      const int64_t mpn = mp - bi;
      const int bpn = pad16(b_next);
      PanelShape shn;
      if (!la_shape(mpn, b_next, &shn)) return RRF_ERR_SHAPE;
      if (!gathered) {
        const double gby = e * mp * b_next * ysplits + 8.0 * mp * b_next;
        RRF_LAUNCH(p, RRF_STAGE_PANEL, 0.0, gby,
                   launch_gather_panel<T>(Yp + yoff, ldb, ldb * 64, ysplits, mp,
                                          (int)b_next, bpn, bi + shn.rows_pad,
                                          p->Ysum, p->sz.ldysum, s));
        spec(RRF_STAGE_PANEL, k_next, 0.0, gby);
      }
      ThinApplyArgs ta{};
      ta.V = V + k + k * ldb; ta.ldv = ldb;
      ta.Tm = Tm + k * kTLd; ta.ldt = kTLd; ta.b = (int)bi; ta.trans = 1;
      ta.Y = p->Ysum; ta.ldy = p->sz.ldysum; ta.mr = mp; ta.ncols = (int)b_next;
      ta.part = p->tx; ta.sums = p->tx + kThinPartWords;
      ta.epoch_base = next_epoch(p); ta.st = p->st;
      const double tfl = 4.0 * mp * bi * b_next, tby = 16.0 * mp * b_next + 8.0 * mp * bi;
      RRF_LAUNCH(p, RRF_STAGE_PANEL, tfl, tby, launch_thin_apply(ta, p->num_cus, s));
      spec(RRF_STAGE_PANEL, k_next, tfl, tby);
      pan.Y = p->Ysum + bi; pan.ldy = p->sz.ldysum;
      pan.m = mpn; pan.b = (int)b_next;
      pan.V = V + k_next + k_next * ldb; pan.ldv = ldb;
      pan.Tm = Tm + k_next * kTLd; pan.ldt = kTLd; pan.tau = tau + k_next;
      pan.red = p->red; pan.rowj = p->rowj; pan.st = p->st; pan.G = shn.G;
      pan_shape = shn;
      pan_flops = panel_flops((double)mpn, (double)b_next);
      pan_bytes = 16.0 * mpn * b_next;
      panel_ready = true;
    }

    // Sketch block sampled by this update (speculative: the stop test comes
    // after the update): Omega_{i+1}, or Omega_{i+2} with look-ahead.
    const int64_t k_s = la ? k_next + b_next : k_next;
    const int64_t b_s = (la ? b_next > 0 : true) ? sub_width(k_s) : 0;
    const int q_s = b_s > 0 ? pad16(b_s) : 0;
    if (b_s > 0) {
      rrf_status rs = sketch_window(k_s, q_s, &om_win);
      if (rs != RRF_OK) return rs;
    }

    // B[k:m, :] -= V_i W, fused with the sample and the norms.
    UpdateArgs<T> ua{};
    ua.src = src + k; ua.lds = lsrc; ua.dst = Bws + k; ua.ldd = ldb;
    ua.mr = mp; ua.n = n; ua.V = V + k + k * ldb; ua.ldv = ldb; ua.bp = bp;
    ua.W = (T*)p->W; ua.ldw = bp; ua.Om = om_win; ua.ldo = kOmLd; ua.qp = q_s;
    ua.P = Yp; ua.ldp = ldb; ua.split_stride = ldb * 64; ua.s0 = bi;
    ua.normpart = p->normpart;
    const bool fused = panel_ready && (la_gram ? update_gram_supported(bp, q_s, pan_shape)
                                               : update_panel_supported(bp, q_s, pan_shape));
    int su0 = upd_splits(mp, n, p->num_cus);
    if (fused) {
      const int occ = la_gram ? update_gram_occupancy<T>(pan_shape)
                              : update_panel_occupancy<T>(pan_shape);
      if (occ > 0)
        su0 = upd_splits_fused(mp, n, (int64_t)occ * p->num_cus - pan_shape.G);
    }
    ua.cols_per_split = round_up(ceil_div(n, su0), 2 * kUpdChunk);
    const int su = (int)ceil_div(n, ua.cols_per_split);
    const double smp_flops = 2.0 * (mp - bi) * n * b_s;
    const double upd_flops = 2.0 * mp * n * bi + smp_flops;
    nparts = (int)(ceil_div(mp, kUpdRows) * su);
    // The stop test runs in the update's last workgroup, except where the
    // spectral estimate of the next block comes between them.
    const bool fin_in_update = !(mode == RRF_STOP_SPECTRAL && at_end && b_next > 0);
    if (fin_in_update)
      set_finalize(p, ua, nparts, at_end ? blk : -1, k_next, kcap, mode, tol, 0);
    if (panel_ready) {
      pan.epoch_base = next_epoch(p);
      if (fused && la_gram) {
        GramPanelArgs ga{};
        ga.p = pan;
        ga.part = p->gx;
        ga.sums = p->gx + kGramPartWords;
        RRF_LAUNCH(p, RRF_STAGE_UPDATE, upd_flops + pan_flops,
                   2.0 * e * mp * n + pan_bytes,
                   launch_update_gram<T>(ua, su, ga, pan_shape, s));
        spec(RRF_STAGE_UPDATE, k_next, pan_flops, pan_bytes);
      } else if (fused) {
        RRF_LAUNCH(p, RRF_STAGE_UPDATE, upd_flops + pan_flops,
                   2.0 * e * mp * n + pan_bytes,
                   launch_update_panel<T>(ua, su, pan, pan_shape, s));
        spec(RRF_STAGE_UPDATE, k_next, pan_flops, pan_bytes);
      } else {
        RRF_LAUNCH(p, RRF_STAGE_UPDATE, upd_flops, 2.0 * e * mp * n,
                   launch_update<T>(ua, su, s));
        RRF_LAUNCH(p, RRF_STAGE_PANEL, pan_flops, pan_bytes,
                   run_panel(p, pan, la_gram ? kPanelGram : kPanelGrid, pan_shape, s));
        spec(RRF_STAGE_PANEL, k_next, pan_flops, pan_bytes);
      }
    } else {
      RRF_LAUNCH(p, RRF_STAGE_UPDATE, upd_flops, 2.0 * e * mp * n,
                 launch_update<T>(ua, su, s));
    }
    if (b_s > 0) spec(RRF_STAGE_UPDATE, k_s, smp_flops, 0.0);
    if (mode == RRF_STOP_SPECTRAL && at_end && b_next > 0) {
      // The sample of the next sub-block (the next block's first columns)
      // is B[k_next:m, :] Omega_next: with look-ahead it is already in Ysum
      // (brought up to date for the panel inside the update's launch),
      // otherwise the update's partials are gathered.
      const double* Yy = p->Ysum + bi;
      if (!la) {
        RRF_LAUNCH(p, RRF_STAGE_FINALIZE, 0.0, e * (mp - bi) * b_next * su,
                   launch_gather_panel<T>(Yp + bi, ldb, ldb * 64, su, mp - bi, (int)b_next,
                                          pad16(b_next), mp - bi, p->Yest, p->sz.ldysum, s));
        Yy = p->Yest;
      }
      rrf_status rs = spectral(k_next, b_next, Yy, p->sz.ldysum, blk);
      if (rs != RRF_OK) return rs;
    }
    if (!fin_in_update)
      RRF_LAUNCH(p, RRF_STAGE_FINALIZE, 0.0, 16.0 * nparts,
                 launch_finalize(p->normpart, nparts, p->st, p->st_mirror, p->trace_trail_d,
                                 p->trace_sub_d, at_end ? blk : -1, k_next, kcap,
                                 mode, tol, 0, s));
    if (!at_end) {
      // Inside a block: the next sub-block runs whatever the norms say (an
      // error recorded meanwhile is read at the end of the block).
      k = k_next;
      ++sub;
      yoff = bi;
      ysplits = su;
      continue;
    }
    // The stop test writes its decision into the pinned host state; the host
    // waits on an event behind that launch alone, with the next block's work
    // that does not depend on the test queued behind the event, so the
    // device keeps working while the host reads the test:
    // without look-ahead the next block's gather and panel (they need only
    // the sample this update took), with look-ahead (the next panel is
    // already factored) its reduce and formW.  It is queued when the
    // stopping quantity, extrapolated geometrically from the last two state
    // reads, stays above sigma^2 after this block; a wrong guess (the run
    // stops here after all) wastes that work, whose results lie past k and
    // are never used.
    const double E_prev = mode == RRF_STOP_TRAILING ? p->st_host->E_trail
                          : (mode == RRF_STOP_SUBTRACT ? p->st_host->E_sub : p->st_host->E_spec);
    const double E_pred =
        E_prev2 > 0.0 ? E_prev * std::min(1.0, E_prev / E_prev2) : E_prev;
    E_prev2 = E_prev;
    const bool more_likely = b_next > 0 && E_pred > p->st_host->sigma2;
    bool next_panel = false, next_w = false;
    PanelShape shn{};
    int route_n = -1;
    if (!la && more_likely) {
      route_n = panel_route(p, m - k_next, (int)b_next, &shn);
      next_panel = route_n >= 0;
    }
    if (la && more_likely && panel_ready) next_w = true;
    if (!p->state_ev) {
      he = hipEventCreateWithFlags(&p->state_ev, hipEventDisableTiming);
      if (he != hipSuccess) return hip_fail(he);
    }
    // The stop test of this launch has written its decision into st_host;
    // the event marks the launch's completion.
    he = hipEventRecord(p->state_ev, s);
    if (he != hipSuccess) return hip_fail(he);
    if (next_w) {
      // Its look-ahead gather reads the partials this update wrote (slab
      // rows from bi, su splits).
      GatherArgs<T> ga{};
      double gby = 0.0;
      w_gathered = la_gather(k_next, b_next, bi, su, &ga, &gby);
      rrf_status rs = issue_w(k_next, b_next, Bws, ldb, true, w_gathered ? &ga : nullptr, gby);
      if (rs != RRF_OK) return rs;
    }
    if (next_panel) {
      const int64_t mpn = m - k_next;
      const double gby = e * mpn * b_next * su + 8.0 * mpn * b_next;
      RRF_LAUNCH(p, RRF_STAGE_PANEL, 0.0, gby,
                 launch_gather_panel<T>(Yp + bi, ldb, ldb * 64, su, mpn, (int)b_next,
                                        pad16(b_next), shn.rows_pad, p->Ysum,
                                        p->sz.ldysum, s));
      PanelArgs pn{};
      pn.Y = p->Ysum; pn.ldy = p->sz.ldysum;
      pn.m = mpn; pn.b = (int)b_next;
      pn.V = V + k_next + k_next * ldb; pn.ldv = ldb;
      pn.Tm = Tm + k_next * kTLd; pn.ldt = kTLd; pn.tau = tau + k_next;
      pn.red = p->red; pn.rowj = p->rowj; pn.st = p->st; pn.G = shn.G;
      if (power > 0) {
        rrf_status rs = power_steps(k_next, b_next, Bws, ldb, shn.rows_pad, true);
        if (rs != RRF_OK) return rs;
      }
      const double pfl = panel_flops((double)mpn, (double)b_next), pby = 16.0 * mpn * b_next;
      RRF_LAUNCH(p, RRF_STAGE_PANEL, pfl, pby, run_panel(p, pn, route_n, shn, s));
      spec(RRF_STAGE_PANEL, k_next, pfl, pby + gby);
    }
    he = hipEventSynchronize(p->state_ev);
    if (he != hipSuccess) return hip_fail(he);
    k = k_next;
    ++blk;
    ++sub;
    yoff = bi;
    ysplits = su;
    if (next_panel) panel_ready = true;
    if (next_w) w_ready = true;
    if (p->st_host->barrier_err) return RRF_ERR_INTERNAL;
    if (p->st_host->nonfinite) return RRF_ERR_NONFINITE;
    stop = p->st_host->stop != 0;
  }
  p->nblocks = blk;

  // Explicit Q = H_0 ... H_{k-1} [I_k; 0], backward over the sub-blocks, in
  // binary64 (float plans round the result once).  Adjacent sub-blocks are
  // applied in groups of up to kGroupMax reflectors, as one block with their
  // merged T (orgqr_groups.hip): a quarter of the passes over Q for 32-column
  // blocks, half for 64-column blocks.
  const int nsub = (int)p->sub_start.size();
  if (k > 0) {
    double* Qd = std::is_same<T, double>::value ? (double*)Q : (double*)p->Q64;
    RRF_LAUNCH(p, RRF_STAGE_ORGQR, 0.0, 8.0 * m * k,
               launch_fill_identity<double>(Qd, ldb, m, k, s));
    // gi: index into the group list (merged T in Tp), or -1 (one block, its
    // own T).
    struct Pass { int64_t k0, b; int gi; };
    std::vector<Pass> passes;
    int ngroups = 0;
    int64_t gram_rows = 0;
    auto width = [&](int i) { return (i + 1 < nsub ? p->sub_start[i + 1] : k) - p->sub_start[i]; };
    for (int i = nsub - 1; i >= 0;) {
      int j = i;
      int64_t w = width(i);
      while (j >= 1 && i - j + 1 < kMaxGroupBlocks && w + width(j - 1) <= kGroupMax) {
        w += width(j - 1);
        --j;
      }
      if (j < i && (size_t)(ngroups + 1) * sizeof(OrgqrGroup) <= p->sz.groups) {
        OrgqrGroup g{};
        g.k0 = p->sub_start[j];
        g.nb = i - j + 1;
        g.w = (int)w;
        for (int c = 0; c < g.nb; ++c) g.off[c] = (int)(p->sub_start[j + c] - g.k0);
        g.off[g.nb] = g.w;
        // Gram tiles with an entry (i, j), block(i) < block(j): blocks are
        // contiguous, so compare the tile's first row and its last column.
        auto blk = [&](int col) {
          int c = 0;
          while (c + 1 < g.nb && col >= g.off[c + 1]) ++c;
          return c;
        };
        g.ntiles = 0;
        for (int ti = 0; 16 * ti < g.w; ++ti)
          for (int tj = 0; 16 * tj < g.w; ++tj)
            if (blk(16 * ti) < blk(std::min(16 * tj + 15, g.w - 1)))
              g.tile[g.ntiles++] = (unsigned char)(8 * ti + tj);
        p->groups_h[ngroups] = g;
        passes.push_back(Pass{g.k0, w, ngroups});
        gram_rows = std::max<int64_t>(gram_rows, m - g.k0);
        ++ngroups;
        i = j - 1;
      } else {
        passes.push_back(Pass{p->sub_start[i], width(i), -1});
        i -= 1;
      }
    }
    if (ngroups > 0) {
      // Row splits of the Gram sums, within the partial buffer (ngroups x
      // (nsplit + 1) matrices of kGroupMax^2).
      const int64_t ent = (int64_t)kGroupMax * kGroupMax;
      const int64_t cap = (int64_t)(p->sz.Zpart / 8) / (ent * ngroups) - 1;
      if (cap < 1) {
        // No room for the partials (tiny plans): every block on its own.
        std::vector<Pass> single;
        for (const Pass& ps : passes) {
          if (ps.gi < 0) { single.push_back(ps); continue; }
          const OrgqrGroup& g = p->groups_h[ps.gi];
          for (int c = g.nb - 1; c >= 0; --c)
            single.push_back(Pass{g.k0 + g.off[c], g.off[c + 1] - g.off[c], -1});
        }
        passes.swap(single);
        ngroups = 0;
      } else {
        he = hipMemcpyAsync(p->groups_d, p->groups_h, ngroups * sizeof(OrgqrGroup),
                            hipMemcpyHostToDevice, s);
        if (he != hipSuccess) return hip_fail(he);
        GroupArgs ga{};
        ga.groups = p->groups_d; ga.ngroups = ngroups;
        ga.V = V; ga.ldv = ldb; ga.m = m;
        ga.Tm = Tm; ga.ldt = kTLd; ga.Tg = p->Tp; ga.ldg = kGroupMax;
        ga.part = (double*)p->Zpart;
        // About two workgroups per compute unit over all groups (each split is
        // a chain of 32-row chunks), splits of at least 256 rows.
        ga.nsplit = (int)std::max<int64_t>(
            1, std::min<int64_t>({ceil_div(gram_rows, 256),
                                  std::max<int64_t>(64, ceil_div(2 * (int64_t)p->num_cus, ngroups)),
                                  cap}));
        RRF_LAUNCH(p, RRF_STAGE_ORGQR, 2.0 * gram_rows * ent * ngroups,
                   8.0 * gram_rows * kGroupMax * ngroups, launch_orgqr_groups(ga, s));
      }
    }
    for (const Pass& ps : passes) {
      const int64_t ki = ps.k0, bi = ps.b;
      const double* Tg = ps.gi >= 0 ? p->Tp + ki * kGroupMax : Tm + ki * kTLd;
      const int64_t ldt = ps.gi >= 0 ? kGroupMax : kTLd;
      if (k - ki <= 64) {
        // The last columns alone: the one-launch thin kernel.
        ThinApplyArgs ta{};
        ta.V = V + ki + ki * ldb; ta.ldv = ldb;
        ta.Tm = Tg; ta.ldt = ldt; ta.b = (int)bi; ta.trans = 0;
        ta.Y = Qd + ki + ki * ldb; ta.ldy = ldb; ta.mr = m - ki; ta.ncols = (int)(k - ki);
        ta.part = p->tx; ta.sums = p->tx + kThinPartWords;
        ta.epoch_base = next_epoch(p); ta.st = p->st;
        RRF_LAUNCH(p, RRF_STAGE_ORGQR, 4.0 * (m - ki) * bi * (k - ki),
                   16.0 * (m - ki) * (k - ki) + 8.0 * (m - ki) * bi,
                   launch_thin_apply(ta, p->num_cus, s));
        continue;
      }
      rrf_status rs = apply_wy<double>(p, 0, V + ki + ki * ldb, ldb, Tg, ldt, (int)bi,
                                       pad_group(bi), Qd + ki + ki * ldb, ldb, m - ki, k - ki,
                                       RRF_STAGE_ORGQR);
      if (rs != RRF_OK) return rs;
    }
    if (!std::is_same<T, double>::value)
      RRF_LAUNCH(p, RRF_STAGE_ORGQR, 0.0, 12.0 * m * k,
                 (launch_convert<double, float>(Qd, ldb, (float*)Q, ldb, m, k, s)));
  }
  he = hipStreamSynchronize(s);
  if (he != hipSuccess) return hip_fail(he);
  if (k > 0) {
    // Errors recorded after the last state read: the thin kernel's grid
    // exchange (last sub-block of Q).
    he = read_state(p);
    if (he != hipSuccess) return hip_fail(he);
    if (p->st_host->barrier_err) return RRF_ERR_INTERNAL;
    if (p->st_host->nonfinite) return RRF_ERR_NONFINITE;
  }
  // Take back the credit of work queued for sub-blocks past k.
  for (const SpecWork& w : p->spec) {
    if (w.col < k) continue;
    p->flops[w.stage] -= w.flops;
    p->bytes[w.stage] -= w.bytes;
  }

  // Trace back to the host.
  if (blk > 0) {
    p->trace_trail.resize(blk);
    p->trace_sub.resize(blk);
    p->trace_spec.assign(blk, std::nan(""));
    he = hipMemcpy(p->trace_trail.data(), p->trace_trail_d, blk * sizeof(double),
                   hipMemcpyDeviceToHost);
    if (he == hipSuccess)
      he = hipMemcpy(p->trace_sub.data(), p->trace_sub_d, blk * sizeof(double),
                     hipMemcpyDeviceToHost);
    // The estimate exists for the blocks that ended below the cap, and only
    // in spectral mode.
    const int nspec = mode == RRF_STOP_SPECTRAL ? (k < kcap ? blk : blk - 1) : 0;
    if (he == hipSuccess && nspec > 0)
      he = hipMemcpy(p->trace_spec.data(), p->trace_spec_d, nspec * sizeof(double),
                     hipMemcpyDeviceToHost);
    if (he != hipSuccess) return hip_fail(he);
  }
  p->E0 = p->st_host->E0;
  p->sigma2 = p->st_host->sigma2;
  // Spectral mode: at the cap there is no estimate; the Frobenius norm (an
  // upper bound of the spectral norm) decides the warning.
  const double E = mode == RRF_STOP_SUBTRACT ? p->st_host->E_sub : p->st_host->E_trail;
  *warn_kmax = k == kcap && kcap < std::min(m, n) && E > p->sigma2;
  *k_out = k;
  return RRF_OK;
}

// The bits of an enum argument as an int.  A C caller may pass any int for
// an enum parameter; reading such a value as the C++ enum type is undefined
// (outside its enumerators' range), so arguments are validated on their bits.
template <typename E>
int enum_bits(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "enum arguments are int-sized");
  int v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}
bool valid_dtype(int d) { return d == RRF_F32 || d == RRF_F64; }

template <typename T>
hipError_t to_plan_type(const double* src, int64_t lds, T* dst, int64_t ldd,
                        int64_t rows, int64_t cols, hipStream_t s) {
  if (std::is_same<T, double>::value)
    return launch_copy<double>(src, lds, (double*)dst, ldd, rows, cols, s);
  return launch_convert<double, float>(src, lds, (float*)dst, ldd, rows, cols, s);
}

template <typename T>
hipError_t from_plan_type(const T* src, int64_t lds, double* dst, int64_t ldd,
                          int64_t rows, int64_t cols, hipStream_t s) {
  if (std::is_same<T, double>::value)
    return launch_copy<double>((const double*)src, lds, dst, ldd, rows, cols, s);
  return launch_convert<float, double>((const float*)src, lds, dst, ldd, rows, cols, s);
}

template <typename T>
rrf_status panel_stage(rrf_plan* p, const T* Y, int64_t m, int64_t b,
                       int64_t ldy, T* Vout, int64_t ldv, T* Tout, int64_t ldt,
                       T* tauout) {
  PanelShape sh;
  const int route = panel_route(p, m, (int)b, &sh);
  if (route < 0) return RRF_ERR_SHAPE;
  hipStream_t s = p->stream;
  hipError_t e = clear_wait_error(p);
  if (e == hipSuccess)
    e = launch_gather_panel<T>(Y, ldy, 0, 1, m, (int)b, sh.bp, sh.rows_pad, p->Ysum,
                               p->sz.ldysum, s);
  if (e != hipSuccess) return hip_fail(e);
  PanelArgs pa{};
  pa.Y = p->Ysum; pa.ldy = p->sz.ldysum;
  pa.m = m; pa.b = (int)b;
  pa.V = p->V; pa.ldv = p->sz.ldb;
  pa.Tm = p->Tm; pa.ldt = kTLd; pa.tau = p->tau;
  pa.red = p->red; pa.rowj = p->rowj; pa.st = p->st; pa.G = sh.G;
  e = run_panel(p, pa, route, sh, s);
  if (e == hipSuccess) e = to_plan_type<T>(p->V, p->sz.ldb, Vout, ldv, m, b, s);
  if (e == hipSuccess) e = to_plan_type<T>(p->Tm, kTLd, Tout, ldt, b, b, s);
  if (e == hipSuccess) e = to_plan_type<T>(p->tau, 1, tauout, 1, b, 1, s);
  // A grid-wide wait that gave up leaves V, T and tau undefined.
  if (e == hipSuccess) e = read_state(p);
  if (e != hipSuccess) return hip_fail(e);
  return p->st_host->barrier_err ? RRF_ERR_INTERNAL : RRF_OK;
}

template <typename T>
rrf_status larfb_stage(rrf_plan* p, int trans, const T* V, int64_t ldv,
                       const T* Tm, int64_t ldt, int64_t b, T* X, int64_t m,
                       int64_t n, int64_t ldx) {
  hipStream_t s = p->stream;
  const int bp = pad16(b);
  const int64_t ldb = p->sz.ldb;
  double* Vw = p->V;
  double* Tw = p->Tm;
  // Zero-padded binary64 copies of V (m x bp) and T (bp x bp).
  hipError_t e = hipMemsetAsync(Vw, 0, (size_t)ldb * bp * sizeof(double), s);
  if (e == hipSuccess) e = hipMemsetAsync(Tw, 0, (size_t)kTLd * bp * sizeof(double), s);
  if (e == hipSuccess) e = from_plan_type<T>(V, ldv, Vw, ldb, m, b, s);
  if (e == hipSuccess) e = from_plan_type<T>(Tm, ldt, Tw, kTLd, b, b, s);
  if (e != hipSuccess) return hip_fail(e);
  stats_reset(p);
  if (std::is_same<T, double>::value && n <= 64) {
    // Thin binary64 X: the one-launch kernel the look-ahead uses.
    ThinApplyArgs ta{};
    ta.V = Vw; ta.ldv = ldb; ta.Tm = Tw; ta.ldt = kTLd; ta.b = (int)b;
    ta.trans = trans ? 1 : 0;
    ta.Y = (double*)X; ta.ldy = ldx; ta.mr = m; ta.ncols = (int)n;
    ta.part = p->tx; ta.sums = p->tx + kThinPartWords;
    ta.epoch_base = next_epoch(p); ta.st = p->st;
    e = clear_wait_error(p);
    if (e == hipSuccess) e = launch_thin_apply(ta, p->num_cus, s);
    if (e == hipSuccess) e = read_state(p);
    if (e != hipSuccess) return hip_fail(e);
    return p->st_host->barrier_err ? RRF_ERR_INTERNAL : RRF_OK;
  }
  return apply_wy<T>(p, trans, Vw, ldb, Tw, kTLd, (int)b, bp, X, ldx, m, n,
                     RRF_STAGE_UPDATE);
}

}  // namespace

extern "C" {

const char* rrf_status_string(rrf_status status) {
  switch (enum_bits(status)) {
    case RRF_OK: return "RRF_OK";
    case RRF_WARN_KMAX: return "RRF_WARN_KMAX: rank cap reached before the tolerance";
    case RRF_ERR_INVALID_ARG: return "RRF_ERR_INVALID_ARG: invalid argument";
    case RRF_ERR_SHAPE: return "RRF_ERR_SHAPE: size exceeds the plan or the panel capacity";
    case RRF_ERR_NONFINITE: return "RRF_ERR_NONFINITE: non-finite input or norm";
    case RRF_ERR_NOMEM: return "RRF_ERR_NOMEM: allocation failed";
    case RRF_ERR_HIP: return "RRF_ERR_HIP: HIP runtime error";
    case RRF_ERR_INTERNAL: return "RRF_ERR_INTERNAL: device-side wait gave up";
  }
  return "RRF: unknown status";
}

rrf_status rrf_workspace_size(rrf_dtype dtype, int64_t m_max, int64_t n_max,
                              int64_t block_b_max, int64_t k_max,
                              size_t* bytes) {
  if (!bytes || !valid_dtype(enum_bits(dtype)) || m_max < 1 || n_max < 1 ||
      block_b_max < 1 || block_b_max > kMaxBlockB || k_max < 0)
    return RRF_ERR_INVALID_ARG;
  *bytes = compute_sizes(dtype, m_max, n_max, block_b_max, k_max).total();
  return RRF_OK;
}

namespace {
rrf_status plan_create(rrf_plan_t* plan, int dtype_bits, int64_t m_max, int64_t n_max,
                       int64_t block_b_max, int64_t k_max, void* hip_stream,
                       void* workspace, size_t workspace_bytes) {
  if (!plan || !valid_dtype(dtype_bits) || m_max < 1 || n_max < 1 ||
      block_b_max < 1 || block_b_max > kMaxBlockB || k_max < 0)
    return RRF_ERR_INVALID_ARG;
  const rrf_dtype dtype = (rrf_dtype)dtype_bits;
  if (workspace) {
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0 ||
        workspace_bytes < compute_sizes(dtype, m_max, n_max, block_b_max, k_max).total())
      return RRF_ERR_INVALID_ARG;
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return RRF_ERR_HIP;
  rrf_plan* p = new (std::nothrow) rrf_plan();
  if (!p) return RRF_ERR_NOMEM;
  p->ws_base = static_cast<char*>(workspace);
  p->ws_bytes = workspace ? workspace_bytes : 0;
  p->dtype = dtype;
  p->elem = dtype == RRF_F32 ? 4 : 8;
  p->m_max = m_max;
  p->n_max = n_max;
  p->b_max = block_b_max;
  p->k_max = k_max;
  p->stream = (hipStream_t)hip_stream;
  p->stop_mode = RRF_STOP_TRAILING;
  // RRF_STOP_MODE (trailing, subtract or spectral) sets the initial stopping
  // quantity; rrf_set_stop_mode changes it.  RRF_LOG=1 logs every run to
  // stderr; the library prints nothing otherwise.
  if (const char* sm = std::getenv("RRF_STOP_MODE")) {
    if (std::strcmp(sm, "subtract") == 0) p->stop_mode = RRF_STOP_SUBTRACT;
    else if (std::strcmp(sm, "spectral") == 0) p->stop_mode = RRF_STOP_SPECTRAL;
  }
  p->log = 0;
  if (const char* lg = std::getenv("RRF_LOG")) p->log = std::atoi(lg) != 0;
  p->power = 0;
  p->timing = 0;
  p->panel_target = 64;
  p->panel_launches = 0;
  if (const char* pt = std::getenv("RRF_PANEL_WGS")) {
    const int v = std::atoi(pt);
    if (v >= 1 && v <= kMaxPanelWGs) p->panel_target = v;
  }
  // RRF_LOOKAHEAD=0 factors every panel after the update that samples it (no
  // overlap); the default factors the next panel during the update.
  p->lookahead = 1;
  if (const char* la = std::getenv("RRF_LOOKAHEAD")) p->lookahead = std::atoi(la) != 0;
  // RRF_PANEL selects the panel algorithm: "grid" (column by column, one
  // grid-wide reduction per column), "gram" (the same reflectors from the
  // Gram matrix, one grid exchange per sweep of columns), "tsqr" (tall-skinny
  // QR with Householder reconstruction); the default picks gram or grid by
  // the block width.  The look-ahead overlaps grid panels and, for blocks of
  // at most 32 columns, gram panels.
  p->panel_mode = kPanelAuto;
  if (const char* pm = std::getenv("RRF_PANEL")) {
    if (std::strcmp(pm, "tsqr") == 0) p->panel_mode = kPanelTsqr;
    else if (std::strcmp(pm, "gram") == 0) p->panel_mode = kPanelGram;
    else if (std::strcmp(pm, "grid") == 0) p->panel_mode = kPanelGrid;
  }
  if (hipGetDevice(&p->device) != hipSuccess ||
      hipDeviceGetAttribute(&p->num_cus, hipDeviceAttributeMultiprocessorCount,
                            p->device) != hipSuccess) {
    free_plan(p);
    return RRF_ERR_HIP;
  }
  // Workgroups the Gram panel may hold inside the update's launch (the
  // look-ahead of blocks of at most 32 columns): half the compute units, so
  // that 4096-row panels take 4 rows per thread (its exchange is one per
  // sweep, so a wider grid costs little; at 4096 x 4096 fp32, b = 32, 128
  // workgroups measured 17.6 ms per run against 17.8 ms for 64 and 18.3 ms
  // for 32); RRF_LA_GRAM_WGS overrides.
  p->gram_fused_max = std::max(1, p->num_cus / 2);
  // Sub-blocks of at most RRF_SUBBLOCK (16, 32 or 64) columns; by default
  // chosen per run from the matrix size (run_impl).
  p->sub_max = 0;
  if (const char* sb = std::getenv("RRF_SUBBLOCK")) {
    const int v = std::atoi(sb);
    if (v == 16 || v == 32 || v == 64) p->sub_max = v;
  }
  if (const char* gw = std::getenv("RRF_LA_GRAM_WGS")) {
    const int v = std::atoi(gw);
    if (v >= 1 && v <= kMaxGramWGs) p->gram_fused_max = v;
  }
  // RRF_TEST_SPIN_LIMIT sets the poll rounds of every grid-wide wait of the
  // plan (tests: 0 makes each wait give up at its first poll, so the
  // give-up path runs while every kernel still drains).
  p->spin_limit = kSpinLimit;
  if (const char* sl = std::getenv("RRF_TEST_SPIN_LIMIT")) {
    const long v = std::atol(sl);
    if (v >= 0 && v <= (long)kSpinLimit) p->spin_limit = (unsigned)v;
  }
  // The first panel has m_max rows; some route must fit it (sub-blocks have
  // at most 64 columns).
  PanelShape sh;
  const int64_t b_sub = std::min<int64_t>(block_b_max, kMaxBlock);
  if (!panel_fits(p, std::max(m_max, b_sub), (int)b_sub, &sh)) {
    free_plan(p);
    return RRF_ERR_SHAPE;
  }
  p->sz = compute_sizes(dtype, m_max, n_max, block_b_max, k_max);
  int counter = 0;
  hipError_t e = hipSuccess;
  void* tmp = nullptr;
#define RRF_ALLOC(field, bytes)                                     \
  do {                                                              \
    if (e == hipSuccess) {                                          \
      e = dev_alloc(p, &tmp, (bytes), &counter);                    \
      p->field = reinterpret_cast<decltype(p->field)>(tmp);         \
    }                                                               \
  } while (0)
  RRF_ALLOC(Bws, p->sz.Bws);
  RRF_ALLOC(V, p->sz.V);
  RRF_ALLOC(Tm, p->sz.Tm);
  RRF_ALLOC(tau, p->sz.tau);
  RRF_ALLOC(Ypart, p->sz.Ypart);
  RRF_ALLOC(Ysum, p->sz.Ysum);
  RRF_ALLOC(Om, p->sz.Om);
  RRF_ALLOC(Zpart, p->sz.Zpart);
  RRF_ALLOC(W, p->sz.W);
  RRF_ALLOC(Q, p->sz.Q);
  if (p->sz.Q64) RRF_ALLOC(Q64, p->sz.Q64);
  RRF_ALLOC(normpart, p->sz.normpart);
  RRF_ALLOC(normtag, p->sz.normtag);
  RRF_ALLOC(tsqr, p->sz.tsqr);
  RRF_ALLOC(red, p->sz.red);
  RRF_ALLOC(rowj, p->sz.rowj);
  RRF_ALLOC(gx, p->sz.gx);
  RRF_ALLOC(tx, p->sz.tx);
  RRF_ALLOC(st, p->sz.st);
  RRF_ALLOC(trace_trail_d, p->sz.trace / 3);
  RRF_ALLOC(trace_sub_d, p->sz.trace / 3);
  RRF_ALLOC(trace_spec_d, p->sz.trace / 3);
  RRF_ALLOC(Yest, p->sz.Yest);
  RRF_ALLOC(spec_part, p->sz.spec);
  RRF_ALLOC(Tpow, p->sz.Tpow);
  RRF_ALLOC(Tp, p->sz.Tp);
  RRF_ALLOC(groups_d, p->sz.groups);
#undef RRF_ALLOC
  if (e == hipSuccess) {
    ++counter;
    const char* f = std::getenv("RRF_FAULT_ALLOC");
    if (f && std::atoi(f) == counter) e = hipErrorOutOfMemory;
    else e = hipHostMalloc((void**)&p->st_host, sizeof(DevState),
                           hipHostMallocMapped | hipHostMallocCoherent);
  }
  // The stop test writes its decision straight into st_host.
  if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&p->st_mirror, p->st_host, 0);
  if (e == hipSuccess) e = hipHostMalloc((void**)&p->groups_h, p->sz.groups, 0);
  if (e == hipSuccess) e = hipMemsetAsync(p->red, 0, p->sz.red, p->stream);
  if (e == hipSuccess) e = hipMemsetAsync(p->rowj, 0, p->sz.rowj, p->stream);
  if (e == hipSuccess) e = hipMemsetAsync(p->gx, 0, p->sz.gx, p->stream);
  if (e == hipSuccess) e = hipMemsetAsync(p->tx, 0, p->sz.tx, p->stream);
  if (e == hipSuccess) e = hipMemsetAsync(p->normtag, 0, p->sz.normtag, p->stream);
  if (e == hipSuccess) {
    std::memset(p->st_host, 0, sizeof(DevState));
    p->st_host->spin_limit = p->spin_limit;
    e = hipMemcpyAsync(p->st, p->st_host, sizeof(DevState), hipMemcpyHostToDevice,
                       p->stream);
  }
  if (e == hipSuccess) e = hipMemsetAsync(p->Om, 0, p->sz.Om, p->stream);
  if (e == hipSuccess) e = hipMemsetAsync(p->V, 0, p->sz.V, p->stream);
  if (e == hipSuccess) e = hipMemsetAsync(p->Yest, 0, p->sz.Yest, p->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(p->stream);
  if (e != hipSuccess) {
    free_plan(p);
    return hip_fail(e);
  }
  stats_reset(p);
  p->last_m = p->last_n = p->last_k = p->nblocks = 0;
  p->last_b = 0;
  p->E0 = p->sigma2 = 0.0;
  *plan = p;
  return RRF_OK;
}
}  // namespace

rrf_status rrf_plan_create(rrf_plan_t* plan, rrf_dtype dtype, int64_t m_max,
                           int64_t n_max, int64_t block_b_max, int64_t k_max,
                           void* hip_stream) {
  return plan_create(plan, enum_bits(dtype), m_max, n_max, block_b_max, k_max, hip_stream,
                     nullptr, 0);
}

rrf_status rrf_plan_create_in(rrf_plan_t* plan, rrf_dtype dtype, int64_t m_max,
                              int64_t n_max, int64_t block_b_max, int64_t k_max,
                              void* hip_stream, void* workspace, size_t workspace_bytes) {
  return plan_create(plan, enum_bits(dtype), m_max, n_max, block_b_max, k_max, hip_stream,
                     workspace, workspace_bytes);
}

rrf_status rrf_destroy(rrf_plan_t plan) {
  if (!plan) return RRF_OK;
  (void)hipStreamSynchronize(plan->stream);
  free_plan(plan);
  return RRF_OK;
}

rrf_status rrf_set_stop_mode(rrf_plan_t plan, rrf_stop_mode mode) {
  const int md = enum_bits(mode);
  if (!plan || (md != RRF_STOP_TRAILING && md != RRF_STOP_SUBTRACT && md != RRF_STOP_SPECTRAL))
    return RRF_ERR_INVALID_ARG;
  plan->stop_mode = mode;
  return RRF_OK;
}

rrf_status rrf_set_power_iterations(rrf_plan_t plan, int q) {
  if (!plan || q < 0 || q > kMaxPower) return RRF_ERR_INVALID_ARG;
  plan->power = q;
  return RRF_OK;
}

rrf_status rrf_set_timing(rrf_plan_t plan, int enable) {
  if (!plan) return RRF_ERR_INVALID_ARG;
  plan->timing = enable ? 1 : 0;
  return RRF_OK;
}

rrf_status rrf_run(rrf_plan_t plan, const void* A, int64_t m, int64_t n,
                   int64_t lda, double tol, int64_t block_b, uint64_t seed,
                   void** Q, int64_t* ldq, int64_t* k, void** B, int64_t* ldb) {
  if (!plan || !A || !Q || !ldq || !k || !B || !ldb) return RRF_ERR_INVALID_ARG;
  if (m < 0 || n < 0 || lda < std::max<int64_t>(1, m)) return RRF_ERR_INVALID_ARG;
  if (!std::isfinite(tol) || tol < 0.0) return RRF_ERR_INVALID_ARG;
  if (block_b < 1 || block_b > plan->b_max) return RRF_ERR_INVALID_ARG;
  // Power iterations act on a whole block's sample at once; blocks wider
  // than one 64-column sub-block would power their second part on the
  // deflated matrix instead.
  if (plan->power > 0 && block_b > kMaxBlock) return RRF_ERR_INVALID_ARG;
  if (m > plan->m_max || n > plan->n_max) return RRF_ERR_SHAPE;
  stats_reset(plan);
  plan->last_m = m;
  plan->last_n = n;
  plan->last_b = block_b;
  plan->last_k = 0;
  plan->nblocks = 0;
  int64_t kk = 0;
  bool warn = false;
  rrf_status st = RRF_OK;
  if (m > 0 && n > 0) {
    if (plan->dtype == RRF_F64)
      st = run_impl<double>(plan, (const double*)A, m, n, lda, tol, block_b,
                            seed, &kk, &warn);
    else
      st = run_impl<float>(plan, (const float*)A, m, n, lda, tol, block_b, seed,
                           &kk, &warn);
    if (st != RRF_OK) {
      (void)hipStreamSynchronize(plan->stream);
      plan->nblocks = 0;
      *k = 0;
      if (plan->log)
        std::fprintf(stderr, "rrf_run: m=%lld n=%lld b=%lld tol=%g: %s\n", (long long)m,
                     (long long)n, (long long)block_b, tol, rrf_status_string(st));
      return st;
    }
    stats_collect(plan);
  }
  plan->last_k = kk;
  if (plan->log) {
    std::fprintf(stderr,
                 "rrf_run: m=%lld n=%lld b=%lld tol=%g mode=%d -> k=%lld blocks=%lld "
                 "||A||_F^2=%.6e sigma^2=%.6e%s\n",
                 (long long)m, (long long)n, (long long)block_b, tol, plan->stop_mode,
                 (long long)kk, (long long)plan->nblocks, plan->E0, plan->sigma2,
                 warn ? " (rank cap)" : "");
    for (int64_t i = 0; i < plan->nblocks; ++i)
      std::fprintf(stderr, "rrf_run:   block %lld: E_trail=%.6e E_sub=%.6e E_spec=%.6e\n",
                   (long long)i, plan->trace_trail[i], plan->trace_sub[i],
                   plan->trace_spec[i]);
  }
  *Q = plan->Q;
  *ldq = plan->sz.ldb;
  *B = plan->Bws;
  *ldb = plan->sz.ldb;
  *k = kk;
  return warn ? RRF_WARN_KMAX : RRF_OK;
}

rrf_status rrf_get_trace(rrf_plan_t plan, int64_t cap, int64_t* nblocks,
                         double* E_trail, double* E_sub, double* E_spec, double* E0,
                         double* sigma2) {
  if (!plan || !nblocks || cap < 0 || (cap > 0 && (!E_trail || !E_sub)))
    return RRF_ERR_INVALID_ARG;
  *nblocks = plan->nblocks;
  const int64_t nw = std::min<int64_t>(cap, plan->nblocks);
  for (int64_t i = 0; i < nw; ++i) {
    E_trail[i] = plan->trace_trail[i];
    E_sub[i] = plan->trace_sub[i];
    if (E_spec) E_spec[i] = plan->trace_spec[i];
  }
  if (E0) *E0 = plan->E0;
  if (sigma2) *sigma2 = plan->sigma2;
  return RRF_OK;
}

rrf_status rrf_get_stage_stats(rrf_plan_t plan, double* ms, int64_t* launches,
                               double* flops, double* bytes) {
  if (!plan) return RRF_ERR_INVALID_ARG;
  for (int i = 0; i < RRF_NUM_STAGES; ++i) {
    if (ms) ms[i] = plan->ms[i];
    if (launches) launches[i] = plan->launches[i];
    if (flops) flops[i] = plan->flops[i];
    if (bytes) bytes[i] = plan->bytes[i];
  }
  return RRF_OK;
}

rrf_status rrf_get_reflectors(rrf_plan_t plan, const void** V, int64_t* ldv,
                              const void** T, int64_t* ldt, const void** tau) {
  if (!plan || !V || !ldv || !T || !ldt || !tau) return RRF_ERR_INVALID_ARG;
  // Zero V above each block (the kernels never touch those rows).
  if (plan->last_k > 0) {
    const int64_t ldb = plan->sz.ldb;
    for (size_t i = 0; i < plan->sub_start.size(); ++i) {
      const int64_t ki = plan->sub_start[i];
      const int64_t bi = (i + 1 < plan->sub_start.size() ? plan->sub_start[i + 1]
                                                            : plan->last_k) - ki;
      if (ki == 0) continue;
      for (int64_t c = 0; c < bi; ++c) {
        hipError_t e = hipMemsetAsync(plan->V + (ki + c) * ldb, 0,
                                      ki * sizeof(double), plan->stream);
        if (e != hipSuccess) return hip_fail(e);
      }
    }
    hipError_t e = hipStreamSynchronize(plan->stream);
    if (e != hipSuccess) return hip_fail(e);
  }
  *V = plan->V;
  *ldv = plan->sz.ldb;
  *T = plan->Tm;
  *ldt = kTLd;
  *tau = plan->tau;
  return RRF_OK;
}

rrf_status rrf_sketch(rrf_dtype dtype, uint64_t seed, int64_t n, int64_t col0,
                      int64_t ncols, void* out, int64_t ldo, void* hip_stream) {
  if (!valid_dtype(enum_bits(dtype)) || !out || n < 0 || col0 < 0 || ncols < 0 ||
      ldo < std::max<int64_t>(1, n))
    return RRF_ERR_INVALID_ARG;
  if (n == 0 || ncols == 0) return RRF_OK;
  hipError_t e;
  if (dtype == RRF_F64)
    e = launch_sketch<double>(seed, n, n, col0, ncols, (double*)out, 1, ldo,
                              (hipStream_t)hip_stream);
  else
    e = launch_sketch<float>(seed, n, n, col0, ncols, (float*)out, 1, ldo,
                             (hipStream_t)hip_stream);
  return e == hipSuccess ? RRF_OK : hip_fail(e);
}


rrf_status rrf_panel_qr(rrf_plan_t plan, const void* Y, int64_t m, int64_t b,
                        int64_t ldy, void* V, int64_t ldv, void* T,
                        int64_t ldt, void* tau) {
  if (!plan || !Y || !V || !T || !tau) return RRF_ERR_INVALID_ARG;
  if (b < 1 || b > std::min<int64_t>(plan->b_max, kMaxBlock) || m < b || ldy < m || ldv < m ||
      ldt < b)
    return RRF_ERR_INVALID_ARG;
  if (m > plan->m_max) return RRF_ERR_SHAPE;
  if (plan->dtype == RRF_F64)
    return panel_stage<double>(plan, (const double*)Y, m, b, ldy, (double*)V,
                               ldv, (double*)T, ldt, (double*)tau);
  return panel_stage<float>(plan, (const float*)Y, m, b, ldy, (float*)V, ldv,
                            (float*)T, ldt, (float*)tau);
}

rrf_status rrf_apply_block_reflector(rrf_plan_t plan, int trans,
                                     const void* V, int64_t ldv,
                                     const void* T, int64_t ldt, int64_t b,
                                     void* X, int64_t m, int64_t n,
                                     int64_t ldx) {
  if (!plan || !V || !T || !X) return RRF_ERR_INVALID_ARG;
  if (b < 1 || b > std::min<int64_t>(plan->b_max, kMaxBlock) || m < 0 || n < 0 ||
      ldv < std::max<int64_t>(1, m) ||
      ldt < b || ldx < std::max<int64_t>(1, m))
    return RRF_ERR_INVALID_ARG;
  if (m > plan->m_max || n > plan->n_max) return RRF_ERR_SHAPE;
  if (m == 0 || n == 0) return RRF_OK;
  if (plan->dtype == RRF_F64)
    return larfb_stage<double>(plan, trans, (const double*)V, ldv,
                               (const double*)T, ldt, b, (double*)X, m, n, ldx);
  return larfb_stage<float>(plan, trans, (const float*)V, ldv, (const float*)T,
                            ldt, b, (float*)X, m, n, ldx);
}

rrf_status rrf_subspace_map(rrf_plan_t plan, const void* Qnew, int64_t ldqn,
                            int64_t r_new, const void* Qold, int64_t ldqo,
                            int64_t r_old, const void* M, int64_t ldm,
                            int64_t m, int64_t n, void* out, int64_t ldo) {
  if (!plan || m < 0 || n < 0 || r_new < 0 || r_old < 0) return RRF_ERR_INVALID_ARG;
  // A pointer may be null only where its matrix is empty.
  if ((!Qnew && m * r_new > 0) || (!Qold && m * r_old > 0) || (!M && r_old * n > 0) ||
      (!out && r_new * n > 0))
    return RRF_ERR_INVALID_ARG;
  if (ldqn < std::max<int64_t>(1, m) ||
      ldqo < std::max<int64_t>(1, m) || ldm < std::max<int64_t>(1, r_old) ||
      ldo < std::max<int64_t>(1, r_new))
    return RRF_ERR_INVALID_ARG;
  const int64_t lim = 2147483647;
  if (m > lim || n > lim || r_new > lim || r_old > lim || ldqn > lim || ldqo > lim ||
      ldm > lim || ldo > lim)
    return RRF_ERR_SHAPE;
  if (r_new == 0 || n == 0) return RRF_OK;
  hipStream_t s = plan->stream;
  const size_t e = plan->dtype == RRF_F64 ? 8 : 4;
  if (r_old == 0 || m == 0) {
    hipError_t he = hipMemset2DAsync(out, (size_t)ldo * e, 0, (size_t)r_new * e, (size_t)n, s);
    return he == hipSuccess ? RRF_OK : hip_fail(he);
  }
  // Grid limits of the tiled kernels (64 x 64 output tiles).
  if (ceil_div(n, 64) > 65535 || ceil_div(r_old, 64) > 65535) return RRF_ERR_SHAPE;
  const int nsplit = map_splits(r_new, r_old, m, plan->num_cus);
  const size_t need = (size_t)(nsplit + 1) * (size_t)r_new * (size_t)r_old * e;
  if (need > plan->map_c_bytes) {
    if (plan->map_c) {
      (void)hipFree(plan->map_c);
      plan->map_c = nullptr;
      plan->map_c_bytes = 0;
    }
    if (hipMalloc(&plan->map_c, need) != hipSuccess) {
      plan->map_c = nullptr;
      return RRF_ERR_NOMEM;
    }
    plan->map_c_bytes = need;
  }
  hipError_t he;
  if (plan->dtype == RRF_F64) {
    double* Cp = (double*)plan->map_c;
    he = launch_subspace_map<double>((const double*)Qnew, ldqn, r_new, (const double*)Qold,
                                     ldqo, r_old, (const double*)M, ldm, m, n, (double*)out,
                                     ldo, Cp, Cp + (size_t)nsplit * r_new * r_old, nsplit, s);
  } else {
    float* Cp = (float*)plan->map_c;
    he = launch_subspace_map<float>((const float*)Qnew, ldqn, r_new, (const float*)Qold, ldqo,
                                    r_old, (const float*)M, ldm, m, n, (float*)out, ldo, Cp,
                                    Cp + (size_t)nsplit * r_new * r_old, nsplit, s);
  }
  return he == hipSuccess ? RRF_OK : hip_fail(he);
}

rrf_status rrf_copy_matrix(rrf_dtype dtype, const void* src, int64_t lds,
                           void* dst, int64_t ldd, int64_t rows, int64_t cols,
                           void* hip_stream) {
  if (!valid_dtype(enum_bits(dtype)) || !src || !dst || rows < 0 || cols < 0 ||
      lds < std::max<int64_t>(1, rows) || ldd < std::max<int64_t>(1, rows))
    return RRF_ERR_INVALID_ARG;
  hipError_t e;
  if (dtype == RRF_F64)
    e = launch_copy<double>((const double*)src, lds, (double*)dst, ldd, rows,
                            cols, (hipStream_t)hip_stream);
  else
    e = launch_copy<float>((const float*)src, lds, (float*)dst, ldd, rows, cols,
                           (hipStream_t)hip_stream);
  return e == hipSuccess ? RRF_OK : hip_fail(e);
}

}  // extern "C"
