// Host runtime of the C ABI declared in include/ds.h: argument validation,
// workspace carve-up, the active-set control loop and the accounting.
//
// Control loop (Sec. 3, Fig. fig:active-loop). Cycle k is two launches:
//   f-half (also the row screen of state k-1 when k-1 is on the audit grid:
//           R_i/a_i = 2^(lse_new - lse_old), a full evaluation of the row
//           marginal);
//   g-half + column check of the screen-positive lanes of state k-1; the last
//           block of each checked lane takes its decision on the device
//           (verifier-gated: the screen alone never retires a lane) and a
//           retired lane's work items stop running at once.
// With guarded release float64 verification launches between the two halves
// (the lanes the outward bound admits, their row marginal, then the column
// marginal of those whose row residual met tol) take the decision instead of
// the float32 column check.
// The host never waits per cycle: the device publishes its control state
// (retirements, survivor widths, a progress word) to pinned host memory, and
// when it shows retirements the host launches the compaction (scan + gather
// into the other bank, with emission of the retired lanes) so later launches
// run at the survivor width. The host runs at most a bounded number of cycles
// ahead of the device. A call may be split into sub-batches (contiguous lane
// ranges), each with this loop on its own host thread and stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "ds.h"
#include "ds_internal.h"

namespace {

thread_local std::string g_last_error;

ds_err fail(ds_err e, const std::string& msg) {
  g_last_error = msg;
  return e;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

constexpr int kMaxParts = 4;   // concurrent sub-batches of one call

bool uses_mfma(const ds_problem* pr, const ds_options* op);
// d > 32: the materialised cost (4 bytes per term from HBM) unless a side has
// more than 16384 points or DS_F_MATRIX_FREE asks for the K-looped matrix-core
// half-step, which recomputes x~ . y~ per tile.
bool uses_mfree(const ds_problem* pr, const ds_options* op) {
  if (pr->d <= ds::kMaxDSmall || (op->flags & DS_F_MATERIALIZE)) return false;
  return (op->flags & DS_F_MATRIX_FREE) || pr->n_max > ds::kMatMaxPts || pr->m_max > ds::kMatMaxPts;
}
bool uses_mat(const ds_problem* pr, const ds_options* op) {
  return (op->flags & DS_F_MATERIALIZE) != 0 || (pr->d > ds::kMaxDSmall && !uses_mfree(pr, op));
}
// The float64 state is the default wherever its kernels exist (matrix-free,
// d <= 16): rounding the scaled coordinates or the potentials to float32
// perturbs exponents of size C/eps by ~C/eps * 2^-24, which moves the residual
// trajectory by 1e-6..1e-5 and with it the completion depths of near-threshold
// lanes. DS_F_FAST32 or a FORCE flag selects the float32 kernels instead.
bool uses_f64(const ds_problem* pr, const ds_options* op) {
  if (uses_mat(pr, op)) return false;
  if (op->flags & DS_F_PRECISE) return true;
  if (op->flags & (DS_F_FAST32 | DS_F_FORCE_VALU | DS_F_FORCE_MFMA)) return false;
  return pr->d <= ds::kMaxDF64;
}

struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    off = align_up(off, 256);
    T* p = reinterpret_cast<T*>(base ? base + off : nullptr);
    off += count * sizeof(T);
    return p;
  }
};

ds::Layout plan(const ds_problem* pr, const ds_options* op, void* ws) {
  ds::Layout L;
  std::memset(&L, 0, sizeof(L));
  L.W = pr->W;
  L.n_max = pr->n_max;
  L.m_max = pr->m_max;
  L.d = pr->d;
  L.dp = pr->d + (pr->d & 1);
  // the matrix-free large-d kernel stages whole kMfreeK-coordinate slices
  if (uses_mfree(pr, op)) L.dp = (int)align_up((size_t)pr->d, ds::kMfreeK);
  L.dh = L.dp / 2;
  L.mat = uses_mat(pr, op) ? 1 : 0;
  L.rows = L.mat ? ds::kRowsValu
                 : uses_f64(pr, op) ? ds::rows_f64(pr->d)
                 : uses_mfree(pr, op) ? ds::kRowsMfmaK
                 : uses_mfma(pr, op) ? ds::kRowsMfma : ds::kRowsValu;
  // every lane-side holds whole work items
  const size_t padq = (size_t)std::max(ds::kPad, L.rows);
  L.pad[0] = (int)align_up((size_t)pr->n_max, padq);
  L.pad[1] = (int)align_up((size_t)pr->m_max, padq);
  L.es = uses_f64(pr, op) ? 2 : 1;
  if (L.mat) L.dp = 0;   // no point records: the cost is materialised
  L.rbmax = std::max(L.pad[0], L.pad[1]) / L.rows;
  const size_t W = (size_t)pr->W;
  Carver c{reinterpret_cast<char*>(ws)};
  for (int b = 0; b < 2; ++b) {
    ds::Bank& B = L.bank[b];
    for (int side = 0; side < 2; ++side) {
      const size_t np = W * (size_t)L.pad[side];
      B.rec[side] = c.take<float>(np * L.dp * L.es);
      B.lm[side] = c.take<float>(np * L.es);
      for (int par = 0; par < 2; ++par) {
        B.lse[side][par] = c.take<float>(np * L.es);
        B.gam[side][par] = c.take<float>(np * L.es);
      }
    }
    B.slot = c.take<ds::SlotInfo>(W);
    for (int role = 0; role < 2; ++role) B.ord[role] = c.take<int>(W);
    B.dec = c.take<ds::Decision>(W);
    for (int k = 0; k < 4; ++k) B.agg[k] = c.take<float4>(W * (size_t)L.rbmax);
  }
  L.center = c.take<float>(W * (size_t)L.d);
  L.vcnt = c.take<int>(W);
  L.nchk = c.take<int>(W);
  L.disc = (op->flags & DS_F_SHADOW) ? c.take<float>(W) : nullptr;
  L.audit = c.take<ds::Audit>(W);
  L.off[0] = c.take<int>(W + 1);
  L.off[1] = c.take<int>(W + 1);
  L.ctrl = c.take<ds::Ctrl>(1);
  L.Q = L.mat ? c.take<float>(W * (size_t)L.pad[0] * (size_t)L.pad[1]) : nullptr;
  L.QT = L.mat ? c.take<float>(W * (size_t)L.pad[0] * (size_t)L.pad[1]) : nullptr;
  L.guard = (op->flags & DS_F_GUARD) ? 1 : 0;
  for (int side = 0; side < 2; ++side) {
    L.agg64[side] = L.guard ? c.take<double2>(W * (size_t)L.rbmax) : nullptr;
    L.gerr[side] = (L.guard && L.es == 2) ? c.take<float4>(W * (size_t)L.rbmax) : nullptr;
  }
  L.row64 = L.guard ? c.take<ds::RowCert>(W) : nullptr;
  L.vpart = L.guard ? c.take<double>(W * (size_t)L.rbmax * ds::kVChunks * (size_t)L.rows)
                    : nullptr;
  L.vscnt = L.guard ? c.take<int>(W * (size_t)L.rbmax) : nullptr;
  for (int role = 0; role < 2; ++role)
    L.vlist[role] = L.guard ? c.take<int>(W * (size_t)L.rbmax) : nullptr;
  L.vlen = L.guard ? c.take<int>(2) : nullptr;
  // partials and arrival words of the launches that split a work item over
  // blocks: the float64 state's narrow launches (at most kSplitSlots items),
  // and every launch of the matrix-free large-d kernel (both passes: at most
  // two items per row block of every lane)
  const bool mfree = uses_mfree(pr, op);
  L.nslots = L.es == 2 ? ds::kSplitSlots : mfree ? (int)(2 * W * (size_t)L.rbmax) : 0;
  L.spart = L.es == 2 ? c.take<double2>((size_t)L.nslots * ds::kGroups * (size_t)L.rows)
                      : nullptr;
  L.kpart = mfree ? c.take<float2>((size_t)L.nslots * ds::kGroups * (size_t)L.rows) : nullptr;
  L.scnt = L.nslots ? c.take<int>((size_t)L.nslots) : nullptr;
  L.bytes = align_up(c.off, 256);
  return L;
}

// Wherever the float32 state runs (DS_F_FAST32, or 16 < d <= 32), the
// matrix-core kernel is the default: even at d = 2 or 3 its augmented
// contraction (K = 2 ceil(d/2) + 2) costs fewer SIMD cycles per term than the
// vector kernel's d fused multiply-adds plus the bias add, and it was measured
// faster at d = 2, 3, 8 and 16.
bool uses_mfma(const ds_problem* pr, const ds_options* op) {
  if (uses_f64(pr, op)) return false;
  if (op->flags & DS_F_FORCE_VALU) return false;
  return true;
}

ds_err check_problem(const ds_problem* pr, const ds_options* op) {
  if (!pr || !op) return fail(DS_E_INVALID, "problem and options must not be NULL");
  if (pr->W < 1 || pr->n_max < 1 || pr->m_max < 1 || pr->d < 1)
    return fail(DS_E_INVALID, "W, n_max, m_max and d must be >= 1");
  if (pr->W > ds::kMaxW) return fail(DS_E_UNSUPPORTED, "W above 4096 is not supported");
  if (pr->d > 512) return fail(DS_E_INVALID, "d must be <= 512");
  if (uses_mat(pr, op)) {
    if (op->flags & (DS_F_PRECISE | DS_F_FAST32 | DS_F_FORCE_VALU | DS_F_FORCE_MFMA))
      return fail(DS_E_UNSUPPORTED, "the materialised cost (d > 32 or DS_F_MATERIALIZE) runs "
                                    "in float32 with its own kernels: no PRECISE / FAST32 / FORCE flags");
    if (pr->n_max > ds::kMatMaxPts || pr->m_max > ds::kMatMaxPts)
      return fail(DS_E_UNSUPPORTED, "the materialised cost supports at most 16384 points per side");
  }
  if ((op->flags & DS_F_GUARD) && (pr->n_max > ds::kMatMaxPts || pr->m_max > ds::kMatMaxPts))
    return fail(DS_E_UNSUPPORTED, "guarded release (DS_F_GUARD) supports at most 16384 points per side");
  if (!(op->tol > 0.f) || !std::isfinite(op->tol)) return fail(DS_E_INVALID, "tol must be finite and > 0");
  if (op->max_iter < 1) return fail(DS_E_INVALID, "max_iter must be >= 1");
  if (op->audit_every < 1) return fail(DS_E_INVALID, "audit_every must be >= 1");
  if (op->mode < DS_MODE_ACTIVE || op->mode > DS_MODE_LOGICAL) return fail(DS_E_INVALID, "unknown mode");
  if (op->streams < 0 || op->streams > kMaxParts) return fail(DS_E_INVALID, "streams must be in 0..4");
  if (op->streams > 1 && op->mode != DS_MODE_ACTIVE)
    return fail(DS_E_INVALID, "sub-batches (streams > 1) need the active mode");
  if ((op->flags & DS_F_MATRIX_FREE) && (op->flags & DS_F_MATERIALIZE))
    return fail(DS_E_INVALID, "DS_F_MATRIX_FREE and DS_F_MATERIALIZE are exclusive");
  if (uses_mfree(pr, op) && (op->flags & DS_F_FORCE_VALU))
    return fail(DS_E_UNSUPPORTED, "the matrix-free large-d half-step runs on the matrix cores");
  if ((op->flags & DS_F_FORCE_VALU) && (op->flags & DS_F_FORCE_MFMA))
    return fail(DS_E_INVALID, "DS_F_FORCE_VALU and DS_F_FORCE_MFMA are exclusive");
  if ((op->flags & DS_F_FORCE_VALU) && pr->d > 16)
    return fail(DS_E_UNSUPPORTED, "the vector-ALU kernels support d <= 16");
  if ((op->flags & DS_F_PRECISE) && (op->flags & (DS_F_FORCE_MFMA | DS_F_FORCE_VALU | DS_F_FAST32)))
    return fail(DS_E_INVALID, "DS_F_PRECISE (float64 state) excludes DS_F_FAST32 and the FORCE flags, "
                              "which select float32 kernels");
  if ((op->flags & DS_F_PRECISE) && pr->d > 16)
    return fail(DS_E_UNSUPPORTED, "the float64 state supports d <= 16");
  // sizes that keep every 32-bit index in range
  const double pts = (double)pr->W * (double)std::max(pr->n_max, pr->m_max);
  if (pts > 2.0e9) return fail(DS_E_UNSUPPORTED, "W * max(n_max, m_max) too large");
  return DS_OK;
}

#define HIP_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t _e = (expr);                                                        \
    if (_e != hipSuccess)                                                          \
      return fail(DS_E_HIP, std::string(#expr) + ": " + hipGetErrorString(_e));  \
  } while (0)

// Host resources of one sub-batch solve, kept for the life of the process in a
// per-device pool (a call takes one per sub-batch and returns them at its end):
// a pinned control snapshot, a join event, timing events, and a stream of
// its own (default priority, not synchronising with the legacy default stream)
// for sub-batches beyond the first.
struct DeviceRes {
  bool busy = false;
  ds::HostSnap* snap = nullptr;      // pinned, device-written control mirror (host view)
  ds::HostSnap* snap_dev = nullptr;  // the same memory as the device addresses it
  hipEvent_t join_ev = nullptr;      // end of this sub-batch's work on its stream
  hipStream_t stream = nullptr;
  std::vector<hipEvent_t> timing;
};
std::mutex g_pool_mu;
std::vector<std::unique_ptr<DeviceRes>> g_pool[64];

// A free resource set of the current device (created on first need).
hipError_t acquire_res(DeviceRes** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  for (auto& r : g_pool[dev])
    if (!r->busy) { r->busy = true; *out = r.get(); return hipSuccess; }
  auto r = std::make_unique<DeviceRes>();
  // a set that cannot be completed is released again, so a failed call leaks nothing
  auto undo = [&](hipError_t err) {
    if (r->stream) (void)hipStreamDestroy(r->stream);
    if (r->join_ev) (void)hipEventDestroy(r->join_ev);
    if (r->snap) (void)hipHostFree(r->snap);
    return err;
  };
  e = hipHostMalloc(reinterpret_cast<void**>(&r->snap), sizeof(ds::HostSnap),
                    hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) return undo(e);
  e = hipHostGetDevicePointer(reinterpret_cast<void**>(&r->snap_dev), r->snap, 0);
  if (e != hipSuccess) return undo(e);
  e = hipEventCreateWithFlags(&r->join_ev, hipEventDisableTiming);
  if (e != hipSuccess) return undo(e);
  e = hipStreamCreateWithFlags(&r->stream, hipStreamNonBlocking);
  if (e != hipSuccess) return undo(e);
  r->busy = true;
  *out = r.get();
  g_pool[dev].push_back(std::move(r));
  return hipSuccess;
}
void release_res(DeviceRes* r) {
  std::lock_guard<std::mutex> lock(g_pool_mu);
  r->busy = false;
}

struct EventTimer {
  bool on = false;
  hipStream_t st = nullptr;
  std::vector<hipEvent_t>* pool = nullptr;
  size_t used = 0;
  std::vector<std::pair<int, int>> spans[3];  // update kernel, compaction, other
  int take() {  // an event of the pool, not yet recorded
    if (used == pool->size()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return -1;
      pool->push_back(e);
    }
    return (int)used++;
  }
  int rec() {
    const int i = take();
    if (i < 0 || hipEventRecord((*pool)[i], st) != hipSuccess) return -1;
    return i;
  }
  double total(int kind) {
    double ms = 0;
    for (auto& sp : spans[kind]) {
      if (sp.first < 0 || sp.second < 0) continue;
      float t = 0;
      if (hipEventElapsedTime(&t, (*pool)[sp.first], (*pool)[sp.second]) == hipSuccess) ms += t;
    }
    return ms;
  }
};

// One sub-batch (or the whole window): ingest, the control loop of cycles,
// the final audit and the emission of its lanes, all on stream st. Fills the
// counters the caller merges into ds_stats.
struct Timed { int cycle, kind; };
struct PartOut {
  ds::Ctrl ctrl;
  int launched = 0, compactions = 0, n_timed = 0;
  int64_t bytes_compacted = 0;
  bool timing = false;
  std::vector<Timed> timed;
  double ms_update = 0.0, ms_compact = 0.0;
  std::vector<int32_t> nchk;
  std::vector<float> disc;   // shadow mode: screen discrepancy per lane
  std::vector<ds::SlotInfo> lanes;
  size_t ws_bytes = 0;
};

// lane_base: the caller's index of this sub-batch's first lane (error messages
// name lanes by the caller's index)
ds_err solve_part(const ds_problem* pr, const ds_options* op, const ds_result* res, void* ws,
                  hipStream_t st, DeviceRes* R, PartOut& out, int lane_base, int parts) {
  using namespace ds;
  Layout L = plan(pr, op, ws);
  const int W = pr->W, d = pr->d;
  const int mode = op->mode;
  const bool active = (mode == DS_MODE_ACTIVE);
  const bool shadow = (op->flags & DS_F_SHADOW) != 0;
  const bool guard = (op->flags & DS_F_GUARD) != 0;
  const bool use_mfma = uses_mfma(pr, op);
  const bool precise = uses_f64(pr, op);
  const bool mat = L.mat != 0;
  const int maxpad = std::max(L.pad[0], L.pad[1]);

  EventTimer tm;
  tm.on = (op->flags & DS_F_TIMING) != 0;
  tm.st = st;
  tm.pool = &R->timing;

  // ---------------------------------------------------------------- ingest
  IngestArgs ia;
  std::memset(&ia, 0, sizeof(ia));
  ia.X = pr->X; ia.Y = pr->Y; ia.a = pr->a; ia.b = pr->b; ia.eps = pr->eps; ia.g0 = pr->g0;
  ia.n = pr->n; ia.m = pr->m;
  ia.W = W; ia.n_max = pr->n_max; ia.m_max = pr->m_max; ia.d = d; ia.dp = L.dp; ia.dh = L.dh;
  ia.pad[0] = L.pad[0]; ia.pad[1] = L.pad[1];
  ia.bank = L.bank[0];
  ia.center = L.center;
  ia.vcnt = L.vcnt; ia.nchk = L.nchk; ia.disc = L.disc; ia.row64 = L.row64; ia.rbmax = L.rbmax;
  ia.precise = precise ? 1 : 0;
  ia.mat = mat ? 1 : 0;
  ia.ctrl = L.ctrl;
  HIP_TRY(launch_ingest(ia, maxpad, st));
  if (L.scnt) HIP_TRY(launch_zero_counters(L.scnt, L.nslots, st));
  if (L.vscnt) HIP_TRY(launch_zero_counters(L.vscnt, W * L.rbmax, st));
  if (L.vlen) HIP_TRY(launch_zero_counters(L.vlen, 2, st));
  HIP_TRY(launch_offsets(L.bank[0].slot, W, L.rows, L.off[0], L.off[1], L.bank[0].ord[0],
                         L.bank[0].ord[1], L.ctrl, st));
  Ctrl ctrl;
  HIP_TRY(hipMemcpyAsync(&ctrl, L.ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, st));
  std::vector<SlotInfo> lanes(W);
  HIP_TRY(hipMemcpyAsync(lanes.data(), L.bank[0].slot, sizeof(SlotInfo) * W, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  if (ctrl.err_lane != 0x7fffffff) {
    const char* what = ctrl.err_code == 1 ? "n out of range [1, n_max]"
                     : ctrl.err_code == 2 ? "m out of range [1, m_max]"
                                          : "eps not finite and > 0";
    return fail(DS_E_INVALID, "lane " + std::to_string(lane_base + ctrl.err_lane) + ": " + what);
  }
  if (mat) {
    CostArgs ca;
    ca.X = pr->X; ca.Y = pr->Y; ca.center = L.center; ca.slot = L.bank[0].slot; ca.Q = L.Q; ca.QT = L.QT;
    ca.W = W; ca.n_max = pr->n_max; ca.m_max = pr->m_max; ca.d = d;
    ca.pad0 = L.pad[0]; ca.pad1 = L.pad[1];
    HIP_TRY(launch_cost(ca, st));
  }
  // uniform lane shapes: work item -> slot is a division, no table lookup
  bool uniform = true;
  for (int t = 1; t < W; ++t)
    uniform = uniform && lanes[t].n == lanes[0].n && lanes[t].m == lanes[0].m;
  const int ipl[2] = {uniform ? row_blocks(lanes[0].n, L.rows) : 0,
                      uniform ? row_blocks(lanes[0].m, L.rows) : 0};

  int A = W, bank = 0;
  int items[2] = {ctrl.items_f, ctrl.items_g};

  auto make_pass = [&](int role, int kind, int par_in, int par_out, int col_par) {
    Pass u;
    std::memset(&u, 0, sizeof(u));
    const Bank& B = L.bank[bank];
    const int rs = role, cs = 1 - role;
    u.rec_row = B.rec[rs]; u.rec_col = B.rec[cs];
    u.lm_row = B.lm[rs];
    u.lse_in = B.lse[rs][par_in];
    u.lse_out = B.lse[rs][par_out];
    u.gam_out = B.gam[rs][par_out];
    u.gam_col = B.gam[cs][col_par];
    u.w_row = role ? pr->b : pr->a;
    u.w_ld = role ? pr->m_max : pr->n_max;
    u.off = L.off[role];
    u.ord = B.ord[role];
    if (kind == 0) {
      u.agg_out = B.agg[role == 0 ? AGG_F : AGG_G];
      u.agg_bound = B.agg[role == 0 ? AGG_G : AGG_F];
    } else {
      u.agg_out = B.agg[role == 0 ? AGG_ROW : AGG_COL];
      u.agg_screen = B.agg[AGG_F];
      u.agg_rowchk = B.agg[AGG_ROW];
    }
    u.A = A; u.ipl = ipl[role];
    u.nr = role ? lanes[0].m : lanes[0].n;   // read only when ipl > 0 (uniform shapes)
    u.nc = role ? lanes[0].n : lanes[0].m;
    u.padr = L.pad[rs]; u.padc = L.pad[cs];
    u.role = role; u.kind = kind;
    return u;
  };
  // float64 verification launches (guarded release), by role: 0 the row
  // marginal (rows = x), 1 the column marginal
  GuardArgs ga;
  std::memset(&ga, 0, sizeof(ga));
  for (int role = 0; role < 2; ++role) {
    ga.w_col[role] = role ? pr->a : pr->b;
    ga.w_ld_col[role] = role ? pr->n_max : pr->m_max;
    ga.xy_row[role] = role ? pr->Y : pr->X;
    ga.xy_col[role] = role ? pr->X : pr->Y;
    ga.ld_row[role] = role ? pr->m_max : pr->n_max;
    ga.ld_col[role] = role ? pr->n_max : pr->m_max;
    ga.agg64[role] = L.agg64[role];
    ga.gerr[role] = L.gerr[role];
  }
  ga.row64 = L.row64;
  ga.vpart = L.vpart; ga.vscnt = L.vscnt;
  ga.vlist[0] = L.vlist[0]; ga.vlist[1] = L.vlist[1]; ga.vlen = L.vlen;
  ga.eps = pr->eps; ga.d = pr->d; ga.es = L.es;
  // with the float64 state the update kernels bound how far rounding to the
  // float32 outputs moves the residual, and only lanes within that bound of
  // tol are verified; a float32 state has no such bound below its own
  // coordinate rounding (about 2^-24 C / eps per exponent), so every audited
  // lane is verified
  ga.bound = L.es == 2 ? 1 : 0;
  auto make_launch = [&]() {
    Launch l;
    std::memset(&l, 0, sizeof(l));
    l.dp = L.dp; l.rbmax = L.rbmax; l.mode = mode; l.rows = L.rows;
    l.tau_screen = op->screen_tol > 0.f ? op->screen_tol : op->tol;
    l.tol = op->tol;
    l.slot = L.bank[bank].slot; l.dec = L.bank[bank].dec;
    l.audit = L.audit; l.vcnt = L.vcnt; l.ctrl = L.ctrl;
    l.hsnap = R->snap_dev; l.nchk = L.nchk; l.disc = L.disc;
    l.progress = &R->snap_dev->progress;
    l.Q = L.Q; l.QT = L.QT; l.q_lane = (size_t)L.pad[0] * L.pad[1]; l.q_ld = L.pad[1];
    l.qt_ld = L.pad[0];
    l.spart = L.spart; l.kpart = L.kpart; l.scnt = L.scnt; l.nslots = L.nslots;
    return l;
  };
  // DS_F_TIMING: both launches of every kSampleEvery-th cycle (and the final
  // audit) carry events in their own dispatch; the rest run untouched. Each
  // timed launch remembers its cycle so its algorithmic (i, j) terms can be
  // counted from the completion depths afterwards (kind 0: update halves of
  // cycle k, kind 1: one marginal pass of the final audit).
  constexpr int kSampleEvery = 32;
  std::vector<Timed> timed_launches;
  // Kernel variant by the width bound of the launch: few items -> more waves
  // per item (shorter sweeps); many items -> more rows per wave (fewer column
  // re-reads). Every variant computes the same bits.
  // Middle widths on the matrix cores: a wave sweeps two groups, or four when
  // a group is at most two column tiles (the launch's columns: the other
  // side's points), so that every wave still sweeps several tiles.
  int tpg[2];
  for (int role = 0; role < 2; ++role) {
    const int cols = uniform ? (role ? lanes[0].n : lanes[0].m) : L.pad[1 - role];
    const int ct = (cols + kColTile - 1) / kColTile;
    tpg[role] = (ct + kGroups - 1) / kGroups;
  }
  auto pick = [&](int items, int role) -> int {
    if (mat) return VAR_MEDIUM;   // one layout: 64-row items, one block each
    // float64 state: few items get one wave per (item, sub-group). The split
    // shortens every sweep from tpg tiles to about tpg / 4 but adds a round
    // trip of the group partials through memory and more blocks per item, so
    // it pays at more items the longer the groups are (measured: up to 64
    // items with 2 tiles per group, 128 with 4, 256 with 32)
    if (precise) {
      const int tg = tpg[role];
      if ((tg >= 16 && items <= 256) || (tg >= 4 && items <= 128) || (tg >= 2 && items <= 64))
        return VAR_SPLIT;
    }
    // (the float64 kernel's items hold 64 to 256 rows: fewer items per width)
    const int medium = use_mfma ? kMediumItemsMfma * kRowsMfma / L.rows
                       : (precise && !uniform) ? kMediumItemsF64Mixed
                       : (precise && parts == 1) ? kMediumItemsF64Solo
                                                 : kMediumItemsValu * kRowsValu / L.rows;
    if (items < medium) return VAR_NARROW;
    return (use_mfma && tpg[role] <= 2) ? VAR_MEDIUM4 : VAR_MEDIUM;
  };
  auto blocks_of = [&](int items) -> int { return std::max(items, 0); };
  int seqno = 0;   // update launches issued (see HostSnap::progress)
  auto run = [&](Launch l, int variant, int blocks, bool sample, int cycle, int kind) -> ds_err {
    l.seqno = ++seqno;
    const bool timed = tm.on && sample && (int)timed_launches.size() < kMaxTimed;
    // the events are part of the kernel's own dispatch: they time the kernel,
    // not the queue around it
    const int e0 = timed ? tm.take() : -1, e1 = timed ? tm.take() : -1;
    hipEvent_t h0 = e0 >= 0 ? (*tm.pool)[e0] : nullptr, h1 = e1 >= 0 ? (*tm.pool)[e1] : nullptr;
    if (mat) HIP_TRY(launch_update_mat(l, blocks, st, h0, h1));
    else if (precise) HIP_TRY(launch_update_f64(l, d, variant, blocks, st, h0, h1));
    else if (d > kMaxDSmall) HIP_TRY(launch_update_mfma_k(l, blocks, st, h0, h1));
    else HIP_TRY(launch_update(l, d, use_mfma, variant, blocks, st, h0, h1));
    if (timed) {
      tm.spans[0].push_back({e0, e1});
      timed_launches.push_back({cycle, kind});
    }
    return DS_OK;
  };

  // ------------------------------------------------------------ main loop
  const int max_iter = op->max_iter, ae = op->audit_every;
  const int kLag = 8;          // cycles the host may run ahead of the device
  volatile HostSnap* hs = R->snap;
  hs->n_active = W; hs->n_retired = 0; hs->compacted = 0; hs->epoch = 0; hs->finished = 0;
  hs->items_act_f = items[0]; hs->items_act_g = items[1];
  hs->progress = 0;
  int epoch = 0;
  int launched = 0;
  int compactions = 0;
  int64_t bytes_compacted = 0;  // upper bound: survivors x per-lane state bytes
  const int64_t lane_bytes = (int64_t)(L.pad[0] + L.pad[1]) * (L.dp + 5) * 4 * L.es +
                             (int64_t)(sizeof(SlotInfo) + sizeof(Decision));
  for (int k = 1; k <= max_iter; ++k) {
    // bounded run-ahead: wait for the device only when too far behind
    // (block 0 of every update launch publishes the launch's sequence
    // number). Only when the word has not moved for a while is the stream
    // queried, so that a failed launch surfaces as an error instead of a wait
    // that never ends; frequent queries from several sub-batch threads would
    // contend with their launches in the runtime.
    if (seqno - hs->progress > 2 * kLag) {
      int seen = hs->progress;
      auto since = std::chrono::steady_clock::now();
      while (seqno - hs->progress > 2 * kLag) {
        const int now_seen = hs->progress;
        if (now_seen != seen) {
          seen = now_seen;
          since = std::chrono::steady_clock::now();
        } else if (std::chrono::steady_clock::now() - since > std::chrono::milliseconds(20)) {
          const hipError_t qe = hipStreamQuery(st);
          if (qe == hipSuccess) break;                // idle: nothing left to wait for
          if (qe != hipErrorNotReady) HIP_TRY(qe);
          since = std::chrono::steady_clock::now();
        }
        std::this_thread::yield();
      }
    }
    const int s_fin = hs->finished, s_ep = hs->epoch, s_ret = hs->n_retired;
    const int s_cmp = hs->compacted, s_act = hs->n_active;
    const int s_itf = hs->items_act_f, s_itg = hs->items_act_g;
    if (s_fin) break;
    if (active && s_ep == epoch && s_ret > s_cmp) {
      // physical compaction: survivors gathered into the other bank
      epoch++;
      ScanArgs sa;
      std::memset(&sa, 0, sizeof(sa));
      sa.slot = L.bank[bank].slot; sa.dec = L.bank[bank].dec;
      sa.off_f = L.off[0]; sa.off_g = L.off[1]; sa.ctrl = L.ctrl; sa.hsnap = R->snap_dev;
      for (int role = 0; role < 2; ++role) {
        sa.ord_src[role] = L.bank[bank].ord[role];
        sa.ord_dst[role] = L.bank[bank ^ 1].ord[role];
      }
      sa.A = A; sa.W = W; sa.compact = 1; sa.rows = L.rows; sa.epoch = epoch;
      const int e0 = tm.on ? tm.rec() : -1;
      HIP_TRY(launch_scan(sa, st));
      MoveArgs ma;
      std::memset(&ma, 0, sizeof(ma));
      ma.src = L.bank[bank]; ma.dst = L.bank[bank ^ 1]; ma.ctrl = L.ctrl;
      ma.A = A; ma.dp = L.dp; ma.compact = 1; ma.emit_all = 0; ma.mode = mode;
      ma.pad[0] = L.pad[0]; ma.pad[1] = L.pad[1];
      ma.n_max = pr->n_max; ma.m_max = pr->m_max; ma.chunk = 1024; ma.es = L.es; ma.rbmax = L.rbmax;
      ma.f = res->f; ma.g = res->g; ma.depth = res->depth; ma.residual = res->residual;
      ma.row_res = res->row_residual; ma.col_res = res->col_residual; ma.status = res->status;
      HIP_TRY(launch_move(ma, A, maxpad, st));
      if (tm.on) tm.spans[1].push_back({e0, tm.rec()});
      bank ^= 1;
      bytes_compacted += (int64_t)s_act * lane_bytes;
      A = std::min(A, s_act);              // upper bound on the survivors
      items[0] = std::min(items[0], s_itf);
      items[1] = std::min(items[1], s_itg);
      compactions++;
    }
    if (A <= 0) break;
    const int pk = k & 1, pk1 = (k - 1) & 1;
    const bool sample = (k % kSampleEvery) == 0;
    const bool audit_prev = (k - 1 >= 1) && ((k - 1) % ae == 0);
    // f-half of cycle k (+ row screen of state k-1)
    Launch lf = make_launch();
    lf.p[0] = make_pass(0, 0, pk1, pk, pk1);
    lf.p[0].depth = k - 1;
    // guarded release: the export rounding of state k-1's f, before its check
    if (audit_prev && guard) lf.p[0].gerr_out = L.gerr[0];
    const int vf = pick(items[0], 0);
    lf.nb0 = blocks_of(items[0]);
    ds_err r = run(lf, vf, lf.nb0, sample, k, 0);
    if (r != DS_OK) return r;
    if (audit_prev && guard) {
      // guarded release: float64 verification of state k-1 (the potentials the
      // emission would write) before the g-half: the row marginal of the lanes
      // the outward bound leaves, then the column marginal of those whose row
      // residual met tol
      Launch lc = make_launch();
      lc.p[0] = make_pass(0, 1, pk1, pk1, pk1);
      lc.p[0].depth = k - 1;
      lc.p[0].verify_all = shadow ? 1 : 0;
      HIP_TRY(launch_vgate(lc, ga, st));
      HIP_TRY(launch_verify64(lc, ga, items[0], st));
      Launch lk = make_launch();
      lk.p[0] = make_pass(1, 1, pk1, pk1, pk1);
      lk.p[0].depth = k - 1;
      HIP_TRY(launch_verify64(lk, ga, items[1], st));
    }
    if (audit_prev && shadow && !guard) {
      // shadow mode: the row marginal of state k-1 recomputed by a dedicated
      // pass, so the decision can record how far the fused screen is from it
      Launch lr = make_launch();
      lr.p[0] = make_pass(0, 1, pk1, pk1, pk1);
      lr.p[0].depth = k - 1;
      lr.p[0].verify_all = 1;
      lr.nb0 = blocks_of(items[0]);
      r = run(lr, pick(items[0], 0), lr.nb0, false, k, 1);
      if (r != DS_OK) return r;
    }
    // g-half of cycle k (+ column check and decision for state k-1)
    // (the check blocks come last: most of them exit at once, and at the front
    // they would delay the update blocks' dispatch)
    Launch lg = make_launch();
    const int vg = pick(items[1], 1);
    const int nbg = blocks_of(items[1]);
    int blocks = nbg;
    if (audit_prev && !guard) {
      lg.p[0] = make_pass(1, 0, pk1, pk, pk);     // g-half of cycle k
      lg.p[1] = make_pass(1, 1, pk1, pk1, pk1);   // column marginal of state k-1
      lg.p[1].decide = 1;
      lg.p[1].verify_all = shadow ? 1 : 0;
      lg.p[1].depth = k - 1;
      lg.nb0 = nbg;
      blocks += nbg;
    } else {
      lg.p[0] = make_pass(1, 0, pk1, pk, pk);
      lg.nb0 = nbg;
    }
    // guarded release: the export rounding of state k's g, for its audit
    if (guard && k % ae == 0) lg.p[0].gerr_out = L.gerr[1];
    r = run(lg, vg, blocks, sample, k, 0);
    if (r != DS_OK) return r;
    launched = k;
  }
  HIP_TRY(hipMemcpyAsync(&ctrl, L.ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  A = ctrl.A;

  // ------------------------------------------------------- final audit
  // max_iter reached with lanes still active (any mode), or static mode's
  // common boundary: both marginals of the returned state, every lane.
  const bool need_final = !ctrl.finished || mode == DS_MODE_STATIC;
  if (need_final) {
    const int K = ctrl.finished ? ctrl.final_cycle : launched;
    const int pK = K & 1;
    HIP_TRY(launch_zero_counters(L.vcnt, W, st));
    int saveA = A;
    if (guard) {
      // both marginals of state K in float64, every lane still running (the
      // column launch decides)
      Launch lc = make_launch(), lk = make_launch();
      lc.p[0] = make_pass(0, 1, pK, pK, pK);
      lk.p[0] = make_pass(1, 1, pK, pK, pK);
      for (Pass* q : {&lc.p[0], &lk.p[0]}) {
        q->final_audit = 1; q->depth = K; q->verify_all = 1; q->decide = 1;
      }
      HIP_TRY(launch_vgate(lc, ga, st));
      HIP_TRY(launch_verify64(lc, ga, ctrl.items_f, st));
      HIP_TRY(launch_verify64(lk, ga, ctrl.items_g, st));
    } else {
      Launch lv = make_launch();
      lv.p[0] = make_pass(0, 1, pK, pK, pK);
      lv.p[0].final_audit = 1; lv.p[0].depth = K; lv.p[0].verify_all = 1;
      const int vv = pick(ctrl.items_f, 0);
      lv.nb0 = blocks_of(ctrl.items_f);
      ds_err r = run(lv, vv, lv.nb0, true, K, 1);
      if (r != DS_OK) return r;
      Launch lw = make_launch();
      lw.p[0] = make_pass(1, 1, pK, pK, pK);
      lw.p[0].final_audit = 1; lw.p[0].decide = 1; lw.p[0].depth = K; lw.p[0].verify_all = 1;
      const int vw = pick(ctrl.items_g, 1);
      lw.nb0 = blocks_of(ctrl.items_g);
      r = run(lw, vw, lw.nb0, true, K, 1);
      if (r != DS_OK) return r;
    }
    A = saveA;
    HIP_TRY(hipMemcpyAsync(&ctrl, L.ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
  }
  // ------------------------------------------------------------ emission
  {
    MoveArgs ma;
    std::memset(&ma, 0, sizeof(ma));
    ma.src = L.bank[bank]; ma.dst = L.bank[bank ^ 1]; ma.ctrl = L.ctrl;
    ma.A = A; ma.dp = L.dp; ma.compact = 0; ma.emit_all = (mode == DS_MODE_STATIC); ma.mode = mode;
    ma.final_par = ctrl.final_cycle & 1;
    ma.pad[0] = L.pad[0]; ma.pad[1] = L.pad[1];
    ma.n_max = pr->n_max; ma.m_max = pr->m_max; ma.chunk = 1024; ma.es = L.es; ma.rbmax = L.rbmax;
    ma.f = res->f; ma.g = res->g; ma.depth = res->depth; ma.residual = res->residual;
    ma.row_res = res->row_residual; ma.col_res = res->col_residual; ma.status = res->status;
    HIP_TRY(launch_move(ma, A, maxpad, st));
  }
  out.nchk.resize(W);
  HIP_TRY(hipMemcpyAsync(out.nchk.data(), L.nchk, sizeof(int32_t) * W, hipMemcpyDeviceToHost, st));
  if (L.disc) {
    out.disc.resize(W);
    HIP_TRY(hipMemcpyAsync(out.disc.data(), L.disc, sizeof(float) * W, hipMemcpyDeviceToHost, st));
  }
  HIP_TRY(hipStreamSynchronize(st));
  out.ctrl = ctrl;
  out.launched = launched;
  out.compactions = compactions;
  out.bytes_compacted = bytes_compacted;
  out.timing = tm.on;
  out.n_timed = (int)tm.spans[0].size();
  if (tm.on) {
    out.ms_update = tm.total(0);
    out.ms_compact = tm.total(1);
  }
  out.timed = std::move(timed_launches);
  out.lanes = std::move(lanes);
  out.ws_bytes = L.bytes;
  return DS_OK;
}

// Sub-batches: contiguous lane ranges solved concurrently, each on its own
// stream with its own workspace part and control loop. Lanes are independent,
// so the results are those of one batch bit for bit; the launch latencies of
// one sub-batch overlap the work of the others. Active mode only (the static
// and logical modes share one final cycle across the window).
// Automatic sub-batch count: two from 32 lanes on. Measured solves (ms) with
// one, two and three sub-batches: mixture window (W = 64, d = 8) 289 / 259 / --,
// telemetry (W = 256, d = 16) 529 / 461 / 469, LiDAR-shaped (W = 1024, d = 3)
// 1870 / 1839 / 1846.
int parts_of(const ds_problem* pr, const ds_options* op) {
  if (op->streams > 0) return std::min(op->streams, pr->W);
  if (op->mode != DS_MODE_ACTIVE || uses_mat(pr, op)) return 1;
  return pr->W < 32 ? 1 : 2;
}
int part_lo(const ds_problem* pr, int parts, int p) {
  return (int)((int64_t)pr->W * p / parts);
}
ds_problem sub_problem(const ds_problem* pr, int lo, int hi) {
  ds_problem s = *pr;
  s.W = hi - lo;
  s.X = pr->X + (size_t)lo * pr->n_max * pr->d;
  s.Y = pr->Y + (size_t)lo * pr->m_max * pr->d;
  s.a = pr->a + (size_t)lo * pr->n_max;
  s.b = pr->b + (size_t)lo * pr->m_max;
  s.eps = pr->eps + lo;
  s.n = pr->n ? pr->n + lo : nullptr;
  s.m = pr->m ? pr->m + lo : nullptr;
  s.g0 = pr->g0 ? pr->g0 + (size_t)lo * pr->m_max : nullptr;
  return s;
}
ds_result sub_result(const ds_problem* pr, const ds_result* res, int lo) {
  ds_result s = *res;
  s.f = res->f + (size_t)lo * pr->n_max;
  s.g = res->g + (size_t)lo * pr->m_max;
  s.depth = res->depth + lo;
  s.residual = res->residual + lo;
  s.row_residual = res->row_residual ? res->row_residual + lo : nullptr;
  s.col_residual = res->col_residual ? res->col_residual + lo : nullptr;
  s.status = res->status + lo;
  s.order = nullptr;
  return s;
}
// workspace offset of every part (and the total, last)
std::vector<size_t> part_offsets(const ds_problem* pr, const ds_options* op, int parts) {
  std::vector<size_t> off(parts + 1, 0);
  for (int p = 0; p < parts; ++p) {
    const ds_problem s = sub_problem(pr, part_lo(pr, parts, p), part_lo(pr, parts, p + 1));
    off[p + 1] = off[p] + align_up(plan(&s, op, nullptr).bytes, 256);
  }
  return off;
}

}  // namespace

extern "C" {

int ds_api_version(void) { return DS_API_VERSION; }

const char* ds_error_string(ds_err e) {
  switch (e) {
    case DS_OK: return "ok";
    case DS_E_INVALID: return "invalid argument";
    case DS_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case DS_E_HIP: return "HIP runtime error";
    case DS_E_UNSUPPORTED: return "unsupported configuration";
    case DS_E_INTERNAL: return "internal error";
  }
  return "unknown error";
}

const char* ds_last_error_message(void) { return g_last_error.c_str(); }

ds_err ds_workspace_bytes(const ds_problem* pr, const ds_options* op, size_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(DS_E_INVALID, "bytes must not be NULL");
  ds_err e = check_problem(pr, op);
  if (e != DS_OK) return e;
  const int parts = parts_of(pr, op);
  *bytes = part_offsets(pr, op, parts)[parts];
  return DS_OK;
}

ds_err ds_solve(const ds_problem* pr, const ds_options* op, const ds_result* res, void* ws,
                size_t ws_bytes, void* stream_v, ds_stats* stats) {
  using namespace ds;
  const auto t_start = std::chrono::steady_clock::now();
  g_last_error.clear();
  ds_err e = check_problem(pr, op);
  if (e != DS_OK) return e;
  if (!res) return fail(DS_E_INVALID, "result must not be NULL");
  if (!pr->X || !pr->Y || !pr->a || !pr->b || !pr->eps)
    return fail(DS_E_INVALID, "X, Y, a, b and eps must not be NULL");
  if (!res->f || !res->g || !res->depth || !res->residual || !res->status)
    return fail(DS_E_INVALID, "f, g, depth, residual and status must not be NULL");
  const int parts = parts_of(pr, op);
  const std::vector<size_t> off = part_offsets(pr, op, parts);
  if (!ws) return fail(DS_E_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(DS_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < off[parts])
    return fail(DS_E_WORKSPACE, "workspace too small: need " + std::to_string(off[parts]) + " bytes");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream_v);
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  const int W = pr->W;
  const int mode = op->mode;
  const bool active = (mode == DS_MODE_ACTIVE);
  const int ae = op->audit_every;

  // resources of every part; parts beyond the first start behind the work
  // already queued on the caller's stream
  std::vector<DeviceRes*> Rs(parts, nullptr);
  struct Releaser {
    std::vector<DeviceRes*>& v;
    ~Releaser() { for (DeviceRes* r : v) if (r) release_res(r); }
  } releaser{Rs};
  for (int p = 0; p < parts; ++p) HIP_TRY(acquire_res(&Rs[p]));
  const bool timing = (op->flags & DS_F_TIMING) != 0;
  if (parts > 1) {
    HIP_TRY(hipEventRecord(Rs[0]->join_ev, st));
    for (int p = 1; p < parts; ++p) HIP_TRY(hipStreamWaitEvent(Rs[p]->stream, Rs[0]->join_ev, 0));
  }
  std::vector<PartOut> outs(parts);
  std::vector<ds_err> errs(parts, DS_OK);
  std::vector<std::string> msgs(parts);
  auto work = [&](int p) {
    if (p > 0) {
      const hipError_t he = hipSetDevice(dev);
      if (he != hipSuccess) { errs[p] = DS_E_HIP; msgs[p] = hipGetErrorString(he); return; }
    }
    const int lo = part_lo(pr, parts, p), hi = part_lo(pr, parts, p + 1);
    const ds_problem sp = sub_problem(pr, lo, hi);
    const ds_result sr = sub_result(pr, res, lo);
    hipStream_t s = p == 0 ? st : Rs[p]->stream;
    errs[p] = solve_part(&sp, op, &sr, static_cast<char*>(ws) + off[p], s, Rs[p], outs[p], lo,
                         parts);
    if (errs[p] != DS_OK) msgs[p] = g_last_error;
    if (p > 0 && errs[p] == DS_OK) {
      const hipError_t he = hipEventRecord(Rs[p]->join_ev, s);
      if (he != hipSuccess) { errs[p] = DS_E_HIP; msgs[p] = hipGetErrorString(he); }
    }
  };
  {
    std::vector<std::thread> th;
    for (int p = 1; p < parts; ++p) th.emplace_back(work, p);
    work(0);
    for (auto& t : th) t.join();
  }
  for (int p = 0; p < parts; ++p) {
    if (errs[p] == DS_OK) continue;
    // drain every sub-batch's stream before its resources go back to the pool
    // (the outputs are undefined after an error, the workspace must be idle)
    (void)hipStreamSynchronize(st);
    for (int q = 1; q < parts; ++q) (void)hipStreamSynchronize(Rs[q]->stream);
    return fail(errs[p], msgs[p]);
  }
  for (int p = 1; p < parts; ++p) HIP_TRY(hipStreamWaitEvent(st, Rs[p]->join_ev, 0));
  if (res->order) HIP_TRY(launch_order(res->depth, W, res->order, st));
  std::vector<int32_t> depth(W), status(W);
  HIP_TRY(hipMemcpyAsync(depth.data(), res->depth, sizeof(int32_t) * W, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipMemcpyAsync(status.data(), res->status, sizeof(int32_t) * W, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  HIP_TRY(hipGetLastError());
  if (stats) {
    ds_stats S;
    std::memset(&S, 0, sizeof(S));
    int lmax = 0;
    int64_t sum_l = 0;
    for (int t = 0; t < W; ++t) { lmax = std::max(lmax, depth[t]); sum_l += depth[t]; }
    S.l_max = lmax;
    S.slots_update = active ? sum_l : (int64_t)W * lmax;
    // (i, j) term counts from the completion depths: a lane runs both halves
    // of every cycle up to its depth (active) or up to l_max (static, logical);
    // speculative halves are not algorithmic work and are not counted here
    std::vector<int64_t> nm(W);
    int64_t upd = 0, chk = 0, retire_events = 0;
    int launched = 0, finished_all = 1;
    for (int p = 0; p < parts; ++p) {
      const int lo = part_lo(pr, parts, p);
      const PartOut& o = outs[p];
      for (size_t u = 0; u < o.lanes.size(); ++u) {
        const int t = lo + (int)u;
        nm[t] = (int64_t)o.lanes[u].n * (int64_t)o.lanes[u].m;
        chk += (int64_t)o.nchk[u] * nm[t];
      }
      retire_events += o.ctrl.retire_events;
      for (float v : o.disc) S.screen_discrepancy = std::max(S.screen_discrepancy, (double)v);
      launched = std::max(launched, o.launched);
      finished_all &= o.ctrl.finished ? 1 : 0;
      S.screen_positive += o.ctrl.screen_pos;
      S.check_failures += o.ctrl.check_fail;
      S.missed_ready += o.ctrl.missed_ready;
      S.guard_missed += o.ctrl.guard_missed;
      S.compactions += o.compactions;
      S.update_launches += o.n_timed;   // timed launches
      S.workspace_bytes += o.ws_bytes;
      S.bytes_compacted += o.bytes_compacted;
    }
    for (int t = 0; t < W; ++t) upd += 2 * (int64_t)(active ? depth[t] : lmax) * nm[t];
    S.pair_evals = upd;
    S.check_pair_evals = chk;
    // every lane ran its l_t cycles; a lane retired at an ordinary audit also
    // ran the cycle after it (its discarded f-half and the g-half that shared
    // the launch with its check)
    S.halfsteps_executed = active ? 2 * sum_l + 2 * retire_events
                                  : 2 * (int64_t)W * (lmax + (finished_all ? 1 : 0));
    S.cycles = launched;
    S.sub_batches = parts;
    S.audits = 0;
    for (int k = 1; k <= launched; ++k) S.audits += (k % ae == 0) ? 1 : 0;
    if (stats->width_trace && stats->width_trace_len > 0) {
      const int cap = stats->width_trace_len;
      int n = 0;
      for (int k = 1; k <= lmax && n < cap; ++k, ++n) {
        int Ak = 0;
        for (int t = 0; t < W; ++t) Ak += (active ? depth[t] >= k : 1);
        stats->width_trace[n] = Ak;
      }
      S.width_trace_len = n;
    }
    S.width_trace = stats->width_trace;
    if (timing) {
      // algorithmic terms of the timed launches: one half-step over the lanes
      // of its sub-batch still running at that cycle, or one marginal pass of
      // the final audit
      int64_t tp = 0;
      for (int p = 0; p < parts; ++p) {
        const int lo = part_lo(pr, parts, p), hi = part_lo(pr, parts, p + 1);
        int plmax = 0;
        for (int t = lo; t < hi; ++t) plmax = std::max(plmax, depth[t]);
        for (const Timed& q : outs[p].timed)
          for (int t = lo; t < hi; ++t) {
            const bool in = q.kind == 0 ? (active ? depth[t] >= q.cycle : q.cycle <= plmax)
                                        : (mode == DS_MODE_STATIC || depth[t] == q.cycle);
            if (in) tp += nm[t];
          }
        S.ms_update += outs[p].ms_update;
        S.ms_compact += outs[p].ms_compact;
      }
      S.timed_pair_evals = tp;
      S.ms_check = 0.0;
    }
    S.ms_total = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    *stats = S;
  }
  return DS_OK;
}

ds_err ds_solve_noalloc(const ds_problem* pr, const ds_options* op, const ds_result* res,
                        void* stream_v, ds_stats* stats) {
  g_last_error.clear();
  ds_err e = check_problem(pr, op);
  if (e != DS_OK) return e;
  if (op->streams > 1)
    return fail(DS_E_INVALID, "ds_solve_noalloc runs one sub-batch on the caller's stream: "
                              "streams must be 0 or 1");
  if (op->flags & DS_F_TIMING)
    return fail(DS_E_INVALID, "ds_solve_noalloc does not time launches (DS_F_TIMING creates events)");
  ds_options one = *op;
  one.streams = 1;
  const size_t need = part_offsets(pr, &one, 1)[1];
  void* ws = nullptr;
  size_t cap = 0;
  HIP_TRY(ds::scratch_area(&ws, &cap));
  if (need > cap)
    return fail(DS_E_UNSUPPORTED, "ds_solve_noalloc: this problem needs " + std::to_string(need) +
                                      " bytes of workspace, above the " + std::to_string(cap) +
                                      "-byte allocation-free workspace; use ds_solve with a "
                                      "caller workspace");
  return ds_solve(pr, &one, res, ws, cap, stream_v, stats);
}

}  // extern "C"
