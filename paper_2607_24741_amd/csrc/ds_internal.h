// Internal layout shared by the host runtime (ds_host.cpp) and the gfx950
// kernels (ds_kernels.hip). Not part of the public ABI.
//
// Representation. Per lane the points are centred (c = mean of the live source
// points and target points, averaged) and scaled by sqrt(2 kappa), where
// kappa = log2(e) / eps. With x~ = sqrt(2 kappa)(x - c) and likewise y~, every
// exponent of the method is an affine function of the dot product x~ . y~ in
// base-2 units:
//     kappa (g_j - C_ij) + kappa |x_i - c|^2 = gam^y_j + x~_i . y~_j,
//     gam^y_j = kappa (g_j - |y_j - c|^2),
// and the f-half of eq:sinkhorn-cycle becomes
//     lse^x_i = log2 sum_j 2^(gam^y_j + x~_i . y~_j),   gam^x_i = log2 a_i - lse^x_i,
// with f_i = (gam^x_i + |x~_i|^2 / 2) / kappa. The g-half is the same with the
// roles of the two sides swapped. Per point the state kept is lse (the row
// role's log-sum, used as the anchor of the next update and for the screen) and
// gam = log2 mass - lse (the column role's operand); both are stored by cycle
// parity so the audited state k survives while cycle k+1 is computed.
//
// The row marginal ratio of the state (f^k, g^k) is exactly
//     R_i / a_i = 2^(lse^x_i(k+1) - lse^x_i(k)),
// so the f-update of cycle k+1 yields the row screen of state k with no extra
// pass over (i, j) (eq:updated-marginal makes the column marginal the current
// one; Sec. 3.1).
//
// Precision. With the float64 state (the default for d <= 16) the records,
// log masses, lse and gam are doubles and every exponent is formed in double
// before one rounding to float32 for the exponential: the terms of the method
// are of size C/eps (thousands in base-2 units), so rounding the scaled
// coordinates or the potentials to float32 perturbs each exponent by
// ~C/eps * 2^-24 and moves the residual trajectory by 1e-6..1e-5, while the
// single rounding of an exponent of magnitude <= 64 costs ~1e-8 on it.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace ds {

constexpr int kPad = 128;        // point padding of every lane-indexed array
constexpr int kColTile = 32;     // columns per MFMA tile
constexpr int kGroups = 8;       // fixed column groups of a lane (whole tiles each)
// Float64-state kernel: each group is cut into kSubGroups fixed sub-groups of
// whole tiles, each summed from a fresh accumulator and folded into the group
// in order, so that a narrow launch can give every (work item, sub-group) a
// wave of its own (k_update_f64_split, one block per group) with the same bits.
constexpr int kSubGroups = 4;
// most work items of one pass of a split launch; a launch holds at most two
// passes, and its partials (in the workspace) are sized for both
constexpr int kSplitItems = 256;
constexpr int kSplitSlots = 2 * kSplitItems;
constexpr int kRowsMfma = 32;    // rows per work item, matrix-core kernel
constexpr int kRowsValu = 64;    // rows per work item, vector-ALU kernel
constexpr int kRowsMfmaK = 128;  // rows per work item, matrix-free large-d kernel
constexpr int kMfreeCols = 128;  // columns per step of the matrix-free large-d kernel
// coordinates per LDS stage of the matrix-free large-d kernel; its point
// records are padded to a multiple of this with zeros
constexpr int kMfreeK = 32;
// Float64 verification (guarded release): the columns of a lane are cut into
// kVChunks fixed chunks, each summed per row on its own and the chunk sums
// added in chunk order; a verification launch strides at most kVerifyBlocks
// blocks over the (row block, chunk) units of the rows it verifies.
constexpr int kVChunks = 8;
constexpr int kVerifyBlocks = 2048;
constexpr int kMaxW = 4096;
constexpr int kMaxDSmall = 32;   // matrix-free kernels
constexpr int kMaxDF64 = 16;     // matrix-free float64-state kernels
constexpr int kMatMaxPts = 16384; // materialised cost: points per lane side (LDS staging, 64 KB)
constexpr float kFastRange = 64.f;  // max spread of the bound (log2 units) for anchored sums
// The same for the float64 state: there the anchored exponent (at most this
// far above the true row maximum) is rounded once to float32 for v_exp_f32,
// a relative error of at most 64 * 2^-24 * ln 2 ~ 2.6e-6 per term.
constexpr float kFastRangePrecise = 64.f;
constexpr int kMaxTimed = 4096;     // timed launches per sub-batch (DS_F_TIMING)
constexpr size_t kScratchBytes = (size_t)64 << 20;  // workspace of ds_solve_noalloc, per GPU
constexpr int kMaxDevices = 64;
// launch-variant thresholds (work items of the launch, see launch_update)
constexpr int kMediumItemsMfma = 384;
constexpr int kMediumItemsValu = 256;
// float64 kernel, mixed lane shapes: eight short-sweep waves per block keep the
// heterogeneous items balanced up to this many items (measured on LiDAR-shaped
// lanes: 8-wave blocks faster up to 8.7k items, 4-wave blocks from 12.6k)
constexpr int kMediumItemsF64Mixed = 10000;
// float64 kernel, uniform shapes, a call of one sub-batch: eight-wave blocks (one
// column group per wave) up to this many items, so that a launch of 17 to 32
// mixture lanes (d = 8, 128-row items) spreads over twice the waves with half
// the sweep each (one-sub-batch mixture solve 274 against 284 ms; the telemetry
// window unchanged). With two sub-batches the streams' launches already share
// the chip, and the four-wave layout stays faster from 128 items (255 against
// 260 ms); 512 or more items were slower either way.
constexpr int kMediumItemsF64Solo = 256;

// Per physical slot lane descriptor; moved by compaction with the rest of the
// lane-indexed state.
struct SlotInfo {
  int lane;        // caller lane id
  int n, m;        // valid prefix sizes
  int done;        // retired (active, logical) -- its work items no longer run
  int passed;      // static mode: first passing audit seen (lane keeps updating)
  float kappa;     // log2(e) / eps
  double kappa64;  // the same in float64 (precise state)
  int pad[2];
};

// Control block (device). Counters written by kernels, read by the host.
struct Ctrl {
  int err_lane;      // first lane failing validation (0x7fffffff none)
  int err_code;      // 1 n out of range, 2 m out of range, 3 eps invalid
  int n_active;      // lanes not yet retired (static: not yet passed)
  int n_retired;     // lanes retired so far (active / logical)
  int finished;      // every lane retired / passed: later work items exit
  int final_cycle;   // audit cycle at which the last lane passed (static)
  int A;             // slots in the current (compacted) layout
  int items_f, items_g;            // work items of the current layout
  int items_act_f, items_act_g;    // work items of the lanes still active
  int screen_pos;    // screen-positive events
  int check_fail;    // screen-positive lanes rejected by the two-sided check
  int missed_ready;  // shadow mode: screen-negative lanes that would pass
  int retire_events; // retirements at ordinary audits (each ran one extra cycle)
  int compacted;     // retired lanes already removed by compaction
  int A_prev;        // width before the latest compaction map
  int guard_missed;  // guarded release + shadow mode: audits whose verified row
                     // residual met tol although the outward bound had excluded them
};

// Best-effort mirror of the control counters in pinned host memory, written
// by the device with system-scope stores (no copy on the stream).
// `progress`: sequence number of the latest update launch that has started on
// the device (its block 0 writes it first thing), so every earlier launch of
// the stream has completed.
struct HostSnap {
  int n_active, n_retired, compacted, epoch, finished, items_act_f, items_act_g, progress;
};

// Guarded release: the float64 row residual of a verified state, by caller lane,
// and the depth of that state (the column check of the same audit reads it).
struct RowCert {
  double r;
  int depth;
  int bad;       // non-finite marginal
};

// Per slot audit scratch (indexed by the slot at audit time).
struct Audit {
  float rhat;    // row residual (fused screen, or row check at the final audit)
  float rcol;    // column residual from the check
  int flag;      // screen-positive at the latest audit
  int pad;
};

// Retirement record of a slot (written when the lane is decided).
struct Decision {
  int status;    // ds_lane_status
  int depth;     // completion depth (cycles)
  float res_row, res_col;
  int new_slot;  // compaction map (scan output), -1 for emitted lanes
  int pad[3];
};

// One bank of lane-indexed state (two banks ping-pong under compaction).
// With the float64 (precise) state every array below holds doubles in the same
// shape (the float pointers are reinterpreted) and records are not
// de-interleaved.
// Row-block aggregates of a pass, by slot: {screen or residual partial sum,
// min and max of the lse change, non-finite flag}. [0] f-half, [1] g-half,
// [2] row check, [3] column check. Slot indexing lets a block fetch its lane's
// aggregates together with its operands, before it has read its slot record;
// compaction carries them to the survivors' new slots.
enum { AGG_F = 0, AGG_G = 1, AGG_ROW = 2, AGG_COL = 3 };

struct Bank {
  float* rec[2];     // side 0 (x), side 1 (y): [W][pad][dp] scaled, centred, de-interleaved
  float* lm[2];      // log2 masses [W][pad]; -inf for dead points
  float* lse[2][2];  // [side][parity] [W][pad]; +inf for dead points
  float* gam[2][2];  // [side][parity] [W][pad]; -inf for dead points
  SlotInfo* slot;    // [W]
  Decision* dec;     // [W]
  float4* agg[4];    // [W][rbmax] row-block aggregates by slot
  // Work item order of the mixed-shape launches, per role (0: f-half and row
  // check, 1: g-half and column check): the slots by decreasing column count
  // (the length of each of the lane's sweeps), then by slot. Launches place
  // the longest sweeps first, so that the short ones fill the end of the
  // launch. Written at ingest, carried through compaction (a stable filter).
  int* ord[2];       // [W]
};

struct Layout {
  int W, n_max, m_max, d, dp, dh;
  int es;            // state element size in floats: 1 float32, 2 float64 (precise)
  int mat;           // materialised cost (no point records; Q below)
  int pad[2];        // npad, mpad
  int rbmax;         // max row blocks of either side
  int rows;          // rows per work item (kernel dependent)
  Bank bank[2];
  float* center;     // [W][d] (ingest only)
  int* vcnt;         // [W] column-check arrival counters
  int* nchk;         // [W] marginal evaluation passes spent on checks, per caller lane
  float* disc;       // [W] shadow mode: max |row screen - recomputed row residual|, per caller lane
  Audit* audit;      // [W]
  int* off[2];       // work item offsets per role [W + 1]
  Ctrl* ctrl;
  float* Q;          // materialised cost [W][pad0][pad1] by caller lane, base-2 units
  float* QT;         // its transpose [W][pad1][pad0]
  double2* agg64[2]; // guarded checks: per row block float64 partials [W][rbmax] (else null)
  float4* gerr[2];   // guarded release, float64 state: per caller lane and row block
                     // [W][rbmax] {sum of mass x export rounding, max export rounding,
                     // sum of mass, 0} of each side's potentials (else null)
  RowCert* row64;    // guarded release: [W] latest verified row residual by caller lane
  double* vpart;     // guarded checks: [W][rbmax][kVChunks][rows] per-row chunk sums (else null)
  int* vscnt;        // and their arrival words [W][rbmax], zero between launches
  int* vlist[2];     // guarded checks: the row blocks to verify per pass [W * rbmax]
  int* vlen;         // and their counts [2]
  double2* spart;    // float64 state: split-launch partials (see Launch::spart)
  float2* kpart;     // matrix-free large d: group partials (see Launch::kpart)
  int* scnt;         // split launches: arrival words [nslots]
  int nslots;        // work items the partials and counters hold
  int guard;
  size_t bytes;
};

// rows per work item of the float64-state kernel: two per lane, so that each
// column value read from LDS serves two terms. At d = 16 one row per lane left
// the sweep bound by those reads (605 against 535 ms per telemetry solve, at
// two waves per SIMD with a few spilled registers); four per lane measured
// slower at d = 3 (2087 against 1980 ms per LiDAR-shaped solve: lower
// occupancy, fewer work items in narrow launches) and at d = 16 (633 against
// 521 ms per telemetry solve: all 256 registers and more spills, half the
// work items per launch)
__host__ __device__ constexpr int rows_f64(int) { return 128; }

// work items of one lane-side: one per block of `rows` rows (all columns)
__host__ __device__ inline int row_blocks(int nrows, int rows) { return (nrows + rows - 1) / rows; }


// ------------------------------------------------------ kernel arguments
// One pass = one half-step (kind 0) or one marginal check (kind 1) over the
// slots of the current bank. A launch runs one or two passes.
struct Pass {
  const float* rec_row;   // [W][padr][dp]
  const float* rec_col;   // [W][padc][dp]
  const float* lm_row;    // [W][padr] log2 masses of the row side
  const float* lse_in;    // [W][padr] row lse of the input state
  float* lse_out;         // [W][padr] (update kind)
  float* gam_out;         // [W][padr] (update kind)
  const float* gam_col;   // [W][padc] column operand
  const float* w_row;     // caller masses of the row side, [W][w_ld] by lane id
  const int* off;         // [A + 1] first work item of each position of `ord` (ipl == 0)
  const int* ord;         // [A] slots in item order (see Bank::ord)
  float4* agg_out;        // [W][rbmax] this pass's row-block aggregates
  float4* gerr_out;       // update kind, guarded release with the float64 state: the
                          // export rounding of this side's potentials, by caller lane
  const float4* agg_bound;   // update: the column side's latest update aggregates
  const float4* agg_screen;  // column check: the f-half aggregates (row screen)
  const float4* agg_rowchk;  // final column check: the row-check aggregates
  int A, ipl;             // slots; uniform items per lane (0: use off)
  int nr, nc;             // uniform lane shapes (ipl > 0): rows and columns of every lane
  int padr, padc, w_ld;
  int role;               // 0: rows are x (f-half), 1: rows are y (g-half)
  int kind;               // 0: update, 1: check (marginal ratio of the input state)
  int verify_all;         // check: every live lane, else screen-positive lanes only
  int decide;             // role 1 check: take the retirement decision
  int final_audit;        // the decision is the max_iter audit
  int depth;              // depth of the audited state
};

struct Launch {
  Pass p[2];
  int nb0;                // blocks of pass 0; the rest belong to pass 1
  int dp, rbmax, mode, rows;
  float tau_screen, tol;
  SlotInfo* slot;
  Decision* dec;
  Audit* audit;
  int* vcnt;
  Ctrl* ctrl;
  HostSnap* hsnap;                // may be null
  int* nchk;                      // [W] check passes per caller lane
  float* disc;                    // [W] shadow mode: screen discrepancy per caller lane (else null)
  const float* Q;                 // materialised cost (caller lane l at Q + l * q_lane)
  const float* QT;                // and its transpose, the same size
  size_t q_lane;                  // floats per lane
  int q_ld;                       // row stride of Q (padded target count)
  int qt_ld;                      // row stride of QT (padded source count)
  int* progress;                  // &hsnap->progress as the device addresses it (may be null)
  int seqno;                      // launch sequence number written there
  double2* spart;                 // split float64 launch: group partials
                                  // [nslots][kGroups][rows]
  float2* kpart;                  // matrix-free large d: group partials [nslots][kGroups][rows]
  int* scnt;                      // and per item its arrival word [nslots], zero between launches
  int nslots;                     // items a launch of either kind may hold (both passes)
};

// Extra arguments of the float64 verification launch (guarded release), per
// pass (p[0] of its Launch: row marginal, rows = x; p[1]: column marginal).
struct GuardArgs {
  const float* w_col[2]; int w_ld_col[2];   // the column side's caller masses
  const float* xy_row[2];                   // caller coordinates of the row side
  const float* xy_col[2];                   // and of the column side, by lane id
  int ld_row[2], ld_col[2];                 // their point strides (n_max / m_max)
  double2* agg64[2];      // [W][rbmax] per row block {sum |marginal - mass|, non-finite}
  const float4* gerr[2];  // export rounding per side (float64 state), see Layout::gerr
  RowCert* row64;         // [W] row residual of the audit, read by its column check
  double* vpart;          // [W][rbmax][kVChunks][rows] per-row chunk sums of a launch
  int* vscnt;             // [W][rbmax] their arrival words (zero between launches)
  int* vlist[2];          // per pass: the items to verify, slot * rbmax + row block
                          // (bit 30: the outward bound had excluded the lane)
  int* vlen;              // [2] the lists' lengths
  const float* eps;       // caller eps [W]
  int d, es;              // point dimension; state element size in floats
  int bound;              // 1: gate the row check by the outward bound (float64
                          // state); 0: verify every audited lane
};

struct ScanArgs {          // compaction map over the slots of the current bank
  SlotInfo* slot;
  Decision* dec;
  int* off_f;             // [W + 1] rewritten for the new layout
  int* off_g;
  const int* ord_src[2];  // item order of the current bank, per role
  int* ord_dst[2];        // and of the other bank (the survivors, order kept)
  Ctrl* ctrl;
  HostSnap* hsnap;
  int A, W, compact, rows, epoch;
};

struct MoveArgs {
  Bank src, dst;
  const Ctrl* ctrl;       // compaction: iterate the slots of the width before the map
  int A, dp, compact, emit_all, mode;
  int pad[2];
  int es;                 // state element size in floats (1 or 2)
  int rbmax;              // row-block aggregates per slot
  int n_max, m_max;
  int final_par;          // parity of the final state (static mode emission)
  int chunk;              // points per block per side
  const Audit* audit;     // static mode: residuals of the final state
  // outputs (caller order)
  float* f; float* g; int* depth; float* residual; float* row_res; float* col_res;
  int* status;
};

struct IngestArgs {
  const float* X; const float* Y; const float* a; const float* b; const float* eps;
  const float* g0;        // proposal g^0 [W][m_max] (null: cold start)
  const int* n; const int* m;
  int W, n_max, m_max, d, dp, dh;
  int pad[2];
  int precise;            // float64 state
  int mat;                // materialised cost: no records, cold start gam^y = 0
  Bank bank;
  float* center;
  int* vcnt;
  int* nchk;
  float* disc;
  RowCert* row64;        // guarded release: cleared (depth 0 matches no audit)
  int rbmax;
  Ctrl* ctrl;
};

// Update kernel variants: how a launch spreads (row tile, column group) work
// over waves. All variants compute identical bits; the host picks one by width.
enum { VAR_NARROW = 0,   // 32-row items, one group per wave (8 waves)
       VAR_MEDIUM = 1,   // 32-row items, two groups per wave (4 waves)
       VAR_MEDIUM4 = 3,  // 32-row items, four groups per wave (2 waves): matrix-core
                         // kernel, lanes of at most 2 column tiles per group
       VAR_SPLIT = 4 };  // float64 kernel: a block per (item, group), a wave per sub-group, at most
                         // kSplitItems items per pass
// e0 / e1 (may be null): events that record the kernel's own start and end
hipError_t launch_update(const Launch& a, int d, bool use_mfma, int variant, int blocks,
                         hipStream_t st, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_update_f64(const Launch& a, int d, int variant, int blocks, hipStream_t st,
                             hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// matrix-free matrix-core half-step for any d (tiled contraction), `blocks`
// work items over both passes
hipError_t launch_update_mfma_k(const Launch& a, int blocks, hipStream_t st,
                                hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_update_mat(const Launch& a, int blocks, hipStream_t st, hipEvent_t e0 = nullptr,
                             hipEvent_t e1 = nullptr);

// Q_ij = kappa_t ||x_i - y_j||^2 for every lane (one launch, before the first cycle)
struct CostArgs {
  const float* X; const float* Y;
  const float* center;
  const SlotInfo* slot;   // ingest layout: slot t = caller lane t
  float* Q;               // [W][pad0][pad1]
  float* QT;              // [W][pad1][pad0] its transpose
  int W, n_max, m_max, d, pad0, pad1;
};
hipError_t launch_cost(const CostArgs& a, hipStream_t st);
// float64 two-sided check of the audited state (both marginals, two passes)
hipError_t launch_vgate(const Launch& a, const GuardArgs& g, hipStream_t st);
hipError_t launch_verify64(const Launch& a, const GuardArgs& g, int items, hipStream_t st);
hipError_t launch_scan(const ScanArgs& a, hipStream_t st);
hipError_t launch_offsets(SlotInfo* slot, int A, int rows, int* off_f, int* off_g, int* ord_f,
                          int* ord_g, Ctrl* ctrl, hipStream_t st);
hipError_t launch_move(const MoveArgs& a, int A, int maxpad, hipStream_t st);
hipError_t launch_ingest(const IngestArgs& a, int maxpad, hipStream_t st);
hipError_t launch_order(const int* depth, int W, int* order, hipStream_t st);
hipError_t launch_zero_counters(int* vcnt, int W, hipStream_t st);
// Device address and size of this device's allocation-free workspace (the
// address is taken once per device, with that device current).
hipError_t scratch_area(void** ptr, size_t* bytes);

}  // namespace ds
