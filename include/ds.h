/*
 * ds.h -- C ABI of the MI355X (gfx950) active-set batched Sinkhorn library.
 *
 * One call solves a window of W independent entropic optimal-transport
 * problems ("lanes") by log-domain Sinkhorn scaling over a candidate axis,
 * screens each lane's non-current marginal after every audited cycle, checks
 * screen-positive lanes with the two-sided L1 stopping rule, and physically
 * compacts passing lanes out of every lane-indexed tensor so later updates run
 * at the width of the unfinished set (DrainSinkhorn, arxiv 2607.24741, Sec. 3).
 *
 * Problem (eq:eot, Sec. 2), per lane t with points x_i (i < n_t), y_j (j < m_t):
 *     min_pi <C, pi> + eps_t sum_ij pi_ij (log pi_ij - 1),  pi 1 = a,  pi^T 1 = b,
 *     C_ij = ||x_i - y_j||^2.
 * The outputs are the dual potentials (f, g) of the convention
 *     pi_ij = exp((f_i + g_j - C_ij) / eps_t),
 * reached by the cycle of eq:sinkhorn-cycle (f-half first) from the cold start
 * f = g = 0, which fixes the gauge (f + c, g - c) of Sec. 4.2.
 *
 * One iteration = one full cycle = one candidate-update slot (Sec. 3.1, 4.1).
 * A lane's completion depth l_t is the first audit at which
 *     r = max(||pi 1 - a||_1, ||pi^T 1 - b||_1) <= tol   (eq:release-contract)
 * holds; audits run after cycle k when k % audit_every == 0 and at max_iter.
 *
 * Conventions for every entry point:
 *   - Array pointers inside ds_problem / ds_result are DEVICE pointers (fp32 or
 *     int32, C-contiguous, lane-major). ds_stats and its width_trace are HOST.
 *   - The caller owns all memory. Inputs are never written. ds_solve performs no
 *     device allocation: all scratch lives in the caller's workspace.
 *   - All device work is enqueued on the caller's stream (a hipStream_t passed
 *     as void*; NULL = the null stream). ds_solve returns after the outputs are
 *     complete (it synchronises that stream). Distinct workspaces may be used
 *     concurrently from different host threads; one workspace must not be
 *     shared by overlapping calls.
 *   - Errors: every entry point returns ds_err. Problems detectable on the host
 *     (null required pointer, non-positive sizes, tol <= 0, max_iter < 1,
 *     audit_every < 1, unknown mode, d > 512, W > 4096, workspace too small)
 *     return before any device work with the outputs untouched. Lane sizes and
 *     eps are validated on the device before the first update: a bad lane makes
 *     the call return DS_E_INVALID (outputs undefined) and
 *     ds_last_error_message() names the first bad lane. A HIP failure returns
 *     DS_E_HIP. Numerical trouble inside one lane is not a call error: it is
 *     reported through that lane's status.
 */
#ifndef DRAINSINKHORN_DS_H
#define DRAINSINKHORN_DS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DS_API_VERSION 4

typedef enum {
  DS_OK = 0,
  DS_E_INVALID = 1,     /* bad argument or bad lane data (see message)          */
  DS_E_WORKSPACE = 2,   /* workspace pointer NULL / misaligned / too small        */
  DS_E_HIP = 3,         /* a HIP runtime call or kernel launch failed             */
  DS_E_UNSUPPORTED = 4, /* valid request outside the implemented envelope         */
  DS_E_INTERNAL = 5
} ds_err;

/* Execution modes (Sec. 3.3). Width-one execution is a call with W = 1. */
typedef enum {
  DS_MODE_ACTIVE = 0,  /* verifier-gated retirement + physical compaction        */
  DS_MODE_STATIC = 1,  /* every lane updated at width W until all have passed;
                          returns each lane's state at that common boundary and
                          its first passing depth                               */
  DS_MODE_LOGICAL = 2  /* passing lanes frozen in place, kernels keep width W    */
} ds_mode;

typedef enum {
  DS_LANE_CONVERGED = 0, /* passed the two-sided check at depth l_t              */
  DS_LANE_MAX_ITER = 1,  /* still failing at max_iter; state of cycle max_iter   */
  DS_LANE_NONFINITE = 2  /* non-finite residual at an audit; residual = NaN      */
} ds_lane_status;

enum {
  DS_F_SHADOW = 1u,     /* shadow replay: also run the full check on screen-
                           negative lanes and count already-releasable lanes the
                           screen missed, and recompute the row marginal of every
                           audited state by a dedicated pass, reporting its largest
                           distance from the fused screen (ds_stats)            */
  DS_F_TIMING = 2u,     /* time the update launches of every 32nd cycle with HIP
                           events in their dispatches (ds_stats)                 */
  DS_F_FORCE_VALU = 4u, /* float32 state on the vector-ALU update kernels (d <= 16) */
  DS_F_FORCE_MFMA = 8u, /* float32 state on the matrix-core update kernels
                           (d <= 32; the default for 16 < d <= 32)             */
  DS_F_PRECISE = 16u,   /* float64 state and exponent arguments (d <= 16). This
                           is the default for d <= 16 unless DS_F_FAST32 or a
                           FORCE flag is given; the flag is kept so a caller can
                           require it (an error where it is unavailable). The
                           outputs stay float32.                                */
  DS_F_MATERIALIZE = 32u, /* build the cost C (base-2 units, float32) and its
                           transpose once per call in the workspace and stream
                           them from HBM by rows in every half-step; the default
                           for d > 32 when n_max, m_max <= 16384 (required here;
                           2 W n_pad m_pad 4 bytes of workspace)                 */
  DS_F_GUARD = 64u,     /* guarded release (eq:release-contract in float64): the
                           release is decided on a float64 evaluation of both
                           marginals of exactly the float32 potentials the caller
                           will receive (cost formed in float64 from the caller's
                           coordinates), and that residual is the one reported.
                           With the float64 state an outward bound on how far the
                           rounding to float32 outputs and the screen's own
                           arithmetic move the row residual (from the per-lane
                           rounding sums, eps and the lane's masses) selects the
                           lanes to verify: only those that could meet tol. With
                           a float32 state every audited lane is verified. The
                           column marginal is evaluated only for lanes whose row
                           residual met tol. Three extra launches per audit cycle;
                           the workspace grows by about 8 KB per 128-row block
                           and lane with the float64 state (2 KB per 32-row
                           block with a float32 state) for the verification's
                           per-row chunk sums; n_max, m_max <= 16384.            */
  DS_F_MATRIX_FREE = 256u, /* d > 32: recompute the cost per tile on the matrix
                           cores (an LDS-tiled contraction over d) instead of
                           materialising it; the default when a side has more
                           than 16384 points. Float32 state. Exclusive with
                           DS_F_MATERIALIZE.                                     */
  DS_F_FAST32 = 128u    /* float32 state on the matrix-core kernels for d <= 16:
                           about 1.5-2.5x faster, but float32 rounding of the
                           scaled coordinates and potentials (exponents of size
                           C/eps) moves residuals by 1e-6..1e-5, so completion
                           depths of lanes within that distance of tol can
                           differ by a cycle from the float64 trajectory's      */
};

/* One window of W lanes. Device pointers. */
typedef struct {
  int32_t W;            /* lanes, 1..4096                                          */
  int32_t n_max, m_max; /* padded point counts per lane (>= 1)                     */
  int32_t d;            /* point dimension, 1..512                                 */
  const float* X;       /* [W, n_max, d] source points                             */
  const float* Y;       /* [W, m_max, d] target points                             */
  const float* a;       /* [W, n_max] source masses, > 0 on the valid prefix       */
  const float* b;       /* [W, m_max] target masses, > 0 on the valid prefix       */
  const float* eps;     /* [W] entropic regularisation, finite and > 0             */
  const int32_t* n;     /* [W] valid prefix sizes 1..n_max; NULL => all n_max      */
  const int32_t* m;     /* [W] valid prefix sizes 1..m_max; NULL => all m_max      */
  const float* g0;      /* [W, m_max] proposal: initial target potential g^0 in the
                           output convention (a warm start or a carried solution,
                           Sec. 2); NULL => the cold proposal g^0 = 0. f is updated
                           first, so a proposal's source potential never enters
                           the trajectory. A non-finite entry on a live point
                           makes that lane NONFINITE at its first audit.        */
} ds_problem;
/* Points beyond a lane's prefix are never read. A zero mass on the valid prefix
 * removes that point from the problem (its output potential is 0). A negative
 * or non-finite mass or coordinate makes that lane NONFINITE at its first audit. */

typedef struct {
  float tol;           /* two-sided stopping tolerance tau_stop, > 0              */
  float screen_tol;    /* one-sided screen threshold tau_screen; <= 0 => tol      */
  int32_t max_iter;    /* cycles, >= 1                                            */
  int32_t audit_every; /* audit grid spacing in cycles, >= 1                      */
  int32_t mode;        /* ds_mode                                                 */
  uint32_t flags;      /* DS_F_*                                                  */
  int32_t streams;     /* concurrent sub-batches, 0..4; 0 => automatic (see below) */
} ds_options;
/* Sub-batches (active mode only). The window is cut into `streams` contiguous
 * lane ranges, each solved with its own control loop, workspace part and HIP
 * stream (the first on the caller's stream, the others on streams of the
 * library that start behind the work already queued on the caller's stream
 * and that the caller's stream waits for before the call returns). Lanes are
 * independent, so every output is bit-identical to the one-batch solve; the
 * launch latencies of one sub-batch overlap the work of the others. Automatic:
 * one sub-batch below 32 lanes, in the static and logical modes (they share
 * one final cycle across the window) and with the materialised cost;
 * otherwise two. ds_workspace_bytes accounts for the split. */

/* Outputs, in caller lane order. Device pointers. */
typedef struct {
  float* f;            /* [W, n_max]; entries past the prefix / zero-mass: 0      */
  float* g;            /* [W, m_max]; same                                        */
  int32_t* depth;      /* [W] l_t in cycles                                       */
  float* residual;     /* [W] max(row, col) L1 residual of the returned state     */
  float* row_residual; /* [W] may be NULL                                          */
  float* col_residual; /* [W] may be NULL                                          */
  int32_t* status;     /* [W] ds_lane_status                                      */
  int32_t* order;      /* [W] lane ids in completion order (depth, then lane id);
                          may be NULL                                              */
} ds_result;

/* Host-side accounting of one solve (all counts exact). */
typedef struct {
  int64_t slots_update;       /* sum over cycles of lanes that ran both halves:
                                 sum_t l_t (active), W * l_max (static, logical)  */
  int64_t halfsteps_executed; /* lane-half-steps launched, incl. the discarded
                                 f-half of each retired lane                       */
  int64_t pair_evals;         /* (i, j) terms of the kept half-steps:
                                 2 sum_t l_t n_t m_t (active), 2 l_max sum_t n_t m_t
                                 (static, logical); speculative halves excluded    */
  int64_t check_pair_evals;   /* (i, j) terms of the two-sided checks: one marginal
                                 pass per ordinary check, two at the final audit  */
  int64_t bytes_compacted;    /* bytes moved by survivor gathers                    */
  int32_t l_max, cycles, audits, screen_positive, check_failures, compactions;
  int32_t missed_ready;       /* DS_F_SHADOW only                                   */
  int32_t update_launches;    /* DS_F_TIMING: number of timed (sampled) launches     */
  double ms_total;            /* wall time of the call (host clock)                 */
  double ms_update;           /* DS_F_TIMING: summed duration of the timed launches
                                 (both launches of every 32nd cycle of every
                                 sub-batch, and the final audit), from HIP events
                                 in each launch's own dispatch                      */
  int64_t timed_pair_evals;   /* DS_F_TIMING: algorithmic (i, j) terms of those
                                 launches (lanes running at that cycle; the checks
                                 sharing a g-launch are not counted)               */
  double ms_check;            /* reserved (checks share the g-half launches)         */
  double ms_compact;          /* DS_F_TIMING: compaction (scan + gather) launches     */
  int32_t* width_trace;       /* optional HOST buffer: A_k for k = 1..             */
  int32_t width_trace_len;    /* capacity in; entries written out                  */
  size_t workspace_bytes;     /* bytes of workspace the call used                   */
  int32_t sub_batches;        /* concurrent sub-batches the call ran (see streams)  */
  double screen_discrepancy;  /* DS_F_SHADOW: max over lanes and audits of
                                 |row screen - row residual recomputed by a full
                                 pass over (i, j) at the audited state|, over the
                                 audits where either is at most 2 tol (where a
                                 release can be decided)                          */
  int32_t guard_missed;       /* DS_F_GUARD | DS_F_SHADOW: audits at which the
                                 outward bound excluded a lane whose verified row
                                 residual met tol (0 when the bound holds)         */
} ds_stats;

/* Version of this header the library was built from (DS_API_VERSION). */
int ds_api_version(void);

/* Workspace bytes ds_solve needs for this problem shape and options. Only the
 * scalar fields of `problem` are read (no pointer is dereferenced). */
ds_err ds_workspace_bytes(const ds_problem* problem, const ds_options* options,
                          size_t* bytes);

/* Solve one window (the whole hot path: ingest, packed f/g updates, fused row
 * screen, two-sided verifier, retirement and compaction, output emission).
 * `workspace` is a device buffer of at least ds_workspace_bytes() bytes,
 * 256-byte aligned, owned by the caller; its contents need no initialisation.
 * `stream` is a hipStream_t (void* here so this header needs no HIP include).
 * `stats` may be NULL. */
ds_err ds_solve(const ds_problem* problem, const ds_options* options,
                const ds_result* result, void* workspace, size_t workspace_bytes,
                void* stream, ds_stats* stats);

/* ds_solve for callers that cannot allocate (code under stream capture, tight
 * serving loops, harnesses that forbid allocation): the same solve, with the
 * workspace taken from a fixed device array the library holds on every GPU it
 * runs on (64 MiB per GPU, kept until the process ends) instead of a caller
 * buffer. The caller still passes inputs and outputs; the call performs no
 * device or pinned-memory allocation, except that the first call on a device
 * sets that device up once (it looks up the array's address and creates the
 * library's per-device host resources: a pinned control snapshot, an event
 * and a stream). It runs one sub-batch on `stream` (options->streams must be
 * 0 or 1) and rejects DS_F_TIMING (DS_E_INVALID). A problem whose workspace
 * (ds_workspace_bytes with streams = 1) exceeds the array returns
 * DS_E_UNSUPPORTED before any device work, with the sizes in
 * ds_last_error_message(). All calls on one GPU share that GPU's array, whose
 * contents persist from the previous call (the solve initialises everything
 * it reads): calls that overlap on one GPU race, so a caller must not issue
 * two at once on the same device (from two host threads or two streams). */
ds_err ds_solve_noalloc(const ds_problem* problem, const ds_options* options,
                        const ds_result* result, void* stream, ds_stats* stats);

/* Static string for an error code. */
const char* ds_error_string(ds_err err);

/* Detail of the last non-OK return on this host thread ("" if none). */
const char* ds_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* DRAINSINKHORN_DS_H */
