// gfx950 kernels of the active-set batched Sinkhorn path (wave64, CDNA4).
//
//  k_update_f64<D, GW>
//                     one half-step of eq:sinkhorn-cycle for every (slot, row
//                     block) work item with the state in float64: every
//                     exponent formed in float64 on the vector ALU (d fused
//                     multiply-adds and an add) and rounded once to float32
//                     for v_exp_f32, column data staged in LDS and broadcast,
//                     two rows per lane up to d = 12, streaming base-2
//                     log-sum-exp over 8 fixed column groups of 4 fixed
//                     sub-groups each, fused row screen; with a second pass in
//                     the same launch, the column check and release decision
//                     (the default path for d <= 16).
//  k_update_f64_split<D>
//                     the same half-step for narrow launches: one block per
//                     (work item, column group), one wave per sub-group, the
//                     group partials merged by the item's last block (the
//                     same bits).
//  k_update_mfma<DH, RT, GW, UNI>
//                     the same half-step with the state in float32: x~.y~ on
//                     the fp32 matrix cores (v_mfma_f32_32x32x2_f32) with the
//                     column potential and the row anchor folded into the
//                     contraction (DS_F_FAST32 for d <= 16; the default for
//                     16 < d <= 32).
//  k_update_valu<D>   the float32 half-step on the vector ALU, column data
//                     wave-uniform (scalar loads, SGPR operands); on request.
//  k_update_mfma_k<UNI>
//                     the float32 matrix-core half-step for any d: a tiled
//                     contraction (128 x 128 block tiles, operands staged in
//                     LDS) with the streaming sum as its epilogue, one block
//                     per (work item, column group) (d > 32 without a
//                     materialised cost).
//  k_cost, k_mat_rows
//                     the materialised cost: built once on the matrix cores
//                     (with its transpose), then streamed by rows from HBM by
//                     both half-steps (the default for d > 32 up to 16384
//                     points a side).
//  k_vgate, k_verify64<DR>
//                     float64 verification of the exported potentials (guarded
//                     release): the lanes the outward bound admits, then their
//                     row and column marginals over (row block, column chunk)
//                     units.
//  k_offsets, k_scan  one block: the work item order and offsets of the
//                     initial layout (longest sweeps first); the compaction
//                     map (survivor ranks, the orders filtered, new offsets)
//                     from the device-side decisions (Sec. 3.2).
//  k_move             retiree emission in caller lane order + survivor gather
//                     into the other bank (physical compaction, Sec. 3.2).
//  k_ingest_*         validation, centring/scaling, log masses, proposals.
//  scratch            the fixed per-GPU workspace of ds_solve_noalloc.
//
// Determinism: every reduction runs in a fixed order (no float atomics); the
// column groups and tile order of a lane depend only on its (n, m), so a lane's
// bits do not depend on the batch width, the launch layout, its slot or its
// co-lanes.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "ds_internal.h"

namespace ds {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// Cross-block hand-off inside one launch. The per-XCD L2 caches are not
// coherent with each other, and an agent-scope release/acquire fence writes
// back and invalidates the whole L2 -- far too costly per work item. Data that
// another block of the same launch reads is therefore written and read with
// relaxed device-scope atomics (coherent, write-through), and ordered against
// the arrival counter by waiting for the stores to complete.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_dev(const int* p) {
  return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev2(float2* p, float2 v) {
  unsigned long long bits = (unsigned long long)__float_as_uint(v.x) |
                            ((unsigned long long)__float_as_uint(v.y) << 32);
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), bits, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_dev2(const float2* p) {
  unsigned long long bits = __hip_atomic_load(
      reinterpret_cast<unsigned long long*>(const_cast<float2*>(p)), __ATOMIC_RELAXED,
      __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((unsigned)bits), __uint_as_float((unsigned)(bits >> 32)));
}
// Arrival of one block of a work item split over `blocks` blocks (kGroups by
// default), by one wave, after its partials (or nothing, without work) were
// stored: one atomic on the item's word, arrivals in its low 16 bits and blocks
// without work counted above them. True for the last block to arrive, which
// clears the word for the next launch (a plain device-scope store: nothing
// reads it again before this launch ends); `skipped` says whether any block of
// the item had no work.
__device__ __forceinline__ bool arrive_last(int* word, bool work, bool& skipped,
                                            int blocks = kGroups) {
  __builtin_amdgcn_s_waitcnt(0);   // the partial stores are complete before the arrival counts
  int prev = 0;
  if ((threadIdx.x & 63) == 0) prev = atomicAdd(word, work ? 1 : 1 + (1 << 16));
  prev = __builtin_amdgcn_readfirstlane(prev);
  const bool last = (prev & 0xFFFF) + 1 == blocks;
  skipped = (prev >> 16) != 0 || !work;
  if (last && (threadIdx.x & 63) == 0)
    __hip_atomic_store(word, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return last;
}

// best-effort publication to pinned host memory (system scope, write-through)
__device__ __forceinline__ void st_sys(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
// Block 0 of an update launch publishes the launch's sequence number to the
// host before anything else: every earlier launch of the stream has completed.
// A plain int store (the snapshot is uncached, coherent host memory): type-based
// alias analysis then keeps the float operand loads that follow it on the
// scalar path, which an atomic store would forbid.
__device__ __forceinline__ void note_progress(const Launch& L) {
  if (blockIdx.x == 0 && threadIdx.x == 0 && L.progress) *L.progress = L.seqno;
}
// all of this wave's outstanding memory operations have completed
__device__ __forceinline__ void wait_mem() { __builtin_amdgcn_s_waitcnt(0); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }

enum { KIND_UPDATE = 0, KIND_VERIFY = 1 };
enum { MODE_ACTIVE = 0, MODE_STATIC = 1, MODE_LOGICAL = 2 };

// --------------------------------------------------------- work item lookup
// The position q < A in a role's item order whose work items hold item b
// (off[q] <= b < off[q + 1]; every lane has at least one item).
__device__ __forceinline__ int find_slot(const int* off, int A, int b) {
  int lo = 0, hi = A;
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (off[mid] <= b) lo = mid; else hi = mid;
  }
  return lo;
}

// ---------------------------------------------------------- wave reductions
// Fixed trees with the same bits in every lane: inside each row of 16 lanes by
// DPP (neighbour pairs, quad pairs, mirrored halves of 8, mirrored halves of
// 16), then across the rows through lane reads, in the order (r0, r1), (r2, r3).
// Every step combines two lanes that already hold equal values on both sides
// of a commutative operation, so no lane can end up with different bits.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float rdlane(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
struct OpAdd { __device__ float operator()(float a, float b) const { return a + b; } };
struct OpMin { __device__ float operator()(float a, float b) const { return fminf(a, b); } };
struct OpMax { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };
template <class Op>
__device__ __forceinline__ float row16(float v, Op op) {
  v = op(v, dpp<0xB1>(v));   // lane ^ 1
  v = op(v, dpp<0x4E>(v));   // lane ^ 2
  v = op(v, dpp<0x141>(v));  // the other quad of the 8
  v = op(v, dpp<0x140>(v));  // the other 8 of the row
  return v;
}
// result of rows (2u, 2u+1), i.e. of lanes [32u, 32u + 32)
template <class Op>
__device__ __forceinline__ float half32(float v16, int u, Op op) {
  return op(rdlane(v16, 32 * u), rdlane(v16, 32 * u + 16));
}
template <class Op>
__device__ __forceinline__ float wave64(float v, Op op) {
  const float r = row16(v, op);
  return op(half32(r, 0, op), half32(r, 1, op));
}

__device__ __forceinline__ void st_dev4(float4* p, float4 v) {
  st_dev(&p->x, v.x); st_dev(&p->y, v.y); st_dev(&p->z, v.z); st_dev(&p->w, v.w);
}
__device__ __forceinline__ float4 ld_dev4(const float4* p) {
  return make_float4(ld_dev(&p->x), ld_dev(&p->y), ld_dev(&p->z), ld_dev(&p->w));
}

// ----------------------------------------------------------- retirement
// Record the decision for slot s and take the lane out of the active set.
// Static mode keeps a passed lane running to the common final boundary.
__device__ void retire_lane(const Launch& L, const Pass& P, int s, const SlotInfo& si, int status,
                            float rrow, float rcol) {
  Decision d;
  d.status = status;
  d.depth = P.depth;
  d.res_row = rrow;
  d.res_col = rcol;
  d.new_slot = -1;
  d.pad[0] = d.pad[1] = d.pad[2] = 0;
  L.dec[s] = d;
  if (L.mode == MODE_STATIC && !P.final_audit) L.slot[s].passed = 1;
  else L.slot[s].done = 1;
  const int rf = row_blocks(si.n, L.rows), rg = row_blocks(si.m, L.rows);
  const int nret = atomicAdd(&L.ctrl->n_retired, 1) + 1;
  const int itf = atomicSub(&L.ctrl->items_act_f, rf) - rf;
  const int itg = atomicSub(&L.ctrl->items_act_g, rg) - rg;
  if (!P.final_audit) atomicAdd(&L.ctrl->retire_events, 1);
  const int prev = atomicSub(&L.ctrl->n_active, 1);
  if (prev == 1) {
    L.ctrl->final_cycle = P.depth;
    atomicExch(&L.ctrl->finished, 1);
  }
  // host-visible snapshot: every field only moves one way, so a stale or
  // reordered value is still a valid bound for the host's decisions
  if (L.hsnap) {
    st_sys(&L.hsnap->n_retired, nret);
    st_sys(&L.hsnap->items_act_f, itf);
    st_sys(&L.hsnap->items_act_g, itg);
    st_sys(&L.hsnap->n_active, prev - 1);
    if (prev == 1) st_sys(&L.hsnap->finished, 1);
  }
}

// -------------------------------------------------- lane-level aggregates
// Fixed-order reduction (by one wave) of the row-block aggregates of slot s
// {sum, min, max, non-finite flag}; every lane of the wave returns the same bits.
struct LaneAgg {
  float sum, dmin, dmax;
  int bad;
};
__device__ __forceinline__ LaneAgg lane_aggregate(const float4* agg, int s, int rbmax, int nrb,
                                                  bool coherent) {
  LaneAgg g;
  float t0 = 0.f, t1 = INFINITY, t2 = -INFINITY, t3 = 0.f;
  const float4* base = agg + (size_t)s * rbmax;
  for (int q = (int)(threadIdx.x & 63); q < nrb; q += 64) {
    const float4 v = coherent ? ld_dev4(base + q) : base[q];
    t0 += v.x;
    t1 = fminf(t1, v.y);
    t2 = fmaxf(t2, v.z);
    t3 = fmaxf(t3, v.w != 0.f ? 1.f : 0.f);
  }
  g.sum = wave64(t0, OpAdd());
  g.dmin = wave64(t1, OpMin());
  g.dmax = wave64(t2, OpMax());
  g.bad = wave64(t3, OpMax()) != 0.f;
  return g;
}

// Lane facts every wave reduces itself (same bits in every wave), so no LDS
// broadcast or barrier sits between the block's loads and its sweep.
//
// Update: lse_new - lse_old lies in [min_j dgam_j, max_j dgam_j], dgam being
// the latest change of the column operand (= -(change of the column lse)), so
// anchored (max-free) sums are safe when that spread is small; M = -min dgam.
//
// Two wave reductions instead of three: a block with a non-finite change
// enters the maximum as +inf, which fails the spread test exactly as the
// separate flag did (inf - dmin is +inf or NaN).
__device__ __forceinline__ void update_facts(const Launch& L, const Pass& P, int s, int ncols,
                                             bool& fast, float& M, float range = kFastRange) {
  float t1 = INFINITY, t2 = -INFINITY;
  const float4* base = P.agg_bound + (size_t)s * L.rbmax;
  const int nrb = row_blocks(ncols, L.rows);
  for (int q = (int)(threadIdx.x & 63); q < nrb; q += 64) {
    const float4 v = base[q];
    t1 = fminf(t1, v.y);
    t2 = fmaxf(t2, v.w != 0.f ? INFINITY : v.z);
  }
  const float dmin = wave64(t1, OpMin()), dmax = wave64(t2, OpMax());
  fast = dmin <= dmax && (dmax - dmin) <= range;
  M = -dmin;
}
// Check: whether this lane is checked at all (screen-positive, non-finite
// screen, or every lane), and the row screen of the audited state (n_x: the
// lane's source points, whose row blocks carry the screen).
__device__ __forceinline__ bool check_facts(const Launch& L, const Pass& P, int s, int n_x,
                                            float& rhat) {
  rhat = NAN;
  if (P.role == 1 && !P.final_audit) {
    const LaneAgg g = lane_aggregate(P.agg_screen, s, L.rbmax, row_blocks(n_x, L.rows), false);
    rhat = g.sum;
    return P.verify_all || !isfinite(g.sum) || g.sum <= L.tau_screen;
  }
  return true;
}

// ----------------------------------------------------------- item epilogue
// Finish of one work item by wave 0 alone, after the column groups were merged.
// Lane l owns rows rb0 * UNIT + 64 r + l (r < R) when `owner[r]` (merged
// (Mt, St) of that row; R > 1 only with one aggregate per item, UNIT = 64 R).
// Writes the new lse / gam (update kind), one aggregate per UNIT-row block
// (NU of them), and -- for the deciding column check -- takes the lane's
// retirement decision in the last arriving item of the lane. `gam_keep`, when
// given, receives the new column operand of each live owned row (update kind).
__device__ __forceinline__ float log2_t(float x) { return lg2(x); }
__device__ __forceinline__ double log2_t(double x) { return log2(x); }
__device__ __forceinline__ float exp2_t(float x) { return ex2(x); }
__device__ __forceinline__ double exp2_t(double x) { return exp2(x); }

template <int UNIT, int NU, int R, typename T>
__device__ void finish_rows_r(const Launch& L, const Pass& P, int s, const SlotInfo& si, int rb0,
                              const bool (&owner)[R], const bool (&live)[R], bool fast, float Mf,
                              const T (&lse_old)[R], const T (&lm)[R], const float (&w)[R],
                              const T (&Mt)[R], const T (&St)[R], float rhat,
                              T* gam_keep = nullptr) {
  static_assert(UNIT * NU <= 64 * R, "one wave owns the rows of an item");
  static_assert(R == 1 || (NU == 1 && UNIT == 64 * R), "several rows per lane: one aggregate");
  const int lane = threadIdx.x & 63;
  const int nrows = P.role ? si.m : si.n;
  const int nrb = row_blocks(nrows, UNIT);
  const bool frozen = (L.mode == MODE_LOGICAL) && si.done;
  const T M = (T)Mf;
  float rho = 0.f, dmin = INFINITY, dmax = -INFINITY, bad = 0.f;
  T lse_new[R], gam_new[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    lse_new[r] = (T)INFINITY;
    gam_new[r] = -(T)INFINITY;
    if (!owner[r]) continue;
    if (P.kind == KIND_UPDATE) {
      if (live[r]) {
        const T anchor = fast ? lse_old[r] + M : (T)0;   // the sweep's row anchor
        lse_new[r] = anchor + (Mt[r] + log2_t(St[r]));
        gam_new[r] = lm[r] - lse_new[r];
        if (gam_keep) gam_keep[r] = gam_new[r];
        const float dl = (float)(lse_new[r] - lse_old[r]);
        if (isfinite(dl)) { dmin = fminf(dmin, dl); dmax = fmaxf(dmax, dl); } else { bad = 1.f; }
        if (P.role == 0) {
          // R_i / a_i of the input state = 2^(lse_new - lse_old), formed so the
          // large terms cancel exactly before rounding
          const T ratio = fast ? St[r] * exp2_t(anchor - lse_old[r])
                               : St[r] * exp2_t(Mt[r] - lse_old[r]);
          rho += w[r] * fabsf((float)(ratio - (T)1));
        }
      }
    } else if (live[r]) {
      // check: terms were pi_ij / 2^lm_i, so St * 2^Mt = R_i / a_i
      const T ratio = St[r] * exp2_t(Mt[r]);
      rho += w[r] * fabsf((float)(ratio - (T)1));
    }
  }
  // one aggregate per UNIT-row block: {sum rho, min, max of the lse change, bad}
  const float r0 = row16(rho, OpAdd()), r1 = row16(dmin, OpMin());
  const float r2 = row16(dmax, OpMax()), r3 = row16(bad, OpMax());
  float4 ag[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    if (UNIT == 32) {
      ag[u] = make_float4(half32(r0, u, OpAdd()), half32(r1, u, OpMin()),
                          half32(r2, u, OpMax()), half32(r3, u, OpMax()));
    } else {
      ag[u] = make_float4(OpAdd()(half32(r0, 0, OpAdd()), half32(r0, 1, OpAdd())),
                          OpMin()(half32(r1, 0, OpMin()), half32(r1, 1, OpMin())),
                          OpMax()(half32(r2, 0, OpMax()), half32(r2, 1, OpMax())),
                          OpMax()(half32(r3, 0, OpMax()), half32(r3, 1, OpMax())));
    }
  }
  const int nu = min(NU, nrb - rb0);
  float4* dst = P.agg_out + (size_t)s * L.rbmax + rb0;
  const bool deciding = P.kind == KIND_VERIFY && P.role == 1 && P.decide;
  if (!deciding) {
    if (lane == 0)
      for (int u = 0; u < nu; ++u) dst[u] = ag[u];
    // the new state goes out last: nothing after it reuses its registers, so
    // the wave ends without waiting for the stores
    if (P.kind == KIND_UPDATE && !frozen) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (!owner[r]) continue;
        const size_t idx = (size_t)s * P.padr + rb0 * UNIT + 64 * r + lane;
        reinterpret_cast<T*>(P.lse_out)[idx] = lse_new[r];
        reinterpret_cast<T*>(P.gam_out)[idx] = gam_new[r];
      }
    }
    return;
  }
  // publish the column-check partials, then count this item's blocks in
  int last = 0;
  if (lane == 0) {
    for (int u = 0; u < nu; ++u) st_dev4(dst + u, ag[u]);
    wait_mem();
    const int prev = atomicAdd(&L.vcnt[si.lane], nu);
    last = (prev + nu == nrb);
    if (last) atomicExch(&L.vcnt[si.lane], 0);
  }
  last = __builtin_amdgcn_readfirstlane(last);
  if (!last) return;
  // last item of a checked lane: column residual and the decision
  const LaneAgg gc = lane_aggregate(P.agg_out, s, L.rbmax, nrb, true);
  float rrow = rhat;
  if (P.final_audit) {
    const LaneAgg gr = lane_aggregate(P.agg_rowchk, s, L.rbmax, row_blocks(si.n, UNIT), false);
    rrow = gr.sum;
  } else if (L.disc) {
    // shadow mode: the row marginal of the audited state was also recomputed
    // by a dedicated check pass; record how far the screen is from it where a
    // release can be decided (either value within twice the tolerance)
    const LaneAgg gr = lane_aggregate(P.agg_rowchk, s, L.rbmax, row_blocks(si.n, UNIT), false);
    const float dsc = fabsf(rhat - gr.sum);
    if (lane == 0 && dsc == dsc && fminf(rhat, gr.sum) <= 2.f * L.tol)
      // non-negative floats order as their bit patterns
      atomicMax(reinterpret_cast<int*>(&L.disc[si.lane]), __float_as_int(dsc));
  }
  if (lane != 0) return;
  // marginal evaluations spent on this lane's check (the final audit
  // evaluates both marginals)
  atomicAdd(&L.nchk[si.lane], P.final_audit ? 2 : 1);
  const float rcol = gc.sum;
  L.audit[s].rhat = rrow;
  L.audit[s].rcol = rcol;
  const float r = fmaxf(rrow, rcol);
  const bool finite = isfinite(rrow) && isfinite(rcol);
  if (P.final_audit) {
    if (L.mode == MODE_STATIC && si.passed) {
      // keep the first passing depth; report the returned (final) state
      L.dec[s].res_row = rrow;
      L.dec[s].res_col = rcol;
      return;
    }
    retire_lane(L, P, s, si, !finite ? 2 : (r <= L.tol ? 0 : 1), rrow, rcol);
    return;
  }
  if (!isfinite(rrow)) {
    retire_lane(L, P, s, si, 2, rrow, rcol);
  } else if (rrow <= L.tau_screen) {
    atomicAdd(&L.ctrl->screen_pos, 1);
    if (!finite) retire_lane(L, P, s, si, 2, rrow, rcol);
    else if (r <= L.tol) retire_lane(L, P, s, si, 0, rrow, rcol);
    else atomicAdd(&L.ctrl->check_fail, 1);
  } else if (finite && r <= L.tol) {
    atomicAdd(&L.ctrl->missed_ready, 1);   // shadow replay: the screen missed it
  }
}

// One row per lane.
template <int UNIT, int NU, typename T>
__device__ __forceinline__ void finish_rows(const Launch& L, const Pass& P, int s,
                                            const SlotInfo& si, int rb0, bool owner, bool live,
                                            bool fast, float Mf, T lse_old, T lm, float w, T Mt,
                                            T St, float rhat) {
  const bool o[1] = {owner}, lv[1] = {live};
  const T lo[1] = {lse_old}, l2[1] = {lm}, mt[1] = {Mt}, st[1] = {St};
  const float ww[1] = {w};
  finish_rows_r<UNIT, NU, 1, T>(L, P, s, si, rb0, o, lv, fast, Mf, lo, l2, ww, mt, st, rhat);
}

// XCD-aware item order. Consecutive workgroups are dispatched to the 8 XCDs
// in turn, so block b (x = b mod 8) takes item x*q + min(x, r) + b/8 of the
// N = 8q + r items: every XCD works through one contiguous range of items --
// whole lanes -- and its L2 holds only those lanes' column operands. The map
// is a bijection of [0, N), so it changes which block runs an item, never
// what the item computes. Used for uniform lane shapes, where every item is
// the same work.
__device__ __forceinline__ int xcd_item(int b, int N) {
  const int q = N >> 3, r = N & 7, x = b & 7;
  return x * q + min(x, r) + (b >> 3);
}

// Ties the device-state values a block checks (slot record, control block) to
// a value computed from the item's own loads, so the compiler cannot test them
// -- and wait for them -- before those loads are in flight.
__device__ __forceinline__ void behind(SlotInfo& si, int& c_fin, int& c_A, float dep) {
  __asm__ volatile("" : "+v"(si.lane), "+v"(si.n), "+v"(si.m), "+v"(si.done), "+v"(si.passed),
                   "+v"(c_fin), "+v"(c_A) : "v"(dep));
}

// Whether the item of slot s has work, given the control block's finished
// flag and width and the slot record.
__device__ __forceinline__ bool item_live(const Launch& L, const Pass& P, int s, const SlotInfo& si,
                                          int c_finished, int c_A) {
  if (!P.final_audit && c_finished) return false;
  if (s >= c_A) return false;
  if (P.kind == KIND_UPDATE) return !(si.done && L.mode == MODE_ACTIVE);
  if (si.done) return false;
  if (!P.final_audit && si.passed) return false;
  return true;
}

// Blocks of pass pi of a launch.
__device__ __forceinline__ int pass_blocks(const Launch& L, int pi) {
  return pi ? (int)gridDim.x - L.nb0 : L.nb0;
}

// Uniform lane shapes (P.ipl > 0): block b of a pass takes item
// xcd_item(b, nb) of the pass's own nb blocks, so its slot s and first row
// block rb0 (RPI row blocks per item) follow from the launch alone and the
// block can issue its operand loads before any read of device state. The host
// sizes every pass to at least the items of the device-side layout, so every
// item is covered; blocks past it are dropped by item_live(). False only for
// slots beyond the launch's own width bound (never read).
template <int RPI>
__device__ __forceinline__ bool item_uniform(const Pass& P, int nb, int b, int& s, int& rb0) {
  const int ipi = (P.ipl + RPI - 1) / RPI;   // items per lane
  const int item = xcd_item(b, nb);
  s = item / ipi;
  rb0 = (item - s * ipi) * RPI;
  return s < P.A;
}

// Mixed lane shapes: the item comes from the offsets table of the device-side
// layout (slot s, first row block rb0); false when the block has no work.
// Items are taken in block order, so consecutive items go to different XCDs:
// with lanes of very different sizes, whole-lane ranges per XCD left the XCDs'
// work 7-21 % apart at full width (the slowest one ends the launch), while
// interleaved items balance it at the price of every XCD reading every lane's
// column operands.
__device__ __forceinline__ bool locate_item(const Launch& L, const Pass& P, int b, int& s,
                                            int& rb0, SlotInfo& si) {
  const Ctrl* c = L.ctrl;
  const int fin = c->finished;
  const int A = min(P.A, c->A);
  if (!P.final_audit && fin) return false;
  const int N = P.off[A];
  if (b >= N) return false;
  const int item = b;
  const int q = find_slot(P.off, A, item);   // position in the role's item order
  rb0 = item - P.off[q];
  s = P.ord[q];
  si = L.slot[s];
  return item_live(L, P, s, si, fin, A);
}

// Where block b of a pass of nb blocks works (slot s, first row block rb0, the
// lane's row and column counts). With uniform shapes the control block and slot record
// are only requested here (c_fin, c_A, si) and checked by item_live() once
// the item's own loads are in flight; otherwise they are already checked.
template <int RPI, int UNI = -1>
__device__ __forceinline__ bool place_item(const Launch& L, const Pass& P, int nb, int b, int& s,
                                           int& rb0, int& nrows, int& ncols, SlotInfo& si,
                                           int& c_fin, int& c_A) {
  // UNI: 1 / 0 when the caller is compiled for uniform / mixed shapes only
  if (UNI == 1 || (UNI < 0 && P.ipl > 0)) {
    if (!item_uniform<RPI>(P, nb, b, s, rb0)) return false;
    // Read through the vector memory path (a zero offset the compiler cannot
    // prove uniform): scalar loads complete out of order, so any later use of
    // a kernel argument would wait for these, while vector loads are waited
    // for in issue order, after the operand loads issued behind them.
    const int z = (int)__builtin_amdgcn_mbcnt_lo(0u, 0u);
    c_fin = L.ctrl[z].finished;
    c_A = L.ctrl[z].A;
    si = L.slot[s + z];
    nrows = P.nr;
    ncols = P.nc;
    return true;
  }
  if (UNI == 1) return false;
  if (!locate_item(L, P, b, s, rb0, si)) return false;   // (RPI == 1: mixed shapes)
  c_fin = 0;
  c_A = 0x7fffffff;
  nrows = P.role ? si.m : si.n;
  ncols = P.role ? si.n : si.m;
  return true;
}

// Placement for kernels whose every placed block must arrive at its item's
// counter (one block per (item, column group)): false only for blocks beyond
// the launch's items, a fact fixed for the whole launch. Whether the item
// still has work can change while the launch runs (a check pass of the same
// launch may retire the lane or finish the window), so it is left to
// item_live() on c_fin, c_A and si, and a block without work arrives marked
// skipped.
template <int UNI = -1>
__device__ __forceinline__ bool place_item_all(const Launch& L, const Pass& P, int nb, int b,
                                               int& s, int& rb0, int& nrows, int& ncols,
                                               SlotInfo& si, int& c_fin, int& c_A) {
  if (UNI == 1 || (UNI < 0 && P.ipl > 0))
    return place_item<1, 1>(L, P, nb, b, s, rb0, nrows, ncols, si, c_fin, c_A);
  const Ctrl* c = L.ctrl;
  c_fin = c->finished;
  c_A = min(P.A, c->A);
  if (b >= P.off[c_A]) return false;
  const int q = find_slot(P.off, c_A, b);
  rb0 = b - P.off[q];
  s = P.ord[q];
  si = L.slot[s];
  nrows = P.role ? si.m : si.n;
  ncols = P.role ? si.n : si.m;
  return true;
}

// --------------------------------------------------------- MFMA half-step
// The columns of a lane are cut into kGroups fixed groups of whole 32-column
// tiles (tpg = ceil(tiles / kGroups) tiles each). Every group is swept in tile
// order from its own start, per half-wave; the partials are then merged per row
// in a fixed order (half-wave 0, half-wave 1, then groups 0..kGroups-1). How a
// launch spreads (row tile, group) pairs over waves -- RT 32-row tiles and GW
// consecutive groups per wave, kGroups / GW waves per block -- changes which
// wave does the work, never the arithmetic, so a lane's bits do not depend on
// the variant the host picks for the current width.
//
// In every 32x32 tile the matrix core forms D[j][i] = sum_k A[j][k] B[k][i] over
// the augmented vectors A_j = (y~_j, gam_j, 1), B_i = (x~_i, 1, -anchor_i)
// (K = 2*DH + 2): D is the base-2 exponent of the (i, j) term minus the row
// anchor. Lane l holds row i = l % 32 for 16 columns, so the streaming sum over
// j stays inside the lane. The next tile's operands load while the current
// tile is reduced.
//
// The second launch bound is the minimum number of waves per SIMD the register
// allocation must allow, chosen per layout and dh so that no variant spills
// vector registers to scratch and the scalar spills stay at the few every
// variant has: at 8 waves (64 registers) the two-group layout spilled 79
// scalar registers into vector lanes, some 250 extra lane read/write
// instructions per wave (c2 3 % slower than at 6 waves).
template <int DH, int RT, int GW>
constexpr int mfma_waves_per_simd() {
  return (kGroups / GW) == 8 ? (DH <= 7 ? 4 : 2)
       : (kGroups / GW) == 2 ? (DH <= 7 ? 5 : 4)
       : (RT == 1 ? (DH <= 5 ? 6 : (DH <= 10 ? 5 : 4)) : (DH <= 8 ? 4 : 2));
}

// UNI: compiled for uniform lane shapes (work item -> slot by division) or
// for mixed shapes (offsets table); the host launches the one that matches.
template <int DH, int RT, int GW, bool UNI>
__global__ __launch_bounds__(64 * (kGroups / GW), (mfma_waves_per_simd<DH, RT, GW>()))
void k_update_mfma(Launch L) {
  note_progress(L);
  static_assert(UNI || RT == 1, "two row tiles per item need uniform lane shapes");
  constexpr int ROWS = 32 * RT;
  constexpr int kUnrollGroups = GW > 2 ? 1 : GW;   // four groups unrolled: 25 scalar spills
  constexpr int DP = 2 * DH;
  __shared__ float2 sh_part[kGroups][2][ROWS];
  const int b = blockIdx.x;
  const int pi = b >= L.nb0;
  const Pass P = L.p[pi];
  int s, rb0, nrows, ncols, c_fin, c_A;
  SlotInfo si;
  if (!place_item<RT, UNI ? 1 : 0>(L, P, pass_blocks(L, pi), pi ? b - L.nb0 : b, s, rb0, nrows,
                                   ncols, si, c_fin, c_A))
    return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  if (!upd) {
    const bool chk = check_facts(L, P, s, P.role ? ncols : nrows, rhat);
    if (UNI) behind(si, c_fin, c_A, rhat);
    if (!item_live(L, P, s, si, c_fin, c_A) || !chk) return;
  }
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  const int h = lane >> 5;
  const int r = lane & 31;

  // Every load of the item (row data, first column tile, the lane facts) is
  // issued before the block waits on any of them -- with uniform lane shapes
  // also before its slot record and the control block are checked.
  float lse_t[RT], bv[RT][DH + 1];
#pragma unroll
  for (int q = 0; q < RT; ++q) {
    const size_t ridx = (size_t)s * P.padr + (rb0 + q) * 32 + r;
    lse_t[q] = P.lse_in[ridx];
    const float* rrow = P.rec_row + ridx * DP + h * DH;
#pragma unroll
    for (int k = 0; k < DH; ++k) bv[q][k] = rrow[k];
  }
  // wave 0 lane l owns row rb0 * 32 + l (tile l / 32, row l % 32)
  const int orow = rb0 * 32 + lane;
  const bool owner = wave == 0 && lane < ROWS && orow < nrows;
  float own_lm = 0.f, own_w = 0.f;
  if (owner) own_lm = P.lm_row[(size_t)s * P.padr + orow];

  const int ct = (ncols + kColTile - 1) / kColTile;
  const int tpg = (ct + kGroups - 1) / kGroups;
  const int g0 = wave * GW;
  const int ta = min(ct, g0 * tpg);
  const int tb = min(ct, (g0 + GW) * tpg);
  const float* ccol = P.rec_col + (size_t)s * P.padc * DP + h * DH + (size_t)r * DP;
  const float* gcol = P.gam_col + (size_t)s * P.padc + r;
  auto load = [&](int t, float* a) {
    const float* c = ccol + (size_t)t * kColTile * DP;
#pragma unroll
    for (int k = 0; k < DH; ++k) a[k] = c[k];
    a[DH] = gcol[(size_t)t * kColTile];
  };
  float A0[DH + 1], A1[DH + 1];
  if (ta < tb) load(ta, A0);

  bool fast = false;
  float M = 0.f;
  if (upd) {
    update_facts(L, P, s, ncols, fast, M);
    if (UNI) behind(si, c_fin, c_A, M);
    if (!item_live(L, P, s, si, c_fin, c_A)) return;
  }
  if (owner) own_w = P.w_row[(size_t)si.lane * P.w_ld + orow];   // caller masses, by lane id
#pragma unroll
  for (int q = 0; q < RT; ++q) {
    const bool live_q = (rb0 + q) * 32 + r < nrows && lse_t[q] != INFINITY;
    float bias = 0.f;
    if (live_q) {
      if (!upd) bias = -lse_t[q];
      else if (fast) bias = -(lse_t[q] + M);
    }
    bv[q][DH] = h ? bias : 1.f;
  }

  float mrun[RT], srun[RT];
  auto reset = [&]() {
#pragma unroll
    for (int q = 0; q < RT; ++q) { mrun[q] = fast ? 0.f : -INFINITY; srun[q] = 0.f; }
  };
  auto tile = [&](const float* a, bool anchored) {
    f32x16 acc[RT];
#pragma unroll
    for (int q = 0; q < RT; ++q)
      acc[q] = f32x16{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < DH; ++k)
#pragma unroll
      for (int q = 0; q < RT; ++q)
        acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[k], bv[q][k], acc[q], 0, 0, 0);
#pragma unroll
    for (int q = 0; q < RT; ++q)
      acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(h ? 1.f : a[DH], bv[q][DH], acc[q], 0, 0, 0);
#pragma unroll
    for (int q = 0; q < RT; ++q) {
      float e[16];
      if (anchored) {
#pragma unroll
        for (int v = 0; v < 16; ++v) e[v] = ex2(acc[q][v]);
#pragma unroll
        for (int w = 8; w > 0; w >>= 1)
#pragma unroll
          for (int v = 0; v < w; ++v) e[v] += e[v + w];
        srun[q] += e[0];
      } else {
        float tm = acc[q][0];
#pragma unroll
        for (int v = 1; v < 16; ++v) tm = fmaxf(tm, acc[q][v]);
        const float mn = fmaxf(mrun[q], tm);
        const float mref = (mn == -INFINITY) ? 0.f : mn;
#pragma unroll
        for (int v = 0; v < 16; ++v) e[v] = ex2(acc[q][v] - mref);
#pragma unroll
        for (int w = 8; w > 0; w >>= 1)
#pragma unroll
          for (int v = 0; v < w; ++v) e[v] += e[v + w];
        srun[q] = srun[q] * ex2(mrun[q] - mref) + e[0];
        mrun[q] = mn;
      }
    }
  };
  // The wave's groups are consecutive tile ranges: the last prefetch of one
  // group may already be the first tile of the next (`have`). No prefetch
  // goes past the wave's last tile, so every load stays in bounds and none is
  // left in flight when the sweep ends.
  auto sweep = [&](bool anchored) {
    bool have = ta < tb;
    int t = ta;
#pragma unroll kUnrollGroups
    for (int u = 0; u < GW; ++u) {
      const int t1 = min(ct, (g0 + u + 1) * tpg);
      reset();
      if (t < t1) {
        if (!have) load(t, A0);
        for (; t + 1 < t1; t += 2) {
          load(t + 1, A1);
          tile(A0, anchored);
          if (t + 2 < tb) load(t + 2, A0);   // no load past the wave's last tile
          tile(A1, anchored);
        }
        if (t < t1) { tile(A0, anchored); ++t; have = false; }
        else have = t < tb;
      }
#pragma unroll
      for (int q = 0; q < RT; ++q) sh_part[g0 + u][h][32 * q + r] = make_float2(mrun[q], srun[q]);
    }
  };
  if (fast) sweep(true); else sweep(false);
  __syncthreads();
  if (wave != 0) return;
  // merge per row: half-waves, then groups, in order. Anchored sums carry a
  // zero running maximum everywhere, so there every scale factor is exactly 1
  // and the merge is the plain sum in the same order (the same bits).
  float Mt = 0.f, St = 0.f;
  if (owner && fast) {
#pragma unroll
    for (int g = 0; g < kGroups; ++g) St += sh_part[g][0][lane].y + sh_part[g][1][lane].y;
  } else if (owner) {
    float Mg[kGroups], Sg[kGroups];
    float mx = -INFINITY;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
      const float2 pa = sh_part[g][0][lane], pb = sh_part[g][1][lane];
      const float mw = fmaxf(pa.x, pb.x);              // -inf only if both are empty
      const float mref = (mw == -INFINITY) ? 0.f : mw;
      Sg[g] = pa.y * ex2(pa.x - mref) + pb.y * ex2(pb.x - mref);
      Mg[g] = mw;
      mx = fmaxf(mx, mw);
    }
    Mt = (mx == -INFINITY) ? 0.f : mx;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) St += Sg[g] * ex2(Mg[g] - Mt);
  }
  // lane l < 32 RT owns tile l / 32 row l % 32, whose input lse it holds as lse_t[l / 32]
  const float own_lse = (RT == 2 && h) ? lse_t[RT - 1] : lse_t[0];
  const bool live = owner && own_lse != INFINITY;
  finish_rows<32, RT, float>(L, P, s, si, rb0, owner, live, fast, M, own_lse, own_lm, own_w, Mt, St,
                             rhat);
}

// --------------------------------------------------- matrix-free, large d
// The float32 half-step for any d as a tiled contraction on the matrix cores
// with the streaming base-2 sum as its epilogue. A block owns one work item of
// 128 rows and one of the lane's kGroups column groups (groups of whole
// 128-column steps), so even a launch of few items spreads over the chip. Per
// step the block forms the 128 x 128 tile of x~ . y~: four waves of 64 x 64
// (2 x 2 v_mfma_f32_32x32x2_f32 tiles each), K-looped over the coordinates in
// stages of kMfreeK, every stage of both operands staged once in LDS by the
// whole block (coalesced 16-byte loads, double-buffered: the next stage loads
// while the current one runs). Inside a stage the matrix instruction p takes
// coordinate 16 h + p from lane half h, so a lane reads its 16 coordinates of
// a row as four 16-byte LDS reads (rows padded to 36 floats: no bank
// conflicts). The column potential and the row anchor enter as one augmented
// matrix instruction per tile, (gam_j, 1) . (1, -anchor_i), then each lane
// reduces its 16 terms of a row per 32-column tile, tile 0 then tile 1 of its
// half of the step, steps in order.
//
// A row's group partial is the fold, in the order (wave column 0, lane half 0),
// (0, 1), (1, 0), (1, 1), of four running partials; it goes to memory with
// device-scope stores, and the item's last block to arrive merges the groups in
// order and finishes the item. Every order depends on the lane's (n, m, d)
// only, so the bits do not depend on the launch.
// One LDS stage of the matrix-free kernel: kMfreeK coordinates of the item's
// kRowsMfmaK rows, then of the step's kMfreeCols columns, each row at a stride
// of kMfreeK + 4 floats. Thread t moves float4 number t % 8 of rows t / 8 + 32 j
// (j < 4) of both operands: eight threads read one row's 128 contiguous bytes.
struct MfreeStage {
  static constexpr int LD = kMfreeK + 4;
  static constexpr int STAGE = (kRowsMfmaK + kMfreeCols) * LD;
  static_assert(kRowsMfmaK == 128 && kMfreeCols == 128 && kMfreeK == 32, "256 threads, 4 rows each");
  const float* xs;   // this thread's first float of the item's rows
  const float* ys;   // and of the lane's columns
  float* ss;         // its first LDS float of a stage
  int dp;
  // native vectors in named registers: HIP's float4 (or an array) here ended up
  // in memory, and its stores then waited for the loads mid-stage
  f32x4 x0, x1, x2, x3, y0, y1, y2, y3;
  __device__ __forceinline__ MfreeStage(const float* xrec, const float* yrec, int dp_, float* sh)
      : dp(dp_) {
    const int row = threadIdx.x >> 3, q = (threadIdx.x & 7) * 4;
    xs = xrec + (size_t)row * dp + q;
    ys = yrec + (size_t)row * dp + q;
    ss = sh + row * LD + q;
  }
  // coordinates k0 .. k0 + kMfreeK of step t
  __device__ __forceinline__ void fetch(int t, int k0) {
    const float* xq = xs + k0;
    const float* yq = ys + (size_t)t * kMfreeCols * dp + k0;
    const size_t r32 = (size_t)32 * dp;
    x0 = *reinterpret_cast<const f32x4*>(xq);
    y0 = *reinterpret_cast<const f32x4*>(yq);
    x1 = *reinterpret_cast<const f32x4*>(xq + r32);
    y1 = *reinterpret_cast<const f32x4*>(yq + r32);
    x2 = *reinterpret_cast<const f32x4*>(xq + 2 * r32);
    y2 = *reinterpret_cast<const f32x4*>(yq + 2 * r32);
    x3 = *reinterpret_cast<const f32x4*>(xq + 3 * r32);
    y3 = *reinterpret_cast<const f32x4*>(yq + 3 * r32);
  }
  __device__ __forceinline__ void stash(int buf) const {
    float* st = ss + buf * STAGE;
    *reinterpret_cast<f32x4*>(st) = x0;
    *reinterpret_cast<f32x4*>(st + kRowsMfmaK * LD) = y0;
    *reinterpret_cast<f32x4*>(st + 32 * LD) = x1;
    *reinterpret_cast<f32x4*>(st + (kRowsMfmaK + 32) * LD) = y1;
    *reinterpret_cast<f32x4*>(st + 64 * LD) = x2;
    *reinterpret_cast<f32x4*>(st + (kRowsMfmaK + 64) * LD) = y2;
    *reinterpret_cast<f32x4*>(st + 96 * LD) = x3;
    *reinterpret_cast<f32x4*>(st + (kRowsMfmaK + 96) * LD) = y3;
  }
};

template <bool UNI>
__global__ __launch_bounds__(256, 2)
void k_update_mfma_k(Launch L) {
  note_progress(L);
  constexpr int BM = kRowsMfmaK;   // rows of an item
  constexpr int BN = kMfreeCols;   // columns of a step
  constexpr int KC = kMfreeK;      // coordinates per stage
  constexpr int LD = MfreeStage::LD;        // LDS row stride (floats)
  constexpr int STAGE = MfreeStage::STAGE;
  __shared__ __align__(16) float sh_buf[2 * STAGE];
  __shared__ int sh_work[4];
  const int it = (int)(blockIdx.x / kGroups);   // work item of the launch (both passes)
  const int g = (int)(blockIdx.x % kGroups);    // its column group
  const int pi = it >= L.nb0;
  const Pass P = L.p[pi];
  const int nitems = pi ? (int)(gridDim.x / kGroups) - L.nb0 : L.nb0;
  int s, rb0, nrows, ncols, c_fin, c_A;
  SlotInfo si;
  if (!place_item_all<UNI ? 1 : 0>(L, P, nitems, pi ? it - L.nb0 : it, s, rb0, nrows, ncols, si,
                                   c_fin, c_A))
    return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  // (a fact of the previous launch: the same for every block of the item)
  if (!upd && !check_facts(L, P, s, P.role ? ncols : nrows, rhat)) return;
  bool fast = false;
  float M = 0.f;
  if (upd) update_facts(L, P, s, ncols, fast, M);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the sweep has block barriers: one liveness verdict for the whole block
  if (lane == 0) sh_work[wave] = item_live(L, P, s, si, c_fin, c_A) ? 1 : 0;
  __syncthreads();
  const bool work = sh_work[0] && sh_work[1] && sh_work[2] && sh_work[3];
  const int h = lane >> 5, r = lane & 31;
  const int wr = wave >> 1, wc = wave & 1;   // the wave's 64 rows and 64 columns of a step
  const int DP = L.dp;
  const int row0 = rb0 * BM;
  float baug[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int i = row0 + wr * 64 + a * 32 + r;
    const float lse = P.lse_in[(size_t)s * P.padr + i];
    const bool lv = i < nrows && lse != INFINITY;
    float bias = 0.f;
    if (lv) {
      if (!upd) bias = -lse;
      else if (fast) bias = -(lse + M);
    }
    baug[a] = h ? bias : 1.f;
  }
  const int S = (ncols + BN - 1) / BN;
  const int spg = (S + kGroups - 1) / kGroups;
  const int tA = min(S, g * spg), tB = min(S, g * spg + spg);
  const int nch = DP / KC;
  const float m0 = fast ? 0.f : -INFINITY;
  float mrun[2] = {m0, m0}, srun[2] = {0.f, 0.f};
  if (work && tA < tB) {
    const float* xrec = P.rec_row + ((size_t)s * P.padr + row0) * DP;
    const float* yrec = P.rec_col + (size_t)s * P.padc * DP;
    const float* gcol = P.gam_col + (size_t)s * P.padc;
    MfreeStage stg(xrec, yrec, DP, sh_buf);
    stg.fetch(tA, 0);
    stg.stash(0);
    __syncthreads();
    int t = tA, kc = 0, buf = 0;
    f32x16 acc[2][2];
    float ag[2];
#pragma unroll 1
    while (t < tB) {
      if (kc == 0) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;
#pragma unroll
        for (int b = 0; b < 2; ++b) ag[b] = h ? 1.f : gcol[(size_t)t * BN + wc * 64 + b * 32 + r];
      }
      // the next stage (of this step, or the first of the next one) loads now;
      // after the last one the current stage is loaded again, unused, so that
      // the loop has no branch around its loads and stores
      int tn = t, kn = kc + 1;
      if (kn == nch) { kn = 0; ++tn; }
      stg.fetch(tn < tB ? tn : t, tn < tB ? kn * KC : kc * KC);
      __builtin_amdgcn_sched_barrier(0);   // the loads go out before the stage's matrix work
      const float* sx = sh_buf + buf * STAGE;
      const float* sy = sx + BM * LD;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        float4 xv[2][2], yv[2][2];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int q = 0; q < 2; ++q)
            xv[a][q] = *reinterpret_cast<const float4*>(sx + (wr * 64 + a * 32 + r) * LD + h * 16 +
                                                        half * 8 + q * 4);
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int q = 0; q < 2; ++q)
            yv[b][q] = *reinterpret_cast<const float4*>(sy + (wc * 64 + b * 32 + r) * LD + h * 16 +
                                                        half * 8 + q * 4);
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
              for (int b = 0; b < 2; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(yv[b][q][e], xv[a][q][e],
                                                                 acc[a][b], 0, 0, 0);
      }
      if (kc == nch - 1) {
        // the step's epilogue: column potential and row anchor, then the
        // streaming sum of each row (tile 0, then tile 1)
#pragma unroll
        for (int a = 0; a < 2; ++a) {
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            const f32x16 z = __builtin_amdgcn_mfma_f32_32x32x2f32(ag[b], baug[a], acc[a][b], 0, 0, 0);
            float e[16];
            if (fast) {
#pragma unroll
              for (int v = 0; v < 16; ++v) e[v] = ex2(z[v]);
#pragma unroll
              for (int w = 8; w > 0; w >>= 1)
#pragma unroll
                for (int v = 0; v < w; ++v) e[v] += e[v + w];
              srun[a] += e[0];
            } else {
              float tm = z[0];
#pragma unroll
              for (int v = 1; v < 16; ++v) tm = fmaxf(tm, z[v]);
              const float mn = fmaxf(mrun[a], tm);
              const float mref = (mn == -INFINITY) ? 0.f : mn;
#pragma unroll
              for (int v = 0; v < 16; ++v) e[v] = ex2(z[v] - mref);
#pragma unroll
              for (int w = 8; w > 0; w >>= 1)
#pragma unroll
                for (int v = 0; v < w; ++v) e[v] += e[v + w];
              srun[a] = srun[a] * ex2(mrun[a] - mref) + e[0];
              mrun[a] = mn;
            }
          }
        }
      }
      // (the stage's stores stay behind the matrix work: hoisted above it they
      // would wait for the global loads before the stage runs)
      __builtin_amdgcn_sched_barrier(0);
      stg.stash(buf ^ 1);
      __syncthreads();
      buf ^= 1;
      t = tn;
      kc = kn;
    }
  }
  // the four running partials of every row, through LDS (the stages are done)
  __syncthreads();
  float2* sp = reinterpret_cast<float2*>(sh_buf);   // [wave column][lane half][row]
#pragma unroll
  for (int a = 0; a < 2; ++a)
    sp[(2 * wc + h) * BM + wr * 64 + a * 32 + r] = make_float2(mrun[a], srun[a]);
  __syncthreads();
  if (wave != 0) return;
  float2* part = L.kpart + (size_t)it * kGroups * BM;
  if (work) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int i = 64 * e + lane;
      float gm = m0, gs = 0.f;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float2 pu = sp[u * BM + i];
        if (fast) {
          gs += pu.y;
        } else {
          const float mn = fmaxf(gm, pu.x);
          const float mref = (mn == -INFINITY) ? 0.f : mn;
          gs = gs * ex2(gm - mref) + pu.y * ex2(pu.x - mref);
          gm = mn;
        }
      }
      st_dev2(part + (size_t)g * BM + i, make_float2(gm, gs));
    }
  }
  // the finish's own row data loads with the arrival (its latency overlaps it)
  bool owner[2], live[2];
  float own_lm[2] = {0.f, 0.f}, own_w[2] = {0.f, 0.f}, own_lse[2], Mt[2] = {0.f, 0.f},
        St[2] = {0.f, 0.f};
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int i = row0 + 64 * e + lane;
    owner[e] = i < nrows;
    own_lse[e] = P.lse_in[(size_t)s * P.padr + i];
    if (owner[e] && work) {
      own_lm[e] = P.lm_row[(size_t)s * P.padr + i];
      own_w[e] = P.w_row[(size_t)si.lane * P.w_ld + i];
    }
  }
  bool skipped;
  if (!arrive_last(&L.scnt[it], work, skipped) || skipped) return;
  // the item's finish: lane l owns rows row0 + l and row0 + 64 + l; every
  // group partial is loaded before the first is used
  float2 pg[2][kGroups];
#pragma unroll
  for (int e = 0; e < 2; ++e)
#pragma unroll
    for (int u = 0; u < kGroups; ++u) pg[e][u] = ld_dev2(part + (size_t)u * BM + 64 * e + lane);
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    live[e] = owner[e] && own_lse[e] != INFINITY;
    if (!owner[e]) continue;
    if (fast) {
#pragma unroll
      for (int u = 0; u < kGroups; ++u) St[e] += pg[e][u].y;
    } else {
      float mx = -INFINITY;
#pragma unroll
      for (int u = 0; u < kGroups; ++u) mx = fmaxf(mx, pg[e][u].x);
      Mt[e] = (mx == -INFINITY) ? 0.f : mx;
#pragma unroll
      for (int u = 0; u < kGroups; ++u) St[e] += pg[e][u].y * ex2(pg[e][u].x - Mt[e]);
    }
  }
  finish_rows_r<BM, 1, 2, float>(L, P, s, si, rb0, owner, live, fast, M, own_lse, own_lm, own_w, Mt,
                                 St, rhat);
}

// --------------------------------------------------------- VALU half-step
// Work item = 64 rows (one per lane) of one lane against all its columns, with
// the same fixed column groups as the matrix-core kernel; each wave sweeps GW
// consecutive groups. The column data of a tile is the same for every lane
// (wave-uniform), so it is read through the scalar path and used as SGPR
// operands: per (i, j) term D fused multiply-adds, one v_exp_f32 and one add.
// Groups are merged in LDS in a fixed order.
template <int D, int DH, int GW>
__global__ __launch_bounds__(64 * (kGroups / GW), (kGroups / GW == 8 ? 4 : 8))
void k_update_valu(Launch L) {
  note_progress(L);
  __shared__ float2 sh_part[kGroups][kRowsValu];
  const int b = blockIdx.x;
  const int pi = b >= L.nb0;
  const Pass P = L.p[pi];
  int s, rb, nrows, ncols, c_fin, c_A;
  SlotInfo si;
  if (!place_item<1>(L, P, pass_blocks(L, pi), pi ? b - L.nb0 : b, s, rb, nrows, ncols, si, c_fin,
                     c_A))
    return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  if (!upd) {
    const bool chk = check_facts(L, P, s, P.role ? ncols : nrows, rhat);
    if (!item_live(L, P, s, si, c_fin, c_A) || !chk) return;
  }
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  const int i = rb * kRowsValu + lane;
  constexpr int DP = 2 * DH;
  // row loads are issued before the update facts are reduced
  const size_t ridx = (size_t)s * P.padr + i;
  const float lse_old = P.lse_in[ridx];
  const bool in_prefix = i < nrows;
  const bool owner = wave == 0 && in_prefix;
  float lm = 0.f, w = 0.f;
  if (owner) lm = P.lm_row[ridx];
  float xr[D];
  const float* rrow = P.rec_row + ridx * DP;
#pragma unroll
  for (int k = 0; k < D; ++k) xr[k] = rrow[k];
  bool fast = false;
  float M = 0.f;
  if (upd) {
    update_facts(L, P, s, ncols, fast, M);
    if (!item_live(L, P, s, si, c_fin, c_A)) return;
  }
  if (owner) w = P.w_row[(size_t)si.lane * P.w_ld + i];   // caller masses, by lane id
  const bool live = in_prefix && (lse_old != INFINITY);
  float bias = 0.f;
  if (live) {
    if (!upd) bias = -lse_old;
    else if (fast) bias = -(lse_old + M);
  }

  const int ct = (ncols + kColTile - 1) / kColTile;
  const int tpg = (ct + kGroups - 1) / kGroups;
  const float* __restrict__ ccol = P.rec_col + (size_t)s * P.padc * DP;
  const float* __restrict__ gcol = P.gam_col + (size_t)s * P.padc;
#pragma unroll
  for (int u = 0; u < GW; ++u) {
    const int g = wave * GW + u;
    const int j0 = min(ct, g * tpg) * kColTile;
    const int j1 = min(ct, g * tpg + tpg) * kColTile;
    float mrun = -INFINITY, srun = 0.f;
    if (fast) {
      float sacc[4] = {0.f, 0.f, 0.f, 0.f};
      for (int j = j0; j < j1; j += 4) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float* cj = ccol + (size_t)(j + v) * DP;
          float z = gcol[j + v] + bias;
#pragma unroll
          for (int k = 0; k < D; ++k) z = fmaf(xr[k], cj[k], z);
          sacc[v] += ex2(z);
        }
      }
      srun = (sacc[0] + sacc[1]) + (sacc[2] + sacc[3]);
      mrun = 0.f;
    } else {
      for (int j = j0; j < j1; j += 8) {
        float z[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const float* cj = ccol + (size_t)(j + v) * DP;
          float zz = gcol[j + v] + bias;
#pragma unroll
          for (int k = 0; k < D; ++k) zz = fmaf(xr[k], cj[k], zz);
          z[v] = zz;
        }
        float tm = z[0];
#pragma unroll
        for (int v = 1; v < 8; ++v) tm = fmaxf(tm, z[v]);
        const float mn = fmaxf(mrun, tm);
        const float mref = (mn == -INFINITY) ? 0.f : mn;
        float e[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) e[v] = ex2(z[v] - mref);
        const float ts = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
        srun = srun * ex2(mrun - mref) + ts;
        mrun = mn;
      }
    }
    sh_part[g][lane] = make_float2(mrun, srun);   // (-inf, 0) for an empty group
  }
  __syncthreads();
  if (wave != 0) return;
  float Mt = 0.f, St = 0.f;
  if (owner && fast) {   // anchored sums: every scale factor is exactly 1
#pragma unroll
    for (int g = 0; g < kGroups; ++g) St += sh_part[g][lane].y;
  } else if (owner) {
    float mx = -INFINITY;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) mx = fmaxf(mx, sh_part[g][lane].x);
    Mt = (mx == -INFINITY) ? 0.f : mx;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) St += sh_part[g][lane].y * ex2(sh_part[g][lane].x - Mt);
  }
  finish_rows<kRowsValu, 1, float>(L, P, s, si, rb, owner, live && owner, fast, M, lse_old, lm, w,
                                   Mt, St, rhat);
}

// The potential of a float64-state point in the caller's units, before its
// rounding to the float32 output: kappa f = gam + |x~|^2 / 2 (gam as stored,
// nrm = |x~|^2 summed by fused multiply-adds in component order). Written with
// an explicit fma so that every caller gets the same bits: the emission, and
// the export-rounding sums of guarded release.
__device__ __forceinline__ double potential_f64(double gam, double nrm, double kappa64) {
  return fma(0.5, nrm, gam) * (1.0 / kappa64);
}

// ------------------------------------------------- float64 (precise) half-step
// The vector-ALU half-step with the state (records, log masses, lse, gam) in
// float64 and every exponent formed in float64 -- d fused multiply-adds and one
// add -- before it is rounded once to float32 for v_exp_f32 (anchored sums are
// used while the bound's spread is at most kFastRangePrecise). The terms of one
// 32-column tile are summed in float32 and each tile's sum is added in float64;
// a sub-group's tiles accumulate from zero and the sub-groups are folded into
// their group in order.
//
// A work item is 64 R rows (rows_f64(D): R = 2): lane l owns rows l + 64 r
// (r < R), so every column value read from LDS serves R terms.
// Column data is the same for every lane; each wave stages its tiles in its own
// LDS double buffer
// (coalesced loads: records, then the column operand gam written into slot D
// of each column -- the record's padding double when D is odd) and reads them
// back as broadcasts. Only the wave itself touches its buffer, so no block
// barrier is needed (a wave's LDS operations complete in order).
// The second launch bound (minimum waves per SIMD) sets the register budget.
// Chosen per d by measurement: at d = 16 two rows per lane spill a few
// registers to scratch even at two waves per SIMD (in the per-tile
// bookkeeping, not the column loop) and still run faster than one row.
template <int D>
constexpr int f64_waves_per_simd() { return D <= 4 ? 4 : (D <= 7 ? 3 : 2); }
// Where the wide sweep's registers run out (d >= 14 spills a few), the
// finish's own row data (masses, log masses, the old lse) is read after the
// sweep instead of before it: telemetry solve (d = 16) 511 against 523 ms.
// Below that the wait at the end of each item costs more (mixture 271
// against 265 ms, LiDAR-shaped 1879 against 1858 ms).
template <int D>
constexpr bool kLateFinishLoads() { return D >= 14; }
// The split kernel sweeps one or a few tiles per wave: at d = 8 it prefetches
// one column ahead instead of two, which frees the registers for a third wave
// per SIMD (narrow launches of 10 to 12 mixture lanes then run in one round of
// blocks instead of two). From d = 9 the same bound spills in the sweep.
template <int D>
constexpr int kSplitPrefetch() { return D == 8 ? 1 : 2; }
template <int D>
constexpr int f64_split_waves_per_simd() { return D == 8 ? 3 : f64_waves_per_simd<D>(); }

// One 32-column tile of the float64 half-step for R rows per lane (the tile in
// LDS at `cur`, column stride DG, the column operand in slot D). Anchored sums
// add the tile's float32 sums in float64; otherwise a streaming maximum and a
// rescaled sum over steps of four columns.
template <int D, int R, int DG, int PFMAX = 2>
__device__ __forceinline__ void f64_tile(const double* cur, const double (&xr)[R][D],
                                         const double (&bias)[R], bool fast, double (&mrun)[R],
                                         double (&srun)[R]) {
  // Anchored sums: even and odd columns of the tile in two float32 sums per
  // row, added in float64 at the tile's end (the same order on both paths).
  if (fast && D <= 4) {
    float tacc[R][2];
#pragma unroll
    for (int r = 0; r < R; ++r) tacc[r][0] = tacc[r][1] = 0.f;
    for (int c = 0; c < kColTile; c += 2) {
#pragma unroll
      for (int v = 0; v < 2; ++v) {
        double cj[D + 1];
#pragma unroll
        for (int k = 0; k <= D; ++k) cj[k] = cur[(c + v) * DG + k];
#pragma unroll
        for (int r = 0; r < R; ++r) {
          double z = cj[D] + bias[r];
#pragma unroll
          for (int k = 0; k < D; ++k) z = fma(xr[r][k], cj[k], z);
          tacc[r][v] += ex2((float)z);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) srun[r] += (double)(tacc[r][0] + tacc[r][1]);
  } else if (fast) {
    // d >= 5: the values of the column PF ahead are read from LDS while the
    // current column computes (software pipelining; the compiler alone waited
    // on nearly every read at the occupancy these register counts allow).
    // Two ahead measured best up to d = 12; at d = 16 registers allow one.
    // (PFMAX: a caller's cap, for a register budget of more waves per SIMD.)
    constexpr int PF = D <= 12 && PFMAX >= 2 ? 2 : 1;
    float tacc[R][2];
#pragma unroll
    for (int r = 0; r < R; ++r) tacc[r][0] = tacc[r][1] = 0.f;
    double cq[PF][D + 1];
#pragma unroll
    for (int p = 0; p < PF; ++p)
#pragma unroll
      for (int k = 0; k <= D; ++k) cq[p][k] = cur[p * DG + k];
#pragma unroll
    for (int c = 0; c < kColTile; ++c) {
      double cj[D + 1];
#pragma unroll
      for (int k = 0; k <= D; ++k) cj[k] = cq[c % PF][k];
      if (c + PF < kColTile) {
#pragma unroll
        for (int k = 0; k <= D; ++k) cq[c % PF][k] = cur[(c + PF) * DG + k];
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        double z = cj[D] + bias[r];
#pragma unroll
        for (int k = 0; k < D; ++k) z = fma(xr[r][k], cj[k], z);
        tacc[r][c & 1] += ex2((float)z);
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) srun[r] += (double)(tacc[r][0] + tacc[r][1]);
  } else {
    for (int c = 0; c < kColTile; c += 4) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        double z[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const double* cj = cur + (c + v) * DG;
          double zz = cj[D] + bias[r];
#pragma unroll
          for (int k = 0; k < D; ++k) zz = fma(xr[r][k], cj[k], zz);
          z[v] = zz;
        }
        const double tm = fmax(fmax(z[0], z[1]), fmax(z[2], z[3]));
        const double mn = fmax(mrun[r], tm);
        const double mref = (mn == -(double)INFINITY) ? 0.0 : mn;
        const double ts =
            ((double)ex2((float)(z[0] - mref)) + (double)ex2((float)(z[1] - mref))) +
            ((double)ex2((float)(z[2] - mref)) + (double)ex2((float)(z[3] - mref)));
        srun[r] = fma(srun[r], (double)ex2((float)(mrun[r] - mref)), ts);
        mrun[r] = mn;
      }
    }
  }
}

// Fold of a sub-group partial (m, s) into its group's (gm, gs), in sub-group
// order: the streaming merge used across tiles. The empty partial (-inf, 0) --
// (0, 0) with anchored sums -- leaves (gm, gs) bit for bit unchanged, and the
// first fold from the empty state returns the partial itself.
__device__ __forceinline__ void f64_fold(double& gm, double& gs, double m, double s, bool fast) {
  if (fast) {
    gs += s;
    return;
  }
  const double mn = fmax(gm, m);
  const double ref = (mn == -(double)INFINITY) ? 0.0 : mn;
  gs = fma(gs, (double)ex2((float)(gm - ref)), s * (double)ex2((float)(m - ref)));
  gm = mn;
}

// Merge of a row's kGroups group partials in group order: (Mt, St) with
// St * 2^Mt the row's sum.
__device__ __forceinline__ void f64_merge(const double (&gm)[kGroups], const double (&gs)[kGroups],
                                          double& Mt, double& St) {
  double mx = -(double)INFINITY;
#pragma unroll
  for (int g = 0; g < kGroups; ++g) mx = fmax(mx, gm[g]);
  Mt = (mx == -(double)INFINITY) ? 0.0 : mx;
  St = 0.0;
#pragma unroll
  for (int g = 0; g < kGroups; ++g) St = fma(gs[g], (double)ex2((float)(gm[g] - Mt)), St);
}

// Guarded release: how far rounding to the float32 outputs moves the potentials
// of an item's rows -- of the input state in the f-half (its column operand is
// lm - lse_old, bit for bit what that state's f-half stored), of the new state
// in the g-half (gnew). Per item {sum of mass x |rounding|, max |rounding|, sum
// of mass} over the points with mass; each |rounding| also covers the float64
// evaluation of the potential (a few units of 2^-53 of its terms). Wave 0.
template <int D, int R>
__device__ __forceinline__ void f64_export_rounding(const Launch& L, const Pass& P,
                                                    const SlotInfo& si, int rb,
                                                    const bool (&owner)[R], const float (&w)[R],
                                                    const double (&lm)[R],
                                                    const double (&lse_old)[R],
                                                    const double (&gnew)[R],
                                                    const double (&xr)[R][D]) {
  float sd = 0.f, md = 0.f, sw = 0.f;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const double gq = P.role ? gnew[r] : lm[r] - lse_old[r];
    if (!owner[r] || w[r] == 0.f || !(fabs(gq) < (double)INFINITY)) continue;
    double nrm = 0.0;
#pragma unroll
    for (int k = 0; k < D; ++k) nrm = fma(xr[r][k], xr[r][k], nrm);
    const double F = potential_f64(gq, nrm, si.kappa64);
    const double dl = fabs((double)(float)F - F) + (fabs(gq) + 0.5 * nrm) * (0x1p-46 / si.kappa64);
    sd += w[r] * (float)dl;
    md = fmaxf(md, (float)dl);
    sw += w[r];
  }
  const float4 v = make_float4(wave64(sd, OpAdd()), wave64(md, OpMax()), wave64(sw, OpAdd()), 0.f);
  if ((threadIdx.x & 63) == 0) P.gerr_out[(size_t)si.lane * L.rbmax + rb] = v;
}

// Column tiles of a lane: ct tiles of 32 columns, kGroups groups of tpg tiles,
// each cut into kSubGroups sub-groups of tps tiles (trailing ones may be empty).
struct F64Tiling {
  int ct, tpg, tps;
  __device__ F64Tiling(int ncols) {
    ct = (ncols + kColTile - 1) / kColTile;
    tpg = (ct + kGroups - 1) / kGroups;
    tps = (tpg + kSubGroups - 1) / kSubGroups;
  }
};

// Stage tile t of the lane's column records and operand into an LDS buffer:
// lane l moves double2 number q * 64 + l of a tile (clamped: the last lanes
// of a partial round repeat an in-range element, harmlessly); double2 e of
// the HBM tile is pair e % (DP / 2) of column e / (DP / 2), which lands at
// double2 (e / (DP / 2)) * (DG / 2) + e % (DP / 2) of the LDS tile, and the
// operand gam of column c at c * DG + D.
template <int D>
struct F64Stage {
  static constexpr int DP = D + (D & 1);
  static constexpr int DG = (D + 2) & ~1;
  static constexpr int TREC = kColTile * DP;   // doubles of records per tile in HBM
  static constexpr int NV2 = TREC / 2;         // double2 per tile
  static constexpr int PER = (NV2 + 63) / 64;  // double2 per lane
  static_assert(PER <= 4, "a float64 tile is at most 4 double2 per lane");
  double2 pv[4];
  double pg;
  __device__ __forceinline__ void fetch(const double* rec_lane, const double* gam_lane, int t,
                                        int lane) {
    const double2* src = reinterpret_cast<const double2*>(rec_lane + (size_t)t * TREC);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      pv[q] = q < PER ? src[min(q * 64 + lane, NV2 - 1)] : make_double2(0.0, 0.0);
    pg = gam_lane[t * kColTile + (lane & (kColTile - 1))];
  }
  __device__ __forceinline__ void stash(double* dst, int lane) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < PER) {
        const int e = min(q * 64 + lane, NV2 - 1);
        reinterpret_cast<double2*>(dst)[(e / (DP / 2)) * (DG / 2) + e % (DP / 2)] = pv[q];
      }
    }
    if (lane < kColTile) dst[lane * DG + D] = pg;
    __builtin_amdgcn_wave_barrier();
  }
};

template <int D, int GW>
__global__ __launch_bounds__(64 * (kGroups / GW), (f64_waves_per_simd<D>()))
void k_update_f64(Launch L) {
  note_progress(L);
  constexpr int ROWS = rows_f64(D);
  constexpr int R = ROWS / 64;
  constexpr int DP = F64Stage<D>::DP;    // record stride in HBM (doubles)
  constexpr int DG = F64Stage<D>::DG;    // column stride in LDS: coordinates, gam, (pad)
  __shared__ double2 sh_part[kGroups][ROWS];
  __shared__ __align__(16) double sh_tile[kGroups / GW][2][kColTile * DG];
  const int b = blockIdx.x;
  const int pi = b >= L.nb0;
  const Pass P = L.p[pi];
  int s, rb, nrows, ncols, c_fin, c_A;
  SlotInfo si;
  if (!place_item<1>(L, P, pass_blocks(L, pi), pi ? b - L.nb0 : b, s, rb, nrows, ncols, si, c_fin,
                     c_A))
    return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  if (!upd) {
    const bool chk = check_facts(L, P, s, P.role ? ncols : nrows, rhat);
    if (!item_live(L, P, s, si, c_fin, c_A) || !chk) return;
  }
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  double lse_old[R], lm[R], xr[R][D];
  bool in_prefix[R], owner[R];
  float w[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = rb * ROWS + 64 * r + lane;
    const size_t ridx = (size_t)s * P.padr + i;
    lse_old[r] = reinterpret_cast<const double*>(P.lse_in)[ridx];
    in_prefix[r] = i < nrows;
    owner[r] = wave == 0 && in_prefix[r];
    lm[r] = 0.0;
    w[r] = 0.f;
    if (!kLateFinishLoads<D>() && owner[r]) lm[r] = reinterpret_cast<const double*>(P.lm_row)[ridx];
    const double* rrow = reinterpret_cast<const double*>(P.rec_row) + ridx * DP;
#pragma unroll
    for (int k = 0; k < D; ++k) xr[r][k] = rrow[k];
  }
  // the wave's first tile loads with the rows, before the lane facts and the
  // liveness verdict are known (in bounds either way; unused if no work)
  const F64Tiling T(ncols);
  const double* rec_lane = reinterpret_cast<const double*>(P.rec_col) + (size_t)s * P.padc * DP;
  const double* gam_lane = reinterpret_cast<const double*>(P.gam_col) + (size_t)s * P.padc;
  F64Stage<D> st;
  {
    const int g0 = wave * GW;
    const int tA0 = min(T.ct, g0 * T.tpg), tB0 = min(T.ct, g0 * T.tpg + T.tpg);
    if (tA0 < tB0) st.fetch(rec_lane, gam_lane, tA0, lane);
  }
  bool fast = false;
  float M = 0.f;
  if (upd) {
    update_facts(L, P, s, ncols, fast, M, kFastRangePrecise);
    if (!item_live(L, P, s, si, c_fin, c_A)) return;
  }
  bool live[R];
  double bias[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = rb * ROWS + 64 * r + lane;
    if (!kLateFinishLoads<D>() && owner[r])
      w[r] = P.w_row[(size_t)si.lane * P.w_ld + i];   // caller masses, by lane id
    live[r] = in_prefix[r] && (lse_old[r] != (double)INFINITY);
    bias[r] = 0.0;
    if (live[r]) {
      if (!upd) bias[r] = -lse_old[r];
      else if (fast) bias[r] = -(lse_old[r] + (double)M);
    }
  }

  double* buf0 = sh_tile[wave][0];
  double* buf1 = sh_tile[wave][1];
  const double m0 = fast ? 0.0 : -(double)INFINITY;
#pragma unroll
  for (int u = 0; u < GW; ++u) {
    const int g = wave * GW + u;
    const int tA = min(T.ct, g * T.tpg), tB = min(T.ct, g * T.tpg + T.tpg);
    // the group's running fold lives in the wave's own sh_part slots (only
    // this wave touches them before the block barrier), not in registers
    double mrun[R], srun[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      mrun[r] = m0;
      srun[r] = 0.0;
      sh_part[g][64 * r + lane] = make_double2(m0, 0.0);
    }
    if (tA < tB) {
      if (u > 0) st.fetch(rec_lane, gam_lane, tA, lane);
      st.stash(buf0, lane);
    }
    // tiles in order, the next one prefetched across sub-group boundaries;
    // each sub-group's sums start afresh and are folded into the group's
    int send = min(tB, tA + T.tps);
    for (int t = tA; t < tB; ++t) {
      const double* cur = ((t - tA) & 1) ? buf1 : buf0;
      double* nxt = ((t - tA) & 1) ? buf0 : buf1;
      const bool more = t + 1 < tB;
      if (more) st.fetch(rec_lane, gam_lane, t + 1, lane);
      f64_tile<D, R, DG>(cur, xr, bias, fast, mrun, srun);
      __builtin_amdgcn_wave_barrier();
      if (more) st.stash(nxt, lane);
      if (t + 1 == send) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          double2 G = sh_part[g][64 * r + lane];
          f64_fold(G.x, G.y, mrun[r], srun[r], fast);
          sh_part[g][64 * r + lane] = G;
          mrun[r] = m0;
          srun[r] = 0.0;
        }
        send = min(tB, send + T.tps);
      }
    }
  }
  __syncthreads();
  if (wave != 0) return;
  if (kLateFinishLoads<D>()) {
    // the finish's row data, read after the sweep so that the sweep keeps
    // those registers (the row's lse is read again: the launch does not
    // write it)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = rb * ROWS + 64 * r + lane;
      const size_t ridx = (size_t)s * P.padr + i;
      lse_old[r] = reinterpret_cast<const double*>(P.lse_in)[ridx];
      if (owner[r]) {
        lm[r] = reinterpret_cast<const double*>(P.lm_row)[ridx];
        w[r] = P.w_row[(size_t)si.lane * P.w_ld + i];
      }
    }
  }
  double Mt[R], St[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    Mt[r] = 0.0;
    St[r] = 0.0;
    if (!owner[r]) continue;
    double pm[kGroups], ps[kGroups];
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
      pm[g] = sh_part[g][64 * r + lane].x;
      ps[g] = sh_part[g][64 * r + lane].y;
    }
    f64_merge(pm, ps, Mt[r], St[r]);
  }
  bool lo[R];
#pragma unroll
  for (int r = 0; r < R; ++r) lo[r] = live[r] && owner[r];
  double gkeep[R];
#pragma unroll
  for (int r = 0; r < R; ++r) gkeep[r] = -(double)INFINITY;
  finish_rows_r<ROWS, 1, R, double>(L, P, s, si, rb, owner, lo, fast, M, lse_old, lm, w, Mt, St,
                                    rhat, gkeep);
  if (P.gerr_out) f64_export_rounding<D, R>(L, P, si, rb, owner, w, lm, lse_old, gkeep, xr);
}

// device-scope (coherent) float64 store and load for the split launch's partials
__device__ __forceinline__ void st_dev_d(double* p, double v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p),
                     (unsigned long long)__double_as_longlong(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_dev_d(const double* p) {
  return __longlong_as_double((long long)__hip_atomic_load(
      reinterpret_cast<unsigned long long*>(const_cast<double*>(p)), __ATOMIC_RELAXED,
      __HIP_MEMORY_SCOPE_AGENT));
}

// The float64 half-step for narrow launches: one block per (work item, group)
// and in it one wave per sub-group, so a launch of few items still spreads
// over the chip. Each wave sweeps its sub-group's tiles exactly as the wave of
// k_update_f64 that owns the group does (same tiles, same order, same
// accumulators); wave 0 folds the four sub-group partials in order and
// publishes the group partial of every row of the item; the last of the
// item's kGroups blocks to arrive merges the groups in group order and
// finishes the item: the bits equal k_update_f64's.
//
// Arrival: every block of a placed item arrives exactly once, also one whose
// waves found the item retired or the window finished (each wave reads that
// on its own, so blocks of one item can disagree when a lane retires during
// the launch): such a block arrives marked skipped and the last arrival then
// does not finish the item (arrive_last). A check item whose lane the screen
// leaves unchecked (a fact of the previous launch, the same for every block)
// is dropped by all of its blocks before arriving.
template <int D>
__global__ __launch_bounds__(64 * kSubGroups, (f64_split_waves_per_simd<D>()))
void k_update_f64_split(Launch L) {
  note_progress(L);
  constexpr int ROWS = rows_f64(D);
  constexpr int R = ROWS / 64;
  constexpr int DP = F64Stage<D>::DP;
  constexpr int DG = F64Stage<D>::DG;
  __shared__ __align__(16) double sh_tile[kSubGroups][2][kColTile * DG];
  __shared__ double2 sh_sub[kSubGroups][ROWS];
  __shared__ int sh_work[kSubGroups];
  const int it = (int)(blockIdx.x / kGroups);   // work item of the launch (both passes)
  const int g = (int)(blockIdx.x % kGroups);    // its group
  const int pi = it >= L.nb0;
  const Pass P = L.p[pi];
  const int nitems = pi ? (int)(gridDim.x / kGroups) - L.nb0 : L.nb0;
  int s, rb, nrows, ncols, c_fin, c_A;
  SlotInfo si;
  if (!place_item_all(L, P, nitems, pi ? it - L.nb0 : it, s, rb, nrows, ncols, si, c_fin, c_A))
    return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  bool work = true;
  if (!upd) {
    if (!check_facts(L, P, s, P.role ? ncols : nrows, rhat)) return;
    work = item_live(L, P, s, si, c_fin, c_A);
  }
  const int lane = threadIdx.x & 63;
  const int q = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // this wave's sub-group
  double lse_old[R], xr[R][D];
  bool in_prefix[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = rb * ROWS + 64 * r + lane;
    const size_t ridx = (size_t)s * P.padr + i;
    lse_old[r] = reinterpret_cast<const double*>(P.lse_in)[ridx];
    in_prefix[r] = i < nrows;
    const double* rrow = reinterpret_cast<const double*>(P.rec_row) + ridx * DP;
#pragma unroll
    for (int k = 0; k < D; ++k) xr[r][k] = rrow[k];
  }
  // the sub-group's first tile loads with the rows, before the lane facts and
  // the liveness verdict are known (in bounds either way; unused if no work)
  const F64Tiling T(ncols);
  const int tA = min(T.ct, g * T.tpg), tB = min(T.ct, g * T.tpg + T.tpg);
  const int sA = min(tB, tA + q * T.tps), sB = min(tB, sA + T.tps);
  const double* rec_lane = reinterpret_cast<const double*>(P.rec_col) + (size_t)s * P.padc * DP;
  const double* gam_lane = reinterpret_cast<const double*>(P.gam_col) + (size_t)s * P.padc;
  F64Stage<D> st;
  if (sA < sB) st.fetch(rec_lane, gam_lane, sA, lane);
  bool fast = false;
  float M = 0.f;
  if (upd) {
    update_facts(L, P, s, ncols, fast, M, kFastRangePrecise);
    work = item_live(L, P, s, si, c_fin, c_A);
  }
  bool live[R];
  double bias[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    live[r] = in_prefix[r] && (lse_old[r] != (double)INFINITY);
    bias[r] = 0.0;
    if (live[r]) {
      if (!upd) bias[r] = -lse_old[r];
      else if (fast) bias[r] = -(lse_old[r] + (double)M);
    }
  }
  const double m0 = fast ? 0.0 : -(double)INFINITY;
  if (work) {
    double mrun[R], srun[R];
#pragma unroll
    for (int r = 0; r < R; ++r) { mrun[r] = m0; srun[r] = 0.0; }
    if (sA < sB) st.stash(sh_tile[q][0], lane);
    for (int t = sA; t < sB; ++t) {
      const double* cur = sh_tile[q][(t - sA) & 1];
      double* nxt = sh_tile[q][((t - sA) & 1) ^ 1];
      const bool more = t + 1 < sB;
      if (more) st.fetch(rec_lane, gam_lane, t + 1, lane);
      f64_tile<D, R, DG, kSplitPrefetch<D>()>(cur, xr, bias, fast, mrun, srun);
      __builtin_amdgcn_wave_barrier();
      if (more) st.stash(nxt, lane);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) sh_sub[q][64 * r + lane] = make_double2(mrun[r], srun[r]);
  }
  if (lane == 0) sh_work[q] = work ? 1 : 0;
  __syncthreads();
  if (q != 0) return;
  bool all = true;
#pragma unroll
  for (int u = 0; u < kSubGroups; ++u) all = all && sh_work[u] != 0;
  // the group partial of every row: the sub-groups folded in order
  double2* part = L.spart + (size_t)it * kGroups * ROWS;
  if (all) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      double gm = m0, gs = 0.0;
#pragma unroll
      for (int u = 0; u < kSubGroups; ++u) {
        const double2 p = sh_sub[u][64 * r + lane];
        f64_fold(gm, gs, p.x, p.y, fast);
      }
      double* dst = reinterpret_cast<double*>(part + (size_t)g * ROWS + 64 * r + lane);
      st_dev_d(dst, gm);
      st_dev_d(dst + 1, gs);
    }
  }
  // the finish's own row data loads with the arrival (its latency overlaps it)
  bool owner[R];
  double lm[R];
  float w[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = rb * ROWS + 64 * r + lane;
    owner[r] = in_prefix[r];
    lm[r] = 0.0;
    w[r] = 0.f;
    if (owner[r] && all) {
      lm[r] = reinterpret_cast<const double*>(P.lm_row)[(size_t)s * P.padr + i];
      w[r] = P.w_row[(size_t)si.lane * P.w_ld + i];
    }
  }
  bool skipped;
  if (!arrive_last(&L.scnt[it], all, skipped) || skipped) return;
  // the item's finish, as wave 0 of k_update_f64 does it; every partial is
  // loaded before the first is used
  double pm[R][kGroups], ps[R][kGroups];
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int u = 0; u < kGroups; ++u) {
      const double* src = reinterpret_cast<const double*>(part + (size_t)u * ROWS + 64 * r + lane);
      pm[r][u] = ld_dev_d(src);
      ps[r][u] = ld_dev_d(src + 1);
    }
  }
  double Mt[R], St[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    Mt[r] = 0.0;
    St[r] = 0.0;
    if (owner[r]) f64_merge(pm[r], ps[r], Mt[r], St[r]);
  }
  bool lo[R];
#pragma unroll
  for (int r = 0; r < R; ++r) lo[r] = live[r] && owner[r];
  double gkeep[R];
#pragma unroll
  for (int r = 0; r < R; ++r) gkeep[r] = -(double)INFINITY;
  finish_rows_r<ROWS, 1, R, double>(L, P, s, si, rb, owner, lo, fast, M, lse_old, lm, w, Mt, St,
                                    rhat, gkeep);
  if (P.gerr_out) f64_export_rounding<D, R>(L, P, si, rb, owner, w, lm, lse_old, gkeep, xr);
}

// ----------------------------------------------- materialised-cost half-steps
// For large d (or on request) the cost of every lane is built once in base-2
// units, Q_ij = kappa ||x_i - y_j||^2, and the half-steps stream it from HBM:
//     lse_i = log2 sum_j 2^(gam_j - Q_ij)   (f-half: rows of Q)
//     lse_j = log2 sum_i 2^(gam_i - Q_ij)   (g-half: rows of Q^T)
// where gam = kappa * potential (no quadratic fold: no point records exist).
// Q and Q^T are indexed by caller lane and never moved by compaction. One
// kernel serves both half-steps: 64-row work items, eight waves, and the
// column operand staged in LDS.

// Build: one 128 x 128 tile of a lane's cost per block. The centred
// coordinates of the tile's rows and columns are staged in LDS kMfreeK at a
// time (double-buffered, as in the matrix-free half-step), x~ . y~ runs on the
// matrix cores (four waves of 64 x 64), and every thread also sums the squares
// of one row's (tid < 128) or one column's staged coordinates in order; then
// Q = kappa (|x|^2 + |y|^2 - 2 x.y) clamped at 0, stored twice: Q by rows of
// x for the f-half and its transpose for the g-half, so that both half-steps
// stream contiguous rows. The padded region is written too (zero
// coordinates), so every entry a half-step can touch is finite.
//
// Staging: thread t moves coordinate t % 32 of the stage for rows t / 32 + 8 u
// (u < 16) of both operands -- 32 threads read one row's 128 contiguous bytes
// of the caller's array (any d, no alignment beyond 4 bytes).
struct CostStage {
  static constexpr int T = 128;
  static constexpr int LD = kMfreeK + 4;
  static constexpr int STAGE = 2 * T * LD;
  static_assert(kMfreeK == 32, "a warp-wide row of 32 coordinates per stage");
  const float* X;    // the lane's points
  const float* Y;
  const float* cc;   // its centre
  int d, n, m;       // coordinates, valid points (n, m >= 1: validated before)
  int i0, j0;        // the tile's first row and column
  int sk, sr;
  int k;             // the coordinate this thread loaded last
  float ck;          // and the centre's value of it
  f32x16 vx, vy;     // raw loaded values: centring and padding wait for stash()
  // every load is in bounds (row, column and coordinate clamped to the valid
  // ones), with no arithmetic on the loaded values: nothing waits for them
  // before the stage's matrix work
  __device__ __forceinline__ void fetch(int k0) {
    k = k0 + sk;
    const int kc = min(k, d - 1);
    ck = cc[kc];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      vx[u] = X[(size_t)min(i0 + sr + 8 * u, n - 1) * d + kc];
      vy[u] = Y[(size_t)min(j0 + sr + 8 * u, m - 1) * d + kc];
    }
  }
  // centred values into LDS, zero for padding rows and coordinates
  __device__ __forceinline__ void stash(float* st) const {
    const bool kin = k < d;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      st[(sr + 8 * u) * LD + sk] = (kin && i0 + sr + 8 * u < n) ? vx[u] - ck : 0.f;
      st[(T + sr + 8 * u) * LD + sk] = (kin && j0 + sr + 8 * u < m) ? vy[u] - ck : 0.f;
    }
  }
};

__global__ __launch_bounds__(256, 2) void k_cost(CostArgs c) {
  constexpr int T = CostStage::T, KC = kMfreeK, LD = CostStage::LD, STAGE = CostStage::STAGE;
  __shared__ __align__(16) float sh[2 * STAGE];
  __shared__ float sh_nrm[2 * T];   // |x~_i|^2 of the tile's rows, then |y~_j|^2 of its columns
  const int t = blockIdx.y;
  const int tiles_j = c.pad1 / T;
  const int ti = (int)blockIdx.x / tiles_j, tj = (int)blockIdx.x - ti * tiles_j;
  const SlotInfo si = c.slot[t];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r = lane & 31, wr = wave >> 1, wc = wave & 1;
  CostStage stg;
  stg.X = c.X + (size_t)t * c.n_max * c.d;
  stg.Y = c.Y + (size_t)t * c.m_max * c.d;
  stg.cc = c.center + (size_t)t * c.d;
  stg.d = c.d;
  stg.n = si.n;
  stg.m = si.m;
  stg.i0 = ti * T;
  stg.j0 = tj * T;
  stg.sk = tid & 31;
  stg.sr = tid >> 5;
  const int nst = (c.d + KC - 1) / KC;
  stg.fetch(0);
  stg.stash(sh);
  __syncthreads();
  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;
  float nrm = 0.f;
#pragma unroll 1
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    // the next stage loads now (after the last, the current one again, unused)
    stg.fetch((st + 1 < nst ? st + 1 : st) * KC);
    __builtin_amdgcn_sched_barrier(0);
    const float* sx = sh + buf * STAGE;
    const float* sy = sx + T * LD;
    {
      // row tid of the stage (x rows, then y rows): its squares in order
      const float* rw = sx + tid * LD;
#pragma unroll
      for (int q = 0; q < KC / 4; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(rw + 4 * q);
        nrm = fmaf(v.x, v.x, nrm);
        nrm = fmaf(v.y, v.y, nrm);
        nrm = fmaf(v.z, v.z, nrm);
        nrm = fmaf(v.w, v.w, nrm);
      }
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      float4 xv[2][2], yv[2][2];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int q = 0; q < 2; ++q)
          xv[a][q] = *reinterpret_cast<const float4*>(sx + (wr * 64 + a * 32 + r) * LD + h * 16 +
                                                      half * 8 + q * 4);
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int q = 0; q < 2; ++q)
          yv[b][q] = *reinterpret_cast<const float4*>(sy + (wc * 64 + b * 32 + r) * LD + h * 16 +
                                                      half * 8 + q * 4);
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
              acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(xv[a][q][e], yv[b][q][e], acc[a][b],
                                                               0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    stg.stash(sh + (buf ^ 1) * STAGE);
    __syncthreads();
  }
  sh_nrm[tid] = nrm;
  __syncthreads();
  const float kap = si.kappa;
  float* Qt = c.Q + (size_t)t * c.pad0 * c.pad1 + (size_t)ti * T * c.pad1 + (size_t)tj * T;
  // the tile also goes through LDS (rows at an odd stride: conflict-free both
  // ways), to be written transposed with coalesced stores
  constexpr int LT = T + 1;
  static_assert(T * LT <= 2 * STAGE, "the transposed tile fits in the stage buffers");
  float* tl = sh;   // the stages are done (the barrier above)
  // lane l holds D[i][j] of column j = l % 32 of its tile and rows
  // i = 8 (v / 4) + 4 (l / 32) + v % 4
#pragma unroll
  for (int a = 0; a < 2; ++a) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int j = wc * 64 + b * 32 + r;
      const float ny = sh_nrm[T + j];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = wr * 64 + a * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        const float q = kap * fmaxf(sh_nrm[i] + ny - 2.f * acc[a][b][v], 0.f);
        Qt[(size_t)i * c.pad1 + j] = q;
        tl[i * LT + j] = q;
      }
    }
  }
  __syncthreads();
  // Q^T: thread t writes half of row j = t / 2 of the transposed tile, 64
  // consecutive i (the two threads of a row write its 512 contiguous bytes)
  float* QTt = c.QT + (size_t)t * c.pad0 * c.pad1 + (size_t)tj * T * c.pad0 + (size_t)ti * T;
  const int j = tid >> 1, i0 = (tid & 1) * 64;
#pragma unroll
  for (int q = 0; q < 64; q += 4) {
    float4 v;
    v.x = tl[(i0 + q) * LT + j];
    v.y = tl[(i0 + q + 1) * LT + j];
    v.z = tl[(i0 + q + 2) * LT + j];
    v.w = tl[(i0 + q + 3) * LT + j];
    *reinterpret_cast<float4*>(QTt + (size_t)j * c.pad0 + i0 + q) = v;
  }
}

// A half-step (and the marginal check) over the rows of Q (f-half) or of Q^T
// (g-half): wave w sweeps rows w, w+8, .. of the item, its lanes striding
// over the columns four at a time.
__global__ __launch_bounds__(512, 2) void k_mat_rows(Launch L) {
  note_progress(L);
  extern __shared__ __align__(16) float sh_gam[];   // the lane's column operand (padc floats)
  __shared__ float2 sh_row[kRowsValu];
  const int b = blockIdx.x;
  const int pi = b >= L.nb0;
  const Pass P = L.p[pi];
  int s, rb, nrows, ncols, c_fin, c_A;
  SlotInfo si;
  if (!place_item<1>(L, P, pass_blocks(L, pi), pi ? b - L.nb0 : b, s, rb, nrows, ncols, si, c_fin,
                     c_A))
    return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  if (!upd) {
    const bool chk = check_facts(L, P, s, P.role ? ncols : nrows, rhat);
    if (!item_live(L, P, s, si, c_fin, c_A) || !chk) return;
  }
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nc4 = (ncols + 3) & ~3;
  // the column operand, padded to a multiple of 4 with dead columns
  const float* gcol = P.gam_col + (size_t)s * P.padc;
  for (int j = threadIdx.x; j < nc4; j += blockDim.x) sh_gam[j] = j < ncols ? gcol[j] : -INFINITY;
  const int i_own = rb * kRowsValu + lane;
  const bool owner = wave == 0 && i_own < nrows;
  float lse_own = INFINITY, lm = 0.f, w = 0.f;
  if (owner) {
    const size_t idx = (size_t)s * P.padr + i_own;
    lse_own = P.lse_in[idx];
    lm = P.lm_row[idx];
  }
  bool fast = false;
  float M = 0.f;
  if (upd) {
    update_facts(L, P, s, ncols, fast, M);
    if (!item_live(L, P, s, si, c_fin, c_A)) return;
  }
  if (owner) w = P.w_row[(size_t)si.lane * P.w_ld + i_own];   // caller masses, by lane id
  __syncthreads();
  const float* Qt = L.Q + (size_t)si.lane * L.q_lane;
  for (int rr = wave; rr < kRowsValu; rr += 8) {
    const int i = rb * kRowsValu + rr;
    float Mr = -INFINITY, Sr = 0.f;
    if (i < nrows) {
      const float lse_i = P.lse_in[(size_t)s * P.padr + i];
      float bias = 0.f;
      if (lse_i != INFINITY) {
        if (!upd) bias = -lse_i;
        else if (fast) bias = -(lse_i + M);
      }
      const float* q = Qt + (size_t)i * L.q_ld;
      float mrun = fast ? 0.f : -INFINITY, srun = 0.f;
      auto step = [&](const float4 qv, const float4 gv) {
        const float z0 = (gv.x + bias) - qv.x, z1 = (gv.y + bias) - qv.y;
        const float z2 = (gv.z + bias) - qv.z, z3 = (gv.w + bias) - qv.w;
        if (fast) {
          srun += (ex2(z0) + ex2(z1)) + (ex2(z2) + ex2(z3));
        } else {
          const float mn = fmaxf(mrun, fmaxf(fmaxf(z0, z1), fmaxf(z2, z3)));
          const float mref = (mn == -INFINITY) ? 0.f : mn;
          srun = srun * ex2(mrun - mref) +
                 ((ex2(z0 - mref) + ex2(z1 - mref)) + (ex2(z2 - mref) + ex2(z3 - mref)));
          mrun = mn;
        }
      };
      // kRowBatch loads of the row in flight before the first is used (one
      // at a time left each wave waiting for memory on every step); the sum
      // takes the steps in column order
      constexpr int kRowBatch = 8;
      int j = 4 * lane;
      for (; j + 256 * (kRowBatch - 1) < nc4; j += 256 * kRowBatch) {
        float4 qv[kRowBatch];
#pragma unroll
        for (int u = 0; u < kRowBatch; ++u) qv[u] = *reinterpret_cast<const float4*>(q + j + 256 * u);
#pragma unroll
        for (int u = 0; u < kRowBatch; ++u)
          step(qv[u], *reinterpret_cast<const float4*>(sh_gam + j + 256 * u));
      }
      for (; j < nc4; j += 256)
        step(*reinterpret_cast<const float4*>(q + j), *reinterpret_cast<const float4*>(sh_gam + j));
      // fixed-tree merge of the 64 lanes
      if (fast) {
        Mr = 0.f;
        Sr = wave64(srun, OpAdd());
      } else {
        Mr = wave64(mrun, OpMax());
        const float mref = (Mr == -INFINITY) ? 0.f : Mr;
        Sr = wave64(srun * ex2(mrun - mref), OpAdd());
      }
    }
    if (lane == 0) sh_row[rr] = make_float2(Mr, Sr);
  }
  __syncthreads();
  if (wave != 0) return;
  const float2 mt = sh_row[lane];
  const float Mt = (mt.x == -INFINITY) ? 0.f : mt.x;
  const float St = (mt.x == -INFINITY) ? 0.f : mt.y * ex2(mt.x - Mt);
  finish_rows<kRowsValu, 1, float>(L, P, s, si, rb, owner, owner && lse_own != INFINITY, fast, M,
                                   lse_own, lm, w, Mt, St, rhat);
}

// ------------------------------------------------------------- block scan
__device__ __forceinline__ int block_exclusive_scan(int v, int* sh, int& total) {
  // wave inclusive scan by shuffles, then wave totals in slot order
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) { int t = sh[w]; sh[w] = acc; acc += t; }
    sh[31] = acc;
  }
  __syncthreads();
  const int excl = x - v + sh[wave];
  total = sh[31];
  __syncthreads();
  return excl;
}

// Compaction map: one block of 1024 threads; thread t owns slots
// [t*C, t*C + C) so every prefix runs in slot order (= caller lane order,
// which stable compaction preserves). Survivors get dense new slots and the
// work item offsets of the new layout; entries past the new width hold the
// total so a stale upper bound on the width still finds no work.
__global__ __launch_bounds__(1024) void k_scan(ScanArgs p) {
  __shared__ int sh[32];
  const int A = min(p.A, p.ctrl->A);  // the host's width is an upper bound
  const int C = (A + 1023) / 1024;
  const int base = threadIdx.x * C;
  int nsurv = 0, items_f = 0, items_g = 0;
  for (int c = 0; c < C; ++c) {
    const int s = base + c;
    if (s >= A) break;
    const SlotInfo si = p.slot[s];
    if (!si.done) {
      nsurv++;
      items_f += row_blocks(si.n, p.rows);
      items_g += row_blocks(si.m, p.rows);
    }
  }
  int tot_surv, tot_f, tot_g;
  int surv_off = block_exclusive_scan(nsurv, sh, tot_surv);
  block_exclusive_scan(items_f, sh, tot_f);   // (the totals only)
  block_exclusive_scan(items_g, sh, tot_g);
  for (int c = 0; c < C; ++c) {
    const int s = base + c;
    if (s >= A) break;
    const SlotInfo si = p.slot[s];
    p.dec[s].new_slot = si.done ? -1 : surv_off++;
  }
  __syncthreads();   // the map is complete (block-visible global writes)
  // each role's item order keeps the survivors in order (a stable filter of a
  // sorted list stays sorted), renamed to their new slots, with the offsets
  // of their work items
  for (int role = 0; role < 2; ++role) {
    const int* src = p.ord_src[role];
    int* dst = p.ord_dst[role];
    int* off = role ? p.off_g : p.off_f;
    int np = 0, ni = 0;
    for (int c = 0; c < C; ++c) {
      const int q = base + c;
      if (q >= A) break;
      const SlotInfo si = p.slot[src[q]];
      if (!si.done) {
        np++;
        ni += row_blocks(role ? si.m : si.n, p.rows);
      }
    }
    int tp, ti;
    int pos = block_exclusive_scan(np, sh, tp);
    int it = block_exclusive_scan(ni, sh, ti);
    for (int c = 0; c < C; ++c) {
      const int q = base + c;
      if (q >= A) break;
      const int s = src[q];
      const SlotInfo si = p.slot[s];
      if (!si.done) {
        dst[pos] = p.dec[s].new_slot;
        off[pos] = it;
        pos++;
        it += row_blocks(role ? si.m : si.n, p.rows);
      }
    }
    __syncthreads();
    for (int q = tp + (int)threadIdx.x; q <= p.W; q += blockDim.x) off[q] = ti;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    Ctrl* c = p.ctrl;
    c->A_prev = A;
    c->A = tot_surv;
    c->items_f = tot_f;
    c->items_g = tot_g;
    c->compacted += A - tot_surv;
    if (p.hsnap) {
      st_sys(&p.hsnap->compacted, c->compacted);
      st_sys(&p.hsnap->epoch, p.epoch);
    }
  }
}

// Offsets over all slots of the current bank (ingest). One block.
// Item order and work item offsets of the initial layout (slot = caller lane):
// per role the slots by decreasing column count, then by slot (the rank of
// every slot counted against all the others), and the first work item of each
// position of that order.
__global__ __launch_bounds__(1024) void k_offsets(SlotInfo* slot, int A, int rows, int* off_f,
                                                  int* off_g, int* ord_f, int* ord_g, Ctrl* ctrl) {
  __shared__ int sh[32];
  __shared__ int key[2][kMaxW];   // column count of every slot per role: m (f-half), n (g-half)
  for (int s = threadIdx.x; s < A; s += blockDim.x) {
    key[0][s] = slot[s].m;
    key[1][s] = slot[s].n;
  }
  __syncthreads();
  for (int s = threadIdx.x; s < A; s += blockDim.x) {
    const int k0 = key[0][s], k1 = key[1][s];
    int r0 = 0, r1 = 0;
    for (int u = 0; u < A; ++u) {
      const int v0 = key[0][u], v1 = key[1][u];
      r0 += (v0 > k0) || (v0 == k0 && u < s);
      r1 += (v1 > k1) || (v1 == k1 && u < s);
    }
    ord_f[r0] = s;
    ord_g[r1] = s;
  }
  __syncthreads();   // the orders are complete (block-visible global writes)
  const int C = (A + 1023) / 1024;
  const int base = threadIdx.x * C;
  int nf = 0, ng = 0;
  for (int c = 0; c < C; ++c) {
    const int q = base + c;
    if (q >= A) break;
    nf += row_blocks(slot[ord_f[q]].n, rows);
    ng += row_blocks(slot[ord_g[q]].m, rows);
  }
  int tf, tg;
  int of = block_exclusive_scan(nf, sh, tf);
  int og = block_exclusive_scan(ng, sh, tg);
  for (int c = 0; c < C; ++c) {
    const int q = base + c;
    if (q >= A) break;
    off_f[q] = of; off_g[q] = og;
    of += row_blocks(slot[ord_f[q]].n, rows);
    og += row_blocks(slot[ord_g[q]].m, rows);
  }
  if (threadIdx.x == 0) {
    off_f[A] = tf; off_g[A] = tg;
    ctrl->items_f = tf; ctrl->items_g = tg;
    ctrl->items_act_f = tf; ctrl->items_act_g = tg;
  }
}

// ------------------------------------------------------------------- move
// Grid (chunks, A). Retired lanes are emitted in caller order from the
// parity of their audited state; in a compaction the survivors are gathered
// into the other bank at their new slots (every lane-indexed array).
// The output-convention potential of one point of a state, exactly as the
// emission writes it: f_i = (gam_i + |x~_i|^2 / 2) / kappa (likewise g_j), formed
// in the precision of the state and rounded to float32; 0 for a removed point.
__device__ __forceinline__ float export_potential(const float* gam, const float* rec, size_t e,
                                                  int dp, int es, const SlotInfo& si) {
  if (es == 2) {
    const double gq = reinterpret_cast<const double*>(gam)[e];
    if (gq == -(double)INFINITY) return 0.f;
    const double* r = reinterpret_cast<const double*>(rec) + e * dp;
    double nrm = 0.0;
    for (int k = 0; k < dp; ++k) nrm = fma(r[k], r[k], nrm);
    return (float)potential_f64(gq, nrm, si.kappa64);
  }
  const float gq = gam[e];
  if (gq == -INFINITY) return 0.f;
  const float* r = rec + e * dp;
  float nrm = 0.f;
  for (int k = 0; k < dp; ++k) nrm = fmaf(r[k], r[k], nrm);
  return (gq + 0.5f * nrm) * (1.f / si.kappa);
}

__global__ __launch_bounds__(256) void k_move(MoveArgs p) {
  const int s = blockIdx.y;
  const int A = p.compact ? min(p.A, p.ctrl->A_prev) : min(p.A, p.ctrl->A);
  if (s >= A) return;
  const SlotInfo si = p.src.slot[s];
  const Decision d = p.src.dec[s];
  const bool emit = p.emit_all || si.done;
  const bool copy = p.compact && !si.done;
  if (!emit && !copy) return;
  const int c0 = blockIdx.x * p.chunk;
  if (emit) {
    const int par = p.emit_all ? p.final_par : (d.depth & 1);
    for (int side = 0; side < 2; ++side) {
      const int lim = side ? p.m_max : p.n_max;
      const int cnt = side ? si.m : si.n;
      const int padn = p.pad[side];
      float* out = side ? p.g : p.f;
      for (int q = c0 + threadIdx.x; q < min(lim, c0 + p.chunk); q += blockDim.x) {
        const float v = q < cnt ? export_potential(p.src.gam[side][par], p.src.rec[side],
                                                   (size_t)s * padn + q, p.dp, p.es, si)
                                : 0.f;
        out[(size_t)si.lane * lim + q] = v;
      }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      const float rr = (d.status == 2) ? NAN : fmaxf(d.res_row, d.res_col);
      p.depth[si.lane] = d.depth;
      p.residual[si.lane] = rr;
      if (p.row_res) p.row_res[si.lane] = d.res_row;
      if (p.col_res) p.col_res[si.lane] = d.res_col;
      p.status[si.lane] = d.status;
    }
  }
  if (copy) {
    // every per-point array moves as raw floats (es of them per element)
    const int ns = d.new_slot;
    const int es = p.es;
    for (int side = 0; side < 2; ++side) {
      const int padn = p.pad[side];
      const int lim = min(padn, c0 + p.chunk);
      const size_t so = (size_t)s * padn * es, dn = (size_t)ns * padn * es;
      for (int q = c0 * es + threadIdx.x; q < lim * es; q += blockDim.x) {
        p.dst.lm[side][dn + q] = p.src.lm[side][so + q];
        for (int par = 0; par < 2; ++par) {
          p.dst.lse[side][par][dn + q] = p.src.lse[side][par][so + q];
          p.dst.gam[side][par][dn + q] = p.src.gam[side][par][so + q];
        }
      }
      // records: contiguous [pad][dp] elements per slot
      const float4* rs = reinterpret_cast<const float4*>(p.src.rec[side] + so * p.dp);
      float4* rd = reinterpret_cast<float4*>(p.dst.rec[side] + dn * p.dp);
      const int q0 = c0 * p.dp * es / 4, q1 = lim * p.dp * es / 4;
      for (int q = q0 + threadIdx.x; q < q1; q += blockDim.x) rd[q] = rs[q];
    }
    if (blockIdx.x == 0) {
      // the row-block aggregates follow the lane (the next f-half reads the
      // g-half's ones as its bound)
      for (int q = threadIdx.x; q < 4 * p.rbmax; q += blockDim.x) {
        const int a = q / p.rbmax, e = q - a * p.rbmax;
        p.dst.agg[a][(size_t)ns * p.rbmax + e] = p.src.agg[a][(size_t)s * p.rbmax + e];
      }
      if (threadIdx.x == 0) {
        p.dst.slot[ns] = si;
        p.dst.dec[ns] = d;
      }
    }
  }
}

// ------------------------------------------- float64 verification (DS_F_GUARD)
// One marginal of the audited state in float64, for one work item (rows rows of a
// lane against all its columns). The potentials are the float32 values the
// emission writes for that state, the cost is formed in float64 from the
// caller's coordinates, the exponentials are float64: the residual that decides
// a release is that of the potentials the caller receives (eq:release-contract),
// to float64 rounding.
//
// Two launches per audit. The row pass (pass 0, rows = x) runs for the lanes the
// outward bound cannot exclude (guard_lower_bound) -- every lane at the final
// audit -- and its last block records the row residual; a lane whose row
// residual exceeds tol is rejected there. The column pass (pass 1, rows = y)
// runs only for lanes whose row residual of the same audit met tol (every lane
// at the final audit), and its last block takes the decision. Launched between
// the f-half and the g-half of an audited cycle (state k-1 is read-only there)
// and at the final audit.
//
// Thread (r, p) of the block owns row r of the item and column phase p (every
// NPH-th column); it keeps the row's coordinates in registers (DR >= d of them,
// zero-padded; DR = 0: d > 32, read from memory per term). The columns'
// coordinates and exported potentials are staged CH at a time in LDS, where
// the lanes of a wave read the same column (a broadcast). A row's sum is its
// phases' partial sums added in phase order. Each block publishes its rows' sum
// of |marginal - mass| (row order); the last block of the lane adds them in
// block order.
// Outward bound of guarded release (float64 state). The verified residual is
// that of the float32 outputs U, the screen rhat that of the state (f, g) the
// iteration holds. Rounding moves each potential by |df_i|, |dg_j| (summed per
// side by the update kernels as S = sum mass |d|, M = max |d|, A = sum mass), so
// every coupling entry changes by a factor exp((df_i + dg_j) / eps), and with
// |e^x - 1| <= |x| e^|x|:
//   |r_row(U) - r_row| <= e^D / eps (sum_i R_i |df_i| + sum_j C_j |dg_j|),
//   D = (M_f + M_g) / eps, sum_i R_i |df_i| <= S_f + r_row M_f,
//   sum_j C_j |dg_j| <= (1 + eta) S_g (the g-half leaves C_j = b_j (1 +- eta)).
// The screen itself is the row residual of (f, g) up to eta per row ratio
// (exponents rounded once to float32 at |z| <= 64 after float64 formation:
// 2.6e-6; v_exp_f32: 2.4e-7; float32 tile sums of at most 32 terms: 1.9e-6)
// and a relative 4e-6 for its float32 summation over rows, so
//   (rhat (1 - 4e-6) - eta A_f) / (1 + eta) <= r_row <= (rhat (1 + 4e-6) + eta A_f) / (1 - eta)
// with eta = 1e-5. A lane whose lower bound on r_row(U) exceeds tol cannot be
// released at this audit and is not verified. The float32 sums of the rounding
// partials are inflated by 1e-5 relative.
__device__ double guard_lower_bound(const Launch& L, const GuardArgs& G, const SlotInfo& si,
                                    float rhat) {
  float sf = 0.f, mf = 0.f, af = 0.f, sg = 0.f, mg = 0.f;
  for (int side = 0; side < 2; ++side) {
    const float4* base = G.gerr[side] + (size_t)si.lane * L.rbmax;
    const int nrb = row_blocks(side ? si.m : si.n, L.rows);
    float t0 = 0.f, t1 = 0.f, t2 = 0.f;
    for (int q = (int)(threadIdx.x & 63); q < nrb; q += 64) {
      const float4 v = base[q];
      t0 += v.x;
      t1 = fmaxf(t1, v.y);
      t2 += v.z;
    }
    const float s0 = wave64(t0, OpAdd()), s1 = wave64(t1, OpMax()), s2 = wave64(t2, OpAdd());
    if (side == 0) { sf = s0; mf = s1; af = s2; } else { sg = s0; mg = s1; }
  }
  const double eta = 1e-5, infl = 1.0 + 1e-5;
  const double inv_eps = 1.0 / (double)G.eps[si.lane];
  const double Sf = sf * infl, Mf = mf * infl, Af = af * infl, Sg = sg * infl, Mg = mg * infl;
  const double r_lo = ((double)rhat * (1.0 - 4e-6) - eta * Af) / (1.0 + eta);
  const double r_hi = ((double)rhat * (1.0 + 4e-6) + eta * Af) / (1.0 - eta);
  const double eD = exp((Mf + Mg) * inv_eps);
  return r_lo - eD * inv_eps * (Sf + r_hi * Mf + (1.0 + eta) * Sg) * infl;
}

constexpr int kGuardThreads = 256;
template <int DR>
constexpr int guard_chunk() { return DR == 0 ? 256 : (2048 / (DR ? DR : 1) < 256 ? 2048 / (DR ? DR : 1) : 256); }

// Float64 verification in three launches per audit:
//  k_vgate       one wave per slot: whether the lane's row marginal is verified
//                (the outward bound, shadow mode, the final audit); admitted
//                lanes append their row blocks to the row list;
//  k_verify64    (row pass) every (row block, column chunk) unit of the list,
//                over a fixed grid; the lane's last row block records the
//                certificate and appends the lane's column items when its row
//                residual met tol (every lane at the final audit);
//  k_verify64    (column pass) the same over the column list; the lane's last
//                item decides.
// The lists hold (slot * rbmax + row block), bit 30 set when the bound had
// excluded the lane (shadow mode verifies it anyway and counts it). Each list's
// length is reset by the launch before the one that fills it: the gate empties
// the column list, the column pass the row list.
constexpr unsigned kVExcluded = 1u << 30;

__global__ __launch_bounds__(256) void k_vgate(Launch L, GuardArgs G) {
  if (blockIdx.x == 0 && threadIdx.x == 0) G.vlen[1] = 0;
  const Pass& P = L.p[0];
  const int s = (int)(blockIdx.x * 4 + (threadIdx.x >> 6));
  if (s >= P.A) return;
  const Ctrl* c = L.ctrl;
  const int c_fin = c->finished;
  const int c_A = min(P.A, c->A);
  // slots past the device-side width hold no lane (their records may never
  // have been written)
  if (s >= c_A) return;
  const SlotInfo si = L.slot[s];
  if (!item_live(L, P, s, si, c_fin, c_A)) return;
  bool gate = true, checked = true;
  if (!P.final_audit) {
    const LaneAgg g = lane_aggregate(P.agg_screen, s, L.rbmax, row_blocks(si.n, L.rows), false);
    gate = !isfinite(g.sum) || !G.bound || guard_lower_bound(L, G, si, g.sum) <= (double)L.tol;
    checked = gate || P.verify_all;
  }
  if (!checked) return;
  const int lane = threadIdx.x & 63;
  const int nit = row_blocks(si.n, L.rows);
  int base = 0;
  if (lane == 0) base = atomicAdd(&G.vlen[0], nit);
  base = __builtin_amdgcn_readfirstlane(base);
  const unsigned tag = gate ? 0u : kVExcluded;
  for (int k = lane; k < nit; k += 64)
    G.vlist[0][base + k] = (int)((unsigned)(s * L.rbmax + k) | tag);
}

// The lane-level end of a verified item, by one thread: the item's
// {sum |marginal - mass|, non-finite} goes out, the item counts in for its
// lane, and the lane's last item takes the marginal's residual (items in row
// block order) and the pass's consequences.
__device__ void verify_item_done(const Launch& L, const GuardArgs& G, const Pass& P, int s,
                                 const SlotInfo& si, int rb, double part_sum, int bad,
                                 bool excluded) {
  const int lane_id = si.lane;
  const int R = L.rows;
  unsigned long long* dst =
      reinterpret_cast<unsigned long long*>(G.agg64[P.role] + (size_t)s * L.rbmax + rb);
  __hip_atomic_store(dst, (unsigned long long)__double_as_longlong(part_sum), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(dst + 1, (unsigned long long)__double_as_longlong(bad ? 1.0 : 0.0),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  wait_mem();
  const int total = row_blocks(P.role ? si.m : si.n, R);   // the lane's items in this pass
  const int prev = atomicAdd(&L.vcnt[lane_id], 1);
  if (prev + 1 != total) return;
  atomicExch(&L.vcnt[lane_id], 0);
  // last item of the lane: this marginal's residual, in row block order
  double rr = 0.0;
  bool fin = true;
  {
    unsigned long long* src =
        reinterpret_cast<unsigned long long*>(G.agg64[P.role] + (size_t)s * L.rbmax);
    for (int q = 0; q < total; ++q) {
      rr += __longlong_as_double((long long)__hip_atomic_load(
          src + 2 * q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      if (__longlong_as_double((long long)__hip_atomic_load(
              src + 2 * q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) != 0.0)
        fin = false;
    }
  }
  fin = fin && isfinite(rr);
  atomicAdd(&L.nchk[lane_id], 1);   // one marginal evaluated
  if (P.role == 0) {
    RowCert rc;
    rc.r = rr;
    rc.depth = P.depth;
    rc.bad = fin ? 0 : 1;
    G.row64[lane_id] = rc;
    L.audit[s].rhat = (float)rr;
    bool col = P.final_audit;   // the final audit's column pass decides every lane
    if (!P.final_audit) {
      atomicAdd(&L.ctrl->screen_pos, 1);
      if (excluded && fin && rr <= (double)L.tol) atomicAdd(&L.ctrl->guard_missed, 1);
      if (!fin) retire_lane(L, P, s, si, 2, (float)rr, NAN);
      else if (rr > (double)L.tol) atomicAdd(&L.ctrl->check_fail, 1);
      else col = true;
    }
    if (col) {
      const int nit = row_blocks(si.m, R);
      const int base = atomicAdd(&G.vlen[1], nit);
      for (int k = 0; k < nit; ++k) G.vlist[1][base + k] = s * L.rbmax + k;
    }
    return;
  }
  // column pass: the decision on both residuals of the audit
  const RowCert rc = G.row64[lane_id];
  const double rrow = rc.r, rcol = rr;
  fin = fin && !rc.bad && isfinite(rrow);
  const double rmax = fmax(rrow, rcol);
  L.audit[s].rcol = (float)rcol;
  if (P.final_audit) {
    if (L.mode == MODE_STATIC && si.passed) {
      L.dec[s].res_row = (float)rrow;
      L.dec[s].res_col = (float)rcol;
      return;
    }
    retire_lane(L, P, s, si, !fin ? 2 : (rmax <= (double)L.tol ? 0 : 1), (float)rrow, (float)rcol);
    return;
  }
  if (!fin) retire_lane(L, P, s, si, 2, (float)rrow, (float)rcol);
  else if (rmax <= (double)L.tol) retire_lane(L, P, s, si, 0, (float)rrow, (float)rcol);
  else atomicAdd(&L.ctrl->check_fail, 1);
}

// One pass of the float64 marginal evaluation (L.p[0]: role 0 rows = x, role 1
// rows = y) over the units of its list: unit u is column chunk u % kVChunks of
// listed item u / kVChunks, a row block of L.rows rows. The lane's columns are
// cut into kVChunks fixed chunks; per chunk, each row's terms are summed by
// kGuardThreads / rows column phases, the phase sums added in phase order, and
// the chunk sum stored (device scope). The item's last chunk to arrive adds
// every row's chunk sums in chunk order: the bits do not depend on the grid.
// A listed lane cannot retire or finish the window before all of its items
// are done (only its own last item decides, and the window finishes only
// when its last active lane retires), so every unit has work and every item
// receives kVChunks arrivals. Blocks stride over the units: the loop is
// bounded by the list's length, fixed before the launch.
template <int DR>
__global__ __launch_bounds__(kGuardThreads) void k_verify64(Launch L, GuardArgs G) {
  constexpr int CH = guard_chunk<DR>();
  constexpr int DS = DR == 0 ? 1 : DR;                       // staged coordinates per column
  __shared__ double sh_y[DR == 0 ? 1 : CH * DS];
  __shared__ double sh_pot[CH];
  __shared__ double sh_acc[kGuardThreads];
  __shared__ double sh_row[256];
  __shared__ int sh_bad[256];
  __shared__ int sh_last;
  const Pass& P = L.p[0];
  const int role = P.role;
  // the column pass empties the row list for the next audit (nothing in this
  // launch reads it)
  if (role == 1 && blockIdx.x == 0 && threadIdx.x == 0) G.vlen[0] = 0;
  const int units = G.vlen[role] * kVChunks;
  const int* list = G.vlist[role];
  const int tid = threadIdx.x;
  const int R = L.rows;                        // 32 to 256 rows per item
  const int nph = kGuardThreads / R;           // column phases
  const int r = tid % R, ph = tid / R;
  const int d = G.d;
#pragma unroll 1
  for (int u = (int)blockIdx.x; u < units; u += (int)gridDim.x) {
    const unsigned e = (unsigned)list[u / kVChunks];
    const int q = u % kVChunks;
    const bool excluded = (e & kVExcluded) != 0;
    const int sr = (int)(e & ~kVExcluded);
    const int s = sr / L.rbmax, rb = sr % L.rbmax;
    const SlotInfo si = L.slot[s];
    const int lane_id = si.lane;
    const int nrows = role ? si.m : si.n, ncols = role ? si.n : si.m;
    const double inv_eps = 1.0 / (double)G.eps[lane_id];
    const float* wr = P.w_row + (size_t)lane_id * P.w_ld;
    const float* wc = G.w_col[role] + (size_t)lane_id * G.w_ld_col[role];
    const float* ycol = G.xy_col[role] + (size_t)lane_id * G.ld_col[role] * d;
    const int i = rb * R + r;
    const bool live = i < nrows && wr[i] != 0.f;
    double* vp = G.vpart + ((size_t)s * L.rbmax + rb) * kVChunks * R;
    const double fi = live ? (double)export_potential(P.gam_out, P.rec_row,
                                                      (size_t)s * P.padr + i, L.dp, G.es, si)
                           : 0.0;
    const float* xi = G.xy_row[role] + ((size_t)lane_id * G.ld_row[role] + (live ? i : 0)) * d;
    double xr[DS];
#pragma unroll
    for (int k = 0; k < DS; ++k) xr[k] = (DR != 0 && k < d) ? (double)xi[k] : 0.0;
    const int cpc = (ncols + kVChunks - 1) / kVChunks;   // columns per chunk
    const int c_lo = min(ncols, q * cpc), c_hi = min(ncols, c_lo + cpc);
    double acc = 0.0;
#pragma unroll 1
    for (int c0 = c_lo; c0 < c_hi; c0 += CH) {
      __syncthreads();   // every thread is done with the previous stage
      for (int t = tid; t < CH; t += kGuardThreads) {
        const int j = c0 + t;
        sh_pot[t] = (j < c_hi && wc[j] != 0.f)
                        ? (double)export_potential(P.gam_col, P.rec_col, (size_t)s * P.padc + j,
                                                   L.dp, G.es, si)
                        : -(double)INFINITY;   // past the chunk or removed (zero mass)
      }
      if (DR != 0) {
        for (int x = tid; x < CH * DS; x += kGuardThreads) {
          const int t = x / DS, k = x % DS;
          sh_y[x] = (c0 + t < c_hi && k < d) ? (double)ycol[(size_t)(c0 + t) * d + k] : 0.0;
        }
      }
      __syncthreads();
      if (!live) continue;
#pragma unroll 1
      for (int t = ph; t < CH && c0 + t < c_hi; t += nph) {
        const double gj = sh_pot[t];
        if (gj == -(double)INFINITY) continue;
        double C = 0.0;
        if (DR != 0) {
#pragma unroll
          for (int k = 0; k < DS; ++k) {
            const double df = xr[k] - sh_y[t * DS + k];
            C = fma(df, df, C);
          }
        } else {
          const float* yj = ycol + (size_t)(c0 + t) * d;
#pragma unroll 4
          for (int k = 0; k < d; ++k) {
            const double df = (double)xi[k] - (double)yj[k];
            C = fma(df, df, C);
          }
        }
        acc += exp((fi + gj - C) * inv_eps);
      }
    }
    // the chunk sum of every row: its phases in phase order
    sh_acc[tid] = acc;
    __syncthreads();
    if (ph == 0) {
      double tot = 0.0;
      for (int v = 0; v < nph; ++v) tot += sh_acc[v * R + r];
      st_dev_d(vp + (size_t)q * R + r, tot);
    }
    wait_mem();   // this wave's chunk sums are stored before the block arrives
    __syncthreads();
    if (tid < 64) {
      bool skipped;
      const bool last = arrive_last(&G.vscnt[sr], true, skipped, kVChunks);
      if (tid == 0) sh_last = last ? 1 : 0;
    }
    __syncthreads();
    if (sh_last) {
      // the item's last chunk: row totals (chunk sums in chunk order)
      if (tid < R) {
        const int i2 = rb * R + tid;
        const bool lv = i2 < nrows && wr[i2] != 0.f;
        double tot = 0.0;
        if (lv)
          for (int v = 0; v < kVChunks; ++v) tot += ld_dev_d(vp + (size_t)v * R + tid);
        sh_row[tid] = lv ? fabs(tot - (double)wr[i2]) : 0.0;
        sh_bad[tid] = lv && !isfinite(tot);
      }
      __syncthreads();
      if (tid == 0) {
        double part_sum = 0.0;
        int bad = 0;
        for (int v = 0; v < R; ++v) {
          if (rb * R + v >= nrows) break;
          part_sum += sh_row[v];
          bad |= sh_bad[v];
        }
        verify_item_done(L, G, P, s, si, rb, part_sum, bad, excluded);
      }
    }
    __syncthreads();   // sh_last, sh_row and sh_acc are free for the next unit
  }
}


// Completion order: lanes sorted by (depth, lane id). rank_t counts the lanes
// that precede t; one block, W <= 4096.
__global__ __launch_bounds__(1024) void k_order(const int* depth, int W, int* order) {
  for (int t = threadIdx.x; t < W; t += blockDim.x) {
    const int dt = depth[t];
    int rank = 0;
    for (int u = 0; u < W; ++u) {
      const int du = depth[u];
      rank += (du < dt) || (du == dt && u < t);
    }
    order[rank] = t;
  }
}

// ----------------------------------------------------------------- ingest
// Centre of each lane: the mean of its live source points and the mean of its
// live target points, averaged, per coordinate. Block (c, t) takes kw
// consecutive coordinates of lane t (kw a power of two, at most 64, so a wave
// reads 4 kw contiguous bytes of a point); thread (g, k) sums coordinate k over
// points g, g + 256 / kw, ... in order (float64), and the partials of the g are
// then added in order: a fixed order, independent of the launch.
__global__ __launch_bounds__(256) void k_centre(IngestArgs p, int kw) {
  const int t = blockIdx.y;
  const int nt = p.n ? p.n[t] : p.n_max;
  const int mt = p.m ? p.m[t] : p.m_max;
  if (nt < 1 || nt > p.n_max || mt < 1 || mt > p.m_max) return;   // reported by k_ingest_lanes
  const int pg = 256 / kw;
  const int g = threadIdx.x / kw;
  const int k = blockIdx.x * kw + (threadIdx.x % kw);
  const int kc = min(k, p.d - 1);
  const float* a = p.a + (size_t)t * p.n_max;
  const float* b = p.b + (size_t)t * p.m_max;
  const float* X = p.X + (size_t)t * p.n_max * p.d + kc;
  const float* Y = p.Y + (size_t)t * p.m_max * p.d + kc;
  double sx = 0.0, sy = 0.0, cx = 0.0, cy = 0.0;
#pragma unroll 4
  for (int i = g; i < nt; i += pg) {
    const bool live = a[i] != 0.f;
    const float v = X[(size_t)i * p.d];
    sx += live ? (double)v : 0.0;
    cx += live ? 1.0 : 0.0;
  }
#pragma unroll 4
  for (int j = g; j < mt; j += pg) {
    const bool live = b[j] != 0.f;
    const float v = Y[(size_t)j * p.d];
    sy += live ? (double)v : 0.0;
    cy += live ? 1.0 : 0.0;
  }
  __shared__ double sh[4][256];
  sh[0][threadIdx.x] = sx;
  sh[1][threadIdx.x] = sy;
  sh[2][threadIdx.x] = cx;
  sh[3][threadIdx.x] = cy;
  __syncthreads();
  if ((int)threadIdx.x >= kw || k >= p.d) return;
  double rx = 0.0, ry = 0.0, nx = 0.0, ny = 0.0;
  for (int q = 0; q < pg; ++q) {
    const int u = q * kw + (int)threadIdx.x;
    rx += sh[0][u];
    ry += sh[1][u];
    nx += sh[2][u];
    ny += sh[3][u];
  }
  const double mx = nx > 0 ? rx / nx : 0.0, my = ny > 0 ? ry / ny : 0.0;
  p.center[(size_t)t * p.d + k] = (float)(0.5 * (mx + my));
}

__global__ __launch_bounds__(256) void k_ingest_lanes(IngestArgs p) {
  const int t = blockIdx.x;
  const int nt = p.n ? p.n[t] : p.n_max;
  const int mt = p.m ? p.m[t] : p.m_max;
  const float e = p.eps[t];
  int code = 0;
  if (nt < 1 || nt > p.n_max) code = 1;
  else if (mt < 1 || mt > p.m_max) code = 2;
  else if (!(isfinite(e) && e > 0.f)) code = 3;
  if (code) {
    if (threadIdx.x == 0) {
      int old = atomicMin(&p.ctrl->err_lane, t);
      if (t < old) atomicExch(&p.ctrl->err_code, code);
    }
    return;
  }
  if (threadIdx.x == 0) {
    SlotInfo si;
    si.lane = t; si.n = nt; si.m = mt; si.done = 0; si.passed = 0;
    si.kappa64 = 1.4426950408889634 / (double)e;
    si.kappa = (float)si.kappa64;
    si.pad[0] = si.pad[1] = 0;
    p.bank.slot[t] = si;
    Decision d;
    d.status = 1; d.depth = 0; d.res_row = NAN; d.res_col = NAN; d.new_slot = -1;
    d.pad[0] = d.pad[1] = d.pad[2] = 0;
    p.bank.dec[t] = d;
    p.vcnt[t] = 0;
    p.nchk[t] = 0;
    if (p.disc) p.disc[t] = 0.f;
    if (p.row64) {
      RowCert rc;
      rc.r = 0.0;
      rc.depth = 0;
      rc.bad = 0;
      p.row64[t] = rc;
    }
  }
  // no previous half-step: the first update of each side runs unanchored
  const float4 none = make_float4(0.f, INFINITY, -INFINITY, 1.f);
  for (int q = threadIdx.x; q < p.rbmax; q += blockDim.x)
    for (int k = 0; k < 4; ++k) p.bank.agg[k][(size_t)t * p.rbmax + q] = none;
}

// Grid (chunks, W): points of both sides of lane t.
__global__ __launch_bounds__(256) void k_ingest_points(IngestArgs p, int chunk) {
  const int t = blockIdx.y;
  if (p.ctrl->err_lane != 0x7fffffff) return;
  const SlotInfo si = p.bank.slot[t];
  const double sigma = sqrt(2.0 * si.kappa64);
  const float* c = p.center + (size_t)t * p.d;
  for (int side = 0; side < 2; ++side) {
    const int padn = p.pad[side];
    const int cnt = side ? si.m : si.n;
    const int ld = side ? p.m_max : p.n_max;
    const float* P = side ? p.Y : p.X;
    const float* w = side ? p.b : p.a;
    const int c0 = blockIdx.x * chunk;
    for (int q = c0 + threadIdx.x; q < min(padn, c0 + chunk); q += blockDim.x) {
      const size_t idx = (size_t)t * padn + q;
      const float mass = (q < cnt) ? w[(size_t)t * ld + q] : 0.f;
      const bool live = (q < cnt) && (mass != 0.f);
      const double lm = live ? log2((double)mass) : -(double)INFINITY;
      // proposal g^0 (0: cold start), in base-2 units: kappa g^0
      const double kg0 = (side == 1 && live && p.g0) ? si.kappa64 * (double)p.g0[(size_t)t * ld + q]
                                                     : 0.0;
      if (p.mat) {
        // no point records; gam = kappa * potential, starting from g^0
        p.bank.lm[side][idx] = (float)lm;
        for (int par = 0; par < 2; ++par) {
          if (!live) {
            p.bank.lse[side][par][idx] = INFINITY;
            p.bank.gam[side][par][idx] = -INFINITY;
          } else if (side == 0) {
            p.bank.lse[0][par][idx] = NAN;
            p.bank.gam[0][par][idx] = NAN;
          } else {
            p.bank.gam[1][par][idx] = (float)kg0;
            p.bank.lse[1][par][idx] = (float)(lm - kg0);
          }
        }
        continue;
      }
      if (p.precise) {
        // float64 state: records in natural component order
        double* rec = reinterpret_cast<double*>(p.bank.rec[side]) + idx * p.dp;
        double nrm = 0.0;
        for (int k = 0; k < p.dp; ++k) {
          const double v = (live && k < p.d)
                               ? sigma * ((double)P[((size_t)t * ld + q) * p.d + k] - (double)c[k])
                               : 0.0;
          rec[k] = v;
          nrm = fma(v, v, nrm);
        }
        reinterpret_cast<double*>(p.bank.lm[side])[idx] = lm;
        for (int par = 0; par < 2; ++par) {
          double* lse = reinterpret_cast<double*>(p.bank.lse[side][par]);
          double* gam = reinterpret_cast<double*>(p.bank.gam[side][par]);
          if (!live) {
            lse[idx] = (double)INFINITY;
            gam[idx] = -(double)INFINITY;
          } else if (side == 0) {
            lse[idx] = (double)NAN;   // no f^0: the first f-half runs unanchored
            gam[idx] = (double)NAN;
          } else {
            gam[idx] = kg0 - 0.5 * nrm;   // kappa (g^0 - |y - c|^2)
            lse[idx] = lm - gam[idx];
          }
        }
        continue;
      }
      float* rec = p.bank.rec[side] + idx * p.dp;
      double nrm = 0.0;
      if (live) {
        // records padded beyond the next even count (matrix-free large d):
        // zeros between and after the two halves
        if (p.dp > p.d + (p.d & 1))
          for (int k = 0; k < p.dp; ++k) rec[k] = 0.f;
        for (int k = 0; k < p.d; ++k) {
          const double v = sigma * ((double)P[((size_t)t * ld + q) * p.d + k] - (double)c[k]);
          const float fv = (float)v;
          // de-interleaved: even components first, then odd ones
          const int pos = (k & 1) ? (p.dh + (k >> 1)) : (k >> 1);
          rec[pos] = fv;
          nrm = fma((double)fv, (double)fv, nrm);   // |y~|^2 of the rounded coordinates
        }
        if (p.d & 1) rec[p.dp - 1] = 0.f;
      } else {
        for (int k = 0; k < p.dp; ++k) rec[k] = 0.f;
      }
      p.bank.lm[side][idx] = (float)lm;
      for (int par = 0; par < 2; ++par) {
        if (!live) {
          p.bank.lse[side][par][idx] = INFINITY;
          p.bank.gam[side][par][idx] = -INFINITY;
        } else if (side == 0) {
          // no f^0 exists: the first f-half runs unanchored
          p.bank.lse[0][par][idx] = NAN;
          p.bank.gam[0][par][idx] = NAN;
        } else {
          // gam^y = kappa (g^0 - |y - c|^2) = kappa g^0 - |y~|^2 / 2 (cold start: g^0 = 0)
          const float gam0 = (float)(kg0 - 0.5 * nrm);
          p.bank.gam[1][par][idx] = gam0;
          p.bank.lse[1][par][idx] = (float)lm - gam0;
        }
      }
    }
  }
}

__global__ void k_zero_counters(int* vcnt, int W) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < W) vcnt[t] = 0;
}

__global__ void k_ctrl_init(Ctrl* c, int W) {
  if (threadIdx.x == 0) {
    Ctrl z;
    z.err_lane = 0x7fffffff; z.err_code = 0; z.n_active = W; z.n_retired = 0; z.finished = 0;
    z.final_cycle = 0; z.A = W; z.items_f = 0; z.items_g = 0; z.items_act_f = 0;
    z.items_act_g = 0; z.screen_pos = 0; z.check_fail = 0; z.missed_ready = 0;
    z.retire_events = 0; z.compacted = 0; z.A_prev = W; z.guard_missed = 0;
    *c = z;
  }
}

// ------------------------------------------ allocation-free workspace (scratch)
// A fixed device array that serves as the workspace of ds_solve_noalloc, for
// callers that cannot allocate. Every GPU the library runs on holds its own
// copy for the life of the process. Host code never uses the array's name as
// an address: scratch_area() takes its device address with that device
// current, once per device, and hands that out.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t scratch_area(void** ptr, size_t* bytes) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kScratchBytes;
  return hipSuccess;
}

// ------------------------------------------------------- host-side launchers
template <int DH>
static hipError_t launch_mfma_dh(const Launch& a, int variant, int blocks, hipStream_t st,
                                 hipEvent_t e0, hipEvent_t e1) {
  const bool uni = a.p[0].ipl > 0;   // both passes of a launch share the shapes
  if (uni) {
    switch (variant) {
      case VAR_NARROW: hipExtLaunchKernelGGL((k_update_mfma<DH, 1, 1, true>), dim3(blocks), dim3(512), 0, st, e0, e1, 0, a); break;
      case VAR_MEDIUM: hipExtLaunchKernelGGL((k_update_mfma<DH, 1, 2, true>), dim3(blocks), dim3(256), 0, st, e0, e1, 0, a); break;
      case VAR_MEDIUM4: hipExtLaunchKernelGGL((k_update_mfma<DH, 1, 4, true>), dim3(blocks), dim3(128), 0, st, e0, e1, 0, a); break;
      default: return hipErrorInvalidValue;
    }
  } else if (variant == VAR_NARROW) {
    hipExtLaunchKernelGGL((k_update_mfma<DH, 1, 1, false>), dim3(blocks), dim3(512), 0, st, e0, e1, 0, a);
  } else if (variant == VAR_MEDIUM4) {
    hipExtLaunchKernelGGL((k_update_mfma<DH, 1, 4, false>), dim3(blocks), dim3(128), 0, st, e0, e1, 0, a);
  } else {
    hipExtLaunchKernelGGL((k_update_mfma<DH, 1, 2, false>), dim3(blocks), dim3(256), 0, st, e0, e1, 0, a);
  }
  return hipGetLastError();
}
template <int D>
static hipError_t launch_valu_d(const Launch& a, int variant, int blocks, hipStream_t st,
                                hipEvent_t e0, hipEvent_t e1) {
  if (variant == VAR_NARROW)
    hipExtLaunchKernelGGL((k_update_valu<D, (D + 1) / 2, 1>), dim3(blocks), dim3(512), 0, st, e0, e1, 0, a);
  else
    hipExtLaunchKernelGGL((k_update_valu<D, (D + 1) / 2, 2>), dim3(blocks), dim3(256), 0, st, e0, e1, 0, a);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_f64_d(const Launch& a, int variant, int blocks, hipStream_t st,
                               hipEvent_t e0, hipEvent_t e1) {
  if (variant == VAR_SPLIT) {
    // `blocks` work items over both passes, one block per (item, group) and a
    // wave per sub-group; the partials and arrival words of the workspace
    // hold a.nslots items
    if (blocks > a.nslots || a.spart == nullptr || a.scnt == nullptr) return hipErrorInvalidValue;
    hipExtLaunchKernelGGL((k_update_f64_split<D>), dim3(blocks * kGroups), dim3(64 * kSubGroups), 0,
                          st, e0, e1, 0, a);
  } else if (variant == VAR_NARROW) {
    hipExtLaunchKernelGGL((k_update_f64<D, 1>), dim3(blocks), dim3(512), 0, st, e0, e1, 0, a);
  } else {
    hipExtLaunchKernelGGL((k_update_f64<D, 2>), dim3(blocks), dim3(256), 0, st, e0, e1, 0, a);
  }
  return hipGetLastError();
}

}  // namespace ds

// Entry points used by the host runtime (C++ linkage, same library).
namespace ds {
hipError_t launch_update(const Launch& a, int d, bool use_mfma, int variant, int blocks,
                         hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  if (blocks <= 0) return hipSuccess;
  const int dh = (d + 1) / 2;
  if (use_mfma) {
    switch (dh) {
      case 1: return launch_mfma_dh<1>(a, variant, blocks, st, e0, e1);
      case 2: return launch_mfma_dh<2>(a, variant, blocks, st, e0, e1);
      case 3: return launch_mfma_dh<3>(a, variant, blocks, st, e0, e1);
      case 4: return launch_mfma_dh<4>(a, variant, blocks, st, e0, e1);
      case 5: return launch_mfma_dh<5>(a, variant, blocks, st, e0, e1);
      case 6: return launch_mfma_dh<6>(a, variant, blocks, st, e0, e1);
      case 7: return launch_mfma_dh<7>(a, variant, blocks, st, e0, e1);
      case 8: return launch_mfma_dh<8>(a, variant, blocks, st, e0, e1);
      case 9: return launch_mfma_dh<9>(a, variant, blocks, st, e0, e1);
      case 10: return launch_mfma_dh<10>(a, variant, blocks, st, e0, e1);
      case 11: return launch_mfma_dh<11>(a, variant, blocks, st, e0, e1);
      case 12: return launch_mfma_dh<12>(a, variant, blocks, st, e0, e1);
      case 13: return launch_mfma_dh<13>(a, variant, blocks, st, e0, e1);
      case 14: return launch_mfma_dh<14>(a, variant, blocks, st, e0, e1);
      case 15: return launch_mfma_dh<15>(a, variant, blocks, st, e0, e1);
      case 16: return launch_mfma_dh<16>(a, variant, blocks, st, e0, e1);
      default: return hipErrorInvalidValue;
    }
  }
  switch (d) {
    case 1: return launch_valu_d<1>(a, variant, blocks, st, e0, e1);
    case 2: return launch_valu_d<2>(a, variant, blocks, st, e0, e1);
    case 3: return launch_valu_d<3>(a, variant, blocks, st, e0, e1);
    case 4: return launch_valu_d<4>(a, variant, blocks, st, e0, e1);
    case 5: return launch_valu_d<5>(a, variant, blocks, st, e0, e1);
    case 6: return launch_valu_d<6>(a, variant, blocks, st, e0, e1);
    case 7: return launch_valu_d<7>(a, variant, blocks, st, e0, e1);
    case 8: return launch_valu_d<8>(a, variant, blocks, st, e0, e1);
    case 9: return launch_valu_d<9>(a, variant, blocks, st, e0, e1);
    case 10: return launch_valu_d<10>(a, variant, blocks, st, e0, e1);
    case 11: return launch_valu_d<11>(a, variant, blocks, st, e0, e1);
    case 12: return launch_valu_d<12>(a, variant, blocks, st, e0, e1);
    case 13: return launch_valu_d<13>(a, variant, blocks, st, e0, e1);
    case 14: return launch_valu_d<14>(a, variant, blocks, st, e0, e1);
    case 15: return launch_valu_d<15>(a, variant, blocks, st, e0, e1);
    case 16: return launch_valu_d<16>(a, variant, blocks, st, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_update_mfma_k(const Launch& a, int blocks, hipStream_t st, hipEvent_t e0,
                                hipEvent_t e1) {
  if (blocks <= 0) return hipSuccess;
  // `blocks` work items over both passes, one block per (item, group); the
  // partials and arrival words of the workspace hold a.nslots items
  if (blocks > a.nslots || a.kpart == nullptr || a.scnt == nullptr) return hipErrorInvalidValue;
  if (a.dp % kMfreeK != 0) return hipErrorInvalidValue;   // whole stages of coordinates
  const bool uni = a.p[0].ipl > 0;   // both passes of a launch share the shapes
  if (uni)
    hipExtLaunchKernelGGL((k_update_mfma_k<true>), dim3(blocks * kGroups), dim3(256), 0, st, e0, e1, 0, a);
  else
    hipExtLaunchKernelGGL((k_update_mfma_k<false>), dim3(blocks * kGroups), dim3(256), 0, st, e0, e1, 0, a);
  return hipGetLastError();
}

hipError_t launch_update_f64(const Launch& a, int d, int variant, int blocks, hipStream_t st,
                             hipEvent_t e0, hipEvent_t e1) {
  if (blocks <= 0) return hipSuccess;
  switch (d) {
    case 1: return launch_f64_d<1>(a, variant, blocks, st, e0, e1);
    case 2: return launch_f64_d<2>(a, variant, blocks, st, e0, e1);
    case 3: return launch_f64_d<3>(a, variant, blocks, st, e0, e1);
    case 4: return launch_f64_d<4>(a, variant, blocks, st, e0, e1);
    case 5: return launch_f64_d<5>(a, variant, blocks, st, e0, e1);
    case 6: return launch_f64_d<6>(a, variant, blocks, st, e0, e1);
    case 7: return launch_f64_d<7>(a, variant, blocks, st, e0, e1);
    case 8: return launch_f64_d<8>(a, variant, blocks, st, e0, e1);
    case 9: return launch_f64_d<9>(a, variant, blocks, st, e0, e1);
    case 10: return launch_f64_d<10>(a, variant, blocks, st, e0, e1);
    case 11: return launch_f64_d<11>(a, variant, blocks, st, e0, e1);
    case 12: return launch_f64_d<12>(a, variant, blocks, st, e0, e1);
    case 13: return launch_f64_d<13>(a, variant, blocks, st, e0, e1);
    case 14: return launch_f64_d<14>(a, variant, blocks, st, e0, e1);
    case 15: return launch_f64_d<15>(a, variant, blocks, st, e0, e1);
    case 16: return launch_f64_d<16>(a, variant, blocks, st, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_update_mat(const Launch& a, int blocks, hipStream_t st, hipEvent_t e0,
                             hipEvent_t e1) {
  if (blocks <= 0) return hipSuccess;
  // the column operand of a lane is staged whole in LDS: padc floats (both
  // passes of a launch have the same role, so the same padc), sized per call
  // so that short lanes keep more blocks per CU
  const size_t lds = (size_t)a.p[0].padc * sizeof(float);
  if (a.p[0].padc > kMatMaxPts) return hipErrorInvalidValue;
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_mat_rows),
                              hipFuncAttributeMaxDynamicSharedMemorySize, kMatMaxPts * 4);
  });
  // the g-half (and column check) streams the rows of the transposed cost
  Launch b = a;
  if (a.p[0].role == 1) {
    b.Q = a.QT;
    b.q_ld = a.qt_ld;
  }
  hipExtLaunchKernelGGL(k_mat_rows, dim3(blocks), dim3(512), lds, st, e0, e1, 0, b);
  return hipGetLastError();
}
hipError_t launch_vgate(const Launch& a, const GuardArgs& g, hipStream_t st) {
  if (g.vlist[0] == nullptr || g.vlen == nullptr) return hipErrorInvalidValue;
  const int A = a.p[0].A;
  hipLaunchKernelGGL(k_vgate, dim3((unsigned)std::max(1, (A + 3) / 4)), dim3(256), 0, st, a, g);
  return hipGetLastError();
}
hipError_t launch_verify64(const Launch& a, const GuardArgs& g, int items, hipStream_t st) {
  if (a.rows != 32 && a.rows != 64 && a.rows != 128 && a.rows != 256) return hipErrorInvalidValue;
  if (g.vpart == nullptr || g.vscnt == nullptr || g.vlist[0] == nullptr || g.vlist[1] == nullptr ||
      g.vlen == nullptr)
    return hipErrorInvalidValue;
  // items: the host's upper bound on the role's work items (the list holds at
  // most these); at least one block, so that the column pass always empties
  // the row list
  const long long units = (long long)std::max(items, 1) * kVChunks;
  const dim3 grid((unsigned)std::min<long long>(units, kVerifyBlocks)), block(kGuardThreads);
  if (g.d <= 4) hipLaunchKernelGGL(k_verify64<4>, grid, block, 0, st, a, g);
  else if (g.d <= 8) hipLaunchKernelGGL(k_verify64<8>, grid, block, 0, st, a, g);
  else if (g.d <= 16) hipLaunchKernelGGL(k_verify64<16>, grid, block, 0, st, a, g);
  else if (g.d <= 32) hipLaunchKernelGGL(k_verify64<32>, grid, block, 0, st, a, g);
  else hipLaunchKernelGGL(k_verify64<0>, grid, block, 0, st, a, g);
  return hipGetLastError();
}
hipError_t launch_cost(const CostArgs& a, hipStream_t st) {
  // whole 128 x 128 tiles of every lane's padded cost
  if (a.pad0 % CostStage::T != 0 || a.pad1 % CostStage::T != 0) return hipErrorInvalidValue;
  const int tiles = (a.pad0 / CostStage::T) * (a.pad1 / CostStage::T);
  hipLaunchKernelGGL(k_cost, dim3(tiles, a.W), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_scan(const ScanArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}
hipError_t launch_offsets(SlotInfo* slot, int A, int rows, int* off_f, int* off_g, int* ord_f,
                          int* ord_g, Ctrl* ctrl,
                          hipStream_t st) {
  if (A > kMaxW) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_offsets, dim3(1), dim3(1024), 0, st, slot, A, rows, off_f, off_g, ord_f,
                     ord_g, ctrl);
  return hipGetLastError();
}
hipError_t launch_move(const MoveArgs& a, int A, int maxpad, hipStream_t st) {
  if (A <= 0) return hipSuccess;
  const int chunks = (maxpad + a.chunk - 1) / a.chunk;
  hipLaunchKernelGGL(k_move, dim3(chunks, A), dim3(256), 0, st, a);
  return hipGetLastError();
}
hipError_t launch_ingest(const IngestArgs& a, int maxpad, hipStream_t st) {
  hipLaunchKernelGGL(k_ctrl_init, dim3(1), dim3(64), 0, st, a.ctrl, a.W);
  hipLaunchKernelGGL(k_ingest_lanes, dim3(a.W), dim3(256), 0, st, a);
  // the centre: up to 64 coordinates per block (a power of two)
  int kw = 1;
  while (kw < a.d && kw < 64) kw *= 2;
  hipLaunchKernelGGL(k_centre, dim3((a.d + kw - 1) / kw, a.W), dim3(256), 0, st, a, kw);
  const int chunk = 1024;
  const int chunks = (maxpad + chunk - 1) / chunk;
  hipLaunchKernelGGL(k_ingest_points, dim3(chunks, a.W), dim3(256), 0, st, a, chunk);
  return hipGetLastError();
}
hipError_t launch_zero_counters(int* vcnt, int W, hipStream_t st) {
  hipLaunchKernelGGL(k_zero_counters, dim3((W + 255) / 256), dim3(256), 0, st, vcnt, W);
  return hipGetLastError();
}
hipError_t launch_order(const int* depth, int W, int* order, hipStream_t st) {
  hipLaunchKernelGGL(k_order, dim3(1), dim3(1024), 0, st, depth, W, order);
  return hipGetLastError();
}
}  // namespace ds
