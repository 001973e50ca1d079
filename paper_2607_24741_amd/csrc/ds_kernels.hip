// gfx950 kernels of the active-set batched Sinkhorn path (wave64, CDNA4).
//
//  k_update_mfma<DH>  one half-step of eq:sinkhorn-cycle for every (slot, row
//                     block, column split) work item, x~.y~ on the fp32 matrix
//                     cores (v_mfma_f32_32x32x2_f32) with the column potential and
//                     the row anchor folded into the contraction, streaming
//                     base-2 log-sum-exp on the vector ALU, fused row screen.
//  k_update_valu<D>   the same half-step for small d on the vector ALU with the
//                     column data wave-uniform (scalar loads, SGPR operands).
//  k_scan             one block: screen/check decisions, wave-ballot +
//                     prefix-sum compaction map, completion ranks, new work
//                     item offsets (Sec. 3.2, Fig. fig:active-loop).
//  k_move             retiree emission in caller lane order + survivor gather
//                     into the other bank (physical compaction, Sec. 3.2).
//  k_ingest_*         validation, centring/scaling, log masses, cold start.
//
// Determinism: every reduction runs in a fixed order (no float atomics); the
// split count and tile order of a lane depend only on its (n, m), so a lane's
// bits do not depend on the batch width, its slot or its co-lanes.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "ds_internal.h"

namespace ds {

typedef float f32x16 __attribute__((ext_vector_type(16)));

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
// best-effort publication to pinned host memory (system scope, write-through)
__device__ __forceinline__ void st_sys(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
// all of this wave's outstanding memory operations have completed
__device__ __forceinline__ void wait_mem() { __builtin_amdgcn_s_waitcnt(0); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }

enum { KIND_UPDATE = 0, KIND_VERIFY = 1 };
enum { MODE_ACTIVE = 0, MODE_STATIC = 1, MODE_LOGICAL = 2 };

// --------------------------------------------------------- work item lookup
__device__ __forceinline__ int find_slot(const int* off, int A, int b) {
  int lo = 0, hi = A;
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (off[mid] <= b) lo = mid; else hi = mid;
  }
  return lo;
}

// ---------------------------------------------------------- wave reductions
// Fixed butterfly over the 64 lanes: identical result in every lane, and the
// order of operations never depends on data or timing.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int wave_or(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o, 64);
  return v;
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
// Fixed-order reduction (by one wave) of one lane's row-block aggregates
// {sum, min, max, non-finite flag}; every lane of the wave returns the same bits.
struct LaneAgg {
  float sum, dmin, dmax;
  int bad;
};
__device__ __forceinline__ LaneAgg lane_aggregate(const float4* agg, int lane_id, int rbmax,
                                                  int nrb, bool coherent) {
  LaneAgg g;
  float t0 = 0.f, t1 = INFINITY, t2 = -INFINITY;
  int t3 = 0;
  const float4* base = agg + (size_t)lane_id * rbmax;
  for (int q = (int)(threadIdx.x & 63); q < nrb; q += 64) {
    const float4 v = coherent ? ld_dev4(base + q) : base[q];
    t0 += v.x;
    t1 = fminf(t1, v.y);
    t2 = fmaxf(t2, v.z);
    t3 |= (v.w != 0.f);
  }
  g.sum = wave_sum(t0);
  g.dmin = wave_min(t1);
  g.dmax = wave_max(t2);
  g.bad = wave_or(t3);
  return g;
}

// Lane facts every wave reduces itself (same bits in every wave), so no LDS
// broadcast or barrier sits between the block's loads and its sweep.
//
// Update: lse_new - lse_old lies in [min_j dgam_j, max_j dgam_j], dgam being
// the latest change of the column operand (= -(change of the column lse)), so
// anchored (max-free) sums are safe when that spread is small; M = -min dgam.
__device__ __forceinline__ void update_facts(const Launch& L, const Pass& P, const SlotInfo& si,
                                             bool& fast, float& M) {
  const int ncols = P.role ? si.n : si.m;
  const LaneAgg g = lane_aggregate(P.agg_bound, si.lane, L.rbmax, row_blocks(ncols, L.rows), false);
  fast = !g.bad && g.dmin <= g.dmax && (g.dmax - g.dmin) <= kFastRange;
  M = -g.dmin;
}
// Check: whether this lane is checked at all (screen-positive, non-finite
// screen, or every lane), and the row screen of the audited state.
__device__ __forceinline__ bool check_facts(const Launch& L, const Pass& P, const SlotInfo& si,
                                            float& rhat) {
  rhat = NAN;
  if (P.role == 1 && !P.final_audit) {
    const LaneAgg g = lane_aggregate(P.agg_screen, si.lane, L.rbmax, row_blocks(si.n, L.rows), false);
    rhat = g.sum;
    return P.verify_all || !isfinite(g.sum) || g.sum <= L.tau_screen;
  }
  return true;
}

// -------------------------------------------------------- block epilogue
// Finish of one work item after the column groups were merged. `owner`
// threads hold one row each (merged (M, sum)). Writes the new lse / gam
// (update), the row-block aggregate, and -- for the column check -- takes
// the lane's retirement decision in the last arriving block of the lane.
// Every thread of the block must call it.
template <int NWAVES>
__device__ void finish_block(const Launch& L, const Pass& P, int s, const SlotInfo& si, int rb,
                             int i, bool owner, bool live, bool fast, float anchor, float lse_old,
                             float lm, float w, float M, float sum, float rhat) {
  __shared__ float sh_red[4][NWAVES];
  __shared__ int sh_last;
  const bool frozen = (L.mode == MODE_LOGICAL) && si.done;
  float rho = 0.f, dmin = INFINITY, dmax = -INFINITY;
  int bad = 0;
  if (owner) {
    const size_t idx = (size_t)s * P.padr + i;
    if (P.kind == KIND_UPDATE) {
      float lse_new, gam_new;
      if (live) {
        lse_new = (fast ? anchor : 0.f) + (M + lg2(sum));
        gam_new = lm - lse_new;
        float dl = lse_new - lse_old;
        if (isfinite(dl)) { dmin = dl; dmax = dl; } else { bad = 1; }
        if (P.role == 0) {
          // R_i / a_i of the input state = 2^(lse_new - lse_old), formed so the
          // large terms cancel exactly before rounding
          float ratio = fast ? sum * ex2(anchor - lse_old) : sum * ex2(M - lse_old);
          rho = w * fabsf(ratio - 1.f);
        }
      } else {
        lse_new = INFINITY;
        gam_new = -INFINITY;
      }
      if (!frozen) {
        P.lse_out[idx] = lse_new;
        P.gam_out[idx] = gam_new;
      }
    } else if (live) {
      // check: terms were pi_ij / 2^lm_i, so sum * 2^M = R_i / a_i
      float ratio = sum * ex2(M);
      rho = w * fabsf(ratio - 1.f);
    }
  }
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  float r0 = wave_sum(rho), r1 = wave_min(dmin), r2 = wave_max(dmax);
  int r3 = wave_or(bad);
  if ((threadIdx.x & 63) == 0) {
    sh_red[0][wave] = r0; sh_red[1][wave] = r1; sh_red[2][wave] = r2;
    sh_red[3][wave] = (float)r3;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float4 a = make_float4(0.f, INFINITY, -INFINITY, 0.f);
    for (int w = 0; w < NWAVES; ++w) {
      a.x += sh_red[0][w];
      a.y = fminf(a.y, sh_red[1][w]);
      a.z = fmaxf(a.z, sh_red[2][w]);
      a.w = fmaxf(a.w, sh_red[3][w]);
    }
    float4* dst = P.agg_out + (size_t)si.lane * L.rbmax + rb;
    if (P.kind == KIND_UPDATE) {
      *dst = a;
      sh_last = 0;
    } else {
      if (P.role == 0 || !P.decide) {
        *dst = a;
        sh_last = 0;
      } else {
        st_dev4(dst, a);
        wait_mem();
        const int nrb = row_blocks(si.m, L.rows);
        const int prev = atomicAdd(&L.vcnt[si.lane], 1);
        sh_last = (prev == nrb - 1);
        if (sh_last) atomicExch(&L.vcnt[si.lane], 0);
      }
    }
  }
  __syncthreads();
  if (!sh_last || threadIdx.x >= 64) return;
  // last block of a checked lane: column residual and the decision
  const LaneAgg gc = lane_aggregate(P.agg_out, si.lane, L.rbmax, row_blocks(si.m, L.rows), true);
  float rrow = rhat;
  if (P.final_audit) {
    const LaneAgg gr = lane_aggregate(P.agg_rowchk, si.lane, L.rbmax, row_blocks(si.n, L.rows), false);
    rrow = gr.sum;
  }
  if (threadIdx.x != 0) return;
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

// XCD-aware item order. Consecutive workgroups are dispatched to the 8 XCDs
// in turn, so block b (x = b mod 8) takes item x*q + min(x, r) + b/8 of the
// N = 8q + r items: every XCD works through one contiguous range of items --
// whole lanes -- and its L2 holds only those lanes' column operands. The map
// is a bijection of [0, N), so it changes which block runs an item, never
// what the item computes.
__device__ __forceinline__ int xcd_item(int b, int N) {
  const int q = N >> 3, r = N & 7, x = b & 7;
  return x * q + min(x, r) + (b >> 3);
}

// Decide what block b of a pass does. Returns false when it has no work.
__device__ __forceinline__ bool locate_item(const Launch& L, const Pass& P, int b, int& s,
                                            int& rb, SlotInfo& si) {
  const Ctrl* c = L.ctrl;
  if (!P.final_audit && c->finished) return false;
  const int A = min(P.A, c->A);
  if (P.ipl > 0) {
    const int N = P.ipl * A;
    if (b >= N) return false;
    const int item = xcd_item(b, N);
    s = item / P.ipl;
    rb = item - s * P.ipl;
  } else {
    const int N = P.off[A];
    if (b >= N) return false;
    const int item = xcd_item(b, N);
    s = find_slot(P.off, A, item);
    rb = item - P.off[s];
  }
  si = L.slot[s];
  if (P.kind == KIND_UPDATE) return !(si.done && L.mode == MODE_ACTIVE);
  if (si.done) return false;
  if (!P.final_audit && si.passed) return false;
  return true;
}

// --------------------------------------------------------- MFMA half-step
// Work item = 32 rows of one lane against all its columns; wave w of the 4
// sweeps column quarter w. In every 32x32 tile the matrix core forms
// D[j][i] = sum_k A[j][k] B[k][i] over the augmented vectors
// A_j = (y~_j, gam_j, 1), B_i = (x~_i, 1, -anchor_i) (K = 2*DH + 2): D is the
// base-2 exponent of the (i, j) term minus the row anchor. Lane l holds row
// i = l % 32 for 16 columns, so the streaming sum over j stays inside the
// lane; half-waves and then the four column quarters are merged (LDS) in a
// fixed order. The next tile's operands load while the current tile reduces.
template <int DH>
__global__ __launch_bounds__(256, (DH <= 7 ? 8 : (DH <= 12 ? 6 : 4))) void k_update_mfma(Launch L) {
  __shared__ float2 sh_part[kColGroups][kRowsMfma];
  const int b = blockIdx.x;
  const int pi = b >= L.nb0;
  const Pass P = pi ? L.p[1] : L.p[0];
  int s, rb;
  SlotInfo si;
  if (!locate_item(L, P, pi ? b - L.nb0 : b, s, rb, si)) return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  if (!upd && !check_facts(L, P, si, rhat)) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  const int h = lane >> 5;
  const int r = lane & 31;
  const int nrows = P.role ? si.m : si.n;
  const int ncols = P.role ? si.n : si.m;
  const int i = rb * kRowsMfma + r;
  constexpr int DP = 2 * DH;

  // Every load of the item (row data, first column tile) is issued before the
  // update facts are reduced, so their latencies overlap.
  const size_t ridx = (size_t)s * P.padr + i;
  const float lse_old = P.lse_in[ridx];
  const float lm = P.lm_row[ridx];
  const bool in_prefix = i < nrows;
  const float w = in_prefix ? P.w_row[(size_t)si.lane * P.w_ld + i] : 0.f;
  float bv[DH + 1];
  const float* rrow = P.rec_row + ridx * DP + h * DH;
#pragma unroll
  for (int k = 0; k < DH; ++k) bv[k] = rrow[k];

  const int ct = (ncols + kColTile - 1) / kColTile;
  const int tpg = (ct + kColGroups - 1) / kColGroups;
  const int t0 = wave * tpg;
  const int t1 = min(ct, t0 + tpg);
  const float* ccol = P.rec_col + (size_t)s * P.padc * DP + h * DH + (size_t)r * DP;
  const float* gcol = P.gam_col + (size_t)s * P.padc + r;
  auto load = [&](int t, float* a) {
    const float* c = ccol + (size_t)t * kColTile * DP;
#pragma unroll
    for (int k = 0; k < DH; ++k) a[k] = c[k];
    a[DH] = gcol[(size_t)t * kColTile];
  };
  float A0[DH + 1], A1[DH + 1];
  if (t0 < t1) load(t0, A0);

  bool fast = false;
  float M = 0.f;
  if (upd) update_facts(L, P, si, fast, M);
  const bool live = in_prefix && (lse_old != INFINITY);
  float anchor = 0.f, bias = 0.f;
  if (live) {
    if (!upd) bias = -lse_old;
    else if (fast) { anchor = lse_old + M; bias = -anchor; }
  }
  bv[DH] = h ? bias : 1.f;

  float mrun = fast ? 0.f : -INFINITY, srun = 0.f;
  auto tile = [&](const float* a, bool anchored) {
    f32x16 acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < DH; ++k) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[k], bv[k], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(h ? 1.f : a[DH], bv[DH], acc, 0, 0, 0);
    float e[16];
    if (anchored) {
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = ex2(acc[v]);
#pragma unroll
      for (int w = 8; w > 0; w >>= 1)
#pragma unroll
        for (int v = 0; v < w; ++v) e[v] += e[v + w];
      srun += e[0];
    } else {
      float tm = acc[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) tm = fmaxf(tm, acc[v]);
      const float mn = fmaxf(mrun, tm);
      const float mref = (mn == -INFINITY) ? 0.f : mn;
#pragma unroll
      for (int v = 0; v < 16; ++v) e[v] = ex2(acc[v] - mref);
#pragma unroll
      for (int w = 8; w > 0; w >>= 1)
#pragma unroll
        for (int v = 0; v < w; ++v) e[v] += e[v + w];
      srun = srun * ex2(mrun - mref) + e[0];
      mrun = mn;
    }
  };
  // operand ping-pong: tile t+1 is in flight while tile t is reduced; the
  // prefetch index is clamped so every load stays in range
  auto sweep = [&](bool anchored) {
    if (t0 >= t1) return;
    int t = t0;
    for (; t + 1 < t1; t += 2) {
      load(t + 1, A1);
      tile(A0, anchored);
      load(min(t + 2, t1 - 1), A0);
      tile(A1, anchored);
    }
    if (t < t1) tile(A0, anchored);
  };
  if (fast) sweep(true); else sweep(false);
  // merge the two half-waves (same rows, different columns) in a canonical
  // order so both halves hold identical bits
  const float mo = __shfl_xor(mrun, 32, 64);
  const float so_ = __shfl_xor(srun, 32, 64);
  const float mA = h ? mo : mrun, sA = h ? so_ : srun;
  const float mB = h ? mrun : mo, sB = h ? srun : so_;
  const float Mw = fmaxf(mA, mB);              // -inf only if both halves are empty
  const float mref = (Mw == -INFINITY) ? 0.f : Mw;
  const float Sw = sA * ex2(mA - mref) + sB * ex2(mB - mref);
  if (h == 0) sh_part[wave][r] = make_float2(Mw, Sw);
  __syncthreads();
  // merge the column quarters in order (wave 0 owns the rows)
  const bool owner = (wave == 0) && (h == 0);
  float Mt = 0.f, St = 0.f;
  if (owner) {
    float mx = -INFINITY;
#pragma unroll
    for (int g = 0; g < kColGroups; ++g) mx = fmaxf(mx, sh_part[g][r].x);
    Mt = (mx == -INFINITY) ? 0.f : mx;
#pragma unroll
    for (int g = 0; g < kColGroups; ++g) St += sh_part[g][r].y * ex2(sh_part[g][r].x - Mt);
  }
  finish_block<4>(L, P, s, si, rb, i, owner, live, fast, anchor, lse_old, lm, w, Mt, St, rhat);
}

// --------------------------------------------------------- VALU half-step
// Work item = 64 rows (one per lane) of one lane against all its columns;
// wave w sweeps column quarter w. The column data of a tile is the same for
// every lane (wave-uniform), so it is read through the scalar path and used
// as SGPR operands: per (i, j) term one subtract, D fused multiply-adds, one
// v_exp_f32 and one add. Column quarters are merged in LDS in a fixed order.
template <int D, int DH>
__global__ __launch_bounds__(256, 8) void k_update_valu(Launch L) {
  __shared__ float2 sh_part[kColGroups][kRowsValu];
  const int b = blockIdx.x;
  const int pi = b >= L.nb0;
  const Pass P = pi ? L.p[1] : L.p[0];
  int s, rb;
  SlotInfo si;
  if (!locate_item(L, P, pi ? b - L.nb0 : b, s, rb, si)) return;
  const bool upd = P.kind == KIND_UPDATE;
  float rhat = NAN;
  if (!upd && !check_facts(L, P, si, rhat)) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform (SGPR)
  const int nrows = P.role ? si.m : si.n;
  const int ncols = P.role ? si.n : si.m;
  const int i = rb * kRowsValu + lane;
  constexpr int DP = 2 * DH;
  // row loads are issued before the update facts are reduced
  const size_t ridx = (size_t)s * P.padr + i;
  const float lse_old = P.lse_in[ridx];
  const float lm = P.lm_row[ridx];
  const bool in_prefix = i < nrows;
  const float w = in_prefix ? P.w_row[(size_t)si.lane * P.w_ld + i] : 0.f;
  float xr[D];
  const float* rrow = P.rec_row + ridx * DP;
#pragma unroll
  for (int k = 0; k < D; ++k) xr[k] = rrow[k];
  bool fast = false;
  float M = 0.f;
  if (upd) update_facts(L, P, si, fast, M);
  const bool live = in_prefix && (lse_old != INFINITY);
  float anchor = 0.f, bias = 0.f;
  if (live) {
    if (!upd) bias = -lse_old;
    else if (fast) { anchor = lse_old + M; bias = -anchor; }
  }

  const int ct = (ncols + kColTile - 1) / kColTile;
  const int tpg = (ct + kColGroups - 1) / kColGroups;
  const int j0 = min(ct, wave * tpg) * kColTile;
  const int j1 = min(ct, wave * tpg + tpg) * kColTile;
  const float* __restrict__ ccol = P.rec_col + (size_t)s * P.padc * DP;
  const float* __restrict__ gcol = P.gam_col + (size_t)s * P.padc;

  float mrun = -INFINITY, srun = 0.f;
  if (fast) {
    float sacc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int j = j0; j < j1; j += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* cj = ccol + (size_t)(j + u) * DP;
        float z = gcol[j + u] + bias;
#pragma unroll
        for (int k = 0; k < D; ++k) z = fmaf(xr[k], cj[k], z);
        sacc[u] += ex2(z);
      }
    }
    srun = (sacc[0] + sacc[1]) + (sacc[2] + sacc[3]);
    mrun = 0.f;
  } else {
    for (int j = j0; j < j1; j += 8) {
      float z[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float* cj = ccol + (size_t)(j + u) * DP;
        float zz = gcol[j + u] + bias;
#pragma unroll
        for (int k = 0; k < D; ++k) zz = fmaf(xr[k], cj[k], zz);
        z[u] = zz;
      }
      float tm = z[0];
#pragma unroll
      for (int u = 1; u < 8; ++u) tm = fmaxf(tm, z[u]);
      const float mn = fmaxf(mrun, tm);
      const float mref = (mn == -INFINITY) ? 0.f : mn;
      float e[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) e[u] = ex2(z[u] - mref);
      const float ts = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
      srun = srun * ex2(mrun - mref) + ts;
      mrun = mn;
    }
  }
  sh_part[wave][lane] = make_float2(mrun, srun);   // (-inf, 0) for an empty quarter
  __syncthreads();
  const bool owner = (wave == 0);
  float Mt = 0.f, St = 0.f;
  if (owner) {
    float mx = -INFINITY;
#pragma unroll
    for (int g = 0; g < kColGroups; ++g) mx = fmaxf(mx, sh_part[g][lane].x);
    Mt = (mx == -INFINITY) ? 0.f : mx;
#pragma unroll
    for (int g = 0; g < kColGroups; ++g) St += sh_part[g][lane].y * ex2(sh_part[g][lane].x - Mt);
  }
  finish_block<4>(L, P, s, si, rb, i, owner, live, fast, anchor, lse_old, lm, w, Mt, St, rhat);
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
  int f_off = block_exclusive_scan(items_f, sh, tot_f);
  int g_off = block_exclusive_scan(items_g, sh, tot_g);
  for (int c = 0; c < C; ++c) {
    const int s = base + c;
    if (s >= A) break;
    const SlotInfo si = p.slot[s];
    if (!si.done) {
      const int ns = surv_off++;
      p.dec[s].new_slot = ns;
      p.off_f[ns] = f_off;
      p.off_g[ns] = g_off;
      f_off += row_blocks(si.n, p.rows);
      g_off += row_blocks(si.m, p.rows);
    } else {
      p.dec[s].new_slot = -1;
    }
  }
  __syncthreads();
  for (int s = tot_surv + (int)threadIdx.x; s <= p.W; s += blockDim.x) {
    p.off_f[s] = tot_f;
    p.off_g[s] = tot_g;
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
__global__ __launch_bounds__(1024) void k_offsets(SlotInfo* slot, int A, int rows, int* off_f,
                                                  int* off_g, Ctrl* ctrl) {
  __shared__ int sh[32];
  const int C = (A + 1023) / 1024;
  const int base = threadIdx.x * C;
  int nf = 0, ng = 0;
  for (int c = 0; c < C; ++c) {
    const int s = base + c;
    if (s >= A) break;
    nf += row_blocks(slot[s].n, rows);
    ng += row_blocks(slot[s].m, rows);
  }
  int tf, tg;
  int of = block_exclusive_scan(nf, sh, tf);
  int og = block_exclusive_scan(ng, sh, tg);
  for (int c = 0; c < C; ++c) {
    const int s = base + c;
    if (s >= A) break;
    off_f[s] = of; off_g[s] = og;
    of += row_blocks(slot[s].n, rows);
    og += row_blocks(slot[s].m, rows);
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
    const float inv_k = 1.f / si.kappa;
    const int par = p.emit_all ? p.final_par : (d.depth & 1);
    for (int side = 0; side < 2; ++side) {
      const int lim = side ? p.m_max : p.n_max;
      const int cnt = side ? si.m : si.n;
      const int padn = p.pad[side];
      float* out = side ? p.g : p.f;
      const float* gam = p.src.gam[side][par] + (size_t)s * padn;
      const float* rec = p.src.rec[side] + (size_t)s * padn * p.dp;
      for (int q = c0 + threadIdx.x; q < min(lim, c0 + p.chunk); q += blockDim.x) {
        float v = 0.f;
        if (q < cnt) {
          const float gq = gam[q];
          if (gq != -INFINITY) {
            float nrm = 0.f;
            for (int k = 0; k < p.dp; ++k) { float x = rec[(size_t)q * p.dp + k]; nrm = fmaf(x, x, nrm); }
            v = (gq + 0.5f * nrm) * inv_k;
          }
        }
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
    const int ns = d.new_slot;
    for (int side = 0; side < 2; ++side) {
      const int padn = p.pad[side];
      const int lim = min(padn, c0 + p.chunk);
      const size_t so = (size_t)s * padn, dn = (size_t)ns * padn;
      for (int q = c0 + threadIdx.x; q < lim; q += blockDim.x) {
        p.dst.lm[side][dn + q] = p.src.lm[side][so + q];
        for (int par = 0; par < 2; ++par) {
          p.dst.lse[side][par][dn + q] = p.src.lse[side][par][so + q];
          p.dst.gam[side][par][dn + q] = p.src.gam[side][par][so + q];
        }
      }
      // records: contiguous [pad][dp] floats per slot
      const float4* rs = reinterpret_cast<const float4*>(p.src.rec[side] + so * p.dp);
      float4* rd = reinterpret_cast<float4*>(p.dst.rec[side] + dn * p.dp);
      const int q0 = c0 * p.dp / 4, q1 = lim * p.dp / 4;
      for (int q = q0 + threadIdx.x; q < q1; q += blockDim.x) rd[q] = rs[q];
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      p.dst.slot[ns] = si;
      p.dst.dec[ns] = d;
    }
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
  // centre: mean of live source points and mean of live target points,
  // averaged; fixed-order double reduction
  __shared__ double sh[256];
  auto reduce = [&](double v) -> double {
    sh[threadIdx.x] = v;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w) sh[threadIdx.x] += sh[threadIdx.x + w];
      __syncthreads();
    }
    double r = sh[0];
    __syncthreads();
    return r;
  };
  double cntx = 0.0, cnty = 0.0;
  for (int i = threadIdx.x; i < nt; i += blockDim.x) cntx += (p.a[(size_t)t * p.n_max + i] != 0.f);
  for (int j = threadIdx.x; j < mt; j += blockDim.x) cnty += (p.b[(size_t)t * p.m_max + j] != 0.f);
  const double nx = reduce(cntx), ny = reduce(cnty);
  for (int k = 0; k < p.d; ++k) {
    double sx = 0.0, sy = 0.0;
    for (int i = threadIdx.x; i < nt; i += blockDim.x)
      if (p.a[(size_t)t * p.n_max + i] != 0.f) sx += p.X[((size_t)t * p.n_max + i) * p.d + k];
    for (int j = threadIdx.x; j < mt; j += blockDim.x)
      if (p.b[(size_t)t * p.m_max + j] != 0.f) sy += p.Y[((size_t)t * p.m_max + j) * p.d + k];
    const double rx = reduce(sx), ry = reduce(sy);
    const double mx = nx > 0 ? rx / nx : 0.0, my = ny > 0 ? ry / ny : 0.0;
    if (threadIdx.x == 0) p.center[(size_t)t * p.d + k] = (float)(0.5 * (mx + my));
  }
  if (threadIdx.x == 0) {
    SlotInfo si;
    si.lane = t; si.n = nt; si.m = mt; si.done = 0; si.passed = 0;
    si.kappa = (float)(1.4426950408889634 / (double)e);
    si.bx_ok = 0; si.by_ok = 0;
    si.bx_min = si.bx_max = si.by_min = si.by_max = 0.f;
    si.pad = 0;
    p.bank.slot[t] = si;
    Decision d;
    d.status = 1; d.depth = 0; d.res_row = NAN; d.res_col = NAN; d.new_slot = -1;
    d.pad[0] = d.pad[1] = d.pad[2] = 0;
    p.bank.dec[t] = d;
    p.vcnt[t] = 0;
    p.nchk[t] = 0;
  }
  // no previous half-step: the first update of each side runs unanchored
  const float4 none = make_float4(0.f, INFINITY, -INFINITY, 1.f);
  for (int q = threadIdx.x; q < p.rbmax; q += blockDim.x)
    for (int k = 0; k < 4; ++k) p.agg[k][(size_t)t * p.rbmax + q] = none;
}

// Grid (chunks, W): points of both sides of lane t.
__global__ __launch_bounds__(256) void k_ingest_points(IngestArgs p, int chunk) {
  const int t = blockIdx.y;
  if (p.ctrl->err_lane != 0x7fffffff) return;
  const SlotInfo si = p.bank.slot[t];
  const double sigma = sqrt(2.0 * (double)si.kappa);
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
      float* rec = p.bank.rec[side] + idx * p.dp;
      const float mass = (q < cnt) ? w[(size_t)t * ld + q] : 0.f;
      const bool live = (q < cnt) && (mass != 0.f);
      float nrm = 0.f;
      if (live) {
        for (int k = 0; k < p.d; ++k) {
          const double v = sigma * ((double)P[((size_t)t * ld + q) * p.d + k] - (double)c[k]);
          const float fv = (float)v;
          // de-interleaved: even components first, then odd ones
          const int pos = (k & 1) ? (p.dh + (k >> 1)) : (k >> 1);
          rec[pos] = fv;
          nrm = fmaf(fv, fv, nrm);
        }
        if (p.d & 1) rec[p.dp - 1] = 0.f;
      } else {
        for (int k = 0; k < p.dp; ++k) rec[k] = 0.f;
      }
      const float lm = live ? (float)log2((double)mass) : -INFINITY;
      p.bank.lm[side][idx] = lm;
      for (int par = 0; par < 2; ++par) {
        if (!live) {
          p.bank.lse[side][par][idx] = INFINITY;
          p.bank.gam[side][par][idx] = -INFINITY;
        } else if (side == 0) {
          // no f^0 exists: the first f-half runs unanchored
          p.bank.lse[0][par][idx] = NAN;
          p.bank.gam[0][par][idx] = NAN;
        } else {
          // cold start g^0 = 0  =>  gam^y = -kappa |y - c|^2 = -|y~|^2 / 2
          const float gam0 = -0.5f * nrm;
          p.bank.gam[1][par][idx] = gam0;
          p.bank.lse[1][par][idx] = lm - gam0;
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
    z.retire_events = 0; z.compacted = 0; z.A_prev = W; z.pad2 = 0;
    *c = z;
  }
}

// ------------------------------------------------------- host-side launchers
template <int DH>
static hipError_t launch_mfma_dh(const Launch& a, int blocks, hipStream_t st) {
  hipLaunchKernelGGL(k_update_mfma<DH>, dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}
template <int D>
static hipError_t launch_valu_d(const Launch& a, int blocks, hipStream_t st) {
  hipLaunchKernelGGL((k_update_valu<D, (D + 1) / 2>), dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace ds

// Entry points used by the host runtime (C++ linkage, same library).
namespace ds {
hipError_t launch_update(const Launch& a, int d, bool use_mfma, int blocks, hipStream_t st) {
  if (blocks <= 0) return hipSuccess;
  const int dh = (d + 1) / 2;
  if (use_mfma) {
    switch (dh) {
      case 1: return launch_mfma_dh<1>(a, blocks, st);
      case 2: return launch_mfma_dh<2>(a, blocks, st);
      case 3: return launch_mfma_dh<3>(a, blocks, st);
      case 4: return launch_mfma_dh<4>(a, blocks, st);
      case 5: return launch_mfma_dh<5>(a, blocks, st);
      case 6: return launch_mfma_dh<6>(a, blocks, st);
      case 7: return launch_mfma_dh<7>(a, blocks, st);
      case 8: return launch_mfma_dh<8>(a, blocks, st);
      case 9: return launch_mfma_dh<9>(a, blocks, st);
      case 10: return launch_mfma_dh<10>(a, blocks, st);
      case 11: return launch_mfma_dh<11>(a, blocks, st);
      case 12: return launch_mfma_dh<12>(a, blocks, st);
      case 13: return launch_mfma_dh<13>(a, blocks, st);
      case 14: return launch_mfma_dh<14>(a, blocks, st);
      case 15: return launch_mfma_dh<15>(a, blocks, st);
      case 16: return launch_mfma_dh<16>(a, blocks, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (d) {
    case 1: return launch_valu_d<1>(a, blocks, st);
    case 2: return launch_valu_d<2>(a, blocks, st);
    case 3: return launch_valu_d<3>(a, blocks, st);
    case 4: return launch_valu_d<4>(a, blocks, st);
    case 5: return launch_valu_d<5>(a, blocks, st);
    case 6: return launch_valu_d<6>(a, blocks, st);
    case 7: return launch_valu_d<7>(a, blocks, st);
    case 8: return launch_valu_d<8>(a, blocks, st);
    case 9: return launch_valu_d<9>(a, blocks, st);
    case 10: return launch_valu_d<10>(a, blocks, st);
    case 11: return launch_valu_d<11>(a, blocks, st);
    case 12: return launch_valu_d<12>(a, blocks, st);
    case 13: return launch_valu_d<13>(a, blocks, st);
    case 14: return launch_valu_d<14>(a, blocks, st);
    case 15: return launch_valu_d<15>(a, blocks, st);
    case 16: return launch_valu_d<16>(a, blocks, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_scan(const ScanArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}
hipError_t launch_offsets(SlotInfo* slot, int A, int rows, int* off_f, int* off_g, Ctrl* ctrl,
                          hipStream_t st) {
  hipLaunchKernelGGL(k_offsets, dim3(1), dim3(1024), 0, st, slot, A, rows, off_f, off_g, ctrl);
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
