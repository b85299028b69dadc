// The one-wave swap planner and the helpers it shares with the workgroup planner (fb_plan_device.hip).
// The one-wave planner also runs inside the predictor's last workgroup (fb_predict.hip), right after
// the counts are complete, so it synchronises its lanes with wave barriers and takes its LDS from
// the caller.  Same algorithm and tie-breaks as the host planner (Sec. "Budgeted Expert-Swap
// Planning", Eq. 6-8, Alg. 1).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fb_internal.h"

namespace fb {
namespace {

constexpr int kMaxRS = FB_MAX_SLOTS_TOTAL;
constexpr int kMaxR = FB_MAX_RANKS;
constexpr int kRankBits = 11;                 // R <= 1024 < 2^11
constexpr int kItemBits = 21;                 // item ids < V + R * S <= 2^21 (checked)
constexpr int kSmallItemBits = 13;            // ... < E + R * S <= 8192 without replicas
constexpr int64_t kLoadCap = (int64_t)1 << 43;  // loads <= 4096 experts * (2^31 - 1) < 2^43

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, 0xF, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, 0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Maximum over the 64 lanes of a wave (every lane must be active); uniform result.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  v = umax64(v, dpp_u64<0xB1>(v));    // quad_perm [1,0,3,2]
  v = umax64(v, dpp_u64<0x4E>(v));    // quad_perm [2,3,0,1]
  v = umax64(v, dpp_u64<0x141>(v));   // row_half_mirror
  v = umax64(v, dpp_u64<0x140>(v));   // row_mirror
  return umax64(umax64(readlane_u64(v, 0), readlane_u64(v, 16)),
                umax64(readlane_u64(v, 32), readlane_u64(v, 48)));
}

// (load, rank) keys: the largest key is the largest load, lowest rank id on ties.
__device__ __forceinline__ uint64_t key_max(int64_t load, int r) {
  return ((uint64_t)load << kRankBits) | (uint64_t)((1 << kRankBits) - 1 - r);
}
// ... and the smallest load, lowest rank id on ties.
__device__ __forceinline__ uint64_t key_min(int64_t load, int r) {
  return ((uint64_t)(kLoadCap - load) << kRankBits) | (uint64_t)((1 << kRankBits) - 1 - r);
}
__device__ __forceinline__ int key_rank(uint64_t key) {
  return (1 << kRankBits) - 1 - (int)(key & ((1u << kRankBits) - 1));
}

// Barrier of the planner's NT threads.  One wave (NT = 64) needs only ordered LDS accesses and a
// wave barrier, so the one-wave planner also runs in a workgroup whose other waves have left.
template <int NT>
__device__ __forceinline__ void plan_sync() {
  if constexpr (NT == 64) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
  } else {
    __syncthreads();
  }
}

// Exclusive prefix sum of v over the NT threads of the workgroup (every thread calls it; wsum holds
// NT / 64 entries): shuffles within each wave, then the totals of the waves before.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int32_t* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if constexpr (NT > 64) {
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    for (int u = 0; u < w; ++u) x += wsum[u];
  }
  return x - v;
}

// Placement check of both kernels (all NT threads of the workgroup call it) on the slot values and
// counts the caller has put in LDS (vals[R * S], cnt[E]; *bad zeroed; all published by the first
// barrier here): every value is -1 or e + E * j with j < R, every expert has replicas 0 .. c_e - 1
// each once, no rank holds two replicas of one expert, every count is >= 0.  A violation sets bit
// 0 of *bad.  On return, after a barrier, reps[e] = c_e, *jmax = the largest c_e, and ej[c] =
// (j << 12) | e for the replica in slot c (-1 for an empty or invalid slot; E <= 4096).
template <int NT>
__device__ void check_placement(int E, int R, int S, const int32_t* vals, const int32_t* cnt,
                                int32_t* ej, int32_t* reps, int32_t* base, int32_t* flag,
                                int32_t* wsum, int32_t* bad, int32_t* jmax) {
  const int tid = threadIdx.x;
  const int RS = R * S;
  for (int e = tid; e < E; e += NT) reps[e] = 0;
  for (int c = tid; c < RS; c += NT) flag[c] = 0;
  if (tid == 0) *jmax = 1;
  plan_sync<NT>();
  for (int c = tid; c < RS; c += NT) {
    const int v = vals[c];
    int x = -1;
    if (v < -1 || v >= E * R) {
      atomicOr(bad, 1);
    } else if (v >= 0) {
      const int j = v / E, e = v - j * E;       // the only division per slot
      x = (j << 12) | e;
      atomicAdd(&reps[e], 1);
    }
    ej[c] = x;
  }
  plan_sync<NT>();
  // exclusive prefix sum of reps over contiguous chunks of experts
  const int chunk = (E + NT - 1) / NT;
  const int e0 = tid * chunk, e1 = e0 + chunk < E ? e0 + chunk : E;
  int acc = 0, jm = 1;
  for (int e = e0; e < e1; ++e) acc += reps[e];
  acc = block_exclusive_scan<NT>(acc, wsum);
  for (int e = e0; e < e1; ++e) {
    base[e] = acc;
    acc += reps[e];
    if (reps[e] == 0 || cnt[e] < 0) atomicOr(bad, 1);
    jm = reps[e] > jm ? reps[e] : jm;
  }
  atomicMax(jmax, jm);
  plan_sync<NT>();
  for (int c = tid; c < RS; c += NT) {
    const int x = ej[c];
    if (x < 0) continue;                         // empty, or flagged above
    const int e = x & 4095, j = x >> 12;
    // base[e] + j < base[e] + reps[e] <= R * S only when j < reps[e]; the entry records the
    // replica's rank + 1, and a second replica with the same ordinal finds it taken
    if (j >= reps[e] || atomicCAS(&flag[base[e] + j], 0, c / S + 1) != 0) atomicOr(bad, 1);
  }
  plan_sync<NT>();
  // no rank holds two replicas of one expert.  Every slot of a pair takes the same branch (it
  // depends on the expert only): with few replicas the later ordinal finds the earlier one's rank
  // among the entries recorded above, otherwise the later slot finds the earlier one on its rank;
  // either way a slot reads at most min(c_e, S) words
  for (int c = tid; c < RS; c += NT) {
    const int x = ej[c];
    if (x < 0) continue;
    const int e = x & 4095, j = x >> 12, k = reps[e];
    if (j >= k) continue;                        // flagged above
    if (k <= S) {
      const int b = base[e], me = c / S + 1;
      for (int w = 0; w < j; ++w)
        if (flag[b + w] == me) atomicOr(bad, 1);
    } else {
      for (int c2 = (c / S) * S; c2 < c; ++c2) {
        const int x2 = ej[c2];
        if (x2 >= 0 && (x2 & 4095) == e) atomicOr(bad, 1);
      }
    }
  }
  plan_sync<NT>();
}

// Expert of the replica id it (it mod E) for 0 <= it < 2^21 and 1 <= E <= 4096, with no integer
// division: the float quotient is within 0.25 of it / E (both roundings are below 2^-24 relative),
// so the truncated estimate is off by at most one, which one correction of the remainder settles.
__device__ __forceinline__ int expert_of(int it, int E, float inv_e) {
  const int q = (int)((float)it * inv_e);
  int r = it - q * E;
  if (r < 0) r += E;
  else if (r >= E) r -= E;
  return r;
}

// Token share of the replica x = (j << 12) | e (as check_placement leaves it; j < c_e).
__device__ __forceinline__ int32_t replica_share(int x, const int32_t* counts, const int32_t* reps) {
  const int e = x & 4095, j = x >> 12;
  const int n = counts[e], k = reps[e];
  if (k == 1) return n;
  return n / k + (j < n % k ? 1 : 0);
}
// ---- time budget: costs and the benefit / cost order (both planners) -------------------------
// ceil(num / beta) for 0 <= num < 2^52 and 1 <= beta <= 2^40, exactly: a double-precision
// quotient is within one of the truncated one (its relative error is below 2^-51), and one
// integer correction step settles it.
__device__ __forceinline__ int64_t ceil_div(int64_t num, int64_t beta, double inv_beta) {
  int64_t q = (int64_t)((double)num * inv_beta);
  int64_t r = num - q * beta;
  if (r < 0) { q -= 1; r += beta; }
  if (r >= beta) { q += 1; r -= beta; }
  return q + (r > 0 ? 1 : 0);
}

// (gain, cost, tie) ordering of the time-budgeted planner; gain 0 means "no candidate".
__device__ __forceinline__ bool ratio_better(uint64_t g1, uint64_t c1, uint64_t t1, uint64_t g2,
                                             uint64_t c2, uint64_t t2) {
  if (g1 == 0) return false;
  if (g2 == 0) return true;
  // the products in double precision decide unless they are within 2^-30 of each other (their
  // relative rounding error is below 2^-51); only then the exact 128-bit products are formed
  const double ld = (double)g1 * (double)c2, rd = (double)g2 * (double)c1;
  const double tol = 0x1p-30 * (ld > rd ? ld : rd);
  if (ld - rd > tol) return true;
  if (rd - ld > tol) return false;
  const unsigned __int128 l = (unsigned __int128)g1 * c2, r = (unsigned __int128)g2 * c1;
  if (l != r) return l > r;
  return t1 < t2;
}

// One step of the time-budgeted reduction (the better (gain, cost, tie) by ratio_better) with the
// lane that DPP control CTRL names.
template <int CTRL>
__device__ __forceinline__ void ratio_step(uint64_t& g, uint64_t& c, uint64_t& t) {
  const uint64_t g2 = dpp_u64<CTRL>(g), c2 = dpp_u64<CTRL>(c), t2 = dpp_u64<CTRL>(t);
  if (ratio_better(g2, c2, t2, g, c, t)) { g = g2; c = c2; t = t2; }
}

// Best (gain, cost, tie) of the wave by ratio_better (every lane takes part; uniform result): each
// row of 16 lanes by DPP (lane ^ 1, lane ^ 2, the mirror within 8 lanes, the mirror within 16),
// then the four rows.
__device__ __forceinline__ void wave_best_ratio(uint64_t& g, uint64_t& c, uint64_t& t) {
  ratio_step<0xB1>(g, c, t);
  ratio_step<0x4E>(g, c, t);
  ratio_step<0x141>(g, c, t);
  ratio_step<0x140>(g, c, t);
  uint64_t bg = readlane_u64(g, 0), bc = readlane_u64(c, 0), bt = readlane_u64(t, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const uint64_t og = readlane_u64(g, 16 * r), oc = readlane_u64(c, 16 * r), ot = readlane_u64(t, 16 * r);
    if (ratio_better(og, oc, ot, bg, bc, bt)) { bg = og; bc = oc; bt = ot; }
  }
  g = bg; c = bc; t = bt;
}

// ---- one-wave frontier planner ------------------------------------------------------------------
constexpr uint32_t kMovedBit = 0x80000000u;

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  v += dpp_u64<0xB1>(v);
  v += dpp_u64<0x4E>(v);
  v += dpp_u64<0x141>(v);
  v += dpp_u64<0x140>(v);
  return readlane_u64(v, 0) + readlane_u64(v, 16) + readlane_u64(v, 32) + readlane_u64(v, 48);
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
  return max(max((uint32_t)__builtin_amdgcn_readlane((int)v, 0), (uint32_t)__builtin_amdgcn_readlane((int)v, 16)),
             max((uint32_t)__builtin_amdgcn_readlane((int)v, 32), (uint32_t)__builtin_amdgcn_readlane((int)v, 48)));
}

// Rounds of the one-wave planner when every rank sits in its own lane (R <= 64), every load fits
// 31 bits and there are no replicas (item ids below E + R * S <= 8192): loads, extremes and tie keys
// are 32-bit, rank ties are resolved by the lowest lane of a
// ballot, and the tie key reduction runs only when two candidates share the best benefit.
// Returns the number of swaps written.
// CPL: candidates per lane (1 when S * S <= 64, else 2).
template <int CPL>
__device__ __forceinline__ int rounds_small(const PlanDeviceLaunch& a, uint2* slot, int32_t* part,
                                            uint32_t& Lu, int64_t g_num, int64_t g_den) {
  const int lane = threadIdx.x;
  const int E = a.E, R = a.R, S = a.S;
  const fb_budget bg = a.budget;
  const bool valid = lane < R;
  // candidates (p, q) = (c / S, c mod S) for c = lane (+ 64)
  int pc[CPL], qc[CPL];
  bool hc[CPL];
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int c = lane + 64 * h;
    hc[h] = c < S * S;
    pc[h] = hc[h] ? c / S : 0;
    qc[h] = hc[h] ? c - pc[h] * S : 0;
  }
  const bool capped = bg.per_rank_cap != 0;
  constexpr uint32_t kMoved = 0x80000000u;
  int ns = 0;
  for (int round = 0; round < bg.max_swaps; ++round) {
    const uint32_t M32 = wave_max_u32(valid ? Lu : 0u);
    const uint32_t Lmin32 = ~wave_max_u32(valid ? ~Lu : 0u);
    const int amax = (int)__builtin_ctzll(__ballot(valid && Lu == M32));
    const int amin = (int)__builtin_ctzll(__ballot(valid && Lu == Lmin32));
    const int64_t M = M32, Lmin = Lmin32;
    if (M - Lmin <= bg.tau) break;
    const uint32_t ko = wave_max_u32(valid && lane != amax && lane != amin ? Lu + 1u : 0u);
    const int64_t other = ko ? (int64_t)ko - 1 : INT64_MIN;

    // this lane's better candidate: larger benefit, then smaller (i, j)
    bool ok = false;
    int64_t gain = 0;
    uint32_t tk = 0;
    uint2 ea = {0u, 0u}, eb = {0u, 0u};
    int pl = 0, ql = 0;
    const bool cap_hit = capped && (part[amax] >= bg.per_rank_cap || part[amin] >= bg.per_rank_cap);
    auto eval = [&](int p, int q, uint2& xa, uint2& xb, int64_t& gh, uint32_t& th) -> bool {
      xa = slot[amax * S + p];
      xb = slot[amin * S + q];
      const uint32_t i = xa.x & ~kMoved, j = xb.x & ~kMoved;
      const int64_t d = (int64_t)(int32_t)xb.y - (int64_t)(int32_t)xa.y;
      const int64_t la = M + d, lb = Lmin - d;
      int64_t m2 = la > lb ? la : lb;
      if (other > m2) m2 = other;
      const int64_t spread = g_num ? g_num * (2 * d * (Lmin - M - d)) : 0;
      gh = g_den * (M - m2) + spread;
      th = (i << kSmallItemBits) | j;
      return !cap_hit && !((xa.x | xb.x) & kMoved) && !(i >= (uint32_t)E && j >= (uint32_t)E) && gh > 0;
    };
    if constexpr (CPL == 1) {
      if (hc[0]) {
        ok = eval(pc[0], qc[0], ea, eb, gain, tk);
        pl = pc[0];
        ql = qc[0];
      }
    } else {
#pragma unroll
      for (int h = 0; h < CPL; ++h) {
        if (!hc[h]) continue;
        uint2 xa, xb;
        int64_t gh;
        uint32_t th;
        const bool okh = eval(pc[h], qc[h], xa, xb, gh, th);
        if (okh && (!ok || gh > gain || (gh == gain && th < tk))) {
          ok = true; gain = gh; tk = th; ea = xa; eb = xb; pl = pc[h]; ql = qc[h];
        }
      }
    }
    // largest benefit as two 32-bit reductions, then the smallest (i, j) among equal benefits
    const uint32_t ghi = wave_max_u32(ok ? (uint32_t)((uint64_t)gain >> 32) : 0u);
    const uint32_t glo = wave_max_u32(ok && (uint32_t)((uint64_t)gain >> 32) == ghi ? (uint32_t)gain : 0u);
    const uint64_t g = ((uint64_t)ghi << 32) | glo;
    if (g == 0) break;                          // no admissible candidate with positive benefit
    const bool best = ok && (uint64_t)gain == g;
    uint64_t win = __ballot(best);
    if (__builtin_popcountll(win) > 1) {
      const uint32_t tmin = ~wave_max_u32(best ? ~tk : 0u);
      win = __ballot(best && tk == tmin);
    }
    const int wl = (int)__builtin_ctzll(win);
    const int wp = __builtin_amdgcn_readlane(pl, wl), wq = __builtin_amdgcn_readlane(ql, wl);
    const uint32_t wi = (uint32_t)__builtin_amdgcn_readlane((int)(ea.x & ~kMoved), wl);
    const uint32_t wj = (uint32_t)__builtin_amdgcn_readlane((int)(eb.x & ~kMoved), wl);
    const int32_t ci = __builtin_amdgcn_readlane((int)ea.y, wl), cj = __builtin_amdgcn_readlane((int)eb.y, wl);
    const int32_t d = cj - ci;
    if (lane == 0) {
      slot[amax * S + wp] = make_uint2(wj | kMoved, (uint32_t)cj);
      slot[amin * S + wq] = make_uint2(wi | kMoved, (uint32_t)ci);
      ++part[amax];
      ++part[amin];
      fb_swap sw;
      sw.src_rank = amax; sw.dst_rank = amin; sw.src_slot = wp; sw.dst_slot = wq;
      sw.expert_src = wi < (uint32_t)E ? (int32_t)wi : -1;
      sw.expert_dst = wj < (uint32_t)E ? (int32_t)wj : -1;
      sw.gain = (int64_t)g;
      a.swaps[ns] = sw;
    }
    Lu += (uint32_t)((lane == amax ? d : 0) - (lane == amin ? d : 0));
    ++ns;
    plan_sync<64>();
  }
  return ns;
}

// Slot capacity of the one-wave planner: R <= 64 * RPL ranks of S <= 8 (CPL 1) or S <= 11 (CPL 2)
// slots, so its LDS follows the launch shape (16.6 KB for 64 ranks of 8 slots) and the workgroup can
// start beside other kernels' workgroups on a CU.
constexpr int wave_cap(int RPL, int CPL) {
  return 64 * RPL * (CPL == 1 ? 8 : 11) < kMaxRS ? 64 * RPL * (CPL == 1 ? 8 : 11) : kMaxRS;
}

// LDS of the one-wave planner, provided by the caller: vals, cnt, ej, reps, base and flag hold at
// least wave_cap(RPL, CPL) entries, slot as many (8-byte aligned), part 64 * RPL; bad and jmax one
// word each.  With one rank per lane (RPL 1) the planner also takes time budgets: ebytes holds the
// expert sizes (as many entries as slots), acc_pair and acc_cost the link and cost of every
// accepted swap (kMaxTimedSwaps); NULL otherwise.
struct PlanWaveLds {
  int32_t *vals, *cnt, *ej, *reps, *base, *flag;
  uint2* slot;
  int32_t* part;
  int32_t *bad, *jmax;
  int64_t* ebytes;
  int64_t* acc_cost;
  int32_t* acc_pair;
};

// Bytes of PlanWaveLds for CAP slots and RPL ranks per lane, laid out as plan_wave_lds carves them.
constexpr size_t plan_wave_lds_bytes(int CAP, int RPL) {
  return (size_t)CAP * 8 + (RPL == 1 ? (size_t)CAP * 8 + (size_t)kMaxTimedSwaps * 12 : 0) +
         (size_t)CAP * 4 * 6 + (size_t)64 * RPL * 4 + 8;
}
// Carves PlanWaveLds out of `mem` (8-byte aligned, plan_wave_lds_bytes(CAP, RPL) bytes).
__device__ __forceinline__ PlanWaveLds plan_wave_lds(char* mem, int CAP, int RPL) {
  PlanWaveLds l;
  l.slot = reinterpret_cast<uint2*>(mem);
  char* m = mem + (size_t)CAP * 8;
  l.ebytes = nullptr;
  l.acc_cost = nullptr;
  l.acc_pair = nullptr;
  if (RPL == 1) {
    l.ebytes = reinterpret_cast<int64_t*>(m);
    m += (size_t)CAP * 8;
    l.acc_cost = reinterpret_cast<int64_t*>(m);
    m += (size_t)kMaxTimedSwaps * 8;
  }
  int32_t* w = reinterpret_cast<int32_t*>(m);
  l.vals = w; w += CAP;
  l.cnt = w; w += CAP;
  l.ej = w; w += CAP;
  l.reps = w; w += CAP;
  l.base = w; w += CAP;
  l.flag = w; w += CAP;
  if (RPL == 1) { l.acc_pair = w; w += kMaxTimedSwaps; }
  l.part = w; w += 64 * RPL;
  l.bad = w; l.jmax = w + 1;
  return l;
}

// RPL: ranks per lane (R <= 64 * RPL); rank r lives in lane r % 64, register r / 64.
// CPL: candidates per lane, 1 for S * S <= 64, 2 for S * S <= 128.
// Runs in the first wave of its workgroup (threadIdx.x < 64); the caller's other waves take no part.
// TABLES_IN_LDS: the caller has already put the counts in lds.cnt, the slot table in lds.vals and,
// under a time budget, the expert sizes in lds.ebytes (all published by a barrier).
// Time budgets (a.timed) need RPL 1: every candidate between the two frontier ranks is costed by
// Eq. 9 on their link, admitted if it fits what is left of both ranks' and of the link's budgets,
// and the round's best is the largest benefit / cost, then the tie key.
template <int RPL, int CPL, bool TABLES_IN_LDS = false>
__device__ void plan_wave_body(const PlanDeviceLaunch& a, const PlanWaveLds& lds) {
  int32_t* const vals = lds.vals;      // the input tables
  int32_t* const cnt = lds.cnt;
  int32_t* const ej = lds.ej;
  int32_t* const reps = lds.reps;      // placement check
  int32_t* const base = lds.base;
  int32_t* const flag = lds.flag;
  uint2* const slot = lds.slot;        // x: item id | moved flag, y: the item's load (token share)
  int32_t* const part = lds.part;
  int32_t& s_bad = *lds.bad;
  int32_t& s_J = *lds.jmax;
  const int lane = threadIdx.x;
  const int E = a.E, R = a.R, S = a.S, RS = R * S;
  const fb_budget bg = a.budget;
  const bool timed = RPL == 1 && a.timed;
  int64_t* const ebytes = lds.ebytes;
  const float inv_e = 1.0f / (float)E;

  // every input table is fetched before the first wait
  for (int e = lane; e < E; e += 64) {
    if (!TABLES_IN_LDS) {
      cnt[e] = a.counts[e];
      if (timed) ebytes[e] = a.expert_bytes[e];
    }
    reps[e] = 0;
  }
  if (!TABLES_IN_LDS)
    for (int c = lane; c < RS; c += 64) vals[c] = a.slot_expert[c];
  for (int r = lane; r < R; r += 64) part[r] = 0;
  // time budget: rank `lane`'s node and what is left of its budget
  const int32_t node_r = timed && lane < R ? a.rank_node[lane] : 0;
  int64_t left_r = a.cost.rank_budget_ns;
  plan_sync<64>();
  // short check of a plain placement (every expert exactly once); a replica (a value >= E) sends the
  // table to the full check
  int bad = 0, replica = 0;
  for (int c = lane; c < RS; c += 64) {
    const int v = vals[c];
    if (v < -1) bad = 1;
    else if (v >= E) replica = 1;
    else if (v >= 0) atomicAdd(&reps[v], 1);
  }
  plan_sync<64>();
  int J = 1;
  if (__ballot(replica)) {
    if (lane == 0) s_bad = 0;
    check_placement<64>(E, R, S, vals, cnt, ej, reps, base, flag, nullptr, &s_bad, &s_J);
    J = s_J;
    bad = s_bad;
  } else {
    for (int e = lane; e < E; e += 64) bad |= (reps[e] != 1) | (cnt[e] < 0);
  }
  if (timed)
    for (int e = lane; e < E; e += 64) bad |= (ebytes[e] < 0) | (ebytes[e] > kCostLimit);
  const int V = E * J;               // slot values are below V; empty-slot ids from V
  const bool any_bad = __ballot(bad) != 0;
  if (any_bad || (int64_t)V + RS > ((int64_t)1 << kItemBits)) {
    if (lane == 0) { *a.n_swaps = 0; *a.status = any_bad ? FB_EINVAL : FB_EUNSUPPORTED; }
    return;
  }
  for (int c = lane; c < RS; c += 64) {
    const int v = vals[c];
    slot[c] = v < 0 ? make_uint2((uint32_t)(V + c), 0u)
                    : make_uint2((uint32_t)v, (uint32_t)(J == 1 ? cnt[v] : replica_share(ej[c], cnt, reps)));
  }
  plan_sync<64>();
  int64_t Lr[RPL];                   // load of rank lane + 64 m (0 past R)
  int64_t mine = 0;
#pragma unroll
  for (int m = 0; m < RPL; ++m) {
    const int r = lane + 64 * m;
    int64_t v = 0;
    if (r < R)
      for (int s = 0; s < S; ++s) v += slot[r * S + s].y;
    Lr[m] = v;
    mine += v;
  }
  const int64_t N = (int64_t)wave_sum_u64((uint64_t)mine);
  int64_t g_num = bg.gamma_num, g_den = bg.gamma_den;
  if (g_den == 0) { g_num = N > 0 ? 1 : 0; g_den = N > 0 ? N : 1; }
  const __int128 bound = (__int128)g_den * N + (__int128)g_num * 4 * (__int128)N * N;
  if (bound > (__int128)INT64_MAX) {
    if (lane == 0) { *a.n_swaps = 0; *a.status = FB_EUNSUPPORTED; }
    return;
  }

  // this lane's candidates (p, q) = (c / S, c mod S) for c = lane (+ 64)
  int pc[CPL], qc[CPL];
  bool hc[CPL];
#pragma unroll
  for (int h = 0; h < CPL; ++h) {
    const int c = lane + 64 * h;
    hc[h] = c < S * S;
    pc[h] = hc[h] ? c / S : 0;
    qc[h] = hc[h] ? c - pc[h] * S : 0;
  }
  const bool capped = bg.per_rank_cap != 0;
  int ns = 0;
  const bool active = N > 0 && bg.max_swaps > 0 && R > 1;
  bool small_done = false;
  if constexpr (RPL == 1) {
    if (active && N < (int64_t)0x7fffffff && J == 1 && !timed) {
      uint32_t Lu = (uint32_t)Lr[0];
      ns = rounds_small<CPL>(a, slot, part, Lu, g_num, g_den);
      Lr[0] = Lu;
      small_done = true;
    }
  }
  for (int round = 0; active && !small_done && round < bg.max_swaps; ++round) {
    uint64_t kmax = 0, kmin = 0;
#pragma unroll
    for (int m = 0; m < RPL; ++m) {
      const int r = lane + 64 * m;
      const bool in = r < R;
      kmax = umax64(kmax, in ? key_max(Lr[m], r) : 0ull);
      kmin = umax64(kmin, in ? key_min(Lr[m], r) : 0ull);
    }
    kmax = wave_max_u64(kmax);
    kmin = wave_max_u64(kmin);
    const int amax = key_rank(kmax), amin = key_rank(kmin);
    const int64_t M = (int64_t)(kmax >> kRankBits);
    const int64_t Lmin = kLoadCap - (int64_t)(kmin >> kRankBits);
    if (M - Lmin <= bg.tau) break;
    uint64_t ko = 0;                  // largest load among the other ranks, plus one (0: none)
#pragma unroll
    for (int m = 0; m < RPL; ++m) {
      const int r = lane + 64 * m;
      const bool in = r < R && r != amax && r != amin;
      ko = umax64(ko, in ? (uint64_t)Lr[m] + 1 : 0ull);
    }
    ko = wave_max_u64(ko);
    const int64_t other = ko ? (int64_t)ko - 1 : INT64_MIN;

    // time budget: the pair's link and the most a candidate may cost there
    int64_t alpha = 0, beta = 1, cap_ns = 0;
    double inv_beta = 1.0;
    const bool link_scan = timed && a.cost.link_budget_ns < a.cost.rank_budget_ns;
    const int key = amax < amin ? amax * kMaxR + amin : amin * kMaxR + amax;
    if (timed) {
      const int tl = __builtin_amdgcn_readlane(node_r, amax) == __builtin_amdgcn_readlane(node_r, amin) ? 0 : 1;
      alpha = a.cost.alpha_ns[tl];
      beta = a.cost.beta_bytes_per_us[tl];
      inv_beta = 1.0 / (double)beta;
      const int64_t left_a = (int64_t)readlane_u64((uint64_t)left_r, amax);
      const int64_t left_b = (int64_t)readlane_u64((uint64_t)left_r, amin);
      cap_ns = left_a < left_b ? left_a : left_b;
      if (link_scan) {
        // a link budget below the rank budget: what the pair's accepted swaps left of it
        uint64_t used = 0;
        for (int s0 = 0; s0 < ns; s0 += 64) {
          const int s = s0 + lane;
          used += s < ns && lds.acc_pair[s] == key ? (uint64_t)lds.acc_cost[s] : 0ull;
        }
        const int64_t left_l = a.cost.link_budget_ns - (int64_t)wave_sum_u64(used);
        cap_ns = left_l < cap_ns ? left_l : cap_ns;
      }
    }
    uint64_t gk = 0, tk = 0, ck = 1;
    int64_t dl = 0;
    uint2 ea = {0u, 0u}, eb = {0u, 0u};
    const bool cap_hit = capped && (part[amax] >= bg.per_rank_cap || part[amin] >= bg.per_rank_cap);
    // with replicas: eq(p, q) says that slot p of amax and slot q of amin hold replicas of one
    // expert.  Candidate (p, q) may not put a replica beside another replica of its expert, nor
    // exchange two replicas of one expert (eq(p, q) itself): row p and column q of eq must be
    // empty.  The wave ballots eq once per round (S <= 11, so a row or column set fits in 32 bits);
    // its set bits are rare and are walked with uniform values
    uint32_t eq_rows = 0, eq_cols = 0;
    if (J > 1) {
#pragma unroll
      for (int h = 0; h < CPL; ++h) {
        bool eqh = false;
        if (hc[h]) {
          const uint32_t ya = slot[amax * S + pc[h]].x & ~kMovedBit;
          const uint32_t yb = slot[amin * S + qc[h]].x & ~kMovedBit;
          eqh = ya < (uint32_t)V && yb < (uint32_t)V &&
                expert_of((int)ya, E, inv_e) == expert_of((int)yb, E, inv_e);
        }
        uint64_t m = __ballot(eqh);
        while (m) {
          const int c = __builtin_ctzll(m) + 64 * h;
          m &= m - 1;
          eq_rows |= 1u << (c / S);
          eq_cols |= 1u << (c % S);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      if (!hc[h]) continue;
      const int pl = pc[h], ql = qc[h];
      const uint2 xa = slot[amax * S + pl], xb = slot[amin * S + ql];
      const uint32_t i = xa.x & ~kMovedBit, j = xb.x & ~kMovedBit;
      bool ok = !cap_hit && !((xa.x | xb.x) & kMovedBit) && !(i >= (uint32_t)V && j >= (uint32_t)V) &&
                !(((eq_rows >> pl) | (eq_cols >> ql)) & 1u);
      const int64_t d = (int64_t)(int32_t)xb.y - (int64_t)(int32_t)xa.y;
      const int64_t la = M + d, lb = Lmin - d;
      int64_t m2 = la > lb ? la : lb;
      if (other > m2) m2 = other;
      const int64_t spread = g_num ? g_num * (2 * d * (Lmin - M - d)) : 0;
      const int64_t gain = g_den * (M - m2) + spread;
      // tie order inside the fixed pair (amax, amin): item ids; the slots ride along below them
      const uint64_t th = ((((uint64_t)i << kItemBits) | j) << 8) | ((uint64_t)pl << 4) | (uint64_t)ql;
      if (!ok || gain <= 0) continue;
      if (timed) {
        const int ei = i >= (uint32_t)V ? -1 : J == 1 ? (int)i : expert_of((int)i, E, inv_e);
        const int ej2 = j >= (uint32_t)V ? -1 : J == 1 ? (int)j : expert_of((int)j, E, inv_e);
        const int64_t bytes = (ei >= 0 ? ebytes[ei] : 0) + (ej2 >= 0 ? ebytes[ej2] : 0);
        const int64_t c = alpha + ceil_div(bytes * 1000, beta, inv_beta);
        if (c > cap_ns || !ratio_better((uint64_t)gain, (uint64_t)c, th, gk, ck, tk)) continue;
        ck = (uint64_t)c;
      } else if (!(gk == 0 || (uint64_t)gain > gk || ((uint64_t)gain == gk && th < tk))) {
        continue;
      }
      gk = (uint64_t)gain;
      tk = th;
      dl = d;
      ea = xa;
      eb = xb;
    }
    uint64_t g, t, cst = 1;
    if (timed) {
      g = gk;
      cst = ck;
      t = tk;
      wave_best_ratio(g, cst, t);
      if (g == 0) break;                        // no admissible candidate with positive benefit
    } else {
      g = wave_max_u64(gk);
      if (g == 0) break;
      t = ~wave_max_u64(gk == g ? ~tk : 0ull);
    }
    const int wp = (int)(t >> 4) & 15, wq = (int)t & 15;
    const int wi = (int)(t >> (8 + kItemBits)) & ((1 << kItemBits) - 1);
    const int wj = (int)(t >> 8) & ((1 << kItemBits) - 1);
    const int wl = __builtin_amdgcn_readfirstlane((wp * S + wq) & 63);   // the lane that holds it
    const int64_t d = (int64_t)readlane_u64((uint64_t)dl, wl);
    const int32_t ci = __builtin_amdgcn_readlane((int)ea.y, wl), cj = __builtin_amdgcn_readlane((int)eb.y, wl);
    if (lane == 0) {
      slot[amax * S + wp] = make_uint2((uint32_t)wj | kMovedBit, (uint32_t)cj);
      slot[amin * S + wq] = make_uint2((uint32_t)wi | kMovedBit, (uint32_t)ci);
      ++part[amax];
      ++part[amin];
      fb_swap sw;
      sw.src_rank = amax; sw.dst_rank = amin; sw.src_slot = wp; sw.dst_slot = wq;
      sw.expert_src = wi < V ? wi : -1;
      sw.expert_dst = wj < V ? wj : -1;
      sw.gain = (int64_t)g;
      a.swaps[ns] = sw;
      if (timed) {
        if (link_scan) { lds.acc_pair[ns] = key; lds.acc_cost[ns] = (int64_t)cst; }
        if (a.swap_cost_ns) a.swap_cost_ns[ns] = (int64_t)cst;
      }
    }
    if (timed && (lane == amax || lane == amin)) left_r -= (int64_t)cst;
#pragma unroll
    for (int m = 0; m < RPL; ++m) {
      const int r = lane + 64 * m;
      Lr[m] += (r == amax ? d : 0) - (r == amin ? d : 0);
    }
    ++ns;
    plan_sync<64>();
  }

  for (int c = lane; c < RS; c += 64) {
    const int it = (int)(slot[c].x & ~kMovedBit);
    a.new_slot_expert[c] = it < V ? it : -1;
    if (it < E) a.new_expert_to_rank[it] = c / S;   // replica 0
  }
#pragma unroll
  for (int m = 0; m < RPL; ++m) {
    const int r = lane + 64 * m;
    if (r < R) a.new_rank_loads[r] = Lr[m];
  }
  if (lane == 0) { *a.n_swaps = ns; *a.status = FB_OK; }
}

}  // namespace
}  // namespace fb
