// Budgeted greedy expert-swap planner as one stream-ordered workgroup (gfx950).
//
// Same algorithm and tie-breaks as the host planner (Sec. "Budgeted Expert-Swap Planning",
// Eq. 6-8, Alg. 1).  Every round: wave 0 finds the most and least loaded ranks and the loads the
// benefit needs (64-bit wave reductions over packed (load, rank) keys), every thread evaluates its
// share of the admissible candidates with the exact integer benefit
//     den * (M - M') + num * 2d (L_b - L_a - d),
// the best candidate under (benefit desc, src rank, dst rank, item ids asc) is found with two
// packed-key reductions, and wave 0 applies it.  State lives in LDS.
//
// The benefit fits an int64: the launcher checks den N + 4 num N^2 <= INT64_MAX once, and each
// term and partial product is bounded by it (0 <= M' <= N, |d| <= N, |L_b - L_a - d| <= N).
//
// Two kernels:
//   * plan_frontier_wave, one wave, for frontier mode with S * S <= 128 (the common case; under a
//     time budget up to 64 ranks).  Rank loads live in registers (ranks lane + 64 m), each lane
//     owns one or two candidates (p, q), slot entries carry the item, its moved flag and its count
//     so that a candidate costs one LDS round trip, and a round is a handful of wave reductions
//     with no workgroup barrier.
//   * plan_general<NT> for everything else (full mode, larger S, a time budget on more ranks): state in LDS,
//     threads split the candidates by rank pair, per-wave reductions combined through LDS.  Full
//     mode on up to 64 ranks of up to 8 slots with gamma > 0 keeps, per rank pair, the few
//     candidates that can still be a round's best and rebuilds only the pairs of the previous
//     swap; other full-mode tables score every pair under a benefit bound.
//
// Under a time budget (the cost form of the same section, Eq. 9-10 enforced per rank and per link)
// every candidate also costs C = alpha + ceil(bytes * 1000 / beta) ns on its link, must fit what is
// left of both ranks' and the link's budgets, and the best candidate is the largest benefit / C,
// compared exactly as gain_1 * C_2 vs gain_2 * C_1 (gains < 2^63, costs < 2^42), then the tie key.
//
// Replicated placements (slot value v = e + E * j is replica j of expert e, as in the host planner):
// an item's id is its slot value, or V + c for the empty slot c (V = E * J, J the largest replica
// count; V = E without replicas), its load is its token share floor(n_e / c_e) + [j < n_e mod c_e],
// held with the item in its slot, and a candidate may not put a replica on a rank that holds
// another replica of the same expert.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fb_internal.h"
#include "fb_plan_wave.h"

namespace fb {
namespace {

constexpr int kMaxSurvivors = 8192;           // full mode: work units listed per round (more are
                                              // evaluated where their bound test ran)
// Tables of at most kSmallRS slots and kSmallR ranks run in a workgroup that holds a fraction of the
// LDS (about 29 KB in frontier mode, 92 KB in full mode, against 153 KB for the largest tables), so
// that it can start on a CU beside another kernel's workgroups, for instance attention's while the
// plan is made on a side stream, instead of waiting for a whole CU to drain.
constexpr int kSmallRS = 512;
constexpr int kSmallR = 64;

// Full mode on tables of at most kSmallR ranks and S <= kFrontS slots per rank: every unordered rank
// pair keeps the candidates that no other candidate of the pair dominates (at most kFrontCap of
// them; kFrontAll when more, and then all of the pair's candidates are scored).
constexpr int kFrontS = 8;
constexpr int kFrontCap = 8;
constexpr uint8_t kFrontAll = 255;

// Tie order after the benefit: (src rank, dst rank, item i, item j) ascending, as one integer.
__device__ __forceinline__ uint64_t tie_key(int a, int b, int i, int j) {
  return ((uint64_t)a << (kRankBits + 2 * kItemBits)) | ((uint64_t)b << (2 * kItemBits)) |
         ((uint64_t)i << kItemBits) | (uint64_t)j;
}

// LDS of plan_general for tables of at most CRS slots and CR ranks; SURV work units listed per
// full-mode round; NPAIR rank pairs with a stored frontier.  E <= R * S <= CRS, so the per-expert
// arrays fit the slot capacity.
template <int CRS, int CR, int SURV, int NPAIR>
struct SharedT {
  static constexpr int kSurv = SURV;
  // full mode with stored frontiers: per unordered pair (index b (b - 1) / 2 + a for a < b) the
  // number of stored candidates (or kFrontAll) and each one's slot pair p * S + q, with p on the
  // more loaded rank of the pair when the frontier was built
  uint8_t fr_n[NPAIR];
  uint8_t fr_pt[NPAIR][kFrontCap];
  int32_t last[2];               // ranks of the swap accepted in the previous round
  int64_t link_used[NPAIR];      // time budget: cost charged to each rank pair's link so far
  int32_t item[CRS];             // slot -> item id (slot value, or V + slot for an empty slot)
  int32_t sload[CRS];            // slot -> load (token share) of its item
  uint8_t mslot[CRS];            // slot -> its item has moved
  union {
    struct {                     // placement check
      int32_t cnt[CRS], ej[CRS], reps[CRS], base[CRS], flag[CRS];
    } chk;
    struct {                     // after the check
      int64_t ebytes[CRS];       // expert sizes (time budget)
      // frontier rounds with replicas: slot p of amax (row) or q of amin (column) holds a replica
      // of an expert that the other rank also holds
      uint8_t mrow[CRS], mcol[CRS];
      // full mode: the smallest and largest load among each rank's items that have not moved
      // (smin > smax when every item has moved), and the work units left after the bound test
      int32_t smin[CR], smax[CR];
      int32_t surv[SURV];
    } run;
  } u;
  int32_t wsum[16];
  int64_t L[CR];
  int32_t part[CR];
  uint64_t wgain[16], wtie[16], wcost[16];
  uint64_t rgain[16], rtie[16], rcost[16];   // full mode: per-wave bests of the first phase
  int64_t cmin[2];               // time budget: the lowest cost of any swap on link type 0 / 1
  int32_t nsurv;                 // full mode: work units that passed this round's bound test
  int64_t N;
  int32_t bad, stop, amax, amin, top[3], ns, J;
  int64_t other;
  // time budget: what is left of every rank's budget, rank nodes, and the accepted swaps' links
  // and costs (the link budgets are charged by scanning them)
  int64_t rank_left[CR];
  int32_t node[CR];
  int32_t acc_pair[kMaxTimedSwaps];   // a * kMaxR + b, a < b
  int64_t acc_cost[kMaxTimedSwaps];
};

// Eq. 9 in whole nanoseconds for a swap moving expert ei off rank ra and expert ej off rank rb
// (-1: an empty slot, which transfers nothing).
template <class SH>
__device__ __forceinline__ int64_t swap_cost(const PlanDeviceLaunch& a, const SH& sh, int ra,
                                             int rb, int ei, int ej) {
  const int t = sh.node[ra] == sh.node[rb] ? 0 : 1;
  const int64_t bytes = (ei >= 0 ? sh.u.run.ebytes[ei] : 0) + (ej >= 0 ? sh.u.run.ebytes[ej] : 0);
  const int64_t beta = a.cost.beta_bytes_per_us[t];
  return a.cost.alpha_ns[t] + ceil_div(bytes * 1000, beta, 1.0 / (double)beta);
}

// Does a swap of cost c between ranks ra and rb fit the remaining rank and link budgets?
template <class SH>
__device__ __forceinline__ bool swap_fits(const PlanDeviceLaunch& a, const SH& sh, int ra,
                                          int rb, int64_t c) {
  if (c > sh.rank_left[ra] || c > sh.rank_left[rb]) return false;
  // every swap on a link also charges both of its ranks, so a link budget at least the rank
  // budget never binds
  if (a.cost.link_budget_ns >= a.cost.rank_budget_ns) return true;
  const int key = ra < rb ? ra * kMaxR + rb : rb * kMaxR + ra;
  int64_t used = 0;
  for (int s = 0; s < sh.ns; ++s) used += sh.acc_pair[s] == key ? sh.acc_cost[s] : 0;
  return c <= a.cost.link_budget_ns - used;
}

// A compile-time flag for generic lambdas.
template <bool B>
struct Flag {
  static constexpr bool value = B;
};

// What a rank pair's candidates share under a time budget: the link's alpha and beta, and the most
// a candidate may cost (what is left of both ranks' budgets and of the pair's link budget).
struct PairCost {
  int64_t alpha, beta, cap_ns;
  double inv_beta;
};

// One step of a lexicographic minimum of (u, c, t) with payload x, with the lane that DPP control
// CTRL names (every lane of the wave takes part).
template <int CTRL>
__device__ __forceinline__ void lex_min_step(uint64_t& u, uint64_t& c, uint64_t& t, int& x) {
  const uint64_t u2 = dpp_u64<CTRL>(u), c2 = dpp_u64<CTRL>(c), t2 = dpp_u64<CTRL>(t);
  const int x2 = __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
  if (u2 < u || (u2 == u && (c2 < c || (c2 == c && t2 < t)))) { u = u2; c = c2; t = t2; x = x2; }
}

// Lexicographic minimum over each group of 8 lanes (8g .. 8g + 7); every lane of a group ends with
// it.  Lane exchanges: lane ^ 1, lane ^ 2, then the mirror within the 8 lanes (lane i and 7 - i).
__device__ __forceinline__ void seg_min8(uint64_t& u, uint64_t& c, uint64_t& t, int& x) {
  lex_min_step<0xB1>(u, c, t, x);    // quad_perm [1,0,3,2]
  lex_min_step<0x4E>(u, c, t, x);    // quad_perm [2,3,0,1]
  lex_min_step<0x141>(u, c, t, x);   // row_half_mirror
}

// Unordered rank pair k = y (y - 1) / 2 + x, x < y.
__device__ __forceinline__ void pair_of(int k, int& x, int& y) {
  int b = (int)((1.0f + sqrtf(8.0f * (float)k + 1.0f)) * 0.5f);
  while (b * (b - 1) / 2 > k) --b;
  while ((b + 1) * b / 2 <= k) ++b;
  y = b;
  x = k - b * (b - 1) / 2;
}

// NT threads (256: frontier mode, 1024: full mode); SMALL: tables of at most kSmallRS slots and
// kSmallR ranks
template <int NT, bool SMALL>
__global__ __launch_bounds__(NT, 1) void plan_general(PlanDeviceLaunch a) {
  constexpr int CRS = SMALL ? kSmallRS : kMaxRS;
  constexpr int CR = SMALL ? kSmallR : kMaxR;
  // the survivor list serves full mode only, the stored frontiers full mode on small tables
  constexpr bool kFront = SMALL && NT == 1024;
  __shared__ SharedT<CRS, CR, NT == 1024 ? kMaxSurvivors : 64, kFront ? CR * (CR - 1) / 2 : 1> sh;
  constexpr int kSurv = decltype(sh)::kSurv;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int E = a.E, R = a.R, S = a.S, RS = R * S;
  const fb_budget bg = a.budget;

  // bits of bad: 1 an invalid table or count, 2 item ids that would not fit the tie keys, 4 a
  // replica (a value >= E) seen by the short check
  if (tid == 0) { sh.bad = 0; sh.ns = 0; sh.N = 0; sh.J = 1; }
  // every input table is fetched before the first wait; item[] holds the raw slot values until the
  // check is done, and the expert sizes of a time budget wait in registers until the check's LDS
  // space is free
  for (int c = tid; c < RS; c += NT) sh.item[c] = a.slot_expert[c];
  for (int e = tid; e < E; e += NT) { sh.u.chk.cnt[e] = a.counts[e]; sh.u.chk.reps[e] = 0; }
  constexpr int kEB = (CRS + NT - 1) / NT;
  int64_t eb[kEB];
#pragma unroll
  for (int u = 0; u < kEB; ++u) {
    const int e = tid + u * NT;
    eb[u] = a.timed && e < E ? a.expert_bytes[e] : 0;
  }
  for (int r = tid; r < R; r += NT) sh.part[r] = 0;
  if constexpr (kFront)
    for (int k = tid; k < R * (R - 1) / 2; k += NT) sh.link_used[k] = 0;
  if (a.timed)
    for (int r = tid; r < R; r += NT) { sh.node[r] = a.rank_node[r]; sh.rank_left[r] = a.cost.rank_budget_ns; }
  __syncthreads();
  // short check of a plain placement: every expert exactly once
  for (int c = tid; c < RS; c += NT) {
    const int v = sh.item[c];
    if (v < -1) atomicOr(&sh.bad, 1);
    else if (v >= E) atomicOr(&sh.bad, 4);
    else if (v >= 0) atomicAdd(&sh.u.chk.reps[v], 1);
  }
  __syncthreads();
  const bool replicated = (sh.bad & 4) != 0;
  __syncthreads();
  if (replicated) {
    if (tid == 0) sh.bad = 0;
    check_placement<NT>(E, R, S, sh.item, sh.u.chk.cnt, sh.u.chk.ej, sh.u.chk.reps, sh.u.chk.base,
                        sh.u.chk.flag, sh.wsum, &sh.bad, &sh.J);
  } else {
    for (int e = tid; e < E; e += NT)
      if (sh.u.chk.reps[e] != 1 || sh.u.chk.cnt[e] < 0) atomicOr(&sh.bad, 1);
    __syncthreads();
  }
  const int J = sh.J;
  const int V = E * J;                       // slot values are below V; empty-slot ids from V
  if (!sh.bad) {
    if ((int64_t)V + RS > ((int64_t)1 << kItemBits)) {
      if (tid == 0) sh.bad = 2;
    } else {
      for (int c = tid; c < RS; c += NT) {
        const int v = sh.item[c];
        sh.item[c] = v >= 0 ? v : V + c;
        sh.sload[c] = v < 0 ? 0
                    : J == 1 ? sh.u.chk.cnt[v]
                             : replica_share(sh.u.chk.ej[c], sh.u.chk.cnt, sh.u.chk.reps);
        sh.mslot[c] = 0;
      }
    }
  }
  __syncthreads();                           // the check's arrays are dead from here on
  if (a.timed) {
#pragma unroll
    for (int u = 0; u < kEB; ++u) {
      const int e = tid + u * NT;
      if (e < E) {
        sh.u.run.ebytes[e] = eb[u];
        if (eb[u] < 0 || eb[u] > kCostLimit) atomicOr(&sh.bad, 1);
      }
    }
  }
  __syncthreads();
  if (sh.bad) {
    if (tid == 0) { *a.n_swaps = 0; *a.status = (sh.bad & 1) ? FB_EINVAL : FB_EUNSUPPORTED; }
    return;
  }

  for (int r = tid; r < R; r += NT) {
    int64_t v = 0;
    for (int s = 0; s < S; ++s) v += sh.sload[r * S + s];
    sh.L[r] = v;
    atomicAdd((unsigned long long*)&sh.N, (unsigned long long)v);
  }
  __syncthreads();
  // does rank r hold a replica of the expert of item it (a replica id below V)?
  const float inv_e = 1.0f / (float)E;
  auto holds = [&](int r, int it) -> bool {
    const int e = expert_of(it, E, inv_e);
    for (int s = 0; s < S; ++s) {
      const int x = sh.item[r * S + s];
      if (x < V && expert_of(x, E, inv_e) == e) return true;
    }
    return false;
  };
  const int64_t N = sh.N;
  int64_t g_num = bg.gamma_num, g_den = bg.gamma_den;
  if (g_den == 0) { g_num = N > 0 ? 1 : 0; g_den = N > 0 ? N : 1; }
  const __int128 bound = (__int128)g_den * N + (__int128)g_num * 4 * (__int128)N * N;
  if (bound > (__int128)INT64_MAX) {
    if (tid == 0) { *a.n_swaps = 0; *a.status = FB_EUNSUPPORTED; }
    return;
  }

  const bool frontier = bg.mode == FB_FRONTIER;
  const bool active = N > 0 && bg.max_swaps > 0 && R > 1;
  const bool marks = frontier && J > 1;
  // full mode with stored frontiers (gamma > 0; with gamma = 0 the benefit stops falling with the
  // load difference once the pair is below the largest load outside it, and the frontiers grow)
  const bool front = kFront && !frontier && S <= kFrontS && g_num > 0;
  if (a.timed && !frontier) {
    // every candidate moves at least one expert, so it costs at least alpha + the smallest
    // expert's transfer time on its link
    int64_t mb = INT64_MAX;
    for (int e = tid; e < E; e += NT) mb = sh.u.run.ebytes[e] < mb ? sh.u.run.ebytes[e] : mb;
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor(mb, off);
      mb = o < mb ? o : mb;
    }
    if (lane == 0) sh.rgain[wave] = (uint64_t)mb;
    __syncthreads();
    if (tid == 0) {
      for (int w = 1; w < NT / 64; ++w) mb = (int64_t)sh.rgain[w] < mb ? (int64_t)sh.rgain[w] : mb;
      for (int t = 0; t < 2; ++t) {
        const int64_t beta = a.cost.beta_bytes_per_us[t];
        sh.cmin[t] = a.cost.alpha_ns[t] + ceil_div(mb * 1000, beta, 1.0 / (double)beta);
      }
    }
    __syncthreads();
  }
  for (int round = 0; active && round < bg.max_swaps; ++round) {
    if (marks)                        // the previous round's reads ended at its last barrier
      for (int s2 = tid; s2 < S; s2 += NT) { sh.u.run.mrow[s2] = 0; sh.u.run.mcol[s2] = 0; }
    // ---- wave 0: argmax, argmin and the loads of the ranks outside a candidate pair ------------
    if (wave == 0) {
      uint64_t kmax = 0, kmin = 0;
      for (int r = lane; r < R; r += 64) {
        kmax = umax64(kmax, key_max(sh.L[r], r));
        kmin = umax64(kmin, key_min(sh.L[r], r));
      }
      kmax = wave_max_u64(kmax);
      kmin = wave_max_u64(kmin);
      const int amax = key_rank(kmax), amin = key_rank(kmin);
      if (frontier) {
        // the largest load among ranks other than amax and amin (0 = there is none)
        uint64_t ko = 0;
        for (int r = lane; r < R; r += 64)
          if (r != amax && r != amin) ko = umax64(ko, (uint64_t)sh.L[r] + 1);
        ko = wave_max_u64(ko);
        if (lane == 0) sh.other = ko ? (int64_t)ko - 1 : INT64_MIN;
      } else {
        // the three largest (load, rank) keys, for the largest load outside any pair
        uint64_t k1 = 0, k2 = 0;
        const int t0 = amax;
        for (int r = lane; r < R; r += 64)
          if (r != t0) k1 = umax64(k1, key_max(sh.L[r], r));
        k1 = wave_max_u64(k1);
        const int t1 = k1 ? key_rank(k1) : -1;
        for (int r = lane; r < R; r += 64)
          if (r != t0 && r != t1) k2 = umax64(k2, key_max(sh.L[r], r));
        k2 = wave_max_u64(k2);
        if (lane == 0) { sh.top[0] = t0; sh.top[1] = t1; sh.top[2] = k2 ? key_rank(k2) : -1; }
      }
      if (lane == 0) {
        sh.amax = amax;
        sh.amin = amin;
        sh.stop = (sh.L[amax] - sh.L[amin] <= bg.tau) ? 1 : 0;
      }
    }
    if (!frontier && !front) {
      for (int r = tid; r < R; r += NT) {
        int32_t lo = INT32_MAX, hi = INT32_MIN;
        for (int q = 0; q < S; ++q) {
          if (sh.mslot[r * S + q]) continue;
          const int32_t l = sh.sload[r * S + q];
          lo = l < lo ? l : lo;
          hi = l > hi ? l : hi;
        }
        sh.u.run.smin[r] = lo;
        sh.u.run.smax[r] = hi;
      }
    }
    // (with stored frontiers the rebuild below needs none of wave 0's results, so the first
    // barrier after it publishes them)
    if (!front) {
      __syncthreads();
      if (sh.stop) break;
    }

    // ---- candidates ----------------------------------------------------------------------------
    const int amax = front ? 0 : sh.amax, amin = front ? 0 : sh.amin;
    if (marks) {
      // candidate (p, q) would put a replica beside another replica of its expert, or exchange two
      // replicas of one expert, exactly when row p or column q of the pair's same-expert matrix
      // has an entry: one pass over the matrix replaces a scan of the other rank per candidate
      for (int idx = tid; idx < S * S; idx += NT) {
        const int p = idx / S, q = idx - p * S;
        const int i = sh.item[amax * S + p], j = sh.item[amin * S + q];
        if (i < V && j < V && expert_of(i, E, inv_e) == expert_of(j, E, inv_e)) {
          sh.u.run.mrow[p] = 1;
          sh.u.run.mcol[q] = 1;
        }
      }
      __syncthreads();
    }
    const int64_t M = sh.L[amax];
    uint64_t bgain = 0, btie = 0;     // gain 0: nothing found (every accepted gain is > 0)
    uint64_t bcost = 1;
    auto consider = [&](int ra, int rb, int p, int q, int64_t other) {
      const int sa = ra * S + p, sb = rb * S + q;
      const int i = sh.item[sa], j = sh.item[sb];
      if (sh.mslot[sa] || sh.mslot[sb] || (i >= V && j >= V)) return;
      if (J > 1) {
        if (marks) {                  // frontier: (ra, rb) = (amax, amin)
          if (sh.u.run.mrow[p] | sh.u.run.mcol[q]) return;
        } else if ((i < V && holds(rb, i)) || (j < V && holds(ra, j))) {
          return;
        }
      }
      const int64_t La = sh.L[ra], Lb = sh.L[rb];
      const int64_t d = (int64_t)sh.sload[sb] - (int64_t)sh.sload[sa];
      const int64_t la = La + d, lb = Lb - d;
      int64_t m2 = la > lb ? la : lb;
      if (other > m2) m2 = other;
      const int64_t spread = g_num ? g_num * (2 * d * (Lb - La - d)) : 0;
      const int64_t gain = g_den * (M - m2) + spread;
      if (gain <= 0) return;
      const uint64_t tk = tie_key(ra, rb, i, j);
      if (a.timed) {
        const int ei = i >= V ? -1 : J == 1 ? i : expert_of(i, E, inv_e);
        const int ej = j >= V ? -1 : J == 1 ? j : expert_of(j, E, inv_e);
        const int64_t c = swap_cost(a, sh, ra, rb, ei, ej);
        if (!swap_fits(a, sh, ra, rb, c)) return;
        if (ratio_better((uint64_t)gain, (uint64_t)c, tk, bgain, bcost, btie)) {
          bgain = (uint64_t)gain; bcost = (uint64_t)c; btie = tk;
        }
        return;
      }
      if ((uint64_t)gain > bgain || ((uint64_t)gain == bgain && tk < btie)) { bgain = (uint64_t)gain; btie = tk; }
    };
    const bool capped = bg.per_rank_cap != 0;
    if (frontier) {
      if (!(capped && (sh.part[amax] >= bg.per_rank_cap || sh.part[amin] >= bg.per_rank_cap))) {
        const int64_t other = sh.other;
        for (int idx = tid; idx < S * S; idx += NT) {
          const int p = idx / S;
          consider(amax, amin, p, idx - p * S, other);
        }
      }
    } else if (front) {
      if constexpr (kFront) {
        // Full mode with stored frontiers (gamma > 0).  In a pair (ra, rb) with D = L_ra - L_rb > 0, a
        // candidate with load difference d = l_j - l_i leaves the two ranks at their mean +- (D +
        // 2d) / 2, so with u = |D + 2d| its benefit is den (M - max(o, (L_ra + L_rb + u) / 2)) +
        // num (D^2 - u^2) / 2, o the largest load outside the pair: it falls strictly as u grows,
        // whatever M and o are.  A candidate (u, C, tk) therefore cannot be the round's best while
        // its pair holds another admissible one with u' <= u, C' <= C and (u', C', tk')
        // lexicographically smaller.  What is left of a pair is a staircase: the lexicographically
        // smallest (u, C, tk), then the smallest among the candidates that cost less than it, and so
        // on (one candidate without a time budget).  Only a swap on a rank of the pair changes
        // what decides it (the pair's loads, items, moved flags, swap counts, rank and link
        // budgets), so each round rebuilds the staircases of the pairs that hold a rank of the
        // previous swap (every pair in the first round) and scores the stored candidates of every
        // pair.
        // Flags REP (a replicated placement) and TIMED (a time budget) are compile-time, so the
        // plain count-budget round is straight-line code.
        // The pair {x, y}: its orientation (ra the more loaded rank), D = L_ra - L_rb, and what its
        // candidates may cost; false when none of them can be admissible.
        auto pair_setup = [&](auto TIMED, int k, int x, int y, int& ra, int& rb, int64_t& D,
                              PairCost& pc) -> bool {
          const int64_t Lx = sh.L[x], Ly = sh.L[y];
          if (Lx == Ly) return false;
          ra = Lx > Ly ? x : y;
          rb = Lx > Ly ? y : x;
          D = Lx > Ly ? Lx - Ly : Ly - Lx;
          if (capped && (sh.part[ra] >= bg.per_rank_cap || sh.part[rb] >= bg.per_rank_cap)) return false;
          pc.alpha = 0; pc.beta = 1; pc.cap_ns = 0; pc.inv_beta = 1.0;
          if constexpr (decltype(TIMED)::value) {
            const int t = sh.node[ra] == sh.node[rb] ? 0 : 1;
            pc.cap_ns = sh.rank_left[ra] < sh.rank_left[rb] ? sh.rank_left[ra] : sh.rank_left[rb];
            // a link budget at least the rank budget never binds (every swap on the link also
            // charges both ranks); else what the pair's accepted swaps left of it
            if (a.cost.link_budget_ns < a.cost.rank_budget_ns) {
              const int64_t left = a.cost.link_budget_ns - sh.link_used[k];
              pc.cap_ns = left < pc.cap_ns ? left : pc.cap_ns;
            }
            if (sh.cmin[t] > pc.cap_ns) return false;      // no swap on this link fits any more
            pc.alpha = a.cost.alpha_ns[t];
            pc.beta = a.cost.beta_bytes_per_us[t];
            pc.inv_beta = 1.0 / (double)pc.beta;
          }
          return true;
        };
        // the expert of item it (below V) and its transfer size
        auto item_bytes = [&](auto REP, int it) -> int64_t {
          if (it >= V) return 0;
          return sh.u.run.ebytes[decltype(REP)::value ? expert_of(it, E, inv_e) : it];
        };
        // candidate (p, q) of the pair (ra, rb): every admissibility test but the benefit's sign;
        // its cost c (1 without a time budget) and its load difference d
        auto cand = [&](auto REP, auto TIMED, int ra, int rb, int p, int q, const PairCost& pc,
                        uint64_t& c, int64_t& d, int& i, int& j) -> bool {
          const int sa = ra * S + p, sb = rb * S + q;
          i = sh.item[sa];
          j = sh.item[sb];
          if (sh.mslot[sa] || sh.mslot[sb] || (i >= V && j >= V)) return false;
          if constexpr (decltype(REP)::value)
            if ((i < V && holds(rb, i)) || (j < V && holds(ra, j))) return false;
          d = (int64_t)sh.sload[sb] - (int64_t)sh.sload[sa];
          c = 1;
          if constexpr (decltype(TIMED)::value) {
            const int64_t cc = pc.alpha + ceil_div((item_bytes(REP, i) + item_bytes(REP, j)) * 1000,
                                                   pc.beta, pc.inv_beta);
            if (cc > pc.cap_ns) return false;
            c = (uint64_t)cc;
          }
          return true;
        };
        // rebuild, one pair per 8 lanes: lane p holds the candidates (p, q) of slot p of the more
        // loaded rank, and each pass stores the group's lexicographically smallest (u, C, tk) among
        // the candidates that cost less than the one stored before.  Groups go to waves 1, 2, ...
        // first: wave 0 finds the extremes meanwhile.
        auto build = [&](auto REP, auto TIMED) {
          constexpr bool rep = decltype(REP)::value, timed = decltype(TIMED)::value;
          const bool all = round == 0;
          const int nd = all ? R * (R - 1) / 2 : 2 * R - 3;
          const int la0 = sh.last[0], lb0 = sh.last[1];
          const int p = lane & 7;
          const int wv = wave == 0 ? NT / 64 - 1 : wave - 1;
          for (int w0 = wv * 8; w0 < nd; w0 += NT / 8) {
            const int w = w0 + (lane >> 3);
            const bool pv = w < nd;
            const int wq = pv ? w : 0;
            int x, y;
            if (all) {
              pair_of(wq, x, y);
            } else {
              int r0 = la0, o;
              if (wq < R - 1) {
                o = wq < la0 ? wq : wq + 1;        // every rank but la0
              } else {
                r0 = lb0;                          // every rank but la0 and lb0
                o = wq - (R - 1);
                const int lo = la0 < lb0 ? la0 : lb0, hi = la0 < lb0 ? lb0 : la0;
                if (o >= lo) ++o;
                if (o >= hi) ++o;
              }
              x = r0 < o ? r0 : o;
              y = r0 < o ? o : r0;
            }
            const int k = y * (y - 1) / 2 + x;
            int ra = 0, rb = 0;
            int64_t D = 0;
            PairCost pc;
            const bool live = pv && pair_setup(TIMED, k, x, y, ra, rb, D, pc);
            // slot p of ra, and the S slots of rb (indices clamped into the rank)
            const int sa = ra * S + (p < S ? p : S - 1), sb0 = rb * S;
            const int ia = sh.item[sa];
            const int64_t lia = sh.sload[sa];
            bool aok = live && p < S && !sh.mslot[sa];
            if constexpr (rep) aok = aok && !(ia < V && holds(rb, ia));
            const int64_t ba = timed ? item_bytes(REP, ia) : 0;
            // the destination slots are read in batches (one LDS wait each): without a time budget
            // items, loads and moved flags once; with one, items and flags, then the sizes, and the
            // items and loads again in every pass (the costs stay in registers)
            int jv[kFrontS], lv[kFrontS];
            bool mv[kFrontS];
#pragma unroll
            for (int q = 0; q < kFrontS; ++q) {
              const int sb = sb0 + (q < S ? q : S - 1);
              jv[q] = sh.item[sb];
              mv[q] = sh.mslot[sb] != 0;
              if constexpr (!timed) lv[q] = sh.sload[sb];
            }
            uint32_t okm = 0;                    // bit q: candidate (p, q) is admissible
#pragma unroll
            for (int q = 0; q < kFrontS; ++q) {
              bool ok = aok && q < S && !mv[q] && !(ia >= V && jv[q] >= V);
              if constexpr (rep) ok = ok && !(jv[q] < V && holds(ra, jv[q]));
              okm |= ok ? 1u << q : 0u;
            }
            uint64_t kc[kFrontS];                // costs (time budget)
            if constexpr (timed) {
              int64_t bv[kFrontS];
#pragma unroll
              for (int q = 0; q < kFrontS; ++q) bv[q] = item_bytes(REP, jv[q]);
#pragma unroll
              for (int q = 0; q < kFrontS; ++q) {
                const int64_t cc = pc.alpha + ceil_div((ba + bv[q]) * 1000, pc.beta, pc.inv_beta);
                if (cc > pc.cap_ns) okm &= ~(1u << q);
                kc[q] = (uint64_t)cc;
              }
            }
            // the group's cheapest admissible candidate: once a stored point costs that little, no
            // candidate can cost less and the staircase is complete
            uint64_t gmin = ~0ull;
            if constexpr (timed) {
#pragma unroll
              for (int q = 0; q < kFrontS; ++q)
                if (((okm >> q) & 1) && kc[q] < gmin) gmin = kc[q];
              uint64_t z0 = 0, z1 = 0;
              int zx = 0;
              seg_min8(gmin, z0, z1, zx);
            }
            uint64_t climit = ~0ull;
            int n = 0;
            bool done = !live;
            for (;;) {
              uint64_t bu = ~0ull, bc = ~0ull, bt = ~0ull;   // tie keys of R <= 64 ranks are below ~0
              int bpq = 0;
              if (!done) {
                if constexpr (timed) {
#pragma unroll
                  for (int q = 0; q < kFrontS; ++q) {
                    const int sb = sb0 + (q < S ? q : S - 1);
                    jv[q] = sh.item[sb];
                    lv[q] = sh.sload[sb];
                  }
                }
#pragma unroll
                for (int q = 0; q < kFrontS; ++q) {
                  const uint64_t c = timed ? kc[q] : 1;
                  const bool in = ((okm >> q) & 1) && c < climit;
                  const int64_t xd = D + 2 * ((int64_t)lv[q] - lia);
                  const uint64_t u = (uint64_t)(xd < 0 ? -xd : xd);
                  const uint64_t tk = tie_key(ra, rb, ia, jv[q]);
                  if (in && (u < bu || (u == bu && (c < bc || (c == bc && tk < bt))))) {
                    bu = u; bc = c; bt = tk; bpq = p * S + q;
                  }
                }
              }
              seg_min8(bu, bc, bt, bpq);
              if (!done) {
                if (bt == ~0ull) {
                  done = true;
                } else if (n == kFrontCap) {
                  n = kFrontAll;
                  done = true;
                } else {
                  if (p == 0) sh.fr_pt[k][n] = (uint8_t)bpq;
                  ++n;
                  climit = bc;
                  done = !timed || bc <= gmin;
                }
              }
              if (__ballot(!done) == 0) break;
            }
            if (pv && p == 0) sh.fr_n[k] = (uint8_t)n;
          }
        };
        // score the stored candidates of every pair, one pair per thread
        auto score = [&](auto REP, auto TIMED, int64_t Mf) {
          for (int k = tid; k < R * (R - 1) / 2; k += NT) {
            const int n = sh.fr_n[k];
            if (n == 0) continue;
            int x, y, ra, rb;
            int64_t D;
            pair_of(k, x, y);
            PairCost pc;
            if (!pair_setup(TIMED, k, x, y, ra, rb, D, pc)) continue;
            int64_t other = INT64_MIN;
            for (int t3 = 0; t3 < 3; ++t3) {
              const int tr = sh.top[t3];
              if (tr >= 0 && tr != ra && tr != rb) { other = sh.L[tr]; break; }
            }
            const int64_t La = sh.L[ra], Lb = sh.L[rb];
            const int cnt = n == kFrontAll ? S * S : n;
            for (int m = 0; m < cnt; ++m) {
              const int pq = n == kFrontAll ? m : sh.fr_pt[k][m];
              const int p = pq / S;
              uint64_t c;
              int64_t d;
              int i, j;
              if (!cand(REP, TIMED, ra, rb, p, pq - p * S, pc, c, d, i, j)) continue;
              const int64_t la = La + d, lb = Lb - d;
              int64_t m2 = la > lb ? la : lb;
              if (other > m2) m2 = other;
              const int64_t gain = g_den * (Mf - m2) + g_num * (2 * d * (Lb - La - d));
              if (gain <= 0) continue;
              const uint64_t tk = tie_key(ra, rb, i, j);
              if constexpr (decltype(TIMED)::value) {
                if (ratio_better((uint64_t)gain, c, tk, bgain, bcost, btie)) {
                  bgain = (uint64_t)gain; bcost = c; btie = tk;
                }
              } else if ((uint64_t)gain > bgain || ((uint64_t)gain == bgain && tk < btie)) {
                bgain = (uint64_t)gain; btie = tk;
              }
            }
          }
        };
        auto with_flags = [&](auto f) {
          if (J > 1) {
            if (a.timed) f(Flag<true>{}, Flag<true>{}); else f(Flag<true>{}, Flag<false>{});
          } else {
            if (a.timed) f(Flag<false>{}, Flag<true>{}); else f(Flag<false>{}, Flag<false>{});
          }
        };
        with_flags(build);
        __syncthreads();                         // the frontiers and wave 0's extremes
        if (sh.stop) break;
        const int64_t Mf = sh.L[sh.amax];
        with_flags([&](auto REP, auto TIMED) { score(REP, TIMED, Mf); });
      }
    } else {
      // Full mode, in two phases.  Phase 1 scores every pair (amax, b); the best of those
      // candidates (they stay in the threads' bests) is the reference.  Phase 2 scores the other
      // pairs, skipping each work unit whose benefit bound divided by the lowest cost on its link
      // falls below the reference's ratio: none of its candidates can be the round's best.  The
      // bound of a unit (pair, slot p) is the benefit at the best load difference d = l_j - l_i
      // that rank b's unmoved items allow.
      // Work units are (rank pair, slot p of the first rank), interleaved over the threads so that
      // skipped pairs spread evenly; what does not depend on the second rank's slot q is taken once
      // per unit.
      uint64_t ref_g = 0, ref_c = 1;
      // unit(..., false) runs the checks and the bound and tells whether the unit can hold the
      // round's best; unit(..., true, q0, qs) also scores its candidates q = q0, q0 + qs, ... (a
      // unit's candidates may be shared among several threads)
      auto unit = [&](int ra, int rb, int p, bool eval, int q0 = 0, int qs = 1) -> bool {
        const int64_t La = sh.L[ra], Lb = sh.L[rb];
        if (!(La > Lb)) return false;
        const int sa = ra * S + p;
        if (sh.mslot[sa]) return false;
        if (capped && (sh.part[ra] >= bg.per_rank_cap || sh.part[rb] >= bg.per_rank_cap)) return false;
        int64_t other = INT64_MIN;
        for (int u = 0; u < 3; ++u) {
          const int tr = sh.top[u];
          if (tr >= 0 && tr != ra && tr != rb) { other = sh.L[tr]; break; }
        }
        const int i = sh.item[sa];
        const int64_t li = sh.sload[sa];
        {
          // d = l_j - l_i lies in [smin_b - l_i, smax_b - l_i]; the benefit is concave in d with
          // its real maximum at d = -D/2 (both terms peak there), so over the integers of that
          // range it is largest at the floor or the ceiling of the clipped optimum
          const int64_t dlo = (int64_t)sh.u.run.smin[rb] - li, dhi = (int64_t)sh.u.run.smax[rb] - li;
          if (dlo > dhi) return false;                     // every item of rank b has moved
          const int64_t D = La - Lb;
          auto bound_at = [&](int64_t d) -> int64_t {
            d = d < dlo ? dlo : d > dhi ? dhi : d;
            const int64_t la = La + d, lb = Lb - d;
            int64_t m2 = la > lb ? la : lb;
            if (other > m2) m2 = other;
            return g_den * (M - m2) + g_num * (2 * d * (-D - d));
          };
          const int64_t dfl = -((D + 1) >> 1), dce = -(D >> 1);   // floor and ceiling of -D/2
          const int64_t b1 = bound_at(dfl), b2 = bound_at(dce);
          const int64_t ub = b1 > b2 ? b1 : b2;
          if (ub <= 0) return false;                       // no positive benefit in this unit
          if (ref_g != 0) {
            const int64_t cmin = a.timed ? sh.cmin[sh.node[ra] == sh.node[rb] ? 0 : 1] : 1;
            if ((unsigned __int128)ub * ref_c < (unsigned __int128)ref_g * (uint64_t)cmin) return false;
          }
        }
        const int ei = i >= V ? -1 : J == 1 ? i : expert_of(i, E, inv_e);
        // time budget: the pair's link, and what the candidate's cost may be at most
        int64_t alpha = 0, beta = 1, cap_ns = 0, bi = 0;
        double inv_beta = 1.0;
        bool link_scan = false;
        if (a.timed) {
          const int t = sh.node[ra] == sh.node[rb] ? 0 : 1;
          alpha = a.cost.alpha_ns[t];
          beta = a.cost.beta_bytes_per_us[t];
          inv_beta = 1.0 / (double)beta;
          cap_ns = sh.rank_left[ra] < sh.rank_left[rb] ? sh.rank_left[ra] : sh.rank_left[rb];
          if (sh.cmin[t] > cap_ns) return false;         // no swap on this link fits any more
          link_scan = a.cost.link_budget_ns < a.cost.rank_budget_ns;
          bi = ei >= 0 ? sh.u.run.ebytes[ei] : 0;
        }
        if (!eval) return true;
        const int64_t spread0 = Lb - La;
        for (int q = q0; q < S; q += qs) {
          const int sb = rb * S + q;
          const int j = sh.item[sb];
          if (sh.mslot[sb] || (i >= V && j >= V)) continue;
          if (J > 1 && ((i < V && holds(rb, i)) || (j < V && holds(ra, j)))) continue;
          const int64_t d = (int64_t)sh.sload[sb] - li;
          const int64_t la = La + d, lb = Lb - d;
          int64_t m2 = la > lb ? la : lb;
          if (other > m2) m2 = other;
          const int64_t gain = g_den * (M - m2) + (g_num ? g_num * (2 * d * (spread0 - d)) : 0);
          if (gain <= 0) continue;
          const uint64_t tk = tie_key(ra, rb, i, j);
          if (a.timed) {
            const int ej = j >= V ? -1 : J == 1 ? j : expert_of(j, E, inv_e);
            const int64_t bytes = bi + (ej >= 0 ? sh.u.run.ebytes[ej] : 0);
            const int64_t c = alpha + ceil_div(bytes * 1000, beta, inv_beta);
            if (c > cap_ns) continue;
            if (link_scan && !swap_fits(a, sh, ra, rb, c)) continue;
            if (ratio_better((uint64_t)gain, (uint64_t)c, tk, bgain, bcost, btie)) {
              bgain = (uint64_t)gain; bcost = (uint64_t)c; btie = tk;
            }
          } else if ((uint64_t)gain > bgain || ((uint64_t)gain == bgain && tk < btie)) {
            bgain = (uint64_t)gain; btie = tk;
          }
        }
        return true;
      };
      // phase 1: the pairs (amax, b), each unit's candidates shared by up to S threads
      {
        const int qp = NT / (R * S) < 1 ? 1 : NT / (R * S) > S ? S : NT / (R * S);
        for (int w = tid; w < R * S * qp; w += NT) {
          const int un = w / qp, rb = un / S;
          unit(amax, rb, un - rb * S, true, w - un * qp, qp);
        }
      }
      if (tid == 0) sh.nsurv = 0;
      {
        uint64_t rg = bgain, rc = bcost, rt = btie;
        for (int off = 32; off > 0; off >>= 1) {
          const uint64_t og = __shfl_xor(rg, off), oc = __shfl_xor(rc, off), ot = __shfl_xor(rt, off);
          const bool better = a.timed ? ratio_better(og, oc, ot, rg, rc, rt)
                                      : (og > rg || (og == rg && og != 0 && ot < rt));
          if (better) { rg = og; rc = oc; rt = ot; }
        }
        if (lane == 0) { sh.rgain[wave] = rg; sh.rcost[wave] = rc; sh.rtie[wave] = rt; }
        __syncthreads();
        rg = sh.rgain[0]; rc = sh.rcost[0]; rt = sh.rtie[0];
        for (int w = 1; w < NT / 64; ++w) {
          const bool better = a.timed ? ratio_better(sh.rgain[w], sh.rcost[w], sh.rtie[w], rg, rc, rt)
                                      : (sh.rgain[w] > rg || (sh.rgain[w] == rg && rg != 0 && sh.rtie[w] < rt));
          if (better) { rg = sh.rgain[w]; rc = sh.rcost[w]; rt = sh.rtie[w]; }
        }
        ref_g = rg;
        ref_c = a.timed ? rc : 1;
      }
      // phase 2: a bound test per pair, over every d = l_j - l_i its unmoved items allow, lists the
      // units of the pairs that pass; the listed units (each with its own, tighter bound test) are
      // then scored spread over all threads, so that a wave's lanes are not left idle behind the
      // few pairs that survive
      for (int pair = tid; pair < R * R; pair += NT) {
        const int ra = pair / R, rb = pair - ra * R;
        if (ra == amax) continue;
        const int64_t La = sh.L[ra], Lb = sh.L[rb];
        if (!(La > Lb)) continue;
        if (capped && (sh.part[ra] >= bg.per_rank_cap || sh.part[rb] >= bg.per_rank_cap)) continue;
        const int t = a.timed ? (sh.node[ra] == sh.node[rb] ? 0 : 1) : 0;
        if (a.timed) {
          const int64_t cap_ns = sh.rank_left[ra] < sh.rank_left[rb] ? sh.rank_left[ra] : sh.rank_left[rb];
          if (sh.cmin[t] > cap_ns) continue;
        }
        const int64_t ia = sh.u.run.smin[ra], xa = sh.u.run.smax[ra];
        const int64_t ib = sh.u.run.smin[rb], xb = sh.u.run.smax[rb];
        if (ia > xa || ib > xb) continue;            // every item of a rank has moved
        int64_t other = INT64_MIN;
        for (int u = 0; u < 3; ++u) {
          const int tr = sh.top[u];
          if (tr >= 0 && tr != ra && tr != rb) { other = sh.L[tr]; break; }
        }
        const int64_t dlo = ib - xa, dhi = xb - ia, D = La - Lb;
        auto bound_at = [&](int64_t d) -> int64_t {
          d = d < dlo ? dlo : d > dhi ? dhi : d;
          const int64_t la = La + d, lb = Lb - d;
          int64_t m2 = la > lb ? la : lb;
          if (other > m2) m2 = other;
          return g_den * (M - m2) + g_num * (2 * d * (-D - d));
        };
        const int64_t b1 = bound_at(-((D + 1) >> 1)), b2 = bound_at(-(D >> 1));
        const int64_t ub = b1 > b2 ? b1 : b2;
        if (ub <= 0) continue;
        if (ref_g != 0) {
          const int64_t cmin = a.timed ? sh.cmin[t] : 1;
          if ((unsigned __int128)ub * ref_c < (unsigned __int128)ref_g * (uint64_t)cmin) continue;
        }
        const int at = atomicAdd(&sh.nsurv, S);
        if (at + S <= kSurv) {
          for (int p = 0; p < S; ++p) sh.u.run.surv[at + p] = pair * S + p;
        } else {
          for (int p = 0; p < S; ++p) unit(ra, rb, p, true);
        }
      }
      __syncthreads();
      // (a pair whose units did not fit was scored where it was tested; the list holds whole
      // pairs, so its length is the largest multiple of S not beyond the capacity)
      const int ns2 = sh.nsurv <= kSurv ? sh.nsurv : (kSurv / S) * S;
      const int qp2 = ns2 == 0 ? 1 : NT / ns2 < 1 ? 1 : NT / ns2 > S ? S : NT / ns2;
      for (int w = tid; w < ns2 * qp2; w += NT) {
        const int k = w / qp2;
        const int un = sh.u.run.surv[k];
        const int pair = un / S, p = un - pair * S;
        const int ra = pair / R;
        unit(ra, pair - ra * R, p, true, w - k * qp2, qp2);
      }
    }
    uint64_t g, t, cst = 1;
    // the best candidate of every wave, then of the waves' bests (lane w reads wave w's): by
    // benefit / cost under a time budget, else by benefit; then by tie key
    constexpr int NW = NT / 64;
    if (a.timed) {
      uint64_t wg = bgain, wc = bcost, wt = btie;
      wave_best_ratio(wg, wc, wt);
      if (lane == 0) { sh.wgain[wave] = wg; sh.wtie[wave] = wt; sh.wcost[wave] = wc; }
      __syncthreads();
      g = lane < NW ? sh.wgain[lane] : 0;
      cst = lane < NW ? sh.wcost[lane] : 1;
      t = lane < NW ? sh.wtie[lane] : ~0ull;
      wave_best_ratio(g, cst, t);
    } else {
      const uint64_t wg = wave_max_u64(bgain);
      const uint64_t wt = ~wave_max_u64((wg != 0 && bgain == wg) ? ~btie : 0ull);
      g = wg; t = wt;
      if (NT > 64) {
        if (lane == 0) { sh.wgain[wave] = wg; sh.wtie[wave] = wt; }
        __syncthreads();
        const uint64_t og = lane < NW ? sh.wgain[lane] : 0;
        const uint64_t ot = lane < NW ? sh.wtie[lane] : ~0ull;
        g = wave_max_u64(og);
        t = ~wave_max_u64((g != 0 && og == g) ? ~ot : 0ull);
      }
    }
    if (g == 0) break;                          // no admissible candidate with positive benefit
    if (wave == 0) {
      const int ca = (int)(t >> (kRankBits + 2 * kItemBits)) & ((1 << kRankBits) - 1);
      const int cb = (int)(t >> (2 * kItemBits)) & ((1 << kRankBits) - 1);
      const int ci = (int)(t >> kItemBits) & ((1 << kItemBits) - 1);
      const int cj = (int)t & ((1 << kItemBits) - 1);
      int sa = ca * S, sb = cb * S;               // the winning items' slots (ids are unique)
      for (int s0 = 0; s0 < S; s0 += 64) {
        const int s = s0 + lane;
        const uint64_t ha = __ballot(s < S && sh.item[ca * S + s] == ci);
        const uint64_t hb = __ballot(s < S && sh.item[cb * S + s] == cj);
        if (ha) sa = ca * S + s0 + __ffsll((unsigned long long)ha) - 1;
        if (hb) sb = cb * S + s0 + __ffsll((unsigned long long)hb) - 1;
      }
      if (lane == 0) {
        const int32_t li = sh.sload[sa], lj = sh.sload[sb];
        const int64_t d = (int64_t)lj - (int64_t)li;
        sh.item[sa] = cj; sh.sload[sa] = lj;
        sh.item[sb] = ci; sh.sload[sb] = li;
        sh.L[ca] += d;
        sh.L[cb] -= d;
        sh.mslot[sa] = 1; sh.mslot[sb] = 1;
        ++sh.part[ca]; ++sh.part[cb];
        if constexpr (kFront) {
          sh.last[0] = ca;
          sh.last[1] = cb;
          if (a.timed) {
            const int lo = ca < cb ? ca : cb, hi = ca < cb ? cb : ca;
            sh.link_used[hi * (hi - 1) / 2 + lo] += (int64_t)cst;
          }
        }
        fb_swap sw;
        sw.src_rank = ca; sw.dst_rank = cb; sw.src_slot = sa - ca * S; sw.dst_slot = sb - cb * S;
        sw.expert_src = ci < V ? ci : -1;
        sw.expert_dst = cj < V ? cj : -1;
        sw.gain = (int64_t)g;
        a.swaps[sh.ns] = sw;
        if (a.timed) {
          sh.rank_left[ca] -= (int64_t)cst;
          sh.rank_left[cb] -= (int64_t)cst;
          sh.acc_pair[sh.ns] = ca < cb ? ca * kMaxR + cb : cb * kMaxR + ca;
          sh.acc_cost[sh.ns] = (int64_t)cst;
          if (a.swap_cost_ns) a.swap_cost_ns[sh.ns] = (int64_t)cst;
        }
        sh.ns = sh.ns + 1;
      }
    }
    __syncthreads();
  }

  __syncthreads();
  for (int c = tid; c < RS; c += NT) {
    const int it = sh.item[c];
    a.new_slot_expert[c] = it < V ? it : -1;
    if (it < E) a.new_expert_to_rank[it] = c / S;   // replica 0
  }
  for (int r = tid; r < R; r += NT) a.new_rank_loads[r] = sh.L[r];
  if (tid == 0) { *a.n_swaps = sh.ns; *a.status = FB_OK; }
}

// ---- one-wave frontier planner (fb_plan_wave.h) as a kernel of its own -----------------------
template <int RPL, int CPL>
__global__ __launch_bounds__(64, 1) void plan_frontier_wave(PlanDeviceLaunch a) {
  constexpr int CAP = wave_cap(RPL, CPL);   // >= R * S >= E
  __shared__ __attribute__((aligned(16))) char lds[plan_wave_lds_bytes(CAP, RPL)];
  plan_wave_body<RPL, CPL>(a, plan_wave_lds(lds, CAP, RPL));
}

}  // namespace

int launch_plan_device(const PlanDeviceLaunch& a) {
  (void)hipGetLastError();
  hipStream_t st = static_cast<hipStream_t>(a.stream);
  if (a.budget.mode == FB_FRONTIER && (int64_t)a.S * a.S <= 128 && (!a.timed || a.R <= 64)) {
    // the routing below keeps R * S within the chosen kernel's slot capacity (time budgets: one
    // rank per lane)
    const int rpl = a.R <= 64 ? 1 : a.R <= 128 ? 2 : a.R <= 256 ? 4 : 16;
    if ((int64_t)a.R * a.S > wave_cap(rpl, (int64_t)a.S * a.S <= 64 ? 1 : 2)) return FB_EUNSUPPORTED;
    if ((int64_t)a.S * a.S <= 64) {
      if (a.R <= 64) hipLaunchKernelGGL((plan_frontier_wave<1, 1>), dim3(1), dim3(64), 0, st, a);
      else if (a.R <= 128) hipLaunchKernelGGL((plan_frontier_wave<2, 1>), dim3(1), dim3(64), 0, st, a);
      else if (a.R <= 256) hipLaunchKernelGGL((plan_frontier_wave<4, 1>), dim3(1), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((plan_frontier_wave<16, 1>), dim3(1), dim3(64), 0, st, a);
    } else {
      if (a.R <= 64) hipLaunchKernelGGL((plan_frontier_wave<1, 2>), dim3(1), dim3(64), 0, st, a);
      else if (a.R <= 128) hipLaunchKernelGGL((plan_frontier_wave<2, 2>), dim3(1), dim3(64), 0, st, a);
      else if (a.R <= 256) hipLaunchKernelGGL((plan_frontier_wave<4, 2>), dim3(1), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((plan_frontier_wave<16, 2>), dim3(1), dim3(64), 0, st, a);
    }
  }
  else {
    const bool small = (int64_t)a.R * a.S <= kSmallRS && a.R <= kSmallR;
    if (a.budget.mode == FB_FRONTIER) {
      if (small) hipLaunchKernelGGL((plan_general<256, true>), dim3(1), dim3(256), 0, st, a);
      else hipLaunchKernelGGL((plan_general<256, false>), dim3(1), dim3(256), 0, st, a);
    } else {
      if (small) hipLaunchKernelGGL((plan_general<1024, true>), dim3(1), dim3(1024), 0, st, a);
      else hipLaunchKernelGGL((plan_general<1024, false>), dim3(1), dim3(1024), 0, st, a);
    }
  }
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

}  // namespace fb
