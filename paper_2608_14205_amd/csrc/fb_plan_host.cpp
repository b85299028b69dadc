// Budgeted greedy expert-swap planner, host implementation (no HIP calls).
//
// Sec. "Budgeted Expert-Swap Planning" and Alg. 1.  A swap of the item in slot p of rank a with
// the item in slot q of rank b changes only those two loads (Eq. 6-7):
//     d = n_j - n_i,  L'_a = L_a + d,  L'_b = L_b - d.
// With N = sum L fixed, sum_r (L_r - mean)^2 = sum L^2 - N^2 / R, so the benefit of Eq. 8 is
//     Delta = (M - M') + gamma * (sum L^2 - sum L'^2) = (M - M') + gamma * 2d (L_b - L_a - d),
// M' = max(L'_a, L'_b, max over the other ranks).  With gamma = num / den the planner ranks the
// exact integer den * Delta = den (M - M') + num * 2d (L_b - L_a - d) in 128-bit arithmetic.
//
// Each round re-enumerates the candidates at the current loads (frontier: the most and the least
// loaded rank, lowest rank id on ties; full: every ordered pair with L_a > L_b), drops items that
// already moved, pairs of empty slots, ranks over their per-rank cap and non-positive benefits, and
// accepts the candidate with the largest benefit, ties broken by (layer, src rank, dst rank, item
// ids).  Empty slots are zero-load items with id E + r * S + s.  The loop ends when the swap cap is
// reached, L_max - L_min <= tau, or no candidate remains.
//
// Under a time budget (fb_plan_swaps_timed) every candidate also costs C = alpha + ceil(bytes *
// 1000 / beta) ns on its link (Eq. 9), must fit what is left of both ranks' and the link's budgets
// (Eq. 10, enforced per participant), and candidates are ranked by benefit / C, compared exactly as
// gain_1 * C_2 vs gain_2 * C_1.
//
// Replicated placements (a history-driven placement that copies hot experts, on top of which the
// paper also runs its planner): slot value v = e + E * j is replica j of expert e.  Replica j of an
// expert with n tokens and c replicas carries floor(n / c) tokens, plus one if j < n mod c, and
// keeps its ordinal when it moves, so Eq. 6-7 hold with these shares as the item loads.  Empty
// slots then take the ids E * J + r * S + s (J = the largest replica count, 1 without replicas).
// A candidate may not put a replica on a rank that already holds one of the same expert.
#include <stdint.h>
#include <math.h>
#include <string.h>

#include <algorithm>
#include <unordered_map>
#include <vector>

#include "fb_internal.h"

namespace {

typedef __int128 i128;


struct Best {
  bool found = false;
  i128 gain = 0;
  int64_t cost = 1;     // 1 for every candidate under a swap-count budget
  int32_t a = 0, b = 0, p = 0, q = 0;
  int64_t i = 0, j = 0;
};

// Candidate ordering: larger gain / cost first (exact cross-multiplication; gains < 2^63 and costs
// < 2^42, so the products fit 128 bits), then lexicographically smaller (a, b, i, j).
bool better(i128 gain, int64_t cost, int32_t a, int32_t b, int64_t i, int64_t j, const Best& cur) {
  if (!cur.found) return true;
  const i128 lhs = gain * cur.cost, rhs = cur.gain * cost;
  if (lhs != rhs) return lhs > rhs;
  if (a != cur.a) return a < cur.a;
  if (b != cur.b) return b < cur.b;
  if (i != cur.i) return i < cur.i;
  return j < cur.j;
}

// The time budget, when there is one: link types from the rank nodes, expert sizes, and what is
// left of every rank's and every used link's budget.
struct TimeBudget {
  fb_cost_model m;
  const int32_t* rank_node;
  const int64_t* expert_bytes;
  int32_t E, R;
  int64_t link_cap;
  std::vector<int64_t> rank_left;
  std::unordered_map<int64_t, int64_t> link_used;   // key a * R + b with a < b

  // Eq. 9 in whole ns for moving experts ei and ej (-1: an empty slot, which transfers nothing)
  int64_t cost(int32_t a, int32_t b, int64_t ei, int64_t ej) const {
    const int t = rank_node[a] == rank_node[b] ? 0 : 1;
    const int64_t bytes = (ei >= 0 ? expert_bytes[ei] : 0) + (ej >= 0 ? expert_bytes[ej] : 0);
    const int64_t beta = m.beta_bytes_per_us[t];
    return m.alpha_ns[t] + (bytes * 1000 + beta - 1) / beta;
  }
  int64_t link_key(int32_t a, int32_t b) const {
    return a < b ? (int64_t)a * R + b : (int64_t)b * R + a;
  }
  bool fits(int32_t a, int32_t b, int64_t c) const {
    if (c > rank_left[a] || c > rank_left[b]) return false;
    const auto it = link_used.find(link_key(a, b));
    return c <= link_cap - (it == link_used.end() ? 0 : it->second);
  }
  void charge(int32_t a, int32_t b, int64_t c) {
    rank_left[a] -= c;
    rank_left[b] -= c;
    link_used[link_key(a, b)] += c;
  }
};

int plan_impl(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R, int32_t S,
              const fb_budget* budget, TimeBudget* tb, fb_swap* swaps, int64_t* swap_cost_ns,
              int32_t swaps_cap, int32_t* n_swaps, int32_t* new_slot_expert,
              int32_t* new_expert_to_rank, int64_t* new_rank_loads) {
  if (!counts || !slot_expert || !budget || !n_swaps || (swaps_cap > 0 && !swaps)) return FB_EINVAL;
  if (E < 1 || R < 1 || S < 1) return FB_EINVAL;
  if ((int64_t)R * S > (int64_t)1 << 30) return FB_EUNSUPPORTED;
  const fb_budget bg = *budget;
  if (bg.max_swaps < 0 || bg.per_rank_cap < 0 || bg.tau < 0 || bg.gamma_num < 0 || bg.gamma_den < 0)
    return FB_EINVAL;
  if (bg.mode != FB_FRONTIER && bg.mode != FB_FULL) return FB_EINVAL;
  if (swaps_cap < bg.max_swaps) return FB_ENOSPC;

  const int64_t RS = (int64_t)R * S;
  if (E > RS) return FB_EINVAL;
  for (int32_t e = 0; e < E; ++e)
    if (counts[e] < 0) return FB_EINVAL;
  // placement rules: every replica once, ordinals 0 .. c_e - 1 of every expert, no rank with two
  // replicas of one expert (so no ordinal reaches R)
  std::vector<int32_t> vals;
  vals.reserve(RS);
  for (int64_t c = 0; c < RS; ++c) {
    const int32_t v = slot_expert[c];
    if (v == -1) continue;
    if (v < 0 || v / E >= R) return FB_EINVAL;
    vals.push_back(v);
  }
  std::sort(vals.begin(), vals.end());
  std::vector<int32_t> reps(E, 0);
  for (size_t u = 0; u < vals.size(); ++u) {
    if (u > 0 && vals[u] == vals[u - 1]) return FB_EINVAL;
    ++reps[vals[u] % E];
  }
  int32_t J = 1;
  for (int32_t e = 0; e < E; ++e) {
    if (reps[e] == 0) return FB_EINVAL;
    J = reps[e] > J ? reps[e] : J;
  }
  // with distinct values, the ordinals of e are 0 .. c_e - 1 iff none reaches c_e
  for (const int32_t v : vals)
    if (v / E >= reps[v % E]) return FB_EINVAL;
  const int64_t V = (int64_t)E * J;                  // slot values are below V
  if (J > 1 && (int64_t)R * E > ((int64_t)1 << 24)) return FB_EUNSUPPORTED;   // held[] <= 16 MB
  std::vector<uint8_t> held(J > 1 ? (size_t)R * E : 0, 0);   // held[r * E + e]: e on rank r
  for (int32_t r = 0; r < R && J > 1; ++r)
    for (int32_t s = 0; s < S; ++s) {
      const int32_t v = slot_expert[(int64_t)r * S + s];
      if (v < 0) continue;
      uint8_t& h = held[(size_t)r * E + v % E];
      if (h) return FB_EINVAL;
      h = 1;
    }

  // items: slot contents; empty slot (r, s) becomes the zero-load item V + r*S + s
  std::vector<int64_t> item(RS);
  for (int64_t c = 0; c < RS; ++c) item[c] = slot_expert[c] >= 0 ? slot_expert[c] : V + c;
  auto expert_of = [&](int64_t it) -> int64_t { return it < V ? it % E : -1; };
  auto load_of = [&](int64_t it) -> int64_t {
    if (it >= V) return 0;
    const int64_t e = it % E, j = it / E, n = counts[e], c = reps[e];
    return n / c + (j < n % c ? 1 : 0);
  };

  std::vector<int64_t> L(R, 0);
  for (int32_t r = 0; r < R; ++r)
    for (int32_t s = 0; s < S; ++s) L[r] += load_of(item[(int64_t)r * S + s]);
  int64_t N = 0;
  for (int32_t r = 0; r < R; ++r) N += L[r];

  i128 g_num = bg.gamma_num, g_den = bg.gamma_den;
  if (g_den == 0) {
    g_num = N > 0 ? 1 : 0;
    g_den = N > 0 ? N : 1;
  }
  // every reported benefit must fit an int64: |den (M - M')| <= den N, |num 2d(...)| <= num 4 N^2
  const i128 bound = g_den * (i128)N + g_num * 4 * (i128)N * (i128)N;
  if (bound > (i128)INT64_MAX) return FB_EUNSUPPORTED;

  std::vector<uint8_t> moved(V + RS, 0);
  std::vector<int32_t> part(R, 0);
  int32_t ns = 0;
  const bool active = N > 0 && bg.max_swaps > 0 && R > 1;
  while (active && ns < bg.max_swaps) {
    int32_t amax = 0, amin = 0;
    for (int32_t r = 1; r < R; ++r) {
      if (L[r] > L[amax]) amax = r;
      if (L[r] < L[amin]) amin = r;
    }
    if (L[amax] - L[amin] <= bg.tau) break;
    // top three loads (lowest rank id first on ties) for max over ranks other than a pair
    int32_t top[3] = {-1, -1, -1};
    for (int32_t r = 0; r < R; ++r) {
      for (int u = 0; u < 3; ++u) {
        if (top[u] < 0 || L[r] > L[top[u]]) {
          for (int v = 2; v > u; --v) top[v] = top[v - 1];
          top[u] = r;
          break;
        }
      }
    }
    const int64_t M = L[amax];
    Best best;
    auto consider = [&](int32_t a, int32_t b) {
      if (bg.per_rank_cap && (part[a] >= bg.per_rank_cap || part[b] >= bg.per_rank_cap)) return;
      int64_t other = INT64_MIN;
      for (int u = 0; u < 3; ++u)
        if (top[u] >= 0 && top[u] != a && top[u] != b) { other = L[top[u]]; break; }
      for (int32_t p = 0; p < S; ++p) {
        const int64_t i = item[(int64_t)a * S + p];
        if (moved[i]) continue;
        for (int32_t q = 0; q < S; ++q) {
          const int64_t j = item[(int64_t)b * S + q];
          if (moved[j] || (i >= V && j >= V)) continue;
          if (J > 1 && ((i < V && held[(size_t)b * E + i % E]) ||
                        (j < V && held[(size_t)a * E + j % E])))
            continue;
          const int64_t d = load_of(j) - load_of(i);
          const int64_t la = L[a] + d, lb = L[b] - d;
          int64_t m2 = la > lb ? la : lb;
          if (other > m2) m2 = other;
          const i128 gain = g_den * (i128)(M - m2) + g_num * 2 * (i128)d * (i128)(L[b] - L[a] - d);
          if (gain <= 0) continue;
          int64_t c = 1;
          if (tb) {
            c = tb->cost(a, b, expert_of(i), expert_of(j));
            if (!tb->fits(a, b, c)) continue;
          }
          if (better(gain, c, a, b, i, j, best)) {
            best.found = true; best.gain = gain; best.cost = c;
            best.a = a; best.b = b; best.p = p; best.q = q; best.i = i; best.j = j;
          }
        }
      }
    };
    if (bg.mode == FB_FRONTIER) {
      consider(amax, amin);
    } else {
      for (int32_t a = 0; a < R; ++a)
        for (int32_t b = 0; b < R; ++b)
          if (L[a] > L[b]) consider(a, b);
    }
    if (!best.found) break;
    const int64_t ca = (int64_t)best.a * S + best.p, cb = (int64_t)best.b * S + best.q;
    const int64_t d = load_of(best.j) - load_of(best.i);
    item[ca] = best.j;
    item[cb] = best.i;
    if (J > 1) {
      if (best.i < V) {
        held[(size_t)best.a * E + best.i % E] = 0;
        held[(size_t)best.b * E + best.i % E] = 1;
      }
      if (best.j < V) {
        held[(size_t)best.b * E + best.j % E] = 0;
        held[(size_t)best.a * E + best.j % E] = 1;
      }
    }
    L[best.a] += d;
    L[best.b] -= d;
    moved[best.i] = moved[best.j] = 1;
    ++part[best.a];
    ++part[best.b];
    fb_swap& sw = swaps[ns++];
    sw.src_rank = best.a;
    sw.dst_rank = best.b;
    sw.src_slot = best.p;
    sw.dst_slot = best.q;
    sw.expert_src = best.i < V ? (int32_t)best.i : -1;
    sw.expert_dst = best.j < V ? (int32_t)best.j : -1;
    sw.gain = (int64_t)best.gain;
    if (tb) {
      tb->charge(best.a, best.b, best.cost);
      if (swap_cost_ns) swap_cost_ns[ns - 1] = best.cost;
    }
  }

  *n_swaps = ns;
  if (new_slot_expert)
    for (int64_t c = 0; c < RS; ++c) new_slot_expert[c] = item[c] < V ? (int32_t)item[c] : -1;
  if (new_expert_to_rank)   // the rank of replica 0
    for (int64_t c = 0; c < RS; ++c)
      if (item[c] < E) new_expert_to_rank[item[c]] = (int32_t)(c / S);
  if (new_rank_loads)
    for (int32_t r = 0; r < R; ++r) new_rank_loads[r] = L[r];
  return FB_OK;
}

}  // namespace

extern "C" int fb_plan_swaps(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                             int32_t S, const fb_budget* budget, fb_swap* swaps, int32_t swaps_cap,
                             int32_t* n_swaps, int32_t* new_slot_expert,
                             int32_t* new_expert_to_rank, int64_t* new_rank_loads) {
  return plan_impl(counts, E, slot_expert, R, S, budget, nullptr, swaps, nullptr, swaps_cap, n_swaps,
                   new_slot_expert, new_expert_to_rank, new_rank_loads);
}

extern "C" int fb_plan_swaps_timed(const int32_t* counts, int32_t E, const int32_t* slot_expert,
                                   int32_t R, int32_t S, const fb_budget* budget,
                                   const fb_cost_model* cost, const int32_t* rank_node,
                                   const int64_t* expert_bytes, fb_swap* swaps,
                                   int64_t* swap_cost_ns, int32_t swaps_cap, int32_t* n_swaps,
                                   int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                                   int64_t* new_rank_loads) {
  if (!cost || !rank_node || !expert_bytes || E < 1 || R < 1) return FB_EINVAL;
  const fb_cost_model m = *cost;
  if (m.rank_budget_ns < 0 || m.link_budget_ns < -1) return FB_EINVAL;
  for (int t = 0; t < 2; ++t)
    if (m.alpha_ns[t] < 1 || m.alpha_ns[t] > fb::kCostLimit || m.beta_bytes_per_us[t] < 1 ||
        m.beta_bytes_per_us[t] > fb::kCostLimit)
      return FB_EINVAL;
  for (int32_t e = 0; e < E; ++e)
    if (expert_bytes[e] < 0 || expert_bytes[e] > fb::kCostLimit) return FB_EINVAL;
  TimeBudget tb;
  tb.m = m;
  tb.rank_node = rank_node;
  tb.expert_bytes = expert_bytes;
  tb.E = E;
  tb.R = R;
  tb.link_cap = m.link_budget_ns < 0 ? m.rank_budget_ns : m.link_budget_ns;
  tb.rank_left.assign(R, m.rank_budget_ns);
  return plan_impl(counts, E, slot_expert, R, S, budget, &tb, swaps, swap_cost_ns, swaps_cap,
                   n_swaps, new_slot_expert, new_expert_to_rank, new_rank_loads);
}

extern "C" int64_t fb_swap_budget_from_cost(double t_attn_us, double delta_us, double alpha_us,
                                            double beta_bytes_per_us, int64_t expert_bytes) {
  const double vals[4] = {t_attn_us, delta_us, alpha_us, beta_bytes_per_us};
  for (double v : vals)
    if (!(v == v) || v > 1e300 || v < -1e300) return FB_EINVAL;  // NaN or infinite
  if (beta_bytes_per_us <= 0.0 || alpha_us < 0.0 || expert_bytes < 0) return FB_EINVAL;
  const double cost = alpha_us + 2.0 * (double)expert_bytes / beta_bytes_per_us;  // Eq. 9
  if (!(cost > 0.0)) return FB_EINVAL;
  const double window = t_attn_us - delta_us > 0.0 ? t_attn_us - delta_us : 0.0;  // Eq. 10
  const double n = window / cost;
  if (n >= 9.0e15) return FB_EINVAL;
  int64_t c = (int64_t)n;  // floor for n >= 0, then corrected against the exact product: the sign of
  // fma(c, cost, -window) is the sign of the exact c * cost - window
  while (c > 0 && fma((double)c, cost, -window) > 0.0) --c;
  while (fma((double)(c + 1), cost, -window) <= 0.0) ++c;
  return c;
}
