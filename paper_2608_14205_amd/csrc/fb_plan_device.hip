// Budgeted greedy expert-swap planner as one stream-ordered workgroup (gfx950).
//
// Same algorithm and tie-breaks as the host planner (Sec. "Budgeted Expert-Swap Planning",
// Eq. 6-8, Alg. 1): every round finds the most and least loaded ranks, evaluates every admissible
// candidate in parallel (one thread per candidate, exact integer benefit
// den * (M - M') + num * 2d (L_b - L_a - d)), reduces to the best candidate under the ordering
// (benefit desc, src rank, dst rank, item ids asc), and one thread applies it.  State lives in LDS;
// the only global traffic is the input tables and the outputs.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fb_internal.h"

namespace fb {
namespace {

constexpr int kPlanThreads = 256;
constexpr int kMaxRS = FB_MAX_SLOTS_TOTAL;
constexpr int kMaxR = FB_MAX_RANKS;

typedef __int128 i128;

struct Cand {
  int64_t gain;   // exact: bounded by the host-side overflow check
  int64_t i, j;   // item ids
  int32_t a, b, p, q;
  int32_t found;
};

__device__ __forceinline__ bool cand_better(const Cand& x, const Cand& y) {
  if (!x.found) return false;
  if (!y.found) return true;
  if (x.gain != y.gain) return x.gain > y.gain;
  if (x.a != y.a) return x.a < y.a;
  if (x.b != y.b) return x.b < y.b;
  if (x.i != y.i) return x.i < y.i;
  return x.j < y.j;
}

// (value, rank) order used for the frontier: larger load first, lower rank id on ties.
__device__ __forceinline__ bool load_before(int64_t lv, int32_t lr, int64_t rv, int32_t rr) {
  return lv > rv || (lv == rv && lr < rr);
}

__global__ __launch_bounds__(kPlanThreads, 1) void plan_kernel(PlanDeviceLaunch a) {
  __shared__ int32_t item[kMaxRS];
  __shared__ int32_t cnt[kMaxRS];
  __shared__ uint8_t moved[2 * kMaxRS];
  __shared__ int64_t L[kMaxR];
  __shared__ int32_t part[kMaxR];
  __shared__ int32_t seen[kMaxRS];
  __shared__ Cand red[kPlanThreads];
  __shared__ int32_t s_bad, s_stop, s_amax, s_amin, s_top[3], s_ns;
  __shared__ int64_t s_N;

  const int tid = threadIdx.x;
  const int E = a.E, R = a.R, S = a.S, RS = R * S;
  const fb_budget bg = a.budget;

  if (tid == 0) { s_bad = 0; s_ns = 0; s_N = 0; }
  for (int e = tid; e < E; e += kPlanThreads) { seen[e] = 0; cnt[e] = a.counts[e]; }
  for (int c = tid; c < E + RS; c += kPlanThreads) moved[c] = 0;
  for (int r = tid; r < R; r += kPlanThreads) part[r] = 0;
  __syncthreads();
  for (int c = tid; c < RS; c += kPlanThreads) {
    const int e = a.slot_expert[c];
    if (e == -1) item[c] = E + c;
    else if (e < 0 || e >= E) s_bad = 1;
    else { item[c] = e; atomicAdd(&seen[e], 1); }
  }
  __syncthreads();
  for (int e = tid; e < E; e += kPlanThreads)
    if (seen[e] != 1 || cnt[e] < 0) s_bad = 1;
  __syncthreads();
  if (s_bad) {
    if (tid == 0) { *a.n_swaps = 0; *a.status = FB_EINVAL; }
    return;
  }

  auto load_of = [&](int64_t it) -> int64_t { return it < E ? (int64_t)cnt[it] : 0; };
  for (int r = tid; r < R; r += kPlanThreads) {
    int64_t v = 0;
    for (int s = 0; s < S; ++s) v += load_of(item[r * S + s]);
    L[r] = v;
    atomicAdd((unsigned long long*)&s_N, (unsigned long long)v);
  }
  __syncthreads();
  const int64_t N = s_N;
  i128 g_num = bg.gamma_num, g_den = bg.gamma_den;
  if (g_den == 0) { g_num = N > 0 ? 1 : 0; g_den = N > 0 ? N : 1; }
  const i128 bound = g_den * (i128)N + g_num * 4 * (i128)N * (i128)N;
  if (bound > (i128)INT64_MAX) {
    if (tid == 0) { *a.n_swaps = 0; *a.status = FB_EUNSUPPORTED; }
    return;
  }

  const bool active = N > 0 && bg.max_swaps > 0 && R > 1;
  for (int round = 0; active && round < bg.max_swaps; ++round) {
    // ---- frontier: wave 0 finds argmax, argmin and the three largest loads --------------------
    if (tid < 64) {
      int64_t bv = INT64_MIN; int32_t br = 0x7fffffff;    // argmax (lowest id on ties)
      int64_t mv = INT64_MAX; int32_t mr = 0x7fffffff;    // argmin (lowest id on ties)
      for (int r = tid; r < R; r += 64) {
        if (load_before(L[r], r, bv, br)) { bv = L[r]; br = r; }
        if (L[r] < mv || (L[r] == mv && r < mr)) { mv = L[r]; mr = r; }
      }
      for (int off = 32; off > 0; off >>= 1) {
        const int64_t ov = __shfl_xor(bv, off); const int32_t orr = __shfl_xor(br, off);
        if (load_before(ov, orr, bv, br)) { bv = ov; br = orr; }
        const int64_t om = __shfl_xor(mv, off); const int32_t omr = __shfl_xor(mr, off);
        if (om < mv || (om == mv && omr < mr)) { mv = om; mr = omr; }
      }
      int32_t top[3] = {br, -1, -1};
      for (int u = 1; u < 3; ++u) {
        int64_t tv = INT64_MIN; int32_t tr = 0x7fffffff;
        for (int r = tid; r < R; r += 64) {
          bool used = false;
          for (int w = 0; w < u; ++w) used |= (top[w] == r);
          if (!used && load_before(L[r], r, tv, tr)) { tv = L[r]; tr = r; }
        }
        for (int off = 32; off > 0; off >>= 1) {
          const int64_t ov = __shfl_xor(tv, off); const int32_t orr = __shfl_xor(tr, off);
          if (load_before(ov, orr, tv, tr)) { tv = ov; tr = orr; }
        }
        top[u] = (tr == 0x7fffffff) ? -1 : tr;
      }
      if (tid == 0) {
        s_amax = br; s_amin = mr;
        s_top[0] = top[0]; s_top[1] = top[1]; s_top[2] = top[2];
        s_stop = (L[br] - L[mr] <= bg.tau) ? 1 : 0;
      }
    }
    __syncthreads();
    if (s_stop) break;

    // ---- candidates, one per thread-iteration --------------------------------------------------
    const int amax = s_amax, amin = s_amin;
    const int64_t M = L[amax];
    Cand best; best.found = 0; best.gain = 0; best.i = best.j = 0; best.a = best.b = best.p = best.q = 0;
    const int64_t ncand = bg.mode == FB_FRONTIER ? (int64_t)S * S : (int64_t)R * R * S * S;
    for (int64_t idx = tid; idx < ncand; idx += kPlanThreads) {
      int ra, rb, p, q;
      if (bg.mode == FB_FRONTIER) {
        ra = amax; rb = amin; p = (int)(idx / S); q = (int)(idx % S);
      } else {
        const int64_t pair = idx / ((int64_t)S * S), pq = idx % ((int64_t)S * S);
        ra = (int)(pair / R); rb = (int)(pair % R); p = (int)(pq / S); q = (int)(pq % S);
        if (!(L[ra] > L[rb])) continue;
      }
      if (bg.per_rank_cap && (part[ra] >= bg.per_rank_cap || part[rb] >= bg.per_rank_cap)) continue;
      const int64_t i = item[ra * S + p], j = item[rb * S + q];
      if (moved[i] || moved[j] || (i >= E && j >= E)) continue;
      int64_t other = INT64_MIN;
      for (int u = 0; u < 3; ++u) {
        const int tr = s_top[u];
        if (tr >= 0 && tr != ra && tr != rb) { other = L[tr]; break; }
      }
      const int64_t d = load_of(j) - load_of(i);
      const int64_t la = L[ra] + d, lb = L[rb] - d;
      int64_t m2 = la > lb ? la : lb;
      if (other > m2) m2 = other;
      const i128 gain = g_den * (i128)(M - m2) + g_num * 2 * (i128)d * (i128)(L[rb] - L[ra] - d);
      if (gain <= 0) continue;
      Cand c; c.found = 1; c.gain = (int64_t)gain; c.i = i; c.j = j; c.a = ra; c.b = rb; c.p = p; c.q = q;
      if (cand_better(c, best)) best = c;
    }
    red[tid] = best;
    __syncthreads();
    for (int stride = kPlanThreads / 2; stride > 0; stride >>= 1) {
      if (tid < stride && cand_better(red[tid + stride], red[tid])) red[tid] = red[tid + stride];
      __syncthreads();
    }
    if (!red[0].found) break;
    if (tid == 0) {
      const Cand c = red[0];
      const int64_t d = load_of(c.j) - load_of(c.i);
      item[c.a * S + c.p] = (int32_t)c.j;
      item[c.b * S + c.q] = (int32_t)c.i;
      L[c.a] += d;
      L[c.b] -= d;
      moved[c.i] = 1; moved[c.j] = 1;
      ++part[c.a]; ++part[c.b];
      fb_swap sw;
      sw.src_rank = c.a; sw.dst_rank = c.b; sw.src_slot = c.p; sw.dst_slot = c.q;
      sw.expert_src = c.i < E ? (int32_t)c.i : -1;
      sw.expert_dst = c.j < E ? (int32_t)c.j : -1;
      sw.gain = c.gain;
      a.swaps[s_ns] = sw;
      s_ns = s_ns + 1;
    }
    __syncthreads();
  }

  __syncthreads();
  for (int c = tid; c < RS; c += kPlanThreads) {
    const int it = item[c];
    a.new_slot_expert[c] = it < E ? it : -1;
    if (it < E) a.new_expert_to_rank[it] = c / S;
  }
  for (int r = tid; r < R; r += kPlanThreads) a.new_rank_loads[r] = L[r];
  if (tid == 0) { *a.n_swaps = s_ns; *a.status = FB_OK; }
}

}  // namespace

int launch_plan_device(const PlanDeviceLaunch& a) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, static_cast<hipStream_t>(a.stream), a);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

}  // namespace fb
