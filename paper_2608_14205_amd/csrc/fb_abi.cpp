// C ABI entry points of libfreebalance.so: argument validation, device check and dispatch to the
// HIP launchers.  Validation happens before any HIP call, so invalid arguments are reported on a
// machine without a GPU as well.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#include "fb_internal.h"

namespace fb {

namespace {
std::atomic<int> g_arch_cache[64];  // 0 unknown, 1 gfx950, 2 other
std::atomic<int> g_cu_cache[64];    // compute units, 0 unknown
}  // namespace

int check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return FB_EDEVICE;
  }
  if (dev < 64) {
    const int c = g_arch_cache[dev].load(std::memory_order_relaxed);
    if (c == 1) return FB_OK;
    if (c == 2) return FB_EUNSUPPORTED;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
    (void)hipGetLastError();
    return FB_EDEVICE;
  }
  const bool ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev < 64) {
    g_cu_cache[dev].store(prop.multiProcessorCount, std::memory_order_relaxed);
    g_arch_cache[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
  }
  return ok ? FB_OK : FB_EUNSUPPORTED;
}

int device_cu_count() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 256;
  }
  const int n = g_cu_cache[dev].load(std::memory_order_relaxed);
  return n > 0 ? n : 256;
}

}  // namespace fb

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

// Host-side checks of the routing rule; see fb_scoring in freebalance.h.
int check_scoring(const fb_scoring& s, int32_t E, const float* select_bias) {
  if (s.kind != FB_SOFTMAX && s.kind != FB_SIGMOID) return FB_EINVAL;
  if (s.kind == FB_SOFTMAX && select_bias) return FB_EINVAL;
  if (s.k < 1 || s.k > E) return FB_EINVAL;
  if (s.n_group < 1 || E % s.n_group != 0) return FB_EINVAL;
  if (s.n_group > 1) {
    if (s.topk_group < 1 || s.topk_group > s.n_group) return FB_EINVAL;
    if (s.group_topn != 1 && s.group_topn != 2) return FB_EINVAL;
    // a sum of logits does not order groups like the sum of their softmax probabilities
    if (s.kind == FB_SOFTMAX && s.group_topn == 2) return FB_EUNSUPPORTED;
    const int gsz = E / s.n_group;
    if ((int64_t)s.k > (int64_t)s.topk_group * gsz) return FB_EINVAL;
    if (s.group_topn > gsz) return FB_EINVAL;
    if (s.n_group > 32) return FB_EUNSUPPORTED;
    const bool lanes_whole = gsz % 16 == 0 && is_pow2(gsz / 16);
    const bool within_lane = gsz < 16 && 16 % gsz == 0;
    if (!lanes_whole && !within_lane) return FB_EUNSUPPORTED;
  }
  if (s.k > FB_MAX_TOPK) return FB_EUNSUPPORTED;
  return FB_OK;
}

}  // namespace

extern "C" {

int fb_abi_version(void) { return FB_ABI_VERSION; }

const char* fb_status_string(int status) {
  switch (status) {
    case FB_OK: return "FB_OK";
    case FB_EINVAL: return "FB_EINVAL: invalid argument";
    case FB_EUNSUPPORTED: return "FB_EUNSUPPORTED: unsupported shape, option or device";
    case FB_EDEVICE: return "FB_EDEVICE: HIP runtime error";
    case FB_ENOSPC: return "FB_ENOSPC: buffer or workspace too small";
    default: return "unknown freebalance status";
  }
}

size_t fb_router_packed_bytes(int32_t E, int32_t H, int32_t dtype) {
  if (E < 1 || E > FB_MAX_EXPERTS || H < 1 || (dtype != FB_BF16 && dtype != FB_F32)) return 0;
  return fb::router_packed_bytes(E, H, dtype);
}

size_t fb_predict_workspace_bytes(int32_t E, int32_t H, int32_t dtype) {
  const size_t packed = fb_router_packed_bytes(E, H, dtype);
  return packed ? fb::kWsBytes + packed : 0;
}

int fb_predict_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || !aligned16(workspace)) return FB_EINVAL;
  if (workspace_bytes < fb::kWsBytes) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_workspace_zero(workspace, fb::kWsBytes, stream);
}

int fb_pack_router_weight(const void* router_w, int32_t E, int32_t H, int32_t dtype, void* packed,
                          size_t packed_bytes, void* stream) {
  if (!router_w || !packed || E < 1 || H < 1) return FB_EINVAL;
  if (dtype != FB_BF16 && dtype != FB_F32) return FB_EINVAL;
  if (E > FB_MAX_EXPERTS) return FB_EUNSUPPORTED;
  if (H % (dtype == FB_BF16 ? 32 : 16) != 0) return FB_EUNSUPPORTED;
  if (!aligned16(router_w) || !aligned16(packed)) return FB_EUNSUPPORTED;
  const size_t need = fb::router_packed_bytes(E, H, dtype);
  if (need >= ((size_t)1 << 31)) return FB_EUNSUPPORTED;   // 32-bit buffer offsets
  if (packed_bytes < need) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_pack(router_w, E, H, dtype, packed, stream);
}

}  // extern "C"

namespace {

// Checks shared by the predictor entry points, except those of the workspace; FB_OK when a launch
// may proceed.
int check_predict_args(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden, int32_t dtype,
                       int32_t E, const float* select_bias, const fb_scoring* scoring,
                       const int32_t* expert_to_rank, int32_t R, const int32_t* counts,
                       const int32_t* rank_loads, const double* max_mean) {
  if (!scoring || !expert_to_rank || !counts || !rank_loads || !max_mean) return FB_EINVAL;
  if (T < 0 || H < 1 || E < 1 || R < 1 || ld_hidden < H) return FB_EINVAL;
  if (T > 0 && !hidden) return FB_EINVAL;
  if (dtype != FB_BF16 && dtype != FB_F32) return FB_EINVAL;
  const int elem = dtype == FB_BF16 ? 2 : 4;
  if (E > FB_MAX_EXPERTS || R > FB_MAX_RANKS) return FB_EUNSUPPORTED;
  if (H % (dtype == FB_BF16 ? 32 : 16) != 0) return FB_EUNSUPPORTED;
  if ((ld_hidden * elem) % 16 != 0 || (hidden && !aligned16(hidden))) return FB_EUNSUPPORTED;
  // 32-bit buffer offsets: one 128-row tile of hidden states and the whole packed router weight
  if (ld_hidden * elem * 128 >= ((int64_t)1 << 31) ||
      fb::router_packed_bytes(E, H, dtype) >= ((size_t)1 << 31))
    return FB_EUNSUPPORTED;
  return check_scoring(*scoring, E, select_bias);
}

// check_predict_args plus the caller's workspace.
int check_predict(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden, int32_t dtype,
                  int32_t E, const float* select_bias, const fb_scoring* scoring,
                  const int32_t* expert_to_rank, int32_t R, const int32_t* counts,
                  const int32_t* rank_loads, const double* max_mean, const void* workspace,
                  size_t workspace_bytes, size_t workspace_need) {
  const int ac = check_predict_args(hidden, T, H, ld_hidden, dtype, E, select_bias, scoring,
                                    expert_to_rank, R, counts, rank_loads, max_mean);
  if (ac != FB_OK) return ac;
  if (!workspace || !aligned16(workspace)) return FB_EINVAL;
  if (workspace_bytes < workspace_need) return FB_ENOSPC;
  return FB_OK;
}

fb::PredictLaunch make_launch(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                              int32_t dtype, const void* router_packed, int32_t E,
                              const float* logit_bias, const float* select_bias,
                              const fb_scoring* scoring, const int32_t* expert_to_rank, int32_t R,
                              int32_t* counts, int32_t* rank_loads, double* max_mean,
                              void* workspace, int32_t* topk_idx, float* logits, void* stream) {
  fb::PredictLaunch a;
  a.hidden = hidden;
  a.T = T;
  a.H = H;
  a.ld_hidden = ld_hidden;
  a.dtype = dtype;
  a.router_packed = router_packed;
  a.E = E;
  a.logit_bias = logit_bias;
  a.select_bias = select_bias;
  a.scoring = *scoring;
  if (a.scoring.n_group == 1) { a.scoring.topk_group = 1; a.scoring.group_topn = 1; }
  a.expert_to_rank = expert_to_rank;
  a.R = R;
  a.counts = counts;
  a.rank_loads = rank_loads;
  a.max_mean = max_mean;
  a.workspace = workspace;
  a.topk_idx = topk_idx;
  a.logits = logits;
  a.stream = stream;
  a.num_cus = fb::device_cu_count();
  a.partial = nullptr;
  a.partial_bytes = 0;
  a.plan = nullptr;
  return a;
}

// Arguments of the swap-count device planner (all but the counts): FB_OK or the status to return.
int check_plan_device(int32_t E, const int32_t* slot_expert, int32_t R, int32_t S,
                      const fb_budget* budget, const fb_swap* swaps, const int32_t* n_swaps,
                      const int32_t* new_slot_expert, const int32_t* new_expert_to_rank,
                      const int64_t* new_rank_loads, const int32_t* status) {
  if (!slot_expert || !budget || !n_swaps || !new_slot_expert || !new_expert_to_rank ||
      !new_rank_loads || !status)
    return FB_EINVAL;
  if (E < 1 || R < 1 || S < 1) return FB_EINVAL;
  if (R > FB_MAX_RANKS || (int64_t)R * S > FB_MAX_SLOTS_TOTAL) return FB_EUNSUPPORTED;
  if (E > R * S) return FB_EINVAL;
  const fb_budget bg = *budget;
  if (bg.max_swaps < 0 || bg.per_rank_cap < 0 || bg.tau < 0 || bg.gamma_num < 0 || bg.gamma_den < 0)
    return FB_EINVAL;
  if (bg.mode != FB_FRONTIER && bg.mode != FB_FULL) return FB_EINVAL;
  if (bg.max_swaps > 0 && !swaps) return FB_EINVAL;
  return FB_OK;
}

fb::PlanDeviceLaunch make_plan_launch(const int32_t* counts, int32_t E, const int32_t* slot_expert,
                                      int32_t R, int32_t S, const fb_budget& bg, fb_swap* swaps,
                                      int32_t* n_swaps, int32_t* new_slot_expert,
                                      int32_t* new_expert_to_rank, int64_t* new_rank_loads,
                                      int32_t* status, void* stream) {
  fb::PlanDeviceLaunch a;
  a.counts = counts;
  a.E = E;
  a.slot_expert = slot_expert;
  a.R = R;
  a.S = S;
  a.budget = bg;
  a.swaps = swaps;
  a.n_swaps = n_swaps;
  a.new_slot_expert = new_slot_expert;
  a.new_expert_to_rank = new_expert_to_rank;
  a.new_rank_loads = new_rank_loads;
  a.status = status;
  a.stream = stream;
  a.timed = 0;
  a.cost = fb_cost_model{};
  a.rank_node = nullptr;
  a.expert_bytes = nullptr;
  a.swap_cost_ns = nullptr;
  return a;
}

// The time budget of a device plan on top of the swap-count planner's arguments: FB_OK with the
// cost model resolved (a link budget of -1 becomes the rank budget), or the status to return.
int check_plan_timed(const fb_budget* budget, const fb_cost_model* cost, const int32_t* rank_node,
                     const int64_t* expert_bytes, fb_cost_model* resolved) {
  if (!cost || !rank_node || !expert_bytes) return FB_EINVAL;
  if (budget->max_swaps > fb::kMaxTimedSwaps) return FB_EUNSUPPORTED;
  fb_cost_model m = *cost;
  if (m.rank_budget_ns < 0 || m.link_budget_ns < -1) return FB_EINVAL;
  for (int t = 0; t < 2; ++t)
    if (m.alpha_ns[t] < 1 || m.alpha_ns[t] > fb::kCostLimit || m.beta_bytes_per_us[t] < 1 ||
        m.beta_bytes_per_us[t] > fb::kCostLimit)
      return FB_EINVAL;
  if (m.link_budget_ns < 0) m.link_budget_ns = m.rank_budget_ns;
  *resolved = m;
  return FB_OK;
}

void set_timed(fb::PlanDeviceLaunch& a, const fb_cost_model& m, const int32_t* rank_node,
               const int64_t* expert_bytes, int64_t* swap_cost_ns) {
  a.timed = 1;
  a.cost = m;
  a.rank_node = rank_node;
  a.expert_bytes = expert_bytes;
  a.swap_cost_ns = swap_cost_ns;
}

// The prediction, then the plan of its counts: the one-wave planner runs in the predictor's last
// workgroup when it serves the plan; any other plan follows as a kernel of its own on the stream.
int predict_then_plan(fb::PredictLaunch& a, const fb::PlanDeviceLaunch& p, size_t workspace_bytes) {
  const size_t sb = fb::split_workspace_bytes(a.T, a.E, a.H, a.dtype, a.num_cus);
  if (sb > 0 && workspace_bytes >= fb::kWsBytes + sb) {
    a.partial = reinterpret_cast<float*>(static_cast<char*>(a.workspace) + fb::kWsBytes);
    a.partial_bytes = workspace_bytes - fb::kWsBytes;
  }
  if (fb::plan_fusable(p)) a.plan = &p;
  const int lc = fb::launch_predict(a);
  if (lc != FB_OK || a.plan != nullptr) return lc;
  return fb::launch_plan_device(p);
}

}  // namespace

extern "C" {

int fb_predict_load(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden, int32_t dtype,
                    const void* router_w, int32_t E, const float* logit_bias,
                    const float* select_bias, const fb_scoring* scoring,
                    const int32_t* expert_to_rank, int32_t R, int32_t* counts,
                    int32_t* rank_loads, double* max_mean, void* workspace,
                    size_t workspace_bytes, int32_t* topk_idx, float* logits, void* stream) {
  if (!router_w) return FB_EINVAL;
  const size_t need = fb_predict_workspace_bytes(E, H, dtype);
  const int vc = check_predict(hidden, T, H, ld_hidden, dtype, E, select_bias, scoring,
                               expert_to_rank, R, counts, rank_loads, max_mean, workspace,
                               workspace_bytes, need);
  if (vc != FB_OK) return vc;
  if (!aligned16(router_w)) return FB_EUNSUPPORTED;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  void* packed = static_cast<char*>(workspace) + fb::kWsBytes;
  const int pc = fb::launch_pack(router_w, E, H, dtype, packed, stream);
  if (pc != FB_OK) return pc;
  return fb::launch_predict(make_launch(hidden, T, H, ld_hidden, dtype, packed, E, logit_bias,
                                        select_bias, scoring, expert_to_rank, R, counts, rank_loads,
                                        max_mean, workspace, topk_idx, logits, stream));
}

int fb_predict_load_packed(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                           int32_t dtype, const void* router_packed, size_t router_packed_bytes,
                           int32_t E, const float* logit_bias, const float* select_bias,
                           const fb_scoring* scoring, const int32_t* expert_to_rank, int32_t R,
                           int32_t* counts, int32_t* rank_loads, double* max_mean,
                           void* workspace, size_t workspace_bytes, int32_t* topk_idx,
                           float* logits, void* stream) {
  if (!router_packed) return FB_EINVAL;
  const int vc = check_predict(hidden, T, H, ld_hidden, dtype, E, select_bias, scoring,
                               expert_to_rank, R, counts, rank_loads, max_mean, workspace,
                               workspace_bytes, fb::kWsBytes);
  if (vc != FB_OK) return vc;
  if (!aligned16(router_packed)) return FB_EUNSUPPORTED;
  if (router_packed_bytes < fb::router_packed_bytes(E, H, dtype)) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  fb::PredictLaunch a = make_launch(hidden, T, H, ld_hidden, dtype, router_packed, E, logit_bias,
                                    select_bias, scoring, expert_to_rank, R, counts, rank_loads,
                                    max_mean, workspace, topk_idx, logits, stream);
  // split mode when the caller's workspace holds the partial logits this batch needs
  const size_t sb = fb::split_workspace_bytes(T, E, H, dtype, a.num_cus);
  if (sb > 0 && workspace_bytes >= fb::kWsBytes + sb) {
    a.partial = reinterpret_cast<float*>(static_cast<char*>(workspace) + fb::kWsBytes);
    a.partial_bytes = workspace_bytes - fb::kWsBytes;
  }
  return fb::launch_predict(a);
}

int fb_predict_plan_packed(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                           int32_t dtype, const void* router_packed, size_t router_packed_bytes,
                           int32_t E, const float* logit_bias, const float* select_bias,
                           const fb_scoring* scoring, const int32_t* expert_to_rank, int32_t R,
                           int32_t* counts, int32_t* rank_loads, double* max_mean,
                           void* workspace, size_t workspace_bytes, const int32_t* slot_expert,
                           int32_t S, const fb_budget* budget, fb_swap* swaps, int32_t* n_swaps,
                           int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                           int64_t* new_rank_loads, int32_t* status, void* stream) {
  if (!router_packed) return FB_EINVAL;
  const int vc = check_predict(hidden, T, H, ld_hidden, dtype, E, select_bias, scoring,
                               expert_to_rank, R, counts, rank_loads, max_mean, workspace,
                               workspace_bytes, fb::kWsBytes);
  if (vc != FB_OK) return vc;
  const int pc = check_plan_device(E, slot_expert, R, S, budget, swaps, n_swaps, new_slot_expert,
                                   new_expert_to_rank, new_rank_loads, status);
  if (pc != FB_OK) return pc;
  if (!aligned16(router_packed)) return FB_EUNSUPPORTED;
  if (router_packed_bytes < fb::router_packed_bytes(E, H, dtype)) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  fb::PredictLaunch a = make_launch(hidden, T, H, ld_hidden, dtype, router_packed, E, logit_bias,
                                    select_bias, scoring, expert_to_rank, R, counts, rank_loads,
                                    max_mean, workspace, nullptr, nullptr, stream);
  const fb::PlanDeviceLaunch p = make_plan_launch(counts, E, slot_expert, R, S, *budget, swaps,
                                                  n_swaps, new_slot_expert, new_expert_to_rank,
                                                  new_rank_loads, status, stream);
  return predict_then_plan(a, p, workspace_bytes);
}

int fb_predict_plan_timed_packed(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                                 int32_t dtype, const void* router_packed,
                                 size_t router_packed_bytes, int32_t E, const float* logit_bias,
                                 const float* select_bias, const fb_scoring* scoring,
                                 const int32_t* expert_to_rank, int32_t R, int32_t* counts,
                                 int32_t* rank_loads, double* max_mean, void* workspace,
                                 size_t workspace_bytes, const int32_t* slot_expert, int32_t S,
                                 const fb_budget* budget, const fb_cost_model* cost,
                                 const int32_t* rank_node, const int64_t* expert_bytes,
                                 fb_swap* swaps, int64_t* swap_cost_ns, int32_t* n_swaps,
                                 int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                                 int64_t* new_rank_loads, int32_t* status, void* stream) {
  if (!router_packed) return FB_EINVAL;
  const int vc = check_predict(hidden, T, H, ld_hidden, dtype, E, select_bias, scoring,
                               expert_to_rank, R, counts, rank_loads, max_mean, workspace,
                               workspace_bytes, fb::kWsBytes);
  if (vc != FB_OK) return vc;
  const int pc = check_plan_device(E, slot_expert, R, S, budget, swaps, n_swaps, new_slot_expert,
                                   new_expert_to_rank, new_rank_loads, status);
  if (pc != FB_OK) return pc;
  fb_cost_model m;
  const int tc = check_plan_timed(budget, cost, rank_node, expert_bytes, &m);
  if (tc != FB_OK) return tc;
  if (!aligned16(router_packed)) return FB_EUNSUPPORTED;
  if (router_packed_bytes < fb::router_packed_bytes(E, H, dtype)) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  fb::PredictLaunch a = make_launch(hidden, T, H, ld_hidden, dtype, router_packed, E, logit_bias,
                                    select_bias, scoring, expert_to_rank, R, counts, rank_loads,
                                    max_mean, workspace, nullptr, nullptr, stream);
  fb::PlanDeviceLaunch p = make_plan_launch(counts, E, slot_expert, R, S, *budget, swaps, n_swaps,
                                            new_slot_expert, new_expert_to_rank, new_rank_loads,
                                            status, stream);
  set_timed(p, m, rank_node, expert_bytes, swap_cost_ns);
  return predict_then_plan(a, p, workspace_bytes);
}

int fb_predict_load_packed_noalloc(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                                   int32_t dtype, const void* router_packed,
                                   size_t router_packed_bytes, int32_t E, const float* logit_bias,
                                   const float* select_bias, const fb_scoring* scoring,
                                   const int32_t* expert_to_rank, int32_t R, int32_t* counts,
                                   int32_t* rank_loads, double* max_mean, int32_t* topk_idx,
                                   float* logits, void* stream) {
  if (!router_packed) return FB_EINVAL;
  const int vc = check_predict_args(hidden, T, H, ld_hidden, dtype, E, select_bias, scoring,
                                    expert_to_rank, R, counts, rank_loads, max_mean);
  if (vc != FB_OK) return vc;
  if (!aligned16(router_packed)) return FB_EUNSUPPORTED;
  if (router_packed_bytes < fb::router_packed_bytes(E, H, dtype)) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  // the split mode's partial logits must fit the scratch; every batch that runs split on a
  // 256-CU device does (the bound is in fb_internal.h)
  const size_t sb = fb::split_workspace_bytes(T, E, H, dtype, fb::device_cu_count());
  if (sb > fb::kNoAllocPartialBytes) return FB_ENOSPC;
  void* scratch = nullptr;
  const int sc = fb::noalloc_scratch(&scratch, stream);
  if (sc != FB_OK) return sc;
  fb::PredictLaunch a = make_launch(hidden, T, H, ld_hidden, dtype, router_packed, E, logit_bias,
                                    select_bias, scoring, expert_to_rank, R, counts, rank_loads,
                                    max_mean, scratch, topk_idx, logits, stream);
  if (sb > 0) {
    a.partial = reinterpret_cast<float*>(static_cast<char*>(scratch) + fb::kWsBytes);
    a.partial_bytes = fb::kNoAllocPartialBytes;
  }
  return fb::launch_predict(a);
}

size_t fb_predict_split_workspace_bytes(int64_t T, int32_t E, int32_t H, int32_t dtype) {
  if (T < 0 || E < 1 || E > FB_MAX_EXPERTS || H < 1 || (dtype != FB_BF16 && dtype != FB_F32))
    return 0;
  const size_t sb = fb::split_workspace_bytes(T, E, H, dtype, fb::device_cu_count());
  return fb::kWsBytes + sb;
}

int fb_plan_swaps_device(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                         int32_t S, const fb_budget* budget, fb_swap* swaps, int32_t* n_swaps,
                         int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                         int64_t* new_rank_loads, int32_t* status, void* stream) {
  if (!counts) return FB_EINVAL;
  const int vc = check_plan_device(E, slot_expert, R, S, budget, swaps, n_swaps, new_slot_expert,
                                   new_expert_to_rank, new_rank_loads, status);
  if (vc != FB_OK) return vc;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_plan_device(make_plan_launch(counts, E, slot_expert, R, S, *budget, swaps,
                                                 n_swaps, new_slot_expert, new_expert_to_rank,
                                                 new_rank_loads, status, stream));
}

int fb_plan_swaps_timed_device(const int32_t* counts, int32_t E, const int32_t* slot_expert,
                               int32_t R, int32_t S, const fb_budget* budget,
                               const fb_cost_model* cost, const int32_t* rank_node,
                               const int64_t* expert_bytes, fb_swap* swaps, int64_t* swap_cost_ns,
                               int32_t* n_swaps, int32_t* new_slot_expert,
                               int32_t* new_expert_to_rank, int64_t* new_rank_loads,
                               int32_t* status, void* stream) {
  if (!counts) return FB_EINVAL;
  const int vc = check_plan_device(E, slot_expert, R, S, budget, swaps, n_swaps, new_slot_expert,
                                   new_expert_to_rank, new_rank_loads, status);
  if (vc != FB_OK) return vc;
  fb_cost_model m;
  const int tc = check_plan_timed(budget, cost, rank_node, expert_bytes, &m);
  if (tc != FB_OK) return tc;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  fb::PlanDeviceLaunch a = make_plan_launch(counts, E, slot_expert, R, S, *budget, swaps, n_swaps,
                                            new_slot_expert, new_expert_to_rank, new_rank_loads,
                                            status, stream);
  set_timed(a, m, rank_node, expert_bytes, swap_cost_ns);
  return fb::launch_plan_device(a);
}

size_t fb_cosine_workspace_bytes(void) { return fb::cosine_workspace_bytes(); }

int fb_topk_hits(const int32_t* topk_pred, const int32_t* topk_actual, int64_t T, int32_t k,
                 int64_t* hits, double* hit_rate, void* stream) {
  if (!hits || T < 0 || k < 1) return FB_EINVAL;
  if (T > 0 && (!topk_pred || !topk_actual)) return FB_EINVAL;
  if (k > FB_MAX_TOPK) return FB_EUNSUPPORTED;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_hits(topk_pred, topk_actual, T, k, hits, hit_rate, stream);
}

int fb_row_cosine_mean(const void* a, const void* b, int64_t rows, int32_t cols, int64_t ld_a,
                       int64_t ld_b, int32_t dtype, double* out, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if (!a || !b || !out || !workspace || rows < 1 || cols < 1 || ld_a < cols || ld_b < cols)
    return FB_EINVAL;
  if (dtype != FB_BF16 && dtype != FB_F32) return FB_EINVAL;
  const int elem = dtype == FB_BF16 ? 2 : 4;
  if ((int64_t)cols * elem % 16 != 0 || ld_a * elem % 16 != 0 || ld_b * elem % 16 != 0 ||
      !aligned16(a) || !aligned16(b))
    return FB_EUNSUPPORTED;
  if (!aligned16(workspace)) return FB_EINVAL;
  if (workspace_bytes < fb::cosine_workspace_bytes()) return FB_ENOSPC;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_cosine(a, b, rows, cols, ld_a, ld_b, dtype, out, workspace, stream);
}

int fb_fold_rank_loads(const int32_t* counts, int32_t E, const int32_t* expert_to_rank, int32_t R,
                       int32_t* rank_loads, double* max_mean, void* stream) {
  if (!counts || !expert_to_rank || !rank_loads || !max_mean || E < 1 || R < 1) return FB_EINVAL;
  if (R > FB_MAX_RANKS) return FB_EUNSUPPORTED;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_fold(counts, E, expert_to_rank, R, rank_loads, max_mean, stream);
}

int fb_fold_slot_loads(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                       int32_t S, int32_t* rank_loads, double* max_mean, void* stream) {
  if (!counts || !slot_expert || !rank_loads || !max_mean || E < 1 || R < 1 || S < 1)
    return FB_EINVAL;
  if (R > FB_MAX_RANKS || (int64_t)R * S > FB_MAX_SLOTS_TOTAL) return FB_EUNSUPPORTED;
  if (E > R * S) return FB_EINVAL;
  const int dc = fb::check_device();
  if (dc != FB_OK) return dc;
  return fb::launch_slot_fold(counts, E, slot_expert, R, S, rank_loads, max_mean, stream);
}

}  // extern "C"
