// Internal declarations shared by the translation units of libfreebalance.so.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "freebalance.h"

namespace fb {

// Arguments of one fused predictor launch, validated by the ABI layer.
struct PlanDeviceLaunch;

struct PredictLaunch {
  const void* hidden;
  int64_t T;
  int32_t H;
  int64_t ld_hidden;  // elements
  int32_t dtype;      // FB_BF16 | FB_F32
  const void* router_packed;  // router weight in the layout written by launch_pack
  int32_t E;
  const float* logit_bias;
  const float* select_bias;
  fb_scoring scoring;
  const int32_t* expert_to_rank;
  int32_t R;
  int32_t* counts;
  int32_t* rank_loads;
  double* max_mean;
  void* workspace;
  int32_t* topk_idx;
  float* logits;
  void* stream;
  int32_t num_cus;    // compute units of the device (tile-height choice)
  float* partial;     // split mode: partial-logit buffer in the workspace, or NULL
  size_t partial_bytes;
  // the swap plan of the counts, made in the predictor's last workgroup (frontier mode, R <= 64,
  // S * S <= 128; see plan_fusable), or NULL
  const PlanDeviceLaunch* plan;
};
// Bytes of partial logits the split mode needs for a batch (0: that batch runs fused).
size_t split_workspace_bytes(int64_t T, int32_t E, int32_t H, int32_t dtype, int num_cus);

// Workspace layout (device): per-expert accumulator and the completion ticket.  Every completed
// launch leaves both at zero.
constexpr size_t kWsAccOffset = 0;
constexpr size_t kWsTicketOffset = 1024;
// split mode: one arrival counter per tile, so the tile's last split finishes it
constexpr size_t kWsTileTicketOffset = 1088;
constexpr int kMaxSplitTiles = 128;
constexpr size_t kWsBytes = 2048;
static_assert(kWsTileTicketOffset + 4 * kMaxSplitTiles <= kWsBytes, "tile tickets fit the header");

// Scratch of fb_predict_load_packed_noalloc: a workspace header, then room for the split mode's
// partial logits of the largest batch that runs split on 256 CUs (at most 128 tiles, 4 splits, 64
// tokens x 256 experts or 128 x 32 per tile: 128 * 4 * 64 * 256 * 4 bytes = 32 MiB).
constexpr size_t kNoAllocPartialBytes = (size_t)32 << 20;
constexpr size_t kNoAllocScratchBytes = kWsBytes + kNoAllocPartialBytes;
// Device address of this device's scratch (set up once per device: symbol lookup, then a fill
// kernel on `stream` that zeroes its header).  FB_OK, FB_EDEVICE or FB_EUNSUPPORTED.
int noalloc_scratch(void** ptr, void* stream);

// Bytes of the packed router weight for E experts of H elements of `dtype`.
size_t router_packed_bytes(int32_t E, int32_t H, int32_t dtype);
// Rewrites the E x H row-major router weight into the fragment-major layout the predictor kernel
// streams (one kernel on `stream`).
int launch_pack(const void* router_w, int32_t E, int32_t H, int32_t dtype, void* packed, void* stream);
int launch_predict(const PredictLaunch& a);
int launch_workspace_zero(void* workspace, size_t bytes, void* stream);

struct PlanDeviceLaunch {
  const int32_t* counts;
  int32_t E;
  const int32_t* slot_expert;
  int32_t R;
  int32_t S;
  fb_budget budget;
  fb_swap* swaps;
  int32_t* n_swaps;
  int32_t* new_slot_expert;
  int32_t* new_expert_to_rank;
  int64_t* new_rank_loads;
  int32_t* status;
  void* stream;
  // time budget (fb_plan_swaps_timed_device); timed == 0 for a swap-count budget
  int32_t timed;
  fb_cost_model cost;            // link_budget_ns already resolved (>= 0)
  const int32_t* rank_node;      // device int32[R]
  const int64_t* expert_bytes;   // device int64[E]
  int64_t* swap_cost_ns;         // device int64[max_swaps] or NULL
};
constexpr int kMaxTimedSwaps = 1024;           // swap cap of the device planner under a time budget
constexpr int64_t kCostLimit = (int64_t)1 << 40;  // alpha, beta and expert sizes
int launch_plan_device(const PlanDeviceLaunch& a);
// Whether the one-wave planner serves this plan with one rank per lane, so that it can run inside
// the predictor's last workgroup: frontier mode (swap-count or time budget), R <= 64 and
// S * S <= 128.
inline bool plan_fusable(const PlanDeviceLaunch& a) {
  return a.budget.mode == FB_FRONTIER && a.R <= 64 && (int64_t)a.S * a.S <= 128;
}

// Prediction-quality diagnostics (fb_quality.hip).
constexpr int kCosineBlocks = 1024;           // grid of the row-cosine kernel (4 waves each)
size_t cosine_workspace_bytes();
int launch_hits(const int32_t* pred, const int32_t* act, int64_t T, int32_t k, int64_t* hits,
                double* rate, void* stream);
int launch_cosine(const void* a, const void* b, int64_t rows, int32_t cols, int64_t lda, int64_t ldb,
                  int32_t dtype, double* out, void* workspace, void* stream);
int launch_fold(const int32_t* counts, int32_t E, const int32_t* e2r, int32_t R, int32_t* rank_loads,
                double* max_mean, void* stream);
int launch_slot_fold(const int32_t* counts, int32_t E, const int32_t* slots, int32_t R, int32_t S,
                     int32_t* rank_loads, double* max_mean, void* stream);

// Current device must be gfx950; cached per device.  FB_OK, FB_EUNSUPPORTED or FB_EDEVICE.
int check_device();
// Compute units of the current device (cached by check_device; 256 if unknown).
int device_cu_count();

}  // namespace fb
