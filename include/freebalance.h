/*
 * freebalance.h -- C ABI of the residual workload predictor and the budgeted expert-swap planner
 * (FreeBalance, arXiv 2608.14205) for AMD Instinct MI355X (gfx950).
 *
 * The predictor is the paper's early router invocation: it applies layer l's router to the residual
 * hidden state h_{l-1} that leaves layer l-1 (Sec. "Residual Workload Prediction", Eq. 2 and the
 * linear router of Eq. 4), applies the routed model's own top-k rule, counts how many tokens chose
 * each expert (the predicted workload, Eq. 5) and folds the counts into per-rank loads under the
 * expert-to-rank placement (Alg. 1, the step that sums expert counts per rank), reporting the
 * max-to-mean rank-load ratio of Sec. "Metrics".  The planner turns counts and a slot table into a
 * budget-feasible list of pairwise expert swaps (Sec. "Budgeted Expert-Swap Planning", Eq. 6-8 and
 * Alg. 1); fb_swap_budget_from_cost converts the cost model of Eq. 9-10 into a swap count.
 *
 * Conventions shared by every entry point
 *   - Every pointer is owned by the caller; the library keeps no reference after a call returns
 *     (host entry points) or after the stream reaches the call (device entry points).
 *   - "device" pointers must be device-accessible on the current HIP device; "host" pointers are
 *     ordinary host memory.
 *   - Device entry points are stream-ordered and asynchronous: they validate their host-visible
 *     arguments, enqueue kernels on `stream` (a hipStream_t passed as void*, NULL = the default
 *     stream) and return.  They allocate no memory, never synchronise, and may run on a side stream
 *     concurrently with other work (the paper overlaps the early pass with attention).
 *   - Return value: FB_OK (0) or a negative FB_E* code.  No exception crosses the ABI.  Arguments are
 *     checked before anything is enqueued, so an error return leaves every output untouched.
 *   - Thread safety: host entry points are reentrant.  Device calls that share a workspace must be
 *     ordered on one stream.
 */
#ifndef FREEBALANCE_H
#define FREEBALANCE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FB_ABI_VERSION 6

/* Status codes. */
#define FB_OK 0
#define FB_EINVAL (-1)        /* an argument is invalid (null pointer, bad size, bad placement...) */
#define FB_EUNSUPPORTED (-2)  /* valid, but outside what this build implements (shape, device) */
#define FB_EDEVICE (-3)       /* the HIP runtime reported an error (no device, launch failure) */
#define FB_ENOSPC (-4)        /* a caller-provided buffer or workspace is too small */

/* Element types of hidden states and router weights. */
#define FB_BF16 0
#define FB_F32 1

/* Scoring rules (the routed model's "original top-k rule"). */
#define FB_SOFTMAX 0 /* softmax over logits; selection = top-k of the logits (softmax is monotone) */
#define FB_SIGMOID 1 /* score = sigmoid(logit) [+ select_bias]; DeepSeek-V3 style */

/* Planner candidate enumeration. */
#define FB_FRONTIER 0 /* only the most and the least loaded rank (Sec. Budgeted Expert-Swap Planning) */
#define FB_FULL 1     /* every ordered rank pair (a, b) with L_a > L_b */

/* Limits of this build. */
#define FB_MAX_EXPERTS 256     /* E of fb_predict_load */
#define FB_MAX_TOPK 32         /* k of fb_predict_load */
#define FB_MAX_RANKS 1024      /* R of fb_predict_load and fb_plan_swaps_device */
#define FB_MAX_SLOTS_TOTAL 4096 /* R * S of fb_plan_swaps_device */

/* Routing rule applied to the early logits.
 *   kind        FB_SOFTMAX or FB_SIGMOID.
 *   k           experts per token, 1 <= k <= min(E, FB_MAX_TOPK).
 *   n_group     1 = plain top-k.  > 1: the E experts form n_group contiguous groups of E / n_group;
 *               each group is scored by the sum of its group_topn best scores, the topk_group best
 *               groups are kept (ties: lower group index) and the k experts are chosen inside them.
 *               Requires E % n_group == 0 and either (E / n_group) % 16 == 0 with (E / n_group) / 16
 *               a power of two, or 16 % (E / n_group) == 0 (FB_EUNSUPPORTED otherwise).
 *   topk_group  1 <= topk_group <= n_group, and k <= topk_group * E / n_group.
 *   group_topn  1 (group max) or 2 (sum of the two best scores); ignored when n_group == 1.
 *               Softmax routing takes group_topn 1 only (FB_EUNSUPPORTED for 2): softmax keeps the
 *               order of single scores, so the group maximum of the logits names the same groups
 *               as that of the probabilities, but it does not keep the order of sums (logits
 *               (10, -100) outrank (5, 5) on probabilities and not on logits). */
typedef struct fb_scoring {
  int32_t kind;
  int32_t k;
  int32_t n_group;
  int32_t topk_group;
  int32_t group_topn;
} fb_scoring;

/* Planner budget and options.
 *   max_swaps     global swap cap B >= 0 (from the configuration or fb_swap_budget_from_cost).
 *   per_rank_cap  0 = none; otherwise the most swaps any one rank may take part in (the paper
 *                 enforces budgets per participant, not only as a global sum).
 *   tau           stop when L_max - L_min <= tau (tokens, >= 0): Alg. 1's imbalance threshold.
 *   gamma_num, gamma_den  gamma of Eq. 8 as a ratio >= 0; gamma_den == 0 selects gamma = 1 / N,
 *                 N = sum of counts.  Benefits are reported as gamma_den * Delta (exact integers).
 *   mode          FB_FRONTIER or FB_FULL.
 *   layer_id      first key of the deterministic tie-break (layer, src rank, dst rank, expert ids). */
typedef struct fb_budget {
  int32_t max_swaps;
  int32_t per_rank_cap;
  int64_t tau;
  int64_t gamma_num;
  int64_t gamma_den;
  int32_t mode;
  int32_t layer_id;
} fb_budget;

/* Migration cost model and time budget of the planner (Sec. "Budgeted Expert-Swap Planning",
 * Eq. 9-10, with the budget enforced per rank and per link).  A swap of the item on rank a with the
 * item on rank b costs, in whole nanoseconds,
 *     C = alpha_ns[t] + ceil((S(e_a) + S(e_b)) * 1000 / beta_bytes_per_us[t]),
 * where t = 0 if the two ranks share a node and 1 otherwise (the paper's intra- and inter-node
 * links) and S(e) is the size of expert e (an empty slot transfers nothing).  A candidate is
 * admissible only if C fits the remaining budget of both ranks and of their link; admissible
 * candidates are ranked by benefit / C (compared exactly, by cross-multiplication), then by the
 * tie-break of fb_budget.layer_id; an accepted swap charges C to both ranks and to the link.
 *   rank_budget_ns     B_l of Eq. 10 for every rank, >= 0 (the profiled attention time of the
 *                      layer's attention type minus the safety margin delta).
 *   link_budget_ns     budget of every rank pair, >= 0; -1 = rank_budget_ns (then the rank budgets
 *                      already bound every link).
 *   alpha_ns           per-swap overhead for link types 0 and 1, 1 .. 2^40.
 *   beta_bytes_per_us  point-to-point bandwidth for link types 0 and 1, 1 .. 2^40. */
typedef struct fb_cost_model {
  int64_t rank_budget_ns;
  int64_t link_budget_ns;
  int64_t alpha_ns[2];
  int64_t beta_bytes_per_us[2];
} fb_cost_model;

/* One accepted swap, in acceptance order.  The expert in src_slot of src_rank (the more loaded
 * rank) trades places with the expert in dst_slot of dst_rank.  expert_* is -1 for an empty slot
 * (then the swap moves a single expert).  gain = gamma_den * (Phi(L) - Phi(L')) > 0. */
typedef struct fb_swap {
  int32_t src_rank;
  int32_t dst_rank;
  int32_t src_slot;
  int32_t dst_slot;
  int32_t expert_src;
  int32_t expert_dst;
  int64_t gain;
} fb_swap;

/* ABI version of the loaded library (FB_ABI_VERSION it was built with). */
int fb_abi_version(void);

/* Static text for a status code; never NULL. */
const char* fb_status_string(int status);

/* Bytes of the packed router weight fb_pack_router_weight writes for E experts of H elements of
 * `dtype`: E rounded up to 32, 64, 128 or 256 rows times H * element size rounded up to a
 * multiple of 256 bytes.  0 if E, H or dtype is invalid or E > FB_MAX_EXPERTS. */
size_t fb_router_packed_bytes(int32_t E, int32_t H, int32_t dtype);

/* Bytes of device workspace fb_predict_load needs: 2048 bytes of accumulators and completion
 * counters plus room for the router weight it packs on every call (fb_router_packed_bytes).
 * fb_predict_load_packed needs only the first 2048 bytes.  0 for invalid arguments as in
 * fb_router_packed_bytes. */
size_t fb_predict_workspace_bytes(int32_t E, int32_t H, int32_t dtype);

/* Prepare a predictor workspace: zero-fills its first 2048 bytes with a kernel on `stream` (no
 * memset node, so the call may be captured into a HIP graph).  Required once before the
 * workspace's first use; every completed predictor call leaves those bytes zeroed again.
 *   workspace  device, >= 2048 bytes, 16-byte aligned. */
int fb_predict_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/* Rewrite a router weight into the layout the predictor kernel streams (one kernel on `stream`).
 * The router weight is a fixed parameter of the routed model, so a caller packs it once when the
 * model is loaded and calls fb_predict_load_packed per batch; fb_predict_load does the same packing
 * into its workspace on every call.  Layout: for each 256-byte stage st of a row, a contiguous
 * block of 1 KB chunks; chunk c = (w * 8 + q) * F + f holds, for lane l of 64, the 16 bytes at
 * byte st * 256 + q * 32 + (l / 32) * 16 of row w * (EP / W) + f * 32 + (l % 32), where EP is E
 * rounded as above, W the number of expert slices of the kernel's tile for EP (4 for EP >= 128, 2
 * for 64, 1 for 32) and F = EP / (32 * W).  Rows >= E and bytes past H read as zero.
 *   router_w      device, E x H row-major, element type `dtype`, 16-byte aligned.
 *   packed        device out, >= fb_router_packed_bytes(E, H, dtype) bytes, 16-byte aligned.
 * FB_EINVAL for null pointers, E < 1, H < 1 or a bad dtype; FB_EUNSUPPORTED for E >
 * FB_MAX_EXPERTS, H not a multiple of 32 (FB_BF16) or 16 (FB_F32), misalignment or a packed
 * weight of 2 GiB or more; FB_ENOSPC if packed_bytes is too small. */
int fb_pack_router_weight(const void* router_w, int32_t E, int32_t H, int32_t dtype, void* packed,
                          size_t packed_bytes, void* stream);

/* Early router pass + top-k + predicted workload + rank fold (Eq. 2, 4, 5; Alg. 1, first two
 * steps).  Packs router_w into the workspace (fb_pack_router_weight), then runs the fused kernel.
 *   hidden          device, T rows of H elements, row stride ld_hidden elements (>= H), element type
 *                   `dtype`; rows 16-byte aligned (ld_hidden * element size % 16 == 0).
 *   T               tokens, >= 0.  T == 0 yields zero counts and *max_mean = 1.0.
 *   H               hidden size; H % 32 == 0 for FB_BF16, H % 16 == 0 for FB_F32.
 *   router_w        device, E x H row-major (row e is expert e's weight column of the paper's
 *                   W in R^{H x E}), same element type, 16-byte aligned.
 *   E               experts, 1 <= E <= FB_MAX_EXPERTS.
 *   logit_bias      device float[E] or NULL: the b of the linear router g(X) = XW + 1b^T, added to
 *                   the logits.
 *   select_bias     device float[E] or NULL: FB_SIGMOID only (FB_EINVAL with FB_SOFTMAX); added to
 *                   the sigmoid score for selection only.
 *   scoring         host, routing rule (see fb_scoring).
 *   expert_to_rank  device int32[E], rank id of each expert in [0, R).  An entry outside [0, R) is
 *                   a precondition violation: the kernel skips that expert in the fold and writes
 *                   *max_mean = -1.0 instead of the ratio.
 *   R               ranks, 1 <= R <= FB_MAX_RANKS.
 *   counts          device int32[E] out: n^_e, tokens whose predicted top-k contains e.
 *   rank_loads      device int32[R] out: L_r = sum of counts of experts placed on r.
 *   max_mean        device double out: max_r L_r / (sum_r L_r / R), 1.0 if every load is 0.
 *   workspace       device, fb_predict_workspace_bytes(E, H, dtype) bytes, prepared by
 *                   fb_predict_workspace_init; must not be used by an overlapping call.
 *   topk_idx        device int32[T * k] out or NULL: the selected experts of each token in
 *                   descending score order (lower index first on equal scores).
 *   logits          device float[T * E] out or NULL: the early logits (incl. logit_bias).
 *   stream          hipStream_t as void*, or NULL.
 * Scores are compared in float32; ties in score go to the lower expert index.  Selection does not
 * depend on whether topk_idx / logits are requested. */
int fb_predict_load(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden, int32_t dtype,
                    const void* router_w, int32_t E, const float* logit_bias,
                    const float* select_bias, const fb_scoring* scoring,
                    const int32_t* expert_to_rank, int32_t R, int32_t* counts,
                    int32_t* rank_loads, double* max_mean, void* workspace,
                    size_t workspace_bytes, int32_t* topk_idx, float* logits, void* stream);

/* fb_predict_load with a router weight packed beforehand by fb_pack_router_weight (same E, H and
 * dtype): the per-batch call of a server that packs its routers at load time.  Results are
 * identical to fb_predict_load's on the same inputs, except in split mode (below).
 *   router_packed        device, as written by fb_pack_router_weight.
 *   router_packed_bytes  its size; FB_ENOSPC if below fb_router_packed_bytes(E, H, dtype).
 *   workspace            device, >= 2048 bytes, prepared by fb_predict_workspace_init.  With at
 *                        least fb_predict_split_workspace_bytes(T, E, H, dtype) bytes, a batch
 *                        too small to occupy the GPU runs in split mode: the hidden dimension of
 *                        every tile is split over several workgroups whose partial logits (kept
 *                        in the workspace past its first 2048 bytes) are added in a fixed order
 *                        by the tile's last workgroup to arrive, still in one launch.  Results
 *                        are then deterministic and within the float32 summation-order
 *                        tolerance of the fused path's.
 * Every other argument, and every error, as in fb_predict_load. */
int fb_predict_load_packed(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                           int32_t dtype, const void* router_packed, size_t router_packed_bytes,
                           int32_t E, const float* logit_bias, const float* select_bias,
                           const fb_scoring* scoring, const int32_t* expert_to_rank, int32_t R,
                           int32_t* counts, int32_t* rank_loads, double* max_mean,
                           void* workspace, size_t workspace_bytes, int32_t* topk_idx,
                           float* logits, void* stream);

/* The whole early pass of one layer in one call: fb_predict_load_packed, then the swap plan of the
 * predicted counts as fb_plan_swaps_device would make it (Alg. 1, Eq. 6-8), stream-ordered with no
 * host round trip.  For a swap-count budget in frontier mode on at most 64 ranks with S * S <= 128
 * (the DeepSeek-V3-shaped 32 x 8 placement, for instance) the plan is made inside the predictor's
 * last workgroup, right after the counts are complete, so that no separate kernel has to wait for
 * a free compute unit when the call runs beside other work (attention on another stream); any
 * other plan runs as its own kernel on the same stream.  Results are identical to the two calls.
 *   hidden ... workspace_bytes   as in fb_predict_load_packed (no debug outputs).
 *   counts                       device int32[E] out: the predicted counts, then the planner's
 *                                input.
 *   slot_expert ... status       as in fb_plan_swaps_device (device arrays; budget a host struct
 *                                read during the call), with this call's E and R.
 * Errors: every argument error of either call, checked on the host before anything runs. */
int fb_predict_plan_packed(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                           int32_t dtype, const void* router_packed, size_t router_packed_bytes,
                           int32_t E, const float* logit_bias, const float* select_bias,
                           const fb_scoring* scoring, const int32_t* expert_to_rank, int32_t R,
                           int32_t* counts, int32_t* rank_loads, double* max_mean,
                           void* workspace, size_t workspace_bytes, const int32_t* slot_expert,
                           int32_t S, const fb_budget* budget, fb_swap* swaps, int32_t* n_swaps,
                           int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                           int64_t* new_rank_loads, int32_t* status, void* stream);

/* fb_predict_plan_packed under a time budget: the prediction, then the plan of its counts as
 * fb_plan_swaps_timed_device would make it (every candidate costed by Eq. 9 on its link type and
 * admitted against the per-rank and per-link budgets of Eq. 10, ranked by benefit / cost).  In
 * frontier mode on at most 64 ranks with S * S <= 128 the plan is made inside the predictor's last
 * workgroup; any other plan runs as its own kernel on the same stream.  Results are identical to
 * fb_predict_load_packed followed by fb_plan_swaps_timed_device.
 *   hidden ... workspace_bytes   as in fb_predict_load_packed (no debug outputs).
 *   counts                       device int32[E] out: the predicted counts, then the planner's
 *                                input.
 *   slot_expert ... status       as in fb_plan_swaps_timed_device (device arrays; budget and cost
 *                                host structs read during the call), with this call's E and R.
 * Errors: every argument error of either call, checked on the host before anything runs. */
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
                                 int64_t* new_rank_loads, int32_t* status, void* stream);

/* fb_predict_load_packed for callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): no workspace argument, no allocation.  The
 * library keeps a fixed scratch array in device memory instead, FB_NOALLOC_SCRATCH_BYTES per device
 * (2048 bytes of accumulators and completion counters, then 32 MiB for split-mode partial logits),
 * held by every device the call runs on until the process ends.  The first call on a device looks
 * up that device's copy and zeroes its header with a fill kernel on `stream`; every completed call
 * leaves the header zeroed again.  All calls on one device share the array: calls that overlap
 * on one device (other streams, other threads) race and give undefined results, so order them on
 * one stream.  Batches too small to occupy the GPU run in split mode as with a large enough
 * workspace; FB_ENOSPC if a batch's split-mode partials would exceed the 32 MiB (no batch on a
 * 256-CU MI355X does).  Results are identical to fb_predict_load_packed's with a workspace of
 * fb_predict_split_workspace_bytes(T, E, H, dtype) bytes.  Every other argument and error as in
 * fb_predict_load_packed; FB_EDEVICE if the scratch cannot be located. */
#define FB_NOALLOC_SCRATCH_BYTES (2048u + (32u << 20))
int fb_predict_load_packed_noalloc(const void* hidden, int64_t T, int32_t H, int64_t ld_hidden,
                                   int32_t dtype, const void* router_packed,
                                   size_t router_packed_bytes, int32_t E, const float* logit_bias,
                                   const float* select_bias, const fb_scoring* scoring,
                                   const int32_t* expert_to_rank, int32_t R, int32_t* counts,
                                   int32_t* rank_loads, double* max_mean, int32_t* topk_idx,
                                   float* logits, void* stream);

/* Workspace bytes that let fb_predict_load_packed run a batch of T tokens in split mode on the
 * current device (2048 when the batch runs fused anyway; 0 for invalid arguments). */
size_t fb_predict_split_workspace_bytes(int64_t T, int32_t E, int32_t H, int32_t dtype);

/* ---- Prediction-quality diagnostics (Sec. "Metrics" and the prediction-quality study) ----------
 * Device-side measurements of how well the early pass predicts the actual routing: run
 * fb_predict_load on h_{l-1} and on the actual router input H_l with topk_idx / logits requested,
 * then compare. All three calls are stream-ordered and deterministic. */

/* Top-k hit count and hit rate: hits = sum over tokens of |predicted set intersect actual set|,
 * hit rate = hits / (T * k) (the fraction of the final top-k assignments the early pass recovers;
 * 1.0 for T = 0).
 *   topk_pred, topk_actual  device int32[T * k], rows of k distinct expert ids in [0, 256).
 *   hits                    device int64 out (overwritten).
 *   hit_rate                device double out (overwritten), or NULL.
 * FB_EINVAL for null pointers, T < 0 or k < 1; FB_EUNSUPPORTED for k > FB_MAX_TOPK. */
int fb_topk_hits(const int32_t* topk_pred, const int32_t* topk_actual, int64_t T, int32_t k,
                 int64_t* hits, double* hit_rate, void* stream);

/* Bytes of device workspace fb_row_cosine_mean needs. */
size_t fb_cosine_workspace_bytes(void);

/* Mean over rows of the cosine similarity of matching rows of a and b (hidden-state cosine for
 * h_{l-1} vs H_l, logit cosine for early vs actual logits). Products and sums in double; per-row
 * cosine = dot / (|a| |b|); the mean sums the rows in a fixed order, so results are reproducible.
 * A zero row gives NaN, as 0/0.
 *   a, b        device, rows x cols row-major with row strides ld_a / ld_b elements, element type
 *               dtype (FB_BF16 or FB_F32), 16-byte aligned rows; cols * element size and the row
 *               strides in bytes must be multiples of 16 (FB_EUNSUPPORTED otherwise).
 *   rows        >= 1.
 *   out         device double out.
 *   workspace   device, >= fb_cosine_workspace_bytes() bytes, 16-byte aligned; no contents kept. */
int fb_row_cosine_mean(const void* a, const void* b, int64_t rows, int32_t cols, int64_t ld_a,
                       int64_t ld_b, int32_t dtype, double* out, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Rank loads and max-to-mean ratio of a count vector under a placement (Alg. 1 aggregation, Sec.
 * "Metrics"): the realised balance of the actual routing under the current or the planned
 * placement.
 *   counts          device int32[E] (>= 0).
 *   expert_to_rank  device int32[E]; an entry outside [0, R) makes *max_mean = -1.0.
 *   rank_loads      device int32[R] out; max_mean device double out (1.0 if every load is 0).
 * FB_EINVAL for null pointers, E < 1 or R < 1; FB_EUNSUPPORTED for R > FB_MAX_RANKS. */
int fb_fold_rank_loads(const int32_t* counts, int32_t E, const int32_t* expert_to_rank, int32_t R,
                       int32_t* rank_loads, double* max_mean, void* stream);

/* Rank loads and max-to-mean ratio of a count vector under a replicated placement, as produced by a
 * history-driven placement that copies hot experts (the starting point of the "EPLB + Ours" runs of
 * Table 1).  The paper leaves the split of an expert's tokens among its copies to the dispatch
 * policy; here replica j of an expert with n tokens and c replicas carries floor(n / c) tokens, plus
 * one if j < n mod c (a round-robin dispatch), and L_r sums the shares on rank r.
 *   counts       device int32[E] (>= 0).
 *   slot_expert  device int32[R * S] row-major: value e + E * j is replica j of expert e, -1 an
 *                empty slot.  Every expert must have replicas 0 .. c_e - 1, each once, and no rank
 *                may hold two replicas of one expert; a placement without replicas (every value
 *                below E) is the plain slot table of fb_plan_swaps.  A violated rule or a negative
 *                count makes *max_mean = -1.0.
 *   rank_loads   device int32[R] out; max_mean device double out (1.0 if every load is 0).
 * FB_EINVAL for null pointers, E, R or S < 1, or E > R * S; FB_EUNSUPPORTED for R > FB_MAX_RANKS or
 * R * S > FB_MAX_SLOTS_TOTAL.  One workgroup, stream-ordered. */
int fb_fold_slot_loads(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                       int32_t S, int32_t* rank_loads, double* max_mean, void* stream);

/* Budgeted greedy expert-swap planner on the host (Sec. Budgeted Expert-Swap Planning, Eq. 6-8,
 * Alg. 1).  Pure and deterministic: identical inputs give a byte-identical plan.
 *   counts            host int32[E] (>= 0): the predicted per-expert workload, not rank loads.
 *   E                 experts, >= 1.
 *   slot_expert       host int32[R * S] row-major: expert in slot s of rank r, -1 = empty slot.
 *                     Every expert 0..E-1 must appear exactly once (FB_EINVAL otherwise), or, for
 *                     a replicated placement (the "EPLB + Ours" setting of Table 1), value e + E * j
 *                     is replica j of expert e: every expert then needs replicas 0 .. c_e - 1, each
 *                     once, and no rank may hold two replicas of one expert.  Replica j carries
 *                     floor(n_e / c_e) tokens, plus one if j < n_e mod c_e (as fb_fold_slot_loads),
 *                     and keeps its ordinal when it moves; a swap may not put a replica on a rank
 *                     that holds another replica of the same expert, and empty slots take the
 *                     tie-break ids E * J + r * S + s (J = the largest c_e).  Swaps and
 *                     new_slot_expert then report slot values, new_expert_to_rank the rank of
 *                     replica 0.
 *   R, S              ranks (>= 1) and slots per rank (>= 1).
 *   budget            host, see fb_budget.
 *   swaps             host fb_swap[swaps_cap] out; swaps_cap >= budget->max_swaps (FB_ENOSPC).
 *   n_swaps           host out: number of swaps written.
 *   new_slot_expert   host int32[R * S] out, may be NULL: slot table after the plan.
 *   new_expert_to_rank host int32[E] out, may be NULL.
 *   new_rank_loads    host int64[R] out, may be NULL: predicted loads after the plan.
 * An empty plan (B = 0, no positive-benefit swap, R = 1, all counts zero) retains the placement. */
int fb_plan_swaps(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                  int32_t S, const fb_budget* budget, fb_swap* swaps, int32_t swaps_cap,
                  int32_t* n_swaps, int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                  int64_t* new_rank_loads);

/* The same planner as one stream-ordered single-workgroup kernel, so that prediction and planning
 * run back to back on the device with no host round trip.  Produces exactly the plan of
 * fb_plan_swaps.  Limits: R <= FB_MAX_RANKS, R * S <= FB_MAX_SLOTS_TOTAL, E <= R * S.
 *   counts, slot_expert   device inputs as in fb_plan_swaps.
 *   budget                host struct, read during the call.
 *   swaps                 device fb_swap[budget->max_swaps] out.
 *   n_swaps               device int32 out.
 *   new_slot_expert       device int32[R * S] out (required).
 *   new_expert_to_rank    device int32[E] out (required).
 *   new_rank_loads        device int64[R] out (required).
 *   status                device int32 out: FB_OK, or FB_EINVAL if the slot table is invalid or a
 *                         count is negative, or FB_EUNSUPPORTED if a replicated placement's item
 *                         ids do not fit the tie keys (E * max c_e + R * S > 2^21); then the plan
 *                         is empty and the placement unchanged.
 * Replicated placements are planned exactly as by fb_plan_swaps. */
int fb_plan_swaps_device(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                         int32_t S, const fb_budget* budget, fb_swap* swaps, int32_t* n_swaps,
                         int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                         int64_t* new_rank_loads, int32_t* status, void* stream);

/* The planner under a time budget (fb_cost_model) on the host: fb_plan_swaps with every candidate
 * costed by Eq. 9 and admitted against the per-rank and per-link budgets, ranked by benefit-to-cost
 * ratio.  budget->max_swaps and budget->per_rank_cap still apply on top of the time budget.  Pure
 * and deterministic.
 *   cost            host, see fb_cost_model.
 *   rank_node       host int32[R]: node id of every rank (link type 0 between equal ids).
 *   expert_bytes    host int64[E]: S(e), 0 .. 2^40.
 *   swap_cost_ns    host int64[swaps_cap] out, may be NULL: C of every accepted swap.
 * Every other argument as in fb_plan_swaps.  FB_EINVAL also for a null cost, rank_node or
 * expert_bytes, or a cost-model value out of range. */
int fb_plan_swaps_timed(const int32_t* counts, int32_t E, const int32_t* slot_expert, int32_t R,
                        int32_t S, const fb_budget* budget, const fb_cost_model* cost,
                        const int32_t* rank_node, const int64_t* expert_bytes, fb_swap* swaps,
                        int64_t* swap_cost_ns, int32_t swaps_cap, int32_t* n_swaps,
                        int32_t* new_slot_expert, int32_t* new_expert_to_rank,
                        int64_t* new_rank_loads);

/* The time-budgeted planner as one stream-ordered single-workgroup kernel: exactly the plan of
 * fb_plan_swaps_timed.  Limits as fb_plan_swaps_device, and budget->max_swaps <= 1024.
 *   counts, slot_expert   device inputs as in fb_plan_swaps.
 *   budget, cost          host structs, read during the call.
 *   rank_node             device int32[R].
 *   expert_bytes          device int64[E].
 *   swaps                 device fb_swap[budget->max_swaps] out.
 *   swap_cost_ns          device int64[budget->max_swaps] out, may be NULL.
 *   n_swaps, new_slot_expert, new_expert_to_rank, new_rank_loads, status  as fb_plan_swaps_device;
 *                         status is FB_EINVAL also for an expert size outside 0 .. 2^40.
 * FB_EUNSUPPORTED for max_swaps > 1024; FB_EINVAL for a cost-model value out of range. */
int fb_plan_swaps_timed_device(const int32_t* counts, int32_t E, const int32_t* slot_expert,
                               int32_t R, int32_t S, const fb_budget* budget,
                               const fb_cost_model* cost, const int32_t* rank_node,
                               const int64_t* expert_bytes, fb_swap* swaps, int64_t* swap_cost_ns,
                               int32_t* n_swaps, int32_t* new_slot_expert,
                               int32_t* new_expert_to_rank, int64_t* new_rank_loads,
                               int32_t* status, void* stream);

/* Swap cap from the cost model: with a uniform expert size S_e and one link type every swap costs
 * C = alpha + 2 * S_e / beta (Eq. 9) and the window is B_l = max(0, t_attn - delta) (Eq. 10); the
 * result is the largest n with n * C <= B_l.  Times in microseconds, beta in bytes per microsecond.
 * Returns the count (>= 0), or FB_EINVAL for beta <= 0, alpha < 0, expert_bytes < 0, a
 * non-positive cost or non-finite inputs. */
int64_t fb_swap_budget_from_cost(double t_attn_us, double delta_us, double alpha_us,
                                 double beta_bytes_per_us, int64_t expert_bytes);

#ifdef __cplusplus
}
#endif

#endif /* FREEBALANCE_H */
