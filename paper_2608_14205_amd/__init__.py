"""MI355X-native residual workload predictor and budgeted expert-swap planner (FreeBalance).

The computation lives in libfreebalance.so (HIP kernels for gfx950 behind the C ABI declared in
include/freebalance.h); this package only binds it.  The library is loaded on first use and its
absence raises an error: nothing here computes on the CPU in its place.
"""
from .api import (  # noqa: F401
    Budget,
    CostModel,
    DevicePlan,
    PackedRouter,
    Quality,
    Plan,
    Prediction,
    Predictor,
    Scoring,
    fold_rank_loads,
    fold_slot_loads,
    pack_router_weight,
    prediction_quality,
    row_cosine_mean,
    topk_hits,
    plan_swaps,
    plan_swaps_device,
    plan_swaps_timed,
    plan_swaps_timed_device,
    predict_load,
    predict_load_packed_noalloc,
    predict_split_workspace_bytes,
    swap_budget_from_cost,
)
from ._lib import FreeBalanceError, LIB_PATH, lib  # noqa: F401
