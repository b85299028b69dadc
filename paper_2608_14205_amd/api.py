"""Python binding of libfreebalance.so over torch tensors.

Argument marshalling only: every step of the predictor and the device planner runs in the library's
HIP kernels; torch provides device memory and the current stream.  Names follow the C ABI
(include/freebalance.h).
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import List, NamedTuple, Optional, Sequence, Tuple

import numpy as np
import torch

from . import _lib as L

SWAP_DTYPE = np.dtype([("src_rank", "<i4"), ("dst_rank", "<i4"), ("src_slot", "<i4"),
                       ("dst_slot", "<i4"), ("expert_src", "<i4"), ("expert_dst", "<i4"),
                       ("gain", "<i8")])
SWAP_BYTES = SWAP_DTYPE.itemsize  # 32 == sizeof(fb_swap)


@dataclasses.dataclass(frozen=True)
class Scoring:
    """The routed model's top-k rule (fb_scoring)."""

    kind: str = "softmax"      # "softmax" | "sigmoid"
    k: int = 2
    n_group: int = 1
    topk_group: int = 1
    group_topn: int = 1

    def to_c(self) -> L.fb_scoring:
        kinds = {"softmax": L.FB_SOFTMAX, "sigmoid": L.FB_SIGMOID}
        if self.kind not in kinds:
            raise ValueError(f"unknown scoring kind {self.kind!r}")
        return L.fb_scoring(kinds[self.kind], self.k, self.n_group, self.topk_group, self.group_topn)


@dataclasses.dataclass(frozen=True)
class Budget:
    """Planner budget (fb_budget).  gamma=None selects 1/N."""

    max_swaps: int
    per_rank_cap: int = 0
    tau: int = 0
    gamma: Optional[Tuple[int, int]] = None
    mode: str = "frontier"     # "frontier" | "full"
    layer_id: int = 0

    def to_c(self) -> L.fb_budget:
        modes = {"frontier": L.FB_FRONTIER, "full": L.FB_FULL}
        if self.mode not in modes:
            raise ValueError(f"unknown planner mode {self.mode!r}")
        num, den = self.gamma if self.gamma is not None else (0, 0)
        return L.fb_budget(self.max_swaps, self.per_rank_cap, self.tau, num, den, modes[self.mode],
                           self.layer_id)


@dataclasses.dataclass(frozen=True)
class CostModel:
    """Migration cost model and time budget (fb_cost_model plus the per-rank node ids and the
    per-expert sizes).  link_budget_ns=None means the rank budget."""

    rank_node: Sequence[int]
    expert_bytes: Sequence[int]
    alpha_ns: Tuple[int, int]
    beta_bytes_per_us: Tuple[int, int]
    rank_budget_ns: int
    link_budget_ns: Optional[int] = None

    def to_c(self) -> L.fb_cost_model:
        m = L.fb_cost_model()
        m.rank_budget_ns = self.rank_budget_ns
        m.link_budget_ns = -1 if self.link_budget_ns is None else self.link_budget_ns
        m.alpha_ns[0], m.alpha_ns[1] = self.alpha_ns
        m.beta_bytes_per_us[0], m.beta_bytes_per_us[1] = self.beta_bytes_per_us
        return m


@dataclasses.dataclass
class Prediction:
    counts: torch.Tensor                 # int32 [E]
    rank_loads: torch.Tensor             # int32 [R]
    max_mean: torch.Tensor               # float64 [1]
    topk: Optional[torch.Tensor] = None  # int32 [T, k]
    logits: Optional[torch.Tensor] = None  # float32 [T, E]


class Plan(NamedTuple):
    swaps: List[tuple]         # (src_rank, dst_rank, src_slot, dst_slot, expert_src, expert_dst, gain)
    slots: np.ndarray          # int32 R x S
    expert_to_rank: np.ndarray  # int32 E
    rank_loads: np.ndarray     # int64 R
    costs: Optional[List[int]] = None  # ns per swap, time-budgeted planning only


@dataclasses.dataclass
class DevicePlan:
    swaps: torch.Tensor        # uint8 [max_swaps * 32]: fb_swap records
    n_swaps: torch.Tensor      # int32 [1]
    slots: torch.Tensor        # int32 [R, S]
    expert_to_rank: torch.Tensor  # int32 [E]
    rank_loads: torch.Tensor   # int64 [R]
    status: torch.Tensor       # int32 [1]
    costs: Optional[torch.Tensor] = None  # int64 [max_swaps]: ns per swap (time budget only)

    def to_host(self) -> Plan:
        st = int(self.status.item())
        L.check(st, "fb_plan_swaps_device (device status)")
        n = int(self.n_swaps.item())
        rec = np.frombuffer(self.swaps.cpu().numpy().tobytes(), dtype=SWAP_DTYPE)[:n]
        costs = None if self.costs is None else [int(v) for v in self.costs.cpu().numpy()[:n]]
        return Plan([tuple(int(v) for v in r) for r in rec], self.slots.cpu().numpy(),
                    self.expert_to_rank.cpu().numpy(), self.rank_loads.cpu().numpy(), costs)


def _fits(checks, what: str) -> None:
    for t, dtype, n, dev in checks:
        if t.dtype != dtype or t.device != dev or not t.is_contiguous() or t.numel() < n:
            raise ValueError(what)


def _check_prediction_out(out: "Prediction", E: int, R: int, T: int, k: int, dev,
                          topk: bool, logits: bool) -> None:
    """A caller's Prediction must have room for what the kernels write: E counts, R rank loads,
    one ratio and, when asked for, T x k selections and T x E logits."""
    checks = [(out.counts, torch.int32, E, dev), (out.rank_loads, torch.int32, R, dev),
              (out.max_mean, torch.float64, 1, dev)]
    if topk:
        checks.append((out.topk, torch.int32, T * k, dev))
    if logits:
        checks.append((out.logits, torch.float32, T * E, dev))
    _fits(checks, "out does not fit this call: contiguous int32[E] counts, int32[R] rank_loads, "
                  "float64[1] max_mean, int32[T * k] topk and float32[T * E] logits on the device")


def _check_plan_out(plan: "DevicePlan", R: int, S: int, E: int, cap: int, dev) -> None:
    """A caller's DevicePlan must have room for what the planner writes: up to max_swaps swap
    records (and costs), the R x S table, E expert ranks, R loads and the two status words."""
    checks = [(plan.swaps, torch.uint8, cap * SWAP_BYTES, dev), (plan.n_swaps, torch.int32, 1, dev),
              (plan.slots, torch.int32, R * S, dev), (plan.expert_to_rank, torch.int32, E, dev),
              (plan.rank_loads, torch.int64, R, dev), (plan.status, torch.int32, 1, dev)]
    if plan.costs is not None:
        checks.append((plan.costs, torch.int64, cap, dev))
    _fits(checks, "plan does not fit this call: contiguous buffers on the device with room for "
                  "max_swaps swaps (and costs), int32[R, S] slots, int32[E] expert ranks and "
                  "int64[R] loads")


def _one_gpu(dev, *tensors) -> None:
    """Every tensor handed to a kernel must be a GPU tensor on the call's device: a host or other
    device's pointer would be dereferenced by the kernel."""
    if torch.device(dev).type != "cuda":
        raise ValueError("tensors must live on a GPU")
    for t in tensors:
        if t is not None and t.device != dev:
            raise ValueError("all tensors of a call must live on one GPU")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(device: torch.device, stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return L.FB_BF16
    if t.dtype == torch.float32:
        return L.FB_F32
    raise TypeError("hidden states and router weights must be bfloat16 or float32")


@dataclasses.dataclass(frozen=True)
class PackedRouter:
    """A router weight rewritten once by fb_pack_router_weight into the predictor's streaming
    layout (a load-time transform of a fixed parameter; see pack_router_weight)."""

    data: torch.Tensor         # uint8 [fb_router_packed_bytes(E, H, dtype)]
    E: int
    H: int
    dtype: torch.dtype


def pack_router_weight(router_w: torch.Tensor,
                       stream: Optional[torch.cuda.Stream] = None) -> PackedRouter:
    """fb_pack_router_weight: E x H router weight -> PackedRouter on the same device."""
    if router_w.dim() != 2 or not router_w.is_contiguous():
        raise ValueError("router_w must be a contiguous E x H tensor")
    E, H = router_w.shape
    code = _dtype_code(router_w)
    _one_gpu(router_w.device, router_w)
    lib = L.lib()
    nbytes = int(lib.fb_router_packed_bytes(E, H, code))
    if nbytes == 0:
        L.check(L.FB_EUNSUPPORTED if E > 0 and H > 0 else L.FB_EINVAL, "fb_router_packed_bytes")
    packed = torch.empty(nbytes, dtype=torch.uint8, device=router_w.device)
    with torch.cuda.device(router_w.device):
        L.check(lib.fb_pack_router_weight(_ptr(router_w), E, H, code, _ptr(packed), nbytes,
                                          _stream_handle(router_w.device, stream)),
                "fb_pack_router_weight")
    return PackedRouter(packed, E, H, router_w.dtype)


def predict_split_workspace_bytes(T: int, E: int, H: int, dtype: torch.dtype,
                                  device=None) -> int:
    """fb_predict_split_workspace_bytes on `device`: the workspace size with which a packed batch
    of T tokens runs in split mode (2048 when it runs fused anyway)."""
    code = L.FB_BF16 if dtype == torch.bfloat16 else L.FB_F32 if dtype == torch.float32 else None
    if code is None:
        raise TypeError("dtype must be bfloat16 or float32")
    dev = torch.device(device) if device is not None else torch.device("cuda")
    with torch.cuda.device(dev):
        n = int(L.lib().fb_predict_split_workspace_bytes(T, E, H, code))
    if n == 0:
        L.check(L.FB_EINVAL, "fb_predict_split_workspace_bytes")
    return n


class Predictor:
    """Holds the device workspace of fb_predict_load for one device.

    Calls on one Predictor must be ordered on one stream (they share the workspace).  The workspace
    grows on demand to what fb_predict_workspace_bytes asks for the largest unpacked router seen
    and, with split=True, to what fb_predict_split_workspace_bytes asks for packed batches too small
    to occupy the GPU (those then run in split mode)."""

    def __init__(self, device=None, stream: Optional[torch.cuda.Stream] = None,
                 split: bool = True):
        dev = torch.device(device) if device is not None else torch.device("cuda")
        if dev.type != "cuda":
            raise ValueError("the predictor runs on a GPU device")
        if dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.split = split
        self.workspace = None
        self._reserve(2048, stream)

    def _reserve(self, nbytes: int, stream) -> None:
        if self.workspace is not None and self.workspace.numel() >= nbytes:
            return
        ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            L.check(L.lib().fb_predict_workspace_init(ws.data_ptr(), nbytes,
                                                      _stream_handle(self.device, stream)),
                    "fb_predict_workspace_init")
        self.workspace = ws

    def predict_load(self, hidden: torch.Tensor, router_w, scoring: Scoring,
                     expert_to_rank: torch.Tensor, R: int, *, logit_bias=None, select_bias=None,
                     out: Optional[Prediction] = None, return_topk: bool = False,
                     return_logits: bool = False,
                     stream: Optional[torch.cuda.Stream] = None) -> Prediction:
        """fb_predict_load (router_w an E x H tensor, packed on every call) or
        fb_predict_load_packed (router_w a PackedRouter)."""
        packed = isinstance(router_w, PackedRouter)
        if hidden.dim() != 2:
            raise ValueError("hidden must be T x H")
        if hidden.numel() > 0 and hidden.stride(1) != 1:
            raise ValueError("hidden rows must be contiguous in H")
        T, H = hidden.shape
        if packed:
            E, wdev = router_w.E, router_w.data.device
            if router_w.H != H or router_w.dtype != hidden.dtype:
                raise ValueError("packed router was built for another H or dtype")
        else:
            if router_w.dim() != 2 or not router_w.is_contiguous():
                raise ValueError("router_w must be a contiguous E x H tensor")
            E, wdev = router_w.shape[0], router_w.device
            if router_w.shape[1] != H or router_w.dtype != hidden.dtype:
                raise ValueError("router_w must be E x H with the hidden states' dtype")
        for t in (hidden, expert_to_rank, logit_bias, select_bias):
            if t is not None and t.device != self.device:
                raise ValueError("all tensors must live on the predictor's device")
        if wdev != self.device:
            raise ValueError("all tensors must live on the predictor's device")
        if (expert_to_rank.dtype != torch.int32 or expert_to_rank.numel() != E
                or not expert_to_rank.is_contiguous()):
            raise ValueError("expert_to_rank must be a contiguous int32[E]")
        for b in (logit_bias, select_bias):
            if b is not None and (b.dtype != torch.float32 or b.numel() != E or not b.is_contiguous()):
                raise ValueError("biases must be contiguous float32[E]")
        code = _dtype_code(hidden)
        lib = L.lib()
        if not packed:
            need = int(lib.fb_predict_workspace_bytes(E, H, code))
            if need == 0:
                L.check(L.FB_EUNSUPPORTED if E > 0 else L.FB_EINVAL, "fb_predict_workspace_bytes")
            self._reserve(need, stream)
        elif self.split:
            with torch.cuda.device(self.device):
                need = int(lib.fb_predict_split_workspace_bytes(T, E, H, code))
            if need > 0:
                self._reserve(need, stream)
        if out is None:
            out = Prediction(torch.empty(E, dtype=torch.int32, device=self.device),
                             torch.empty(R, dtype=torch.int32, device=self.device),
                             torch.empty(1, dtype=torch.float64, device=self.device))
        if return_topk and out.topk is None:
            out.topk = torch.empty((T, scoring.k), dtype=torch.int32, device=self.device)
        if return_logits and out.logits is None:
            out.logits = torch.empty((T, E), dtype=torch.float32, device=self.device)
        _check_prediction_out(out, E, R, T, scoring.k, self.device, return_topk, return_logits)
        sc = scoring.to_c()
        ld = hidden.stride(0) if T > 0 else H
        topk = _ptr(out.topk) if return_topk else None
        logits = _ptr(out.logits) if return_logits else None
        sh = _stream_handle(self.device, stream)
        with torch.cuda.device(self.device):
            if packed:
                st = lib.fb_predict_load_packed(
                    _ptr(hidden), T, H, ld, code, _ptr(router_w.data), router_w.data.numel(), E,
                    _ptr(logit_bias), _ptr(select_bias), ctypes.byref(sc), _ptr(expert_to_rank), R,
                    _ptr(out.counts), _ptr(out.rank_loads), _ptr(out.max_mean),
                    _ptr(self.workspace), self.workspace.numel(), topk, logits, sh)
            else:
                st = lib.fb_predict_load(
                    _ptr(hidden), T, H, ld, code, _ptr(router_w), E, _ptr(logit_bias),
                    _ptr(select_bias), ctypes.byref(sc), _ptr(expert_to_rank), R, _ptr(out.counts),
                    _ptr(out.rank_loads), _ptr(out.max_mean), _ptr(self.workspace),
                    self.workspace.numel(), topk, logits, sh)
        L.check(st, "fb_predict_load_packed" if packed else "fb_predict_load")
        return out

    def predict_plan(self, hidden: torch.Tensor, router: PackedRouter, scoring: Scoring,
                     expert_to_rank: torch.Tensor, slots: torch.Tensor, budget: Budget, *,
                     logit_bias=None, select_bias=None, out: Optional[Prediction] = None,
                     plan: Optional[DevicePlan] = None, cost: Optional[CostModel] = None,
                     stream: Optional[torch.cuda.Stream] = None):
        """fb_predict_plan_packed (fb_predict_plan_timed_packed with a cost model): the prediction
        and the swap plan of its counts in one call (the plan inside the predictor's last workgroup
        where the one-wave planner serves it).  slots is the int32[R, S] placement; the cost
        model's node ids and expert sizes as in plan_swaps_timed_device.  Returns (Prediction,
        DevicePlan)."""
        if not isinstance(router, PackedRouter):
            raise ValueError("predict_plan takes a packed router (pack_router_weight)")
        if hidden.dim() != 2 or (hidden.numel() > 0 and hidden.stride(1) != 1):
            raise ValueError("hidden must be T x H with rows contiguous in H")
        if slots.dtype != torch.int32 or slots.dim() != 2 or not slots.is_contiguous():
            raise ValueError("slots must be a contiguous int32[R, S] tensor")
        T, H = hidden.shape
        E = router.E
        if router.H != H or router.dtype != hidden.dtype:
            raise ValueError("packed router was built for another H or dtype")
        R, S = slots.shape
        for t in (hidden, expert_to_rank, slots, logit_bias, select_bias, router.data):
            if t is not None and t.device != self.device:
                raise ValueError("all tensors must live on the predictor's device")
        if (expert_to_rank.dtype != torch.int32 or expert_to_rank.numel() != E
                or not expert_to_rank.is_contiguous()):
            raise ValueError("expert_to_rank must be a contiguous int32[E]")
        for b in (logit_bias, select_bias):
            if b is not None and (b.dtype != torch.float32 or b.numel() != E or not b.is_contiguous()):
                raise ValueError("biases must be contiguous float32[E]")
        code = _dtype_code(hidden)
        lib = L.lib()
        if self.split:
            with torch.cuda.device(self.device):
                need = int(lib.fb_predict_split_workspace_bytes(T, E, H, code))
            if need > 0:
                self._reserve(need, stream)
        else:
            self._reserve(2048, stream)
        dev = self.device
        if out is None:
            out = Prediction(torch.empty(E, dtype=torch.int32, device=dev),
                             torch.empty(R, dtype=torch.int32, device=dev),
                             torch.empty(1, dtype=torch.float64, device=dev))
        cap = max(budget.max_swaps, 1)
        if plan is None:
            plan = DevicePlan(torch.empty(cap * SWAP_BYTES, dtype=torch.uint8, device=dev),
                              torch.empty(1, dtype=torch.int32, device=dev),
                              torch.empty((R, S), dtype=torch.int32, device=dev),
                              torch.empty(E, dtype=torch.int32, device=dev),
                              torch.empty(R, dtype=torch.int64, device=dev),
                              torch.empty(1, dtype=torch.int32, device=dev),
                              None if cost is None else torch.zeros(cap, dtype=torch.int64, device=dev))
        _check_prediction_out(out, E, R, T, scoring.k, dev, False, False)
        _check_plan_out(plan, R, S, E, cap, dev)
        sc = scoring.to_c()
        bg = budget.to_c()
        ld = hidden.stride(0) if T > 0 else H
        head = (_ptr(hidden), T, H, ld, code, _ptr(router.data), router.data.numel(), E,
                _ptr(logit_bias), _ptr(select_bias), ctypes.byref(sc), _ptr(expert_to_rank), R,
                _ptr(out.counts), _ptr(out.rank_loads), _ptr(out.max_mean), _ptr(self.workspace),
                self.workspace.numel(), slots.data_ptr(), S, ctypes.byref(bg))
        tail = (plan.n_swaps.data_ptr(), plan.slots.data_ptr(), plan.expert_to_rank.data_ptr(),
                plan.rank_loads.data_ptr(), plan.status.data_ptr(), _stream_handle(dev, stream))
        if cost is None:
            with torch.cuda.device(dev):
                st = lib.fb_predict_plan_packed(*head, plan.swaps.data_ptr(), *tail)
            L.check(st, "fb_predict_plan_packed")
            return out, plan
        nodes = torch.as_tensor(cost.rank_node, dtype=torch.int32, device=dev).contiguous()
        nbytes = torch.as_tensor(cost.expert_bytes, dtype=torch.int64, device=dev).contiguous()
        if nodes.numel() != R or nbytes.numel() != E:
            raise ValueError("cost model does not match the placement")
        cm = cost.to_c()
        with torch.cuda.device(dev):
            st = lib.fb_predict_plan_timed_packed(*head, ctypes.byref(cm), nodes.data_ptr(),
                                                  nbytes.data_ptr(), plan.swaps.data_ptr(),
                                                  _ptr(plan.costs), *tail)
        L.check(st, "fb_predict_plan_timed_packed")
        return out, plan


def predict_load_packed_noalloc(hidden: torch.Tensor, router: PackedRouter, scoring: Scoring,
                                expert_to_rank: torch.Tensor, R: int, out: Prediction, *,
                                logit_bias=None, select_bias=None,
                                stream: Optional[torch.cuda.Stream] = None) -> Prediction:
    """fb_predict_load_packed_noalloc: the packed prediction with the library's fixed device
    scratch instead of a workspace.  Allocates nothing: every output lives in `out` (counts,
    rank_loads, max_mean, and topk / logits when they are not None).  Calls on one device share the
    scratch, so they must be ordered on one stream."""
    if hidden.dim() != 2 or (hidden.numel() > 0 and hidden.stride(1) != 1):
        raise ValueError("hidden must be T x H with contiguous rows")
    T, H = hidden.shape
    if router.H != H or router.dtype != hidden.dtype:
        raise ValueError("packed router was built for another H or dtype")
    dev = hidden.device
    _one_gpu(dev, hidden, router.data, expert_to_rank, logit_bias, select_bias, out.counts,
             out.rank_loads, out.max_mean, out.topk, out.logits)
    E = router.E
    if (expert_to_rank.dtype != torch.int32 or expert_to_rank.numel() != E
            or not expert_to_rank.is_contiguous()):
        raise ValueError("expert_to_rank must be a contiguous int32[E]")
    _check_prediction_out(out, E, R, T, scoring.k, dev, out.topk is not None, out.logits is not None)
    for b in (logit_bias, select_bias):
        if b is not None and (b.dtype != torch.float32 or b.numel() != E or not b.is_contiguous()):
            raise ValueError("biases must be contiguous float32[E]")
    sc = scoring.to_c()
    with torch.cuda.device(dev):
        st = L.lib().fb_predict_load_packed_noalloc(
            _ptr(hidden), T, H, hidden.stride(0) if T > 0 else H, _dtype_code(hidden),
            _ptr(router.data), router.data.numel(), E, _ptr(logit_bias), _ptr(select_bias),
            ctypes.byref(sc), _ptr(expert_to_rank), R, _ptr(out.counts), _ptr(out.rank_loads),
            _ptr(out.max_mean), _ptr(out.topk), _ptr(out.logits), _stream_handle(dev, stream))
    L.check(st, "fb_predict_load_packed_noalloc")
    return out


_default_predictors = {}


def predict_load(hidden: torch.Tensor, router_w: torch.Tensor, scoring: Scoring,
                 expert_to_rank: torch.Tensor, R: int, **kw) -> Prediction:
    """fb_predict_load on the current stream with a per-device default workspace."""
    dev = hidden.device
    key = (dev.index if dev.index is not None else torch.cuda.current_device())
    pred = _default_predictors.get(key)
    if pred is None:
        pred = _default_predictors[key] = Predictor(torch.device("cuda", key))
    return pred.predict_load(hidden, router_w, scoring, expert_to_rank, R, **kw)


def plan_swaps(counts, slots, budget: Budget) -> Plan:
    """fb_plan_swaps (host planner) on host arrays."""
    c = np.ascontiguousarray(np.asarray(counts), dtype=np.int32)
    sl = np.ascontiguousarray(np.asarray(slots), dtype=np.int32)
    if sl.ndim != 2:
        raise ValueError("slots must be R x S")
    R, S = sl.shape
    E = c.size
    bg = budget.to_c()
    cap = max(budget.max_swaps, 1)
    swaps = (L.fb_swap * cap)()
    n = ctypes.c_int32(0)
    new_slots = np.empty((R, S), np.int32)
    new_e2r = np.empty(E, np.int32)
    new_L = np.empty(R, np.int64)
    st = L.lib().fb_plan_swaps(c.ctypes.data, E, sl.ctypes.data, R, S, ctypes.byref(bg),
                               ctypes.addressof(swaps), cap, ctypes.addressof(n),
                               new_slots.ctypes.data, new_e2r.ctypes.data, new_L.ctypes.data)
    L.check(st, "fb_plan_swaps")
    out = [(s.src_rank, s.dst_rank, s.src_slot, s.dst_slot, s.expert_src, s.expert_dst, s.gain)
           for s in swaps[:n.value]]
    return Plan(out, new_slots, new_e2r, new_L)


def plan_swaps_timed(counts, slots, budget: Budget, cost: CostModel) -> Plan:
    """fb_plan_swaps_timed (host planner under a time budget) on host arrays."""
    c = np.ascontiguousarray(np.asarray(counts), dtype=np.int32)
    sl = np.ascontiguousarray(np.asarray(slots), dtype=np.int32)
    if sl.ndim != 2:
        raise ValueError("slots must be R x S")
    R, S = sl.shape
    E = c.size
    nodes = np.ascontiguousarray(np.asarray(cost.rank_node), dtype=np.int32)
    nbytes = np.ascontiguousarray(np.asarray(cost.expert_bytes), dtype=np.int64)
    if nodes.size != R or nbytes.size != E:
        raise ValueError("cost model does not match the placement")
    bg = budget.to_c()
    cm = cost.to_c()
    cap = max(budget.max_swaps, 1)
    swaps = (L.fb_swap * cap)()
    costs = np.zeros(cap, np.int64)
    n = ctypes.c_int32(0)
    new_slots = np.empty((R, S), np.int32)
    new_e2r = np.empty(E, np.int32)
    new_L = np.empty(R, np.int64)
    st = L.lib().fb_plan_swaps_timed(c.ctypes.data, E, sl.ctypes.data, R, S, ctypes.byref(bg),
                                     ctypes.byref(cm), nodes.ctypes.data, nbytes.ctypes.data,
                                     ctypes.addressof(swaps), costs.ctypes.data, cap,
                                     ctypes.addressof(n), new_slots.ctypes.data, new_e2r.ctypes.data,
                                     new_L.ctypes.data)
    L.check(st, "fb_plan_swaps_timed")
    out = [(s.src_rank, s.dst_rank, s.src_slot, s.dst_slot, s.expert_src, s.expert_dst, s.gain)
           for s in swaps[:n.value]]
    return Plan(out, new_slots, new_e2r, new_L, [int(v) for v in costs[:n.value]])


def plan_swaps_device(counts: torch.Tensor, slots: torch.Tensor, budget: Budget,
                      out: Optional[DevicePlan] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> DevicePlan:
    """fb_plan_swaps_device: the planner as a stream-ordered kernel on device tensors."""
    if counts.dtype != torch.int32 or slots.dtype != torch.int32 or slots.dim() != 2:
        raise ValueError("counts must be int32[E] and slots int32[R, S]")
    if not (counts.is_contiguous() and slots.is_contiguous()):
        raise ValueError("counts and slots must be contiguous")
    dev = counts.device
    _one_gpu(dev, counts, slots)
    R, S = slots.shape
    E = counts.numel()
    if out is None:
        out = DevicePlan(torch.empty(max(budget.max_swaps, 1) * SWAP_BYTES, dtype=torch.uint8, device=dev),
                         torch.empty(1, dtype=torch.int32, device=dev),
                         torch.empty((R, S), dtype=torch.int32, device=dev),
                         torch.empty(E, dtype=torch.int32, device=dev),
                         torch.empty(R, dtype=torch.int64, device=dev),
                         torch.empty(1, dtype=torch.int32, device=dev))
    _check_plan_out(out, R, S, E, max(budget.max_swaps, 1), dev)
    bg = budget.to_c()
    with torch.cuda.device(dev):
        st = L.lib().fb_plan_swaps_device(
            counts.data_ptr(), E, slots.data_ptr(), R, S, ctypes.byref(bg), out.swaps.data_ptr(),
            out.n_swaps.data_ptr(), out.slots.data_ptr(), out.expert_to_rank.data_ptr(),
            out.rank_loads.data_ptr(), out.status.data_ptr(), _stream_handle(dev, stream))
    L.check(st, "fb_plan_swaps_device")
    return out


def plan_swaps_timed_device(counts: torch.Tensor, slots: torch.Tensor, budget: Budget,
                            cost: CostModel, out: Optional[DevicePlan] = None,
                            stream: Optional[torch.cuda.Stream] = None) -> DevicePlan:
    """fb_plan_swaps_timed_device: the time-budgeted planner as a stream-ordered kernel.  The
    cost model's node ids and expert sizes may be sequences (copied to the device on every call)
    or device tensors (int32[R] and int64[E], used as they are: the form for repeated calls)."""
    if counts.dtype != torch.int32 or slots.dtype != torch.int32 or slots.dim() != 2:
        raise ValueError("counts must be int32[E] and slots int32[R, S]")
    if not (counts.is_contiguous() and slots.is_contiguous()):
        raise ValueError("counts and slots must be contiguous")
    dev = counts.device
    _one_gpu(dev, counts, slots)
    R, S = slots.shape
    E = counts.numel()
    nodes = torch.as_tensor(cost.rank_node, dtype=torch.int32, device=dev).contiguous()
    nbytes = torch.as_tensor(cost.expert_bytes, dtype=torch.int64, device=dev).contiguous()
    if nodes.numel() != R or nbytes.numel() != E:
        raise ValueError("cost model does not match the placement")
    cap = max(budget.max_swaps, 1)
    if out is None:
        out = DevicePlan(torch.empty(cap * SWAP_BYTES, dtype=torch.uint8, device=dev),
                         torch.empty(1, dtype=torch.int32, device=dev),
                         torch.empty((R, S), dtype=torch.int32, device=dev),
                         torch.empty(E, dtype=torch.int32, device=dev),
                         torch.empty(R, dtype=torch.int64, device=dev),
                         torch.empty(1, dtype=torch.int32, device=dev),
                         torch.zeros(cap, dtype=torch.int64, device=dev))
    _check_plan_out(out, R, S, E, cap, dev)
    bg = budget.to_c()
    cm = cost.to_c()
    with torch.cuda.device(dev):
        st = L.lib().fb_plan_swaps_timed_device(
            counts.data_ptr(), E, slots.data_ptr(), R, S, ctypes.byref(bg), ctypes.byref(cm),
            nodes.data_ptr(), nbytes.data_ptr(), out.swaps.data_ptr(), _ptr(out.costs),
            out.n_swaps.data_ptr(), out.slots.data_ptr(), out.expert_to_rank.data_ptr(),
            out.rank_loads.data_ptr(), out.status.data_ptr(), _stream_handle(dev, stream))
    L.check(st, "fb_plan_swaps_timed_device")
    return out


def swap_budget_from_cost(t_attn_us: float, delta_us: float, alpha_us: float,
                          beta_bytes_per_us: float, expert_bytes: int) -> int:
    """fb_swap_budget_from_cost (Eq. 9-10 as a swap count)."""
    n = int(L.lib().fb_swap_budget_from_cost(t_attn_us, delta_us, alpha_us, beta_bytes_per_us,
                                             int(expert_bytes)))
    L.check(n if n < 0 else L.FB_OK, "fb_swap_budget_from_cost")
    return n


@dataclasses.dataclass
class Quality:
    """Prediction quality of one layer (device-computed)."""

    hits: int
    hit_rate: float
    logit_cosine: Optional[float]
    hidden_cosine: Optional[float]


_cosine_workspaces = {}


def _cosine_workspace(device: torch.device) -> torch.Tensor:
    key = device.index if device.index is not None else torch.cuda.current_device()
    ws = _cosine_workspaces.get(key)
    if ws is None:
        n = int(L.lib().fb_cosine_workspace_bytes())
        ws = _cosine_workspaces[key] = torch.empty(n, dtype=torch.uint8, device=device)
    return ws


def row_cosine_mean(a: torch.Tensor, b: torch.Tensor,
                    stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """fb_row_cosine_mean: mean over rows of cos(a[r], b[r]) as a device float64 scalar."""
    if a.dim() != 2 or a.shape != b.shape or a.dtype != b.dtype or a.device != b.device:
        raise ValueError("a and b must be matching 2-D tensors on one device")
    if a.stride(1) != 1 or b.stride(1) != 1:
        raise ValueError("rows must be contiguous")
    _one_gpu(a.device, a, b)
    out = torch.empty(1, dtype=torch.float64, device=a.device)
    ws = _cosine_workspace(a.device)
    with torch.cuda.device(a.device):
        L.check(L.lib().fb_row_cosine_mean(_ptr(a), _ptr(b), a.shape[0], a.shape[1], a.stride(0),
                                           b.stride(0), _dtype_code(a), _ptr(out), _ptr(ws), ws.numel(),
                                           _stream_handle(a.device, stream)), "fb_row_cosine_mean")
    return out


def topk_hits(topk_pred: torch.Tensor, topk_actual: torch.Tensor,
              stream: Optional[torch.cuda.Stream] = None,
              with_rate: bool = False):
    """fb_topk_hits: sum over tokens of the predicted and actual sets' intersection size (device
    int64); with_rate=True also returns the device-computed hit rate hits / (T k) (float64)."""
    if topk_pred.shape != topk_actual.shape or topk_pred.dim() != 2:
        raise ValueError("top-k tables must both be T x k")
    for t in (topk_pred, topk_actual):
        if t.dtype != torch.int32 or not t.is_contiguous():
            raise ValueError("top-k tables must be contiguous int32")
    _one_gpu(topk_pred.device, topk_pred, topk_actual)
    out = torch.empty(1, dtype=torch.int64, device=topk_pred.device)
    rate = torch.empty(1, dtype=torch.float64, device=topk_pred.device) if with_rate else None
    with torch.cuda.device(topk_pred.device):
        L.check(L.lib().fb_topk_hits(_ptr(topk_pred), _ptr(topk_actual), topk_pred.shape[0],
                                     topk_pred.shape[1], _ptr(out), _ptr(rate),
                                     _stream_handle(topk_pred.device, stream)), "fb_topk_hits")
    return (out, rate) if with_rate else out


def fold_rank_loads(counts: torch.Tensor, expert_to_rank: torch.Tensor, R: int,
                    stream: Optional[torch.cuda.Stream] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """fb_fold_rank_loads: (rank_loads int32[R], max_mean float64[1]) on the device."""
    if counts.dtype != torch.int32 or expert_to_rank.dtype != torch.int32:
        raise ValueError("counts and expert_to_rank must be int32")
    if counts.numel() != expert_to_rank.numel():
        raise ValueError("counts and expert_to_rank must have E entries each")
    if not (counts.is_contiguous() and expert_to_rank.is_contiguous()):
        raise ValueError("counts and expert_to_rank must be contiguous")
    dev = counts.device
    _one_gpu(dev, counts, expert_to_rank)
    loads = torch.empty(R, dtype=torch.int32, device=dev)
    mm = torch.empty(1, dtype=torch.float64, device=dev)
    with torch.cuda.device(dev):
        L.check(L.lib().fb_fold_rank_loads(_ptr(counts), counts.numel(), _ptr(expert_to_rank), R,
                                           _ptr(loads), _ptr(mm), _stream_handle(dev, stream)),
                "fb_fold_rank_loads")
    return loads, mm


def fold_slot_loads(counts: torch.Tensor, slots: torch.Tensor,
                    stream: Optional[torch.cuda.Stream] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """fb_fold_slot_loads: rank loads of a (possibly replicated) R x S slot table, as
    (rank_loads int32[R], max_mean float64[1]) on the device; max_mean is -1 for a table that breaks
    the placement rules."""
    if counts.dtype != torch.int32 or slots.dtype != torch.int32 or slots.dim() != 2:
        raise ValueError("counts must be int32[E] and slots an int32 R x S table")
    if not (counts.is_contiguous() and slots.is_contiguous()) or counts.device != slots.device:
        raise ValueError("counts and slots must be contiguous and on one device")
    dev = counts.device
    _one_gpu(dev, counts, slots)
    R, S = slots.shape
    loads = torch.empty(R, dtype=torch.int32, device=dev)
    mm = torch.empty(1, dtype=torch.float64, device=dev)
    with torch.cuda.device(dev):
        L.check(L.lib().fb_fold_slot_loads(_ptr(counts), counts.numel(), _ptr(slots), R, S,
                                           _ptr(loads), _ptr(mm), _stream_handle(dev, stream)),
                "fb_fold_slot_loads")
    return loads, mm


def prediction_quality(pred: Prediction, actual: Prediction, hidden_prev: Optional[torch.Tensor] = None,
                       hidden_target: Optional[torch.Tensor] = None) -> Quality:
    """Hit rate and cosines of an early pass against the actual routing; both Predictions must
    carry topk (and logits for the logit cosine)."""
    if pred.topk is None or actual.topk is None:
        raise ValueError("both passes need return_topk=True")
    hits, rate = topk_hits(pred.topk, actual.topk, with_rate=True)
    lc = row_cosine_mean(pred.logits, actual.logits) if pred.logits is not None and actual.logits is not None else None
    hc = row_cosine_mean(hidden_prev, hidden_target) if hidden_prev is not None and hidden_target is not None else None
    return Quality(int(hits.item()), float(rate.item()), None if lc is None else float(lc.item()),
                   None if hc is None else float(hc.item()))
