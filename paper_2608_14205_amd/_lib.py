"""ctypes view of libfreebalance.so (declarations mirror include/freebalance.h).

The library is loaded from the package directory only.  A missing or unloadable library raises
immediately: there is no CPU fallback behind this binding.
"""
from __future__ import annotations

import ctypes
import os
import threading

LIB_NAME = "libfreebalance.so"
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

FB_OK, FB_EINVAL, FB_EUNSUPPORTED, FB_EDEVICE, FB_ENOSPC = 0, -1, -2, -3, -4
FB_BF16, FB_F32 = 0, 1
FB_SOFTMAX, FB_SIGMOID = 0, 1
FB_FRONTIER, FB_FULL = 0, 1
ABI_VERSION = 6


class fb_scoring(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("k", ctypes.c_int32), ("n_group", ctypes.c_int32),
                ("topk_group", ctypes.c_int32), ("group_topn", ctypes.c_int32)]


class fb_budget(ctypes.Structure):
    _fields_ = [("max_swaps", ctypes.c_int32), ("per_rank_cap", ctypes.c_int32),
                ("tau", ctypes.c_int64), ("gamma_num", ctypes.c_int64),
                ("gamma_den", ctypes.c_int64), ("mode", ctypes.c_int32),
                ("layer_id", ctypes.c_int32)]


class fb_cost_model(ctypes.Structure):
    _fields_ = [("rank_budget_ns", ctypes.c_int64), ("link_budget_ns", ctypes.c_int64),
                ("alpha_ns", ctypes.c_int64 * 2), ("beta_bytes_per_us", ctypes.c_int64 * 2)]


class fb_swap(ctypes.Structure):
    _fields_ = [("src_rank", ctypes.c_int32), ("dst_rank", ctypes.c_int32),
                ("src_slot", ctypes.c_int32), ("dst_slot", ctypes.c_int32),
                ("expert_src", ctypes.c_int32), ("expert_dst", ctypes.c_int32),
                ("gain", ctypes.c_int64)]


class FreeBalanceError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


_VP, _I32, _I64, _SZ, _D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_double

SIGNATURES = {
    "fb_abi_version": (ctypes.c_int, []),
    "fb_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "fb_router_packed_bytes": (_SZ, [_I32, _I32, _I32]),
    "fb_predict_workspace_bytes": (_SZ, [_I32, _I32, _I32]),
    "fb_predict_workspace_init": (ctypes.c_int, [_VP, _SZ, _VP]),
    "fb_predict_load": (ctypes.c_int, [_VP, _I64, _I32, _I64, _I32, _VP, _I32, _VP, _VP,
                                       ctypes.POINTER(fb_scoring), _VP, _I32, _VP, _VP, _VP, _VP,
                                       _SZ, _VP, _VP, _VP]),
    "fb_pack_router_weight": (ctypes.c_int, [_VP, _I32, _I32, _I32, _VP, _SZ, _VP]),
    "fb_predict_load_packed": (ctypes.c_int, [_VP, _I64, _I32, _I64, _I32, _VP, _SZ, _I32, _VP,
                                              _VP, ctypes.POINTER(fb_scoring), _VP, _I32, _VP,
                                              _VP, _VP, _VP, _SZ, _VP, _VP, _VP]),
    "fb_predict_plan_packed": (ctypes.c_int, [_VP, _I64, _I32, _I64, _I32, _VP, _SZ, _I32, _VP,
                                              _VP, ctypes.POINTER(fb_scoring), _VP, _I32, _VP,
                                              _VP, _VP, _VP, _SZ, _VP, _I32,
                                              ctypes.POINTER(fb_budget), _VP, _VP, _VP, _VP, _VP,
                                              _VP, _VP]),
    "fb_predict_plan_timed_packed": (ctypes.c_int, [_VP, _I64, _I32, _I64, _I32, _VP, _SZ, _I32,
                                                    _VP, _VP, ctypes.POINTER(fb_scoring), _VP, _I32,
                                                    _VP, _VP, _VP, _VP, _SZ, _VP, _I32,
                                                    ctypes.POINTER(fb_budget),
                                                    ctypes.POINTER(fb_cost_model), _VP, _VP, _VP,
                                                    _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "fb_predict_load_packed_noalloc": (ctypes.c_int, [_VP, _I64, _I32, _I64, _I32, _VP, _SZ, _I32,
                                                      _VP, _VP, ctypes.POINTER(fb_scoring), _VP,
                                                      _I32, _VP, _VP, _VP, _VP, _VP, _VP]),
    "fb_predict_split_workspace_bytes": (_SZ, [_I64, _I32, _I32, _I32]),
    "fb_plan_swaps": (ctypes.c_int, [_VP, _I32, _VP, _I32, _I32, ctypes.POINTER(fb_budget), _VP,
                                     _I32, _VP, _VP, _VP, _VP]),
    "fb_plan_swaps_device": (ctypes.c_int, [_VP, _I32, _VP, _I32, _I32, ctypes.POINTER(fb_budget),
                                            _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "fb_plan_swaps_timed": (ctypes.c_int, [_VP, _I32, _VP, _I32, _I32, ctypes.POINTER(fb_budget),
                                           ctypes.POINTER(fb_cost_model), _VP, _VP, _VP, _VP, _I32,
                                           _VP, _VP, _VP, _VP]),
    "fb_plan_swaps_timed_device": (ctypes.c_int, [_VP, _I32, _VP, _I32, _I32,
                                                  ctypes.POINTER(fb_budget),
                                                  ctypes.POINTER(fb_cost_model), _VP, _VP, _VP,
                                                  _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "fb_swap_budget_from_cost": (_I64, [_D, _D, _D, _D, _I64]),
    "fb_topk_hits": (ctypes.c_int, [_VP, _VP, _I64, _I32, _VP, _VP, _VP]),
    "fb_cosine_workspace_bytes": (_SZ, []),
    "fb_row_cosine_mean": (ctypes.c_int, [_VP, _VP, _I64, _I32, _I64, _I64, _I32, _VP, _VP, _SZ, _VP]),
    "fb_fold_rank_loads": (ctypes.c_int, [_VP, _I32, _VP, _I32, _VP, _VP, _VP]),
    "fb_fold_slot_loads": (ctypes.c_int, [_VP, _I32, _VP, _I32, _I32, _VP, _VP, _VP]),
}

_lock = threading.Lock()
_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it is missing (build it with paper_2608_14205_amd.build)."""
    global _lib
    if _lib is None:
        with _lock:
            if _lib is None:
                if not os.path.exists(LIB_PATH):
                    raise ImportError(f"{LIB_PATH} is missing: build the HIP library first "
                                      "(python -m paper_2608_14205_amd.build)")
                handle = ctypes.CDLL(LIB_PATH)
                for name, (res, args) in SIGNATURES.items():
                    fn = getattr(handle, name)
                    fn.restype = res
                    fn.argtypes = args
                if handle.fb_abi_version() != ABI_VERSION:
                    raise ImportError("libfreebalance.so ABI version mismatch")
                _lib = handle
    return _lib


def status_string(status: int) -> str:
    return lib().fb_status_string(int(status)).decode()


def check(status: int, where: str) -> None:
    if status != FB_OK:
        raise FreeBalanceError(status, where)
