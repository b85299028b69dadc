"""fb_predict_load_packed_noalloc (the prediction with the library's fixed device scratch, for
callers that cannot allocate) against fb_predict_load_packed with a caller workspace, through the C
ABI: calls in a row on one stream, each smaller than the one before (fused, then split-mode
batches), every output bit for bit, and every call against the oracle."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2608_14205_amd as fb
from gpu_util import check_prediction, scoring_of, to_device
from workloads import CONFIGS, contiguous_placement, make_layer

pytestmark = pytest.mark.gpu


def _run_both(wl, li, e2r, pred):
    dev = torch.device("cuda", torch.cuda.current_device())
    x = to_device(li.x, wl.dtype)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    sb = None if li.select_bias is None else torch.from_numpy(li.select_bias).cuda()
    e2r_t = torch.from_numpy(np.asarray(e2r, np.int32)).cuda()
    ref = pred.predict_load(x, wp, scoring_of(wl), e2r_t, wl.R, select_bias=sb, return_topk=True,
                            return_logits=True)
    out = fb.Prediction(torch.empty(wl.E, dtype=torch.int32, device=dev),
                        torch.empty(wl.R, dtype=torch.int32, device=dev),
                        torch.empty(1, dtype=torch.float64, device=dev),
                        torch.empty((wl.T, wl.k), dtype=torch.int32, device=dev),
                        torch.empty((wl.T, wl.E), dtype=torch.float32, device=dev))
    fb.predict_load_packed_noalloc(x, wp, scoring_of(wl), e2r_t, wl.R, out, select_bias=sb)
    torch.cuda.synchronize()
    return ref, out


def test_noalloc_matches_the_workspace_entry_point():
    pred = fb.Predictor()
    base = CONFIGS["dsv3"]
    _, e2r = contiguous_placement(base.E, base.R, base.S)
    for i, T in enumerate((20000, 5000, 300)):
        wl = dataclasses.replace(base, T=T)
        split = fb.predict_split_workspace_bytes(T, wl.E, wl.H, torch.bfloat16) > 2048
        print(f"[noalloc] call {i}: T={T} split={split}", flush=True)
        assert split == (T < 20000)
        li = make_layer(wl, 4 + i)
        ref, out = _run_both(wl, li, e2r, pred)
        for name in ("counts", "rank_loads", "topk"):
            assert torch.equal(getattr(ref, name), getattr(out, name)), name
        assert torch.equal(ref.logits.view(torch.int32), out.logits.view(torch.int32))
        assert ref.max_mean.item() == out.max_mean.item()
        got = {"counts": out.counts.cpu().numpy().astype(np.int64),
               "rank_loads": out.rank_loads.cpu().numpy().astype(np.int64),
               "max_mean": float(out.max_mean.item()), "topk": out.topk.cpu().numpy(),
               "logits": out.logits.cpu().numpy()}
        check_prediction(got, li, wl, e2r, label=f"noalloc/T={T}")


def test_noalloc_empty_batch():
    wl = dataclasses.replace(CONFIGS["qwen3"], T=0, H=256)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    dev = torch.device("cuda", torch.cuda.current_device())
    li = make_layer(dataclasses.replace(wl, T=1), 0)
    wp = fb.pack_router_weight(to_device(li.w, wl.dtype))
    out = fb.Prediction(torch.full((wl.E,), 7, dtype=torch.int32, device=dev),
                        torch.full((wl.R,), 7, dtype=torch.int32, device=dev),
                        torch.zeros(1, dtype=torch.float64, device=dev))
    x = torch.empty((0, wl.H), dtype=torch.bfloat16, device=dev)
    fb.predict_load_packed_noalloc(x, wp, scoring_of(wl), torch.from_numpy(e2r).cuda(), wl.R, out)
    torch.cuda.synchronize()
    assert int(out.counts.sum()) == 0 and int(out.rank_loads.sum()) == 0
    assert out.max_mean.item() == 1.0
