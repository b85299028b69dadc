"""Seeded synthetic input generator: determinism, bf16 rounding and the input recipe."""
import hashlib

import numpy as np
import pytest
import torch

import workloads
from workloads import CONFIGS, bf16_bits_from_f32, contiguous_placement, make_layer
from workloads.synth import truncated_zipf_probs


def _h(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def test_bf16_rne_matches_torch_cast():
    g = np.random.default_rng(0)
    x = np.concatenate([
        g.standard_normal(200000).astype(np.float32) * np.float32(3.0),
        g.standard_normal(1000).astype(np.float32) * np.float32(1e-30),
        np.array([0.0, -0.0, 1.0, -1.0, 65504.0, 3.0e38, 1.0e-38, 1.00390625, 1.01171875],
                 dtype=np.float32),
    ])
    # values exactly half-way between two bf16 neighbours exercise the ties-to-even rule
    halfway = (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    x = np.concatenate([x, halfway])
    ours = bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_rejects_non_finite():
    with pytest.raises(ValueError):
        bf16_bits_from_f32(np.array([np.inf], np.float32))


def test_layer_generation_is_deterministic():
    wl = CONFIGS["tiny"]
    a = make_layer(wl, 3, with_target=True)
    b = make_layer(wl, 3, with_target=True)
    assert _h(a.x) == _h(b.x) and _h(a.w) == _h(b.w) and _h(a.h_target) == _h(b.h_target)
    c = make_layer(wl, 4)
    assert _h(a.w) != _h(c.w) and _h(a.x) != _h(c.x)


def test_sampled_rows_match_full_generation():
    wl = CONFIGS["mixtral"].with_T(5000)
    full = make_layer(wl, 1, with_target=True)
    rows = [0, 17, 2047, 2048, 4999]
    part = make_layer(wl, 1, with_target=True, rows=rows)
    assert np.array_equal(part.x, full.x[rows])
    assert np.array_equal(part.h_target, full.h_target[rows])
    assert np.array_equal(part.clusters, full.clusters[rows])


def test_zero_sigma_target_equals_input():
    import dataclasses
    wl = dataclasses.replace(CONFIGS["qwen3"], T=300, sigma=0.0)
    li = make_layer(wl, 0, with_target=True)
    assert np.array_equal(li.x, li.h_target)


def test_dtypes_and_shapes():
    t = make_layer(CONFIGS["tiny"], 0)
    assert t.x.dtype == np.float32 and t.x.shape == (512, 1024) and t.w.shape == (16, 1024)
    m = make_layer(CONFIGS["mixtral"].with_T(64), 0)
    assert m.x.dtype == np.uint16 and m.w.dtype == np.uint16 and m.select_bias is None
    d = make_layer(CONFIGS["dsv3"].with_T(64), 0)
    assert d.select_bias is not None and d.select_bias.dtype == np.float32 and d.select_bias.shape == (256,)


def test_router_weight_and_bias_statistics():
    w = make_layer(CONFIGS["tiny"], 0).w
    assert abs(float(w.std()) - 0.02) < 0.001 and abs(float(w.mean())) < 0.001
    b = make_layer(CONFIGS["dsv3"].with_T(1), 0).select_bias
    assert abs(float(b.std()) - 0.01) < 0.003


def test_truncated_zipf():
    p = truncated_zipf_probs(1.2, 16)
    assert abs(p.sum() - 1.0) < 1e-12 and np.all(np.diff(p) < 0)
    assert abs(p[0] / p[1] - 2 ** 1.2) < 1e-9
    q = truncated_zipf_probs(0.0, 5)
    assert np.allclose(q, 0.2)


def test_cluster_frequencies_follow_zipf():
    wl = CONFIGS["tiny"].with_T(200000)
    cl = workloads.synth._token_clusters(wl, wl.T)
    freq = np.bincount(cl, minlength=16) / wl.T
    assert np.max(np.abs(freq - truncated_zipf_probs(1.2, 16))) < 0.005


def test_sweep_mixture():
    wl = workloads.sweep_workload(4096)
    assert wl.tasks == 4 and wl.layers == 58 and wl.budgets == (0, 4, 8, 16)
    assert np.allclose(wl.zipf_s, [0.8, 1.0666666666666667, 1.3333333333333333, 1.6])
    cl = workloads.synth._token_clusters(wl, wl.T)
    assert cl.min() >= 0 and cl.max() < 256 and len(np.unique(cl)) > 64


def test_contiguous_placement():
    slots, e2r = contiguous_placement(256, 32, 8)
    assert slots.shape == (32, 8) and slots[3].tolist() == list(range(24, 32))
    assert e2r[24] == 3 and e2r[255] == 31
    slots, e2r = contiguous_placement(8, 8, 2)
    assert slots[5].tolist() == [5, -1] and e2r.tolist() == list(range(8))
    with pytest.raises(ValueError):
        contiguous_placement(10, 4, 4)
