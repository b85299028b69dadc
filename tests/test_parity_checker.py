"""The comparison rules of the GPU parity tests (tests/parity.py), checked on the CPU: the oracle's
own outputs pass, outputs perturbed within the rigorous logit bound pass (their differing tokens are
exempt and valid), and planted mistakes of each kind are caught."""
import dataclasses

import numpy as np
import pytest

import parity as P
from oracle import predictor as OP
from workloads import CONFIGS, make_layer


def _oracle_outputs(name, T, layer=0, **over):
    wl = dataclasses.replace(CONFIGS[name].with_T(T), **over)
    li = make_layer(wl, layer)
    z = OP.router_logits(li.x, li.w, wl.dtype)
    topk, s, _ = OP.select(z, wl.k, wl.kind, li.select_bias, wl.n_group, wl.topk_group, wl.group_topn)
    return wl, li, z, topk, s


@pytest.mark.parametrize("name", ["tiny", "mixtral", "qwen3", "dsv3"])
def test_oracle_outputs_pass(name):
    wl, li, z, topk, _ = _oracle_outputs(name, 300, H=512 if name != "tiny" else 1024)
    st, fails, hist = P.compare_prediction(z, topk, li.x, li.w, li.select_bias, wl)
    assert not fails and st["mismatch"] == 0 and st["mismatch_on_gpu_logits"] == 0
    assert np.array_equal(hist, OP.expert_histogram(topk, wl.E))


@pytest.mark.parametrize("name", ["qwen3", "dsv3"])
def test_perturbation_within_the_bound_passes(name):
    """Logits moved by up to 0.9 of the rigorous bound, then selected by the rule: differing tokens
    are exempt and valid, and the histogram rule holds."""
    wl, li, z, topk, _ = _oracle_outputs(name, 600, H=512)
    bound = P.logit_bounds(li.x, li.w, wl)
    g = np.random.default_rng(5)
    zp = (z.astype(np.float64) + 0.9 * bound * g.uniform(-1, 1, z.shape)).astype(np.float32)
    tp, _, _ = OP.select(zp, wl.k, wl.kind, li.select_bias, wl.n_group, wl.topk_group, wl.group_topn)
    st, fails, _ = P.compare_prediction(zp, tp, li.x, li.w, li.select_bias, wl)
    assert not fails, fails
    assert st["counts_l1_vs_oracle"] <= 2 * wl.k * st["mismatch"]


def _planted(name, mutate, T=300):
    wl, li, z, topk, s = _oracle_outputs(name, T, H=512)
    z2, t2 = z.copy(), topk.copy()
    mutate(wl, z2, t2, s)
    _, fails, _ = P.compare_prediction(z2, t2, li.x, li.w, li.select_bias, wl)
    return fails


def test_catches_a_low_scoring_expert():
    def m(wl, z, t, s):
        outside = np.setdiff1d(np.arange(wl.E), t[7])
        t[7, -1] = outside[np.argmin(s[7, outside])]
    fails = _planted("qwen3", m)
    assert any("rule on the GPU's own logits" in f for f in fails)
    assert any("invalid selection" in f for f in fails)


def test_catches_an_expert_outside_the_kept_groups():
    def m(wl, z, t, s):
        gsz = wl.E // wl.n_group
        gs = OP.group_scores(s[11:12], wl.n_group, wl.group_topn)[0]
        worst = int(np.argmin(gs))
        # the best expert of the worst group: high enough to pass a pure score test
        e = worst * gsz + int(np.argmax(s[11, worst * gsz:(worst + 1) * gsz]))
        t[11, -1] = e
    fails = _planted("dsv3", m)
    assert any("cannot be kept" in f for f in fails), fails


def test_catches_a_repeated_expert():
    def m(wl, z, t, s):
        t[3, 1] = t[3, 0]
    assert any("distinct" in f for f in _planted("dsv3", m))


def test_catches_a_list_out_of_order():
    def m(wl, z, t, s):
        t[4] = t[4][::-1]
    assert any("descending score order" in f for f in _planted("qwen3", m))


def test_catches_logits_beyond_the_bound():
    def m(wl, z, t, s):
        z[9, 3] += 1e-3 * max(1.0, abs(float(z[9, 3])))
    assert any("summation error bound" in f for f in _planted("mixtral", m))


def test_catches_a_selection_that_ignores_the_logits():
    """A selection that is valid for the oracle's logits but not for the logits reported next to it."""
    def m(wl, z, t, s):
        z[2, t[2, 0]] = -30.0
    fails = _planted("qwen3", m)
    assert any("rule on the GPU's own logits" in f for f in fails)
