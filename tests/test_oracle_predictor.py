"""Pins of the predictor oracle against the paper's definitions (no GPU).

The oracle is checked against things other than itself: hand-worked cases, an exact-rational
micro-oracle, brute-force selection by explicit sorting, an explicit float64 softmax, and invariants and
metamorphic relations that the definitions (Eq. 4, Eq. 5, the top-k rule, Alg. 1's rank aggregation)
imply.
"""
import json
import os

import numpy as np
import pytest

from oracle import exact
from oracle import predictor as P
from workloads import CONFIGS, bf16_bits_from_f32, contiguous_placement, make_layer


def _load_golden(golden_dir):
    with open(os.path.join(golden_dir, "predictor_hand.json")) as f:
        return json.load(f)["cases"]


def test_hand_worked_cases(golden_dir):
    for c in _load_golden(golden_dir):
        x = np.array(c["x"], np.float32)
        w = np.array(c["w"], np.float32)
        sb = None if c.get("select_bias") is None else np.array(c["select_bias"], np.float32)
        lb = None if c.get("logit_bias") is None else np.array(c["logit_bias"], np.float32)
        out = P.predict_load(x, w, "f32", c["k"], c["kind"], np.array(c["expert_to_rank"]), c["R"],
                             select_bias=sb, logit_bias=lb, n_group=c.get("n_group", 1),
                             topk_group=c.get("topk_group", 1), group_topn=c.get("group_topn", 1))
        assert out["logits"].tolist() == c["logits"], c["name"]
        assert out["topk"].tolist() == c["topk"], c["name"]
        assert out["counts"].tolist() == c["counts"], c["name"]
        assert out["rank_loads"].tolist() == c["rank_loads"], c["name"]
        assert out["max_mean"] == pytest.approx(c["max_mean"], abs=1e-15), c["name"]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_float64_gemm_matches_exact_rationals(dtype):
    g = np.random.default_rng(11)
    T, H, E = 6, 48, 5
    x = g.standard_normal((T, H)).astype(np.float32) * np.float32(2.0)
    w = g.standard_normal((E, H)).astype(np.float32) * np.float32(0.05)
    b = g.standard_normal(E).astype(np.float32) * np.float32(0.1)
    if dtype == "bf16":
        x, w = bf16_bits_from_f32(x), bf16_bits_from_f32(w)
    z = P.router_logits(x, w, dtype, b)
    zx = exact.exact_logits(x, w, dtype, b)
    assert np.array_equal(z.view(np.uint32), zx.view(np.uint32))


def test_logits_follow_router_orientation():
    # w is stored E x H (row e = column e of the paper's W); a one-hot hidden picks out column h
    H, E = 8, 3
    w = np.arange(E * H, dtype=np.float32).reshape(E, H)
    x = np.zeros((1, H), np.float32)
    x[0, 5] = 1.0
    assert P.router_logits(x, w, "f32").tolist() == [[5.0, 13.0, 21.0]]


def _random_case(seed, T, E, ties=False):
    g = np.random.default_rng(seed)
    z = g.standard_normal((T, E)).astype(np.float32)
    if ties:
        z = np.round(z * 2) / 2   # many exact ties
    return z


@pytest.mark.parametrize("kind", ["softmax", "sigmoid"])
@pytest.mark.parametrize("groups", [(1, 1, 1), (4, 2, 2), (8, 4, 2), (4, 3, 1)])
@pytest.mark.parametrize("ties", [False, True])
def test_selection_matches_brute_force(kind, groups, ties):
    n_group, topk_group, topn = groups
    E, T, k = 16 if n_group <= 4 else 32, 40, 3
    z = _random_case(7 + n_group, T, E, ties)
    if kind == "softmax" and n_group > 1 and topn > 1:
        # sums of logits do not rank groups like sums of probabilities: refused on both sides
        with pytest.raises(ValueError):
            P.select(z, k, kind, None, n_group, topk_group, topn)
        with pytest.raises(ValueError):
            exact.brute_select(z[0].tolist(), k, kind, None, n_group, topk_group, topn)
        return
    g = np.random.default_rng(5)
    bias = (g.standard_normal(E) * 0.01).astype(np.float32) if kind == "sigmoid" else None
    if ties and bias is not None:
        bias = np.round(bias * 256) / 256
    topk, _, _ = P.select(z, k, kind, bias, n_group, topk_group, topn)
    for t in range(T):
        ref = exact.brute_select(z[t].tolist(), k, kind, None if bias is None else bias.tolist(),
                                 n_group, topk_group, topn)
        assert topk[t].tolist() == ref


def test_softmax_selection_equals_probability_selection():
    g = np.random.default_rng(3)
    z = (g.standard_normal((500, 128)) * 2).astype(np.float32)
    z64 = z.astype(np.float64)
    p = np.exp(z64 - z64.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    eid = np.broadcast_to(np.arange(128), p.shape)
    by_prob = np.lexsort((eid, -p), axis=-1)[:, :8]
    topk, _, _ = P.select(z, 8, "softmax")
    assert np.array_equal(np.sort(by_prob, 1), np.sort(topk, 1))


def test_softmax_group_max_ranks_groups_like_probabilities():
    """Softmax with groups scored by their maximum: groups kept and experts chosen on logits equal
    those chosen on explicit float64 probabilities (brute force per token)."""
    g = np.random.default_rng(11)
    z = (g.standard_normal((300, 32)) * 3).astype(np.float32)
    topk, _, _ = P.select(z, 4, "softmax", None, 8, 3, 1)
    z64 = z.astype(np.float64)
    p = np.exp(z64 - z64.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    for t in range(z.shape[0]):
        gmax = [max(p[t, 4 * q:4 * q + 4]) for q in range(8)]
        kept = sorted(range(8), key=lambda q: (-gmax[q], q))[:3]
        ref = sorted((e for e in range(32) if e // 4 in kept), key=lambda e: (-p[t, e], e))[:4]
        assert topk[t].tolist() == ref


def test_softmax_group_sum_is_not_a_logit_rule():
    """Why softmax routing refuses group sums: logits (10, -100) outrank (5, 5) on the sum of
    probabilities and not on the sum of logits."""
    z = np.array([10.0, -100.0, 5.0, 5.0])
    p = np.exp(z - z.max())
    p /= p.sum()
    assert p[0] + p[1] > p[2] + p[3] and z[0] + z[1] < z[2] + z[3]


def test_group_limit_degenerates_to_plain_topk():
    z = _random_case(21, 64, 32)
    plain, _, _ = P.select(z, 4, "sigmoid")
    for ng in (1, 2, 4, 8):
        all_kept, _, _ = P.select(z, 4, "sigmoid", None, ng, ng, 2)
        assert np.array_equal(all_kept, plain)


def test_sigmoid_scores_are_correctly_rounded():
    z = np.array([0.0, -1.5, 2.25, 10.0, -30.0], np.float32)
    s = P.router_scores(z, "sigmoid")
    for v, sv in zip(z.tolist(), s.tolist()):
        assert sv == exact.f32_round(1.0 / (1.0 + np.exp(-v)))
    assert s[0] == 0.5
    # sigma(-z) = 1 - sigma(z) up to one float32 rounding of each side
    zz = np.linspace(-6, 6, 101).astype(np.float32)
    a, b = P.router_scores(zz, "sigmoid"), P.router_scores(-zz, "sigmoid")
    assert np.max(np.abs(a.astype(np.float64) + b - 1.0)) < 1.2e-7


def _predict(li, wl, e2r):
    return P.predict_load(li.x, li.w, wl.dtype, wl.k, wl.kind, e2r, wl.R,
                          select_bias=li.select_bias, n_group=wl.n_group,
                          topk_group=wl.topk_group, group_topn=wl.group_topn)


@pytest.mark.parametrize("name,T", [("tiny", 512), ("mixtral", 700), ("qwen3", 600), ("dsv3", 300)])
def test_invariants_on_workloads(name, T):
    wl = CONFIGS[name].with_T(T)
    li = make_layer(wl, 0)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    out = _predict(li, wl, e2r)
    topk, counts, L = out["topk"], out["counts"], out["rank_loads"]
    assert topk.shape == (T, wl.k)
    assert all(len(set(r.tolist())) == wl.k for r in topk)          # k distinct experts per token
    assert counts.sum() == T * wl.k and np.all(counts <= T) and np.all(counts >= 0)
    assert L.sum() == T * wl.k
    assert 1.0 <= out["max_mean"] <= wl.R
    if wl.n_group > 1:   # every selected expert lies in a kept group, at most topk_group groups used
        gsz = wl.E // wl.n_group
        for r in topk:
            assert len(set((r // gsz).tolist())) <= wl.topk_group
    # clustered hidden states give real routing skew
    assert out["max_mean"] > 1.05


def test_uniform_counts_balance():
    counts = np.full(256, 10, np.int64)
    _, e2r = contiguous_placement(256, 32, 8)
    L = P.rank_loads(counts, e2r, 32)
    assert L.tolist() == [80] * 32 and P.max_to_mean(L) == 1.0
    assert P.max_to_mean(np.zeros(4, np.int64)) == 1.0


def test_rank_fold_rejects_bad_rank():
    with pytest.raises(ValueError):
        P.rank_loads(np.ones(4), np.array([0, 1, 2, 4]), 4)


def test_token_permutation_keeps_counts():
    wl = CONFIGS["qwen3"].with_T(400)
    li = make_layer(wl, 2)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    a = _predict(li, wl, e2r)
    perm = np.random.default_rng(0).permutation(wl.T)
    li.x = li.x[perm]
    b = _predict(li, wl, e2r)
    assert np.array_equal(a["counts"], b["counts"])
    assert np.array_equal(a["topk"][perm], b["topk"])


def test_expert_relabelling_permutes_counts():
    # permute whole groups and experts within groups: a relabelling that keeps the group structure
    wl = CONFIGS["dsv3"].with_T(256)
    li = make_layer(wl, 1)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    a = _predict(li, wl, e2r)
    g = np.random.default_rng(9)
    gsz = wl.E // wl.n_group
    gperm = g.permutation(wl.n_group)
    perm = np.concatenate([gp * gsz + g.permutation(gsz) for gp in gperm])  # new e -> old perm[e]
    li.w = li.w[perm]
    li.select_bias = li.select_bias[perm]
    b = _predict(li, wl, e2r[perm])
    assert np.array_equal(b["counts"], a["counts"][perm])
    assert np.array_equal(b["rank_loads"], a["rank_loads"])


def test_prediction_equals_actual_when_inputs_coincide():
    import dataclasses
    wl = dataclasses.replace(CONFIGS["dsv3"], T=128, sigma=0.0)
    li = make_layer(wl, 0, with_target=True)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    pred = _predict(li, wl, e2r)
    li.x = li.h_target
    act = _predict(li, wl, e2r)
    assert np.array_equal(pred["topk"], act["topk"]) and np.array_equal(pred["counts"], act["counts"])
    assert P.hit_rate(pred["topk"], act["topk"]) == 1.0


def test_prediction_quality_metrics_are_sane():
    wl = CONFIGS["qwen3"].with_T(512)
    li = make_layer(wl, 0, with_target=True)
    zp = P.router_logits(li.x, li.w, wl.dtype)
    za = P.router_logits(li.h_target, li.w, wl.dtype)
    tp, _, _ = P.select(zp, wl.k, wl.kind)
    ta, _, _ = P.select(za, wl.k, wl.kind)
    hr = P.hit_rate(tp, ta)
    assert 0.3 < hr < 1.0
    assert 0.9 < P.mean_cosine(zp, za) <= 1.0
    assert P.mean_cosine(za, za) == pytest.approx(1.0)
    assert P.hit_rate(tp, tp) == 1.0


def test_softmax_rejects_selection_bias():
    with pytest.raises(ValueError):
        P.router_scores(np.zeros((1, 4), np.float32), "softmax", np.zeros(4, np.float32))


def test_topk_requires_enough_allowed():
    s = np.zeros((1, 4), np.float32)
    with pytest.raises(ValueError):
        P.topk_experts(s, 3, np.array([[True, True, False, False]]))


def test_quality_metrics_hand_worked():
    """Hand-worked values of the prediction-quality metrics (Sec. "Metrics"): the hit rate counts set
    intersections, the cosine is the mean of the per-row cosines."""
    tp = np.array([[0, 1], [2, 3], [1, 0]])
    ta = np.array([[1, 0], [2, 4], [3, 2]])
    # row 0: {0,1} & {0,1} = 2; row 1: {2,3} & {2,4} = 1; row 2: {0,1} & {2,3} = 0 -> 3 / 6
    assert P.hit_rate(tp, ta) == 0.5
    a = np.array([[1.0, 0.0], [1.0, 1.0], [3.0, 4.0]])
    b = np.array([[2.0, 0.0], [1.0, 0.0], [-3.0, -4.0]])
    # cosines 1, 1/sqrt(2), -1
    assert P.mean_cosine(a, b) == pytest.approx((1.0 + 2 ** -0.5 - 1.0) / 3.0, rel=1e-15)
