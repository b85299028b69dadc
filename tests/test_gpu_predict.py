"""Parity of the HIP predictor (through the C ABI) with the CPU oracle, on MI355X.

Small cases span several workgroup tiles and a ragged tail; the full DeepSeek-V3-shaped workload
runs in the launch configuration the benchmark times (no debug outputs) and is checked through
properties that hold at any size plus oracle recomputation of sampled tokens.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import paper_2608_14205_amd as fb
from oracle import predictor as OP
from workloads import CONFIGS, contiguous_placement, make_layer
from gpu_util import (check_counts_consistent, check_prediction, run_gpu, scoring_of, to_device)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _case(name, T, **over):
    wl = dataclasses.replace(CONFIGS[name].with_T(T), **over)
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S) if wl.E % wl.R == 0 else (None, np.arange(wl.E) % wl.R)
    return wl, e2r


@pytest.mark.parametrize("name,T,dtype", [("tiny", 512, "f32"), ("tiny", 512, "bf16"), ("tiny", 77, "f32"),
                                          ("mixtral", 1000, "bf16"), ("qwen3", 1091, "bf16"),
                                          ("dsv3", 1100, "bf16")])
def test_config_parity(name, T, dtype):
    """Every config at an oracle-sized T (Tiny also in bf16): every token against the oracle, counts,
    rank loads and max/mean against the oracle's, and the device swap plan of the GPU's counts under
    the config's budget against the oracle's plan (and the host planner's)."""
    from oracle import planner as OPL
    _say(f"[parity] {name} T={T} {dtype}")
    wl, e2r = _case(name, T, dtype=dtype)
    slots, _ = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 1)
    gpu = run_gpu(li, wl, e2r)
    stats = check_prediction(gpu, li, wl, e2r, label=f"{name}/T={T}/{dtype}")
    check_counts_consistent(gpu, wl, e2r)
    ref = OP.predict_load(li.x, li.w, wl.dtype, wl.k, wl.kind, e2r, wl.R, select_bias=li.select_bias,
                          n_group=wl.n_group, topk_group=wl.topk_group, group_topn=wl.group_topn)
    # counts differ from the oracle's only through (exempt) tokens whose selection differs
    assert np.abs(gpu["counts"] - ref["counts"]).sum() <= 2 * wl.k * stats["mismatch"]
    if stats["mismatch"] == 0:
        assert np.array_equal(gpu["counts"], ref["counts"])
        assert np.array_equal(gpu["rank_loads"], ref["rank_loads"])
        assert gpu["max_mean"] == ref["max_mean"]
    counts_d = torch.from_numpy(gpu["counts"].astype(np.int32)).cuda()
    dev = fb.plan_swaps_device(counts_d, torch.from_numpy(slots).cuda(), fb.Budget(wl.budget)).to_host()
    host = fb.plan_swaps(gpu["counts"], slots, fb.Budget(wl.budget))
    oplan = OPL.plan_swaps(gpu["counts"], slots, wl.budget)
    for p in (dev, host):
        assert [tuple(x) for x in p.swaps] == [tuple(x) for x in oplan.swaps]
        assert np.array_equal(p.slots, oplan.slots)
    if name == "mixtral":
        assert not oplan.swaps        # one expert per rank: no swap lowers the maximum
    _say(f"[parity] {name} T={T} {dtype} ok {stats}; plan {len(oplan.swaps)} swaps")


@pytest.mark.parametrize("E,k,kind,groups", [
    (8, 1, "softmax", (1, 1, 1)), (8, 2, "softmax", (1, 1, 1)), (16, 2, "sigmoid", (1, 1, 1)),
    (24, 3, "softmax", (1, 1, 1)), (32, 6, "sigmoid", (4, 2, 2)), (64, 6, "softmax", (1, 1, 1)),
    (64, 6, "sigmoid", (8, 3, 2)), (96, 8, "sigmoid", (3, 2, 1)), (128, 8, "softmax", (1, 1, 1)),
    (160, 6, "sigmoid", (10, 3, 2)), (256, 8, "sigmoid", (8, 4, 2)), (256, 8, "sigmoid", (8, 4, 1)),
    (256, 8, "softmax", (1, 1, 1)), (256, 1, "sigmoid", (1, 1, 1)), (256, 32, "sigmoid", (4, 2, 2)),
])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_shape_sweep(E, k, kind, groups, dtype):
    n_group, topk_group, topn = groups
    _say(f"[sweep] E={E} k={k} {kind} groups={groups} {dtype}")
    R = 8 if E % 8 == 0 else 4
    wl = dataclasses.replace(CONFIGS["dsv3"], name=f"sweep-E{E}", cfg_id=9, T=300, H=320, E=E, k=k,
                             dtype=dtype, kind=kind, n_group=n_group, topk_group=topk_group,
                             group_topn=topn, select_bias=(kind == "sigmoid"), R=R,
                             S=max(1, E // R), n_clusters=E)
    e2r = np.arange(E, dtype=np.int32) % R
    li = make_layer(wl, 0)
    gpu = run_gpu(li, wl, e2r)
    check_prediction(gpu, li, wl, e2r, label=f"E={E},k={k},{kind},{groups},{dtype}")
    check_counts_consistent(gpu, wl, e2r)


def _random_shape(g, i):
    E = int(g.choice([8, 16, 24, 32, 40, 64, 96, 128, 160, 192, 256]))
    kind = "sigmoid" if g.random() < 0.5 else "softmax"
    # group sizes the kernel takes: powers of two (whole 16-expert lane blocks, or within a lane)
    n_group = int(g.choice([d for d in (1, 2, 4, 8) if E % d == 0 and
                            (d == 1 or (E // d) & (E // d - 1) == 0)]))
    gsz = E // n_group
    topk_group = int(g.integers(1, n_group + 1))
    topn = int(g.integers(1, min(2, gsz) + 1))
    if kind == "softmax":
        topn = 1            # softmax groups are scored by their maximum only
    k = int(g.integers(1, min(32, topk_group * gsz) + 1))
    dtype = "f32" if g.random() < 0.25 else "bf16"
    H = int(g.integers(1, 129)) * (16 if dtype == "f32" else 32)
    T = int(g.integers(1, 2500))
    R = int(g.choice([d for d in (1, 2, 4, 8) if E % d == 0]))
    return dataclasses.replace(CONFIGS["dsv3"], name=f"rand{i}", cfg_id=100 + i, T=T, H=H, E=E, k=k,
                               dtype=dtype, kind=kind, n_group=n_group, topk_group=topk_group,
                               group_topn=topn, select_bias=(kind == "sigmoid"), R=R,
                               S=max(1, E // R), n_clusters=E)


def test_random_shapes():
    """Seeded random shapes (E, k, scoring, groups, dtype, H, T, ranks), fused and split launches,
    each against the oracle on every token."""
    g = np.random.default_rng(2608)
    pred = fb.Predictor()
    for i in range(40):
        wl = _random_shape(g, i)
        packed = bool(i % 2)
        _say(f"[random {i}] T={wl.T} H={wl.H} E={wl.E} k={wl.k} {wl.kind} groups=({wl.n_group},"
             f"{wl.topk_group},{wl.group_topn}) {wl.dtype} R={wl.R} packed={packed}")
        e2r = (np.arange(wl.E) * wl.R // wl.E).astype(np.int32)
        li = make_layer(wl, 0)
        gpu = run_gpu(li, wl, e2r, predictor=pred, packed=packed)
        check_prediction(gpu, li, wl, e2r, label=wl.name)
        check_counts_consistent(gpu, wl, e2r)


@pytest.mark.parametrize("T", [0, 1, 63, 64, 65, 127, 128, 129, 255, 257])
def test_token_edges(T):
    _say(f"[edges] T={T}")
    for name in ("dsv3", "qwen3", "tiny"):
        wl, e2r = _case(name, T, H=256 if name != "tiny" else 128)
        li = make_layer(wl, 2)
        gpu = run_gpu(li, wl, e2r)
        if T == 0:
            assert gpu["counts"].sum() == 0 and gpu["rank_loads"].sum() == 0 and gpu["max_mean"] == 1.0
            continue
        check_prediction(gpu, li, wl, e2r, label=f"{name}/T={T}")
        check_counts_consistent(gpu, wl, e2r)


@pytest.mark.parametrize("H", [32, 96, 160, 7168 + 32])
def test_hidden_size_tails(H):
    # H % 64 == 32 exercises the half-width last pipeline stage
    _say(f"[H] H={H}")
    wl, e2r = _case("dsv3", 200, H=H)
    li = make_layer(wl, 0)
    gpu = run_gpu(li, wl, e2r)
    check_prediction(gpu, li, wl, e2r, label=f"H={H}")
    check_counts_consistent(gpu, wl, e2r)


def test_strided_hidden_and_router_bias():
    _say("[ld] strided rows + router bias")
    wl, e2r = _case("qwen3", 333, H=512)
    li = make_layer(wl, 0)
    pad = np.zeros((wl.T, wl.H + 64), np.uint16)
    pad[:, :wl.H] = li.x
    lb = (np.random.default_rng(1).standard_normal(wl.E) * 0.5).astype(np.float32)
    x_dev = to_device(pad, "bf16")[:, :wl.H]
    assert x_dev.stride(0) == wl.H + 64
    out = fb.Predictor().predict_load(x_dev, to_device(li.w, "bf16"), scoring_of(wl),
                                      torch.from_numpy(e2r.astype(np.int32)).cuda(), wl.R,
                                      logit_bias=torch.from_numpy(lb).cuda(), return_topk=True,
                                      return_logits=True)
    torch.cuda.synchronize()
    gpu = {"counts": out.counts.cpu().numpy().astype(np.int64), "rank_loads": out.rank_loads.cpu().numpy(),
           "max_mean": float(out.max_mean.item()), "topk": out.topk.cpu().numpy(),
           "logits": out.logits.cpu().numpy()}
    check_prediction(gpu, li, wl, e2r, logit_bias=lb, label="strided+bias")
    check_counts_consistent(gpu, wl, e2r)


def test_deterministic_and_debug_independent():
    _say("[det] repeated runs")
    wl, e2r = _case("dsv3", 2000)
    li = make_layer(wl, 3)
    pred = fb.Predictor()
    runs = [run_gpu(li, wl, e2r, debug=(i % 2 == 0), predictor=pred) for i in range(4)]
    for r in runs[1:]:
        assert np.array_equal(r["counts"], runs[0]["counts"])
        assert np.array_equal(r["rank_loads"], runs[0]["rank_loads"])
        assert r["max_mean"] == runs[0]["max_mean"]
    assert np.array_equal(runs[0]["topk"], runs[2]["topk"])
    assert np.array_equal(runs[0]["logits"].view(np.uint32), runs[2]["logits"].view(np.uint32))


def test_prediction_equals_actual_when_inputs_coincide():
    _say("[sigma0] predicted == actual")
    wl, e2r = _case("dsv3", 700, sigma=0.0)
    li = make_layer(wl, 0, with_target=True)
    assert np.array_equal(li.x, li.h_target)
    a = run_gpu(li, wl, e2r)
    li.x = li.h_target
    b = run_gpu(li, wl, e2r)
    assert np.array_equal(a["topk"], b["topk"]) and np.array_equal(a["counts"], b["counts"])


def _zero_hidden(wl, layer=0, select_bias=None):
    """The layer's router weight with hidden states that are exactly zero, so every logit is zero."""
    li = make_layer(wl, layer)
    x = np.zeros_like(li.x)
    return dataclasses.replace(li, x=x, select_bias=select_bias)


@pytest.mark.parametrize("E,k,dtype,packed", [(128, 8, "bf16", False), (128, 8, "bf16", True),
                                              (16, 2, "f32", False), (16, 16, "bf16", True),
                                              (256, 1, "bf16", True), (8, 8, "bf16", True),
                                              (256, 32, "f32", False)])
def test_all_tied_logits_take_the_lowest_indices(E, k, dtype, packed):
    """Zero hidden states make every logit exactly zero: every expert ties with every other, so each
    token takes experts 0 .. k-1 (ties go to the lower index, Sec. "Residual Workload Prediction",
    the model's top-k rule) and the counts are T for those experts and zero elsewhere.  Checked
    exactly on every token of a batch that spans several tiles and a ragged tail, in fused and
    split launches; no near-tie exemption applies."""
    T = 300
    wl = dataclasses.replace(CONFIGS["tiny"].with_T(T), H=256, E=E, k=k, dtype=dtype, R=8,
                             S=max(1, E // 8), n_clusters=E)
    e2r = (np.arange(E) * 8 // E).astype(np.int32)
    li = _zero_hidden(wl)
    gpu = run_gpu(li, wl, e2r, packed=packed)
    _say(f"[ties] E={E} k={k} {dtype} packed={packed}")
    assert not gpu["logits"].any()
    assert np.array_equal(np.sort(gpu["topk"], axis=1), np.tile(np.arange(k), (T, 1)))
    want = np.where(np.arange(E) < k, T, 0)
    assert np.array_equal(gpu["counts"], want)
    assert np.array_equal(gpu["rank_loads"], np.bincount(e2r, weights=want, minlength=8).astype(np.int64))
    check_counts_consistent(gpu, wl, e2r)


def _tied_group_bias():
    """A selection bias of multiples of 1/1024 (the sigmoid scores 0.5 + b are exact in float32 and
    float64) for 8 groups of 32 experts, built so that the group rule meets exact ties: the best two
    scores of groups 3, 4 and 6 sum to the same value at the fourth place (group 3, the lowest index,
    is kept), and the eighth and ninth experts of the kept groups tie (the lower index is taken).
    Returns the bias and the eight experts the rule selects."""
    g = np.random.default_rng(77)
    j = np.zeros(256, np.int64)
    tops = {0: (60, 40, 30), 1: (50, 40), 2: (45, 35), 3: (40, 30), 4: (35, 35), 5: (31, 29),
            6: (60, 10), 7: (25, 25)}
    chosen = []
    for grp, vals in tops.items():
        pos = g.permutation(32)
        rest = g.integers(-100, 10, size=32)       # below every group's second best: no effect
        j[32 * grp: 32 * grp + 32] = rest
        for v, p in zip(vals, pos):
            j[32 * grp + p] = v
        if grp <= 3:
            chosen += [(v, 32 * grp + p) for v, p in zip(vals, pos)]
    # kept groups 0-3 (sums 100, 90, 80, 70; groups 4 and 6 also sum to 70); the eight best by
    # (score desc, index asc): 60, 50, 45, the three 40s, 35, then group 0's 30 before group 3's
    chosen.sort(key=lambda t: (-t[0], t[1]))
    want = sorted(int(e) for _, e in chosen[:8])
    return (j / 1024.0).astype(np.float32), want


@pytest.mark.parametrize("packed", [False, True])
def test_tied_groups_and_experts_follow_the_lower_index(packed):
    """Zero hidden states under the DeepSeek-V3 rule (sigmoid plus selection bias, 8 groups, the 4
    with the largest sum of their best two scores kept, top-8) with the bias above: exact ties
    between group scores and at the k-th expert.  Every token must select exactly the experts the
    rule gives (worked out by hand and by the oracle)."""
    T = 333
    wl = dataclasses.replace(CONFIGS["dsv3"].with_T(T), H=256)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    sb, want = _tied_group_bias()
    oracle_topk = OP.select(np.zeros((1, wl.E), np.float32), wl.k, wl.kind, sb, wl.n_group,
                            wl.topk_group, wl.group_topn)[0]
    assert sorted(oracle_topk[0].tolist()) == want
    li = _zero_hidden(wl, select_bias=sb)
    gpu = run_gpu(li, wl, e2r, packed=packed)
    _say(f"[ties] DS-V3 rule, tied groups, packed={packed}: {want}")
    assert np.array_equal(np.sort(gpu["topk"], axis=1), np.tile(want, (T, 1)))
    counts = np.zeros(wl.E, np.int64)
    counts[want] = T
    assert np.array_equal(gpu["counts"], counts)
    check_counts_consistent(gpu, wl, e2r)


@pytest.mark.parametrize("E,n_group,topk_group,kind,topn", [(64, 8, 2, "sigmoid", 2),
                                                           (128, 4, 1, "softmax", 1),
                                                           (32, 4, 4, "sigmoid", 1)])
def test_k_fills_the_kept_groups(E, n_group, topk_group, kind, topn):
    """k = topk_group x group size: each token selects every expert of its kept groups, so its
    selection is a union of whole groups (with every group kept, all E experts and counts of T)."""
    gsz = E // n_group
    k = topk_group * gsz
    T = 400
    wl = dataclasses.replace(CONFIGS["dsv3"].with_T(T), H=320, E=E, k=k, kind=kind,
                             n_group=n_group, topk_group=topk_group, group_topn=topn,
                             select_bias=(kind == "sigmoid"), R=8, S=E // 8, n_clusters=E)
    e2r = (np.arange(E) % 8).astype(np.int32)
    li = make_layer(wl, 1)
    gpu = run_gpu(li, wl, e2r)
    _say(f"[ties] k={k} fills {topk_group} of {n_group} groups, E={E} {kind}")
    check_prediction(gpu, li, wl, e2r, label=f"k fills groups E={E}")
    check_counts_consistent(gpu, wl, e2r)
    sel = np.sort(gpu["topk"], axis=1)
    groups = sel // gsz
    for t in range(T):
        kept = np.unique(groups[t])
        assert kept.size == topk_group
        assert np.array_equal(sel[t], np.concatenate([np.arange(gg * gsz, gg * gsz + gsz) for gg in kept]))
    if topk_group == n_group:
        assert np.array_equal(gpu["counts"], np.full(E, T))


def test_bad_rank_table_is_reported():
    _say("[e2r] out-of-range rank id")
    wl, e2r = _case("qwen3", 100, H=128)
    bad = e2r.copy()
    bad[5] = wl.R + 3
    li = make_layer(wl, 0)
    gpu = run_gpu(li, wl, bad, debug=False)
    assert gpu["max_mean"] == -1.0
    good = run_gpu(li, wl, e2r, debug=False)
    assert np.array_equal(gpu["counts"], good["counts"])


def test_workspace_is_left_clean_across_shapes():
    _say("[ws] workspace reuse across shapes")
    pred = fb.Predictor()
    for name, T in (("dsv3", 500), ("tiny", 33), ("qwen3", 900), ("mixtral", 1), ("dsv3", 129)):
        wl, e2r = _case(name, T, H=256 if name != "tiny" else 64)
        li = make_layer(wl, 0)
        a = run_gpu(li, wl, e2r, predictor=pred)
        check_counts_consistent(a, wl, e2r)
    ws = pred.workspace[:2048].cpu().numpy()    # accumulators + ticket; the rest holds the packed weight
    assert not ws.any()


@pytest.mark.parametrize("layer", [0, 1])
def test_full_size_dsv3(layer):
    """The benchmarked configuration: T=32768, H=7168, E=256, sigmoid + bias, 8 groups keep 4.  The
    bench launch (packed router, no debug outputs) and a debug run give the same counts; every token
    is compared with the oracle, and the counts with the oracle's histogram."""
    wl = CONFIGS["dsv3"]
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    _say(f"[full] dsv3 layer {layer}: generating inputs")
    li = make_layer(wl, layer)
    _say("[full] bench-configuration run (packed router, no debug outputs)")
    plain = run_gpu(li, wl, e2r, debug=False, packed=True)
    dbg = run_gpu(li, wl, e2r, debug=True)
    assert np.array_equal(plain["counts"], dbg["counts"])
    assert np.array_equal(plain["rank_loads"], dbg["rank_loads"]) and plain["max_mean"] == dbg["max_mean"]
    check_counts_consistent(dbg, wl, e2r)
    assert plain["counts"].sum() == wl.T * wl.k
    _say(f"[full] oracle on all {wl.T} tokens")
    stats = check_prediction(dbg, li, wl, e2r, label=f"dsv3-full/l{layer}")
    _say(f"[full] ok {stats}")


def _pack_reference(w_bytes: np.ndarray, E: int, row_bytes: int) -> np.ndarray:
    """The packed layout of fb_pack_router_weight, written from its description in the header."""
    epad = next(p for p in (32, 64, 128, 256) if E <= p)
    W = 4 if epad >= 128 else (2 if epad == 64 else 1)
    F = epad // (32 * W)
    nst = -(-row_bytes // 256)
    src = np.zeros((epad, nst * 256), np.uint8)
    src[:E, :row_bytes] = w_bytes.reshape(E, row_bytes)
    out = np.zeros((nst, epad // 4, 64, 16), np.uint8)
    for st in range(nst):
        for c in range(epad // 4):
            f, q, w = c % F, (c // F) % 8, c // (8 * F)
            for l in range(64):
                row = w * (epad // W) + f * 32 + (l % 32)
                b = st * 256 + q * 32 + (l // 32) * 16
                out[st, c, l] = src[row, b:b + 16]
    return out.reshape(-1)


@pytest.mark.parametrize("E,H,dtype", [(8, 4096, "bf16"), (20, 96, "f32"), (60, 2048, "bf16"),
                                       (128, 2080, "bf16"), (256, 7168, "bf16"), (256, 160, "f32")])
def test_pack_layout_and_packed_predict(E, H, dtype):
    """fb_pack_router_weight writes exactly the documented layout (byte-exact), and
    fb_predict_load_packed returns bit-identical results to fb_predict_load."""
    _say(f"[pack] E={E} H={H} {dtype}")
    base = CONFIGS["dsv3" if E == 256 else "qwen3"]
    wl = dataclasses.replace(base.with_T(300), H=H, E=E, dtype=dtype, n_clusters=E,
                             k=min(base.k, max(1, E // 4)))
    e2r = np.arange(E, dtype=np.int32) % wl.R
    li = make_layer(wl, 0)
    w = to_device(li.w, dtype)
    pk = fb.pack_router_weight(w)
    torch.cuda.synchronize()
    got = pk.data.cpu().numpy()
    ref = _pack_reference(np.ascontiguousarray(li.w).view(np.uint8), E, H * (2 if dtype == "bf16" else 4))
    assert got.size == ref.size and np.array_equal(got, ref)
    a = run_gpu(li, wl, e2r, packed=False)
    b = run_gpu(li, wl, e2r, packed=True, predictor=fb.Predictor(split=False))
    for key in ("counts", "rank_loads", "topk"):
        assert np.array_equal(a[key], b[key]), key
    assert a["max_mean"] == b["max_mean"]
    assert np.array_equal(a["logits"].view(np.uint32), b["logits"].view(np.uint32))


@pytest.mark.parametrize("name,T", [("tiny", 77), ("tiny", 512), ("mixtral", 1000), ("qwen3", 1091),
                                    ("dsv3", 300), ("dsv3", 1100)])
def test_split_mode_parity(name, T):
    """Packed batches too small to occupy the GPU run in split mode (partial logits of stage ranges
    on several workgroups, added in split order by the tile's last split to arrive): oracle parity,
    repeats that are bit-identical, the workspace header (accumulators, ticket and the per-tile
    arrival counters) left at zero, and the fused path's selections where both match the oracle on
    every token."""
    wl, e2r = _case(name, T)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    need = fb.predict_split_workspace_bytes(T, wl.E, wl.H, dt)
    _say(f"[split] {name} T={T} workspace {need}")
    assert need > 2048, "this batch is expected to run in split mode"
    li = make_layer(wl, 1)
    pred = fb.Predictor()
    a = run_gpu(li, wl, e2r, predictor=pred, packed=True)
    assert pred.workspace.numel() >= need
    stats = check_prediction(a, li, wl, e2r, label=f"split {name}/T={T}")
    check_counts_consistent(a, wl, e2r)
    b = run_gpu(li, wl, e2r, predictor=pred, packed=True)
    for key in ("counts", "rank_loads", "topk"):
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(a["logits"].view(np.uint32), b["logits"].view(np.uint32))
    assert not pred.workspace[:2048].cpu().numpy().any()
    fused = run_gpu(li, wl, e2r, predictor=fb.Predictor(split=False), packed=True)
    fstats = check_prediction(fused, li, wl, e2r, label=f"fused {name}/T={T}")
    if stats["mismatch"] == 0 and fstats["mismatch"] == 0:
        assert np.array_equal(a["counts"], fused["counts"])
        assert np.array_equal(np.sort(a["topk"], 1), np.sort(fused["topk"], 1))
    _say(f"[split] {name} T={T} ok {stats}")


def test_qwen3_layers_back_to_back():
    """Qwen3-MoE-shaped layers (every token against the oracle) and the device plan of each layer's
    counts under the config's budget against the oracle's plan.  All 48 layers run in bench.py's
    report mode."""
    from oracle import planner as OPL
    wl = CONFIGS["qwen3"]
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    pred = fb.Predictor()
    slots_d = torch.from_numpy(slots).cuda()
    for layer in (0, 23, 47):
        _say(f"[qwen3] layer {layer}")
        li = make_layer(wl, layer)
        gpu = run_gpu(li, wl, e2r, predictor=pred)
        check_counts_consistent(gpu, wl, e2r)
        check_prediction(gpu, li, wl, e2r, label=f"qwen3/l{layer}")
        dev = fb.plan_swaps_device(torch.from_numpy(gpu["counts"].astype(np.int32)).cuda(), slots_d,
                                   fb.Budget(wl.budget, layer_id=layer)).to_host()
        ref = OPL.plan_swaps(gpu["counts"], slots, wl.budget, layer_id=layer)
        assert [tuple(x) for x in dev.swaps] == [tuple(x) for x in ref.swaps]
        assert np.array_equal(dev.slots, ref.slots)


def test_mixtral_full_size():
    wl = CONFIGS["mixtral"]
    _, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    _say("[mixtral] full size")
    li = make_layer(wl, 0)
    gpu = run_gpu(li, wl, e2r)
    check_counts_consistent(gpu, wl, e2r)
    stats = check_prediction(gpu, li, wl, e2r, label="mixtral-full")
    _say(f"[mixtral] ok {stats}")


@pytest.mark.parametrize("T,layers", [(4096, (0, 29, 57)), (16384, (0, 57)), (65536, (0,))])
def test_sweep_config(T, layers):
    """Multi-task skew sweep: DeepSeek-V3 shapes, 4-task mixture, per-layer routers.  Predicted and
    actual passes (H_l = h_{l-1} + residual) on the GPU, oracle parity on sampled tokens, and the
    plans for every budget of the sweep: device = host = oracle on the predicted counts.  Every
    token is compared with the oracle.  All 58 layers at each T run in bench.py's report mode."""
    from oracle import planner as OPL
    from workloads import sweep_workload
    wl = sweep_workload(T)
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    pred = fb.Predictor()
    for layer in layers:
        _say(f"[sweep] T={T} layer {layer}: generating inputs")
        li = make_layer(wl, layer, with_target=True)
        got = run_gpu(li, wl, e2r, predictor=pred, packed=True)
        check_counts_consistent(got, wl, e2r)
        stats = check_prediction(got, li, wl, e2r, label=f"sweep T={T} l{layer}")
        act_li = dataclasses.replace(li, x=li.h_target)
        act = run_gpu(act_li, wl, e2r, predictor=pred, debug=False, packed=True)
        assert act["counts"].sum() == T * wl.k
        counts_d = torch.from_numpy(got["counts"].astype(np.int32)).cuda()
        slots_d = torch.from_numpy(slots).cuda()
        for B in wl.budgets:
            bg = fb.Budget(B, layer_id=layer)
            dev = fb.plan_swaps_device(counts_d, slots_d, bg).to_host()
            host = fb.plan_swaps(got["counts"], slots, bg)
            ref = OPL.plan_swaps(got["counts"], slots, B, layer_id=layer)
            for p in (dev, ref):
                assert [tuple(s) for s in p.swaps] == [tuple(s) for s in host.swaps]
                assert np.array_equal(p.slots, host.slots)
            assert len(host.swaps) <= B
            assert host.rank_loads.max() <= got["rank_loads"].max()
            # realised balance of the actual pass under the planned placement (diagnostic)
            act_after = OP.max_to_mean(OP.rank_loads(act["counts"], host.expert_to_rank, wl.R))
            _say(f"[sweep] T={T} l{layer} B={B}: predicted max/mean {got['max_mean']:.3f} -> "
                 f"{host.rank_loads.max() * wl.R / host.rank_loads.sum():.3f}; actual {act['max_mean']:.3f} "
                 f"-> {act_after:.3f}")
        _say(f"[sweep] T={T} l{layer} ok {stats}")
