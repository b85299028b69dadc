"""Benchmark of the residual workload predictor + swap planner on one MI355X.

A step is one pass of the whole hot path over one batch, one fb_predict_plan_packed call: the fused
predictor kernel (router GEMM, scoring, top-k, histogram, rank fold, max/mean) whose last workgroup
then makes the swap plan of the counts.  The workload is the DeepSeek-V3-shaped prefill batch: T=32768 tokens, H=7168, E=256
routed experts, sigmoid scoring with a per-expert selection bias, group-limited top-8 (8 groups,
4 kept, group score = sum of the top-2), 32 ranks x 8 slots, swap cap 8.  Inputs are seeded
synthetic data resident in HBM before timing starts; hidden-state buffers rotate so every step reads
its 470 MB from HBM rather than the 256 MB last-level cache.

Prints one JSON line (see the fields below).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "predict_dsv3_counters.txt")
# the predictor kernel's sources: its own file and the headers compiled into it (the one-wave
# planner of its last workgroup among them)
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_14205_amd", "csrc", f)
                  for f in ("fb_predict.hip", "fb_plan_wave.h", "fb_internal.h")]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(wl) -> int:
    """Bytes the predictor must move once per launch: hidden states and router weight read, the
    per-expert bias and placement read, counts / rank loads / max-mean written."""
    elem = 2 if wl.dtype == "bf16" else 4
    return (wl.T * wl.H + wl.E * wl.H) * elem + wl.E * 4 * 3 + wl.R * 4 + 8


def traffic_from_profile():
    """HBM bytes per launch from the committed rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE
    scaled by a plain copy of known size), or None if it was taken on another kernel source."""
    try:
        with open(PROFILE_COUNTERS) as f:
            rec = dict(l.split(":", 1) for l in f if ":" in l and not l.startswith("#"))
    except OSError:
        return None
    if rec.get("kernel_source_sha256_16", "").strip() != kernel_source_hash():
        return None
    try:
        return int(rec["hbm_bytes_per_launch"].strip())
    except (KeyError, ValueError):
        return None


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, li, e2r, slots, target_s: float, gpu_topk, gpu_counts):
    """The CPU oracle, as it stands, on the same workload: whole batches repeated for about
    target_s seconds over the BLAS threads NumPy uses, plus one-thread passes of the Tiny and
    Mixtral-shaped configs.  Also checks the timed layer's GPU counts against the oracle's: the
    difference is exactly the histogram difference of the tokens whose selections differ, so
    ||n_gpu - n_oracle||_1 <= 2k * #differing, and at most 0.2% of the tokens may differ."""
    import oracle.planner as OPL
    import oracle.predictor as OPR
    from threadpoolctl import threadpool_info, threadpool_limits
    from workloads import CONFIGS, contiguous_placement, make_layer

    info = threadpool_info()
    blas = [{"api": i.get("internal_api"), "version": i.get("version"),
             "threads": int(i.get("num_threads", 1))} for i in info if i.get("user_api") == "blas"]
    cores = max([b["threads"] for b in blas] or [1])

    def run(w, l, e2r_, slots_, B):
        t0 = time.perf_counter()
        out = OPR.predict_load(l.x, l.w, w.dtype, w.k, w.kind, e2r_, w.R, select_bias=l.select_bias,
                               n_group=w.n_group, topk_group=w.topk_group, group_topn=w.group_topn)
        OPL.plan_swaps(out["counts"], slots_, B)
        return time.perf_counter() - t0, out

    reps, dt, ref = 0, 0.0, None
    while reps == 0 or dt < target_s:
        d, ref = run(wl, li, e2r, slots, wl.budget)
        dt += d
        reps += 1
    # the timed layer's GPU result against the oracle
    differ = int(np.count_nonzero(np.any(np.sort(gpu_topk, 1) != np.sort(ref["topk"], 1), axis=1)))
    l1 = int(np.abs(np.asarray(gpu_counts, np.int64) - ref["counts"]).sum())
    assert np.array_equal(np.bincount(gpu_topk.reshape(-1), minlength=wl.E)[:wl.E], gpu_counts), \
        "GPU counts are not the histogram of its selections"
    assert differ <= 0.002 * wl.T and l1 <= 2 * wl.k * differ, \
        f"GPU counts against the oracle: {differ} tokens differ, L1 {l1}"
    single = {}
    with threadpool_limits(limits=1):
        for name in ("tiny", "mixtral"):
            w = CONFIGS[name]
            sl, er = contiguous_placement(w.E, w.R, w.S)
            lw = make_layer(w, 0)
            n, t = 0, 0.0
            while n == 0 or t < 1.0:
                t += run(w, lw, er, sl, w.budget)[0]
                n += 1
            single[name] = {"tokens_per_s": n * w.T / t, "passes": n, "T": w.T, "H": w.H, "E": w.E}
    return {"value": reps * wl.T / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"the whole {wl.T}-token DeepSeek-V3-shaped batch (layer 0), {reps} passes: "
                      f"float64 router GEMM, scoring, group-limited top-8, histogram, rank fold and "
                      f"the frontier planner (B={wl.budget}); {dt:.1f} s",
            "cpu_model": _cpu_model(), "blas": blas,
            "single_thread": single,
            "gpu_vs_oracle": {"tokens_differing": differ, "counts_l1": l1}}


def attention_standin(torch, dev, seqs=4, seq_len=8192, heads=128, head_dim=128, group=16,
                      window=None):
    """An attention-shaped stand-in for one DeepSeek-V3-shaped prefill layer: for each of `seqs`
    sequences of seq_len tokens and each of `heads` heads of head_dim, S = Q K^T and O = S V as bf16
    batched GEMMs (groups of `group` heads per call).  With `window`, a sliding-window attention
    type: every block of `window` queries meets a band of 2 * window keys.  Returns (run(stream),
    flops); run enqueues one layer of it.  Every operand is a contiguous tensor of its own (K is
    stored transposed; the band tensors stand in for the per-block key and value slices)."""
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    n = seqs * heads
    rows = seq_len if window is None else window
    keys = seq_len if window is None else 2 * window
    blocks = 1 if window is None else seq_len // window
    q = torch.randn((n, rows, head_dim), generator=g, device=dev, dtype=torch.bfloat16)
    kt = torch.randn((n, head_dim, keys), generator=g, device=dev, dtype=torch.bfloat16)
    v = torch.randn((n, keys, head_dim), generator=g, device=dev, dtype=torch.bfloat16)
    sc = torch.empty((group, rows, keys), device=dev, dtype=torch.bfloat16)
    o = torch.empty((group, rows, head_dim), device=dev, dtype=torch.bfloat16)
    flops = 2 * 2.0 * n * blocks * rows * keys * head_dim

    def run(stream):
        with torch.cuda.stream(stream):
            for _ in range(blocks):
                for i in range(0, n, group):
                    torch.bmm(q[i:i + group], kt[i:i + group], out=sc)
                    torch.bmm(sc, v[i:i + group], out=o)
    return run, flops


def measure_overlap(fb, torch, wl, x, wp, scoring, budget, e2r_t, slots_t, sb, counts_for_plan):
    """The paper's overlap (Fig. 1, stages 1-2 under attention) and its budget (Eq. 10).

    * Budget per attention type: each attention stand-in of one DeepSeek-V3-shaped prefill layer
      (full attention, and sliding-window attention) is timed alone; B_l = max(0, T_attn - delta),
      delta = the prediction + planning time that the same window must also hold, and the
      time-budgeted device planner spends B_l.
    * Overlap: a one-sequence stand-in (short enough that its run-to-run noise stays below the early
      pass's own time) on the main stream with prediction + planning on a side stream, enqueued
      after the attention and before it; medians of alternating repetitions."""
    dev = x.device
    main = torch.cuda.current_stream(dev)
    side = torch.cuda.Stream(dev)
    pred = fb.Predictor(dev, stream=side)
    out, plan = pred.predict_plan(x, wp, scoring, e2r_t, slots_t, budget, select_bias=sb,
                                  stream=side)
    torch.cuda.synchronize()
    lat = []                          # the early pass's own latency in the last run_once
    timed_pass = {}                   # the time-budgeted early pass: its outputs and cost model

    def early_pass(timed=False):
        p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        p0.record(side)
        if timed:
            tp = timed_pass
            pred.predict_plan(x, wp, scoring, e2r_t, slots_t, tp["budget"], select_bias=sb,
                              out=tp["out"], plan=tp["plan"], cost=tp["cost"], stream=side)
        else:
            pred.predict_plan(x, wp, scoring, e2r_t, slots_t, budget, select_bias=sb, out=out,
                              plan=plan, stream=side)
        p1.record(side)
        lat[:] = [(p0, p1)]

    def run_once(attn, use_attn, use_pp, pp_first=False, timed=False):
        st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e_side = torch.cuda.Event()
        torch.cuda.synchronize()
        st.record(main)
        side.wait_event(st)
        if use_pp and pp_first:
            early_pass(timed)
        if use_attn:
            attn(main)
        if use_pp and not pp_first:
            early_pass(timed)
        e_side.record(side)
        main.wait_event(e_side)
        en.record(main)
        torch.cuda.synchronize()
        return st.elapsed_time(en)

    def alone(attn, reps=3):
        run_once(attn, True, False)
        return min(run_once(attn, True, False) for _ in range(reps))

    t_pp = min(run_once(None, False, True) for _ in range(5))
    nodes_t = torch.tensor([r // 8 for r in range(wl.R)], dtype=torch.int32, device=dev)
    sizes_t = torch.full((wl.E,), 3 * 7168 * 2048 * 2, dtype=torch.int64, device=dev)

    def spend(t_ms):
        B_ns = max(0, int((t_ms - t_pp) * 1e6))
        cm = fb.CostModel(nodes_t, sizes_t, (20_000, 50_000), (100_000, 25_000), B_ns)
        tplan = fb.plan_swaps_timed_device(counts_for_plan, slots_t, fb.Budget(64), cm).to_host()
        return {"B_l_ns": B_ns, "timed_plan_swaps": len(tplan.swaps),
                "timed_plan_cost_ns": sum(tplan.costs or [])}

    per_type = {}
    for name, kw in (("full", {}), ("sliding_window_2048", {"window": 2048})):
        attn, flops = attention_standin(torch, dev, **kw)
        t = alone(attn)
        per_type[name] = {"t_attn_ms": t, "tflops": flops / (t * 1e-3) / 1e12, **spend(t)}
        del attn
    # the overlap itself, on one sequence of the full stand-in: each repetition times the attention
    # alone and with the early pass enqueued after it and before it, in a rotating order, and keeps
    # the differences to the run alone, which cancels the slow drift of the clocks between
    # repetitions
    attn, _ = attention_standin(torch, dev, seqs=1)
    run_once(attn, True, True)
    reps = 15
    ta, d_after, d_first, l_after, l_first = [], [], [], [], []
    for i in range(reps):
        kinds = ["alone", "after", "first"]
        kinds = kinds[i % 3:] + kinds[:i % 3]
        t = {}
        for k in kinds:
            t[k] = run_once(attn, True, k != "alone", pp_first=(k == "first"))
            if k != "alone":
                (l_after if k == "after" else l_first).append(lat[0][0].elapsed_time(lat[0][1]))
        ta.append(t["alone"])
        d_after.append(t["after"] - t["alone"])
        d_first.append(t["first"] - t["alone"])
    med = lambda v: sorted(v)[len(v) // 2]
    quart = lambda v: [sorted(v)[len(v) // 4], sorted(v)[(3 * len(v)) // 4]]
    # the early pass under the time budget of that layer's own window (Eq. 10) in one call
    # (fb_predict_plan_timed_packed), enqueued before the attention: its latency beside it, and its
    # plan against the time-budgeted device planner's on the same counts
    B1 = max(0, int((med(ta) - t_pp) * 1e6))
    tb = fb.Budget(64)
    cm1 = fb.CostModel(nodes_t, sizes_t, (20_000, 50_000), (100_000, 25_000), B1)
    o1, p1_ = pred.predict_plan(x, wp, scoring, e2r_t, slots_t, tb, select_bias=sb, cost=cm1,
                                stream=side)
    timed_pass.update(budget=tb, cost=cm1, out=o1, plan=p1_)
    l_timed = []
    for _ in range(7):
        run_once(attn, True, True, pp_first=True, timed=True)
        l_timed.append(lat[0][0].elapsed_time(lat[0][1]))
    got = p1_.to_host()
    ref = fb.plan_swaps_timed_device(o1.counts, slots_t, tb, cm1).to_host()
    assert [tuple(v) for v in got.swaps] == [tuple(v) for v in ref.swaps] and got.costs == ref.costs, \
        "the one-call timed early pass disagrees with the time-budgeted device planner"
    full = per_type["full"]
    return {"attention_standin": "4 sequences x 8192 tokens x 128 heads x 128 dims: S = QK^T and "
                                 "O = SV as bf16 batched GEMMs (hipBLASLt via torch.bmm), main stream; "
                                 "sliding window: blocks of 2048 queries x bands of 4096 keys",
            "t_predict_plan_ms": t_pp,
            "per_attention_type": per_type,
            "B_l_rule": "max(0, T_attn - delta), delta = predict + plan time",
            "B_l_ns": full["B_l_ns"], "timed_plan_swaps": full["timed_plan_swaps"],
            "overlap_one_sequence": {
                "t_attn_ms": med(ta),
                "added_ms_pass_after": med(d_after), "added_ms_pass_after_quartiles": quart(d_after),
                "added_ms_pass_first": med(d_first), "added_ms_pass_first_quartiles": quart(d_first),
                "hidden_fraction_pass_after": 1.0 - med(d_after) / t_pp,
                "hidden_fraction_pass_first": 1.0 - med(d_first) / t_pp,
                "early_pass_latency_ms_pass_after": med(l_after),
                "early_pass_latency_ms_pass_first": med(l_first),
                "timed_early_pass": {"B_l_ns": B1, "swaps": len(got.swaps),
                                     "cost_ns": sum(got.costs or []),
                                     "latency_ms_pass_first": med(l_timed),
                                     "what": "fb_predict_plan_timed_packed with B_l = this "
                                             "attention's time minus t_predict_plan, 7 runs "
                                             "enqueued before it; plan = the time-budgeted "
                                             "device planner's"},
                "what": f"{reps} repetitions, each timing the attention alone and with the early pass "
                        "(fb_predict_plan_packed) enqueued after and before it (rotating order); "
                        "added = that repetition's difference to the attention alone, median and "
                        "quartiles; hidden fraction = 1 - added / t_predict_plan; early-pass "
                        "latency = its own start-to-end on the side stream beside the attention"}}

def measure_sequence(fb, torch, wl, x0, w, scoring, budget, e2r_t, slots_t, sb, layers, nbytes):
    """The early passes of `layers` distinct layers back to back on one stream, as a forward pass
    issues them (each layer: `fb_predict_plan_packed` on its own hidden states with its own packed
    router).  Layer l's hidden states are the batch's rows rotated by l * 997 and its router the
    weight's rows permuted by a seeded permutation: the same statistics, distinct bytes, so every
    layer reads its hidden states from HBM.  Reported against `layers` x the algorithmic bytes at
    the HBM peak."""
    dev = x0.device
    g = torch.Generator(device="cpu")
    g.manual_seed(7)
    xs = [torch.roll(x0, shifts=(l * 997) % max(wl.T, 1), dims=0).contiguous() for l in range(layers)]
    wps = [fb.pack_router_weight(w[torch.randperm(wl.E, generator=g).to(dev)].contiguous())
           for _ in range(layers)]
    pred = fb.Predictor(dev)
    outs, plans = [], []
    for l in range(layers):
        o, p = pred.predict_plan(xs[l], wps[l], scoring, e2r_t, slots_t, budget, select_bias=sb)
        outs.append(o)
        plans.append(p)
    torch.cuda.synchronize()
    for o in outs:
        assert int(o.counts.sum().item()) == wl.T * wl.k, "a layer failed the count invariant"

    def once():
        for l in range(layers):
            pred.predict_plan(xs[l], wps[l], scoring, e2r_t, slots_t, budget, select_bias=sb,
                              out=outs[l], plan=plans[l])

    for _ in range(3):
        once()
    torch.cuda.synchronize()
    times = []
    for _ in range(7):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        once()
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    ms = sorted(times)[len(times) // 2]
    roof_ms = layers * nbytes / (PEAK_HBM_GBS * 1e9) * 1e3
    return {"layers": layers, "ms": ms, "us_per_layer": ms / layers * 1e3,
            "roofline_ms": roof_ms, "frac": roof_ms / ms,
            "what": "median of 7 passes over the layers, each layer's fb_predict_plan_packed call "
                    "back to back on one stream; roofline = layers x algorithmic bytes at 8 TB/s"}


def _time_ms(torch, stream, fn, K):
    """Average duration of K back-to-back calls of fn, bracketed by events on the stream."""
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    fn(0)
    torch.cuda.synchronize()
    a.record(stream)
    for i in range(K):
        fn(i)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / K


def _smi_sample():
    """Socket power (amd-smi) and shader clock (rocm-smi) of GPU 0; read-only queries."""
    import subprocess
    out = {}
    try:
        r = subprocess.run(["amd-smi", "metric", "--power", "--json"], capture_output=True,
                           text=True, timeout=20)
        out["socket_power_w"] = json.loads(r.stdout)["gpu_data"][0]["power"]["socket_power"]["value"]
    except Exception:
        pass
    try:
        r = subprocess.run(["rocm-smi", "-c", "--json"], capture_output=True, text=True, timeout=20)
        card = next(iter(json.loads(r.stdout).values()))
        out["sclk_mhz"] = int(card["sclk clock speed:"].strip("()Mhz"))
    except Exception:
        pass
    return out


def measure_power(torch, xs, nbuf, run_pred, wt, stream, seconds):
    """Board power and shader clock while the predictor runs back to back on the benchmark's hidden
    states, on all-zero hidden states of the same shape, and while hipBLASLt runs the plain router
    GEMM on the benchmark's hidden states and the one-sequence attention stand-in of the overlap
    measurement: evidence for what bounds the kernel (the chip's power limit versus its own design)
    and for how much of the early pass attention can hide.  Each phase runs for `seconds`; sampling
    starts after one second."""
    import statistics
    import threading
    zeros = [torch.zeros_like(xs[0]) for _ in range(2)]
    attn, _ = attention_standin(torch, xs[0].device, seqs=1)
    phases = [("predictor", lambda i: run_pred(xs[i % nbuf])),
              ("predictor_all_zero_hidden", lambda i: run_pred(zeros[i % 2])),
              ("hipblaslt_router_gemm", lambda i: torch.matmul(xs[i % nbuf], wt)),
              ("attention_standin_one_sequence", lambda i: attn(stream))]
    res = {"idle": _smi_sample()}
    for name, fn in phases:
        stop = threading.Event()
        samples = []

        def poll():
            time.sleep(1.0)
            while not stop.is_set():
                samples.append(_smi_sample())

        th = threading.Thread(target=poll)
        th.start()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        n = n0 = 0
        started = False
        while time.perf_counter() - t0 < seconds:
            if not started and time.perf_counter() - t0 > 1.0:
                a.record(stream)
                n0, started = n, True
            for i in range(20):
                fn(n + i)
            n += 20
            torch.cuda.synchronize()
        b.record(stream)
        torch.cuda.synchronize()
        stop.set()
        th.join()
        pw = [x["socket_power_w"] for x in samples if "socket_power_w" in x]
        ck = [x["sclk_mhz"] for x in samples if "sclk_mhz" in x]
        res[name] = {"us_per_launch": a.elapsed_time(b) / max(1, n - n0) * 1e3,
                     "socket_power_w_median": statistics.median(pw) if pw else None,
                     "sclk_mhz_median": statistics.median(ck) if ck else None,
                     "samples": len(samples)}
    return res


def measure_extras(args, fb, torch, wl, xs, nbuf, wp, w, scoring, budget, e2r_t, slots_t, sb, pred,
                   out, stream):
    """The rest of the hot path's entry points on the same workload, each timed back to back:
    the step replayed from a HIP graph (one node, and predict -> plan as two), the
    prediction-quality diagnostics (row cosine of two hidden-state batches, top-k hits, rank fold),
    the time-budgeted planner and the fold and plan of a replicated placement."""
    K = max(10, args.steps // 4)
    res = {}
    # the step (fb_predict_plan_packed, one node) captured once per hidden-state buffer, replayed
    # in rotation; and predict -> plan as two nodes
    try:
        side = torch.cuda.Stream()
        plan_g = fb.plan_swaps_device(out.counts, slots_t, budget)
        graphs, graphs2 = [], []
        with torch.cuda.stream(side):
            for i in range(nbuf):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=side):
                    pred.predict_plan(xs[i], wp, scoring, e2r_t, slots_t, budget, select_bias=sb,
                                      out=out, plan=plan_g)
                graphs.append(g)
                g2 = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g2, stream=side):
                    pred.predict_load(xs[i], wp, scoring, e2r_t, wl.R, select_bias=sb, out=out)
                    fb.plan_swaps_device(out.counts, slots_t, budget, out=plan_g)
                graphs2.append(g2)
        torch.cuda.synchronize()
        res["graph_ms_per_step"] = _time_ms(torch, stream, lambda i: graphs[i % nbuf].replay(), K)
        res["graph_two_nodes_ms_per_step"] = _time_ms(torch, stream,
                                                      lambda i: graphs2[i % nbuf].replay(), K)
    except Exception as ex:  # graph capture is context, never a reason to lose the bench line
        res["graph_ms_per_step"] = None
        res["graph_error"] = str(ex)[:200]
    # mean row cosine of two T x H bf16 batches: reads both once (the hidden-state cosine of the
    # prediction-quality study), HBM-bound
    a_, b_ = xs[0], xs[1 % nbuf]
    cos_ms = _time_ms(torch, stream, lambda i: fb.row_cosine_mean(a_, b_), K)
    nbytes = 2 * a_.numel() * a_.element_size()
    res["row_cosine_mean"] = {"ms": cos_ms, "bytes": nbytes, "achieved_gbs": nbytes / cos_ms / 1e6,
                              "frac_of_hbm_peak": nbytes / cos_ms / 1e6 / PEAK_HBM_GBS}
    # top-k hits between two T x k selections, and the rank fold of a count vector
    dbg = pred.predict_load(xs[0], wp, scoring, e2r_t, wl.R, select_bias=sb, return_topk=True)
    dbg2 = pred.predict_load(xs[1 % nbuf], wp, scoring, e2r_t, wl.R, select_bias=sb, return_topk=True)
    res["topk_hits_ms"] = _time_ms(torch, stream, lambda i: fb.topk_hits(dbg.topk, dbg2.topk), K)
    res["fold_rank_loads_ms"] = _time_ms(torch, stream,
                                         lambda i: fb.fold_rank_loads(out.counts, e2r_t, wl.R), K)
    # time-budgeted planner: 32 ranks on 4 nodes of 8, 88 MB experts (three 7168 x 2048 bf16
    # matrices), 20 us / 100 GB/s inside a node, 50 us / 25 GB/s across, 8 ms per rank
    nodes_t = torch.tensor([r // 8 for r in range(wl.R)], dtype=torch.int32, device=out.counts.device)
    sizes_t = torch.full((wl.E,), 3 * 7168 * 2048 * 2, dtype=torch.int64, device=out.counts.device)
    cm = fb.CostModel(nodes_t, sizes_t, (20_000, 50_000), (100_000, 25_000), 8_000_000)
    for mode in ("frontier", "full"):
        bg_t = fb.Budget(64, mode=mode)
        tplan = fb.plan_swaps_timed_device(out.counts, slots_t, bg_t, cm)
        res[f"plan_timed_{mode}_ms"] = _time_ms(
            torch, stream, lambda i: fb.plan_swaps_timed_device(out.counts, slots_t, bg_t, cm, out=tplan), K)
        res[f"plan_timed_{mode}_swaps"] = len(tplan.to_host().swaps)
    # a placement that replicates popular experts (32 ranks x 9 slots: the 32 most popular experts
    # twice): the GPU fold and the device plan of the predicted counts
    from workloads import replicated_placement, truncated_zipf_probs
    rslots = torch.from_numpy(replicated_placement(truncated_zipf_probs(wl.zipf_s[0], wl.E), wl.R,
                                                   wl.S + 1)).to(out.counts.device)
    res["fold_slot_loads_ms"] = _time_ms(torch, stream, lambda i: fb.fold_slot_loads(out.counts, rslots), K)
    rplan = fb.plan_swaps_device(out.counts, rslots, budget)
    res["plan_replicated_ms"] = _time_ms(
        torch, stream, lambda i: fb.plan_swaps_device(out.counts, rslots, budget, out=rplan), K)
    res["plan_replicated_swaps"] = len(rplan.to_host().swaps)
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    # The chip needs roughly 20-40 ms of sustained load before its clocks settle (the first launches
    # take up to 1.5x the steady-state time), and the CPU leg leaves it idle for seconds: before the
    # warm-up steps, steps run for at least this long (not counted as warm-up or timed steps).
    ap.add_argument("--settle-ms", type=float, default=300.0)
    ap.add_argument("--streams", type=int, default=2,
                    help="independent batches in flight during the timed steps (1 = one stream)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    # instead of the bench line: board power and shader clock while the predictor runs on the
    # benchmark's hidden states and on all-zero ones, and while hipBLASLt runs the router GEMM
    ap.add_argument("--power", action="store_true")
    ap.add_argument("--power-seconds", type=float, default=5.0)
    # The bench line is the DeepSeek-V3-shaped batch.  The other input shapes can be timed the same
    # way for context (same step, roofline fields without counter traffic, no extras or CPU leg).
    ap.add_argument("--workload", default="deepseek-v3",
                    choices=["deepseek-v3", "mixtral", "qwen3", "sweep-4096", "sweep-16384",
                             "sweep-65536"])
    # the multi-layer workloads (48 Qwen3-shaped layers, 58 sweep layers): also time that many
    # distinct layers back to back, as a forward pass issues their early passes
    ap.add_argument("--layers", type=int, default=0)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the predictor shards over tokens with one 1 KB count "
              "all-reduce, which this single-GPU build does not run; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_14205_amd as fb
    from workloads import CONFIGS, contiguous_placement, make_layer, sweep_workload

    default = args.workload == "deepseek-v3"
    if args.workload.startswith("sweep-"):
        wl = sweep_workload(int(args.workload.split("-")[1]))
    else:
        wl = CONFIGS[{"deepseek-v3": "dsv3", "mixtral": "mixtral", "qwen3": "qwen3"}[args.workload]]
    slots, e2r = contiguous_placement(wl.E, wl.R, wl.S)
    li = make_layer(wl, 0)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    x0 = torch.from_numpy(li.x.view(np.int16)).to(dev).view(torch.bfloat16)
    w = torch.from_numpy(li.w.view(np.int16)).to(dev).view(torch.bfloat16)
    sb = torch.from_numpy(li.select_bias).to(dev) if li.select_bias is not None else None
    e2r_t = torch.from_numpy(e2r).to(dev)
    slots_t = torch.from_numpy(slots).to(dev)
    nbuf = max(2, math.ceil(768e6 / x0.numel() / 2))
    xs = [x0] + [x0.clone() for _ in range(nbuf - 1)]
    scoring = fb.Scoring(wl.kind, wl.k, wl.n_group, wl.topk_group, wl.group_topn)
    budget = fb.Budget(wl.budget)
    pred = fb.Predictor(dev)
    # the router weight is a fixed model parameter: packed once, as a server does at load time
    wp = fb.pack_router_weight(w)
    out = fb.Prediction(torch.empty(wl.E, dtype=torch.int32, device=dev),
                        torch.empty(wl.R, dtype=torch.int32, device=dev),
                        torch.empty(1, dtype=torch.float64, device=dev))
    plan = fb.plan_swaps_device(out.counts, slots_t, budget)   # allocates the plan buffers once

    def step(i, router):
        if isinstance(router, fb.PackedRouter):
            pred.predict_plan(xs[i % nbuf], router, scoring, e2r_t, slots_t, budget, select_bias=sb,
                              out=out, plan=plan)
        else:
            pred.predict_load(xs[i % nbuf], router, scoring, e2r_t, wl.R, select_bias=sb, out=out)
            fb.plan_swaps_device(out.counts, slots_t, budget, out=plan)

    if args.power:
        res = measure_power(torch, xs, nbuf,
                            lambda x: pred.predict_load(x, wp, scoring, e2r_t, wl.R, select_bias=sb,
                                                        out=out),
                            w.t(), stream, args.power_seconds)
        print(json.dumps({"power_probe": res, "workload": args.workload,
                          "what": "amd-smi socket power and rocm-smi shader clock, medians of the "
                                  "samples taken while each load ran back to back"}))
        return

    # The timed steps keep `streams` independent batches in flight: step i runs on stream
    # i mod streams with that stream's own workspace, outputs and plan, so one batch's planning and
    # tail overlap the next batch's prediction.  Every step still predicts and plans its own batch.
    lanes = []
    for j in range(args.streams):
        s_j = stream if args.streams == 1 else torch.cuda.Stream(dev)
        o_j = fb.Prediction(torch.empty(wl.E, dtype=torch.int32, device=dev),
                            torch.empty(wl.R, dtype=torch.int32, device=dev),
                            torch.empty(1, dtype=torch.float64, device=dev))
        lanes.append((s_j, fb.Predictor(dev, stream=s_j), o_j,
                      fb.plan_swaps_device(o_j.counts, slots_t, budget, stream=s_j)))

    def steps(first, n):
        if args.streams > 1:
            ev = torch.cuda.Event()
            ev.record(stream)
            for s_j, _, _, _ in lanes:
                s_j.wait_event(ev)
        for i in range(first, first + n):
            s_j, p_j, o_j, pl_j = lanes[i % args.streams]
            p_j.predict_plan(xs[i % nbuf], wp, scoring, e2r_t, slots_t, budget, select_bias=sb,
                             out=o_j, plan=pl_j, stream=s_j)
        if args.streams > 1:
            for s_j, _, _, _ in lanes:
                e = torch.cuda.Event()
                e.record(s_j)
                stream.wait_event(e)

    # the timed layer once with its selections, for the check against the oracle in the CPU leg
    dbg = pred.predict_load(x0, wp, scoring, e2r_t, wl.R, select_bias=sb, return_topk=True)
    torch.cuda.synchronize()
    gpu_topk, gpu_counts = dbg.topk.cpu().numpy(), dbg.counts.cpu().numpy().astype(np.int64)
    cpu = None
    if not args.no_cpu_baseline and default:
        cpu = cpu_baseline(wl, li, e2r, slots, args.cpu_seconds, gpu_topk, gpu_counts)
    extras = None
    if default:
        extras = measure_extras(args, fb, torch, wl, xs, nbuf, wp, w, scoring, budget, e2r_t,
                                slots_t, sb, pred, out, stream)
        extras["overlap"] = measure_overlap(fb, torch, wl, x0, wp, scoring, budget, e2r_t, slots_t,
                                            sb, dbg.counts)

    # clocks to their sustained state, then the warm-up steps
    t0 = time.perf_counter()
    n_settle = 0
    while (time.perf_counter() - t0) * 1e3 < args.settle_ms:
        steps(n_settle, 20)
        n_settle += 20
        torch.cuda.synchronize()
    steps(0, args.warmup)
    torch.cuda.synchronize()

    # the timed steps
    K = args.steps
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    steps(0, K)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    # every batch's result: the same counts and plan as the checked run
    for _, _, o_j, pl_j in lanes:
        assert np.array_equal(o_j.counts.cpu().numpy().astype(np.int64), gpu_counts), \
            "a timed step disagrees with the checked run"
        assert len(pl_j.to_host().swaps) <= wl.budget

    # the same K steps on one stream, one batch after the other (for reference)
    o_start = torch.cuda.Event(enable_timing=True)
    o_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    o_start.record(stream)
    for i in range(K):
        step(i, wp)
    o_end.record(stream)
    torch.cuda.synchronize()
    one_stream_ms = o_start.elapsed_time(o_end) / K

    # the predictor kernel alone: K launches back to back right after the timed steps, bracketed by
    # events on its stream (a marker between every launch would add several microseconds of its
    # own to each bracketed launch).  Three launches go first so that the start marker is reached
    # with the following launches already queued: the GPU never waits for the host in between.
    k_start = torch.cuda.Event(enable_timing=True)
    k_end = torch.cuda.Event(enable_timing=True)
    for i in range(3):
        pred.predict_load(xs[i % nbuf], wp, scoring, e2r_t, wl.R, select_bias=sb, out=out)
    k_start.record(stream)
    for i in range(K):
        pred.predict_load(xs[i % nbuf], wp, scoring, e2r_t, wl.R, select_bias=sb, out=out)
    k_end.record(stream)
    torch.cuda.synchronize()
    avg_kernel_s = k_start.elapsed_time(k_end) / K / 1e3

    # the device planner alone, K launches back to back on the final counts
    p_start = torch.cuda.Event(enable_timing=True)
    p_end = torch.cuda.Event(enable_timing=True)
    p_start.record(stream)
    for i in range(K):
        fb.plan_swaps_device(out.counts, slots_t, budget, out=plan)
    p_end.record(stream)
    torch.cuda.synchronize()
    plan_ms = p_start.elapsed_time(p_end) / K

    # context: the vendor library's plain router GEMM (hipBLASLt through torch.matmul, bf16 in and
    # out, no scoring or selection) on the same hidden buffers, timed the same way
    g_start = torch.cuda.Event(enable_timing=True)
    g_end = torch.cuda.Event(enable_timing=True)
    wt = w.t()
    for i in range(20):
        torch.matmul(xs[i % nbuf], wt)
    g_start.record(stream)
    for i in range(K):
        torch.matmul(xs[i % nbuf], wt)
    g_end.record(stream)
    torch.cuda.synchronize()
    gemm_ms = g_start.elapsed_time(g_end) / K

    counts = out.counts.cpu().numpy()
    host_plan = plan.to_host()

    # the same step with fb_predict_load, which repacks the router weight on every call
    u_start = torch.cuda.Event(enable_timing=True)
    u_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    u_start.record(stream)
    for i in range(K):
        step(i, w)
    u_end.record(stream)
    torch.cuda.synchronize()
    unpacked_ms = u_start.elapsed_time(u_end) / K
    split_mode = fb.predict_split_workspace_bytes(wl.T, wl.E, wl.H, torch.bfloat16, dev) > 2048
    rep_counts = out.counts.cpu().numpy()
    assert int(rep_counts.sum()) == wl.T * wl.k, "repacking path failed its invariant"
    if not split_mode:
        # the same kernel on the same bytes; in split mode the packed path adds partial sums in
        # another order, so near-tie tokens may legitimately differ
        assert np.array_equal(rep_counts, counts), "packed and repacking paths disagree"
    assert np.array_equal(counts.astype(np.int64), gpu_counts), "timed steps disagree with the checked run"
    assert int(counts.sum()) == wl.T * wl.k, "predictor output failed its invariant"
    assert len(host_plan.swaps) <= wl.budget

    nbytes = algorithmic_bytes(wl)
    flops = 2.0 * wl.T * wl.H * wl.E
    achieved = nbytes / avg_kernel_s / 1e9
    tflops = flops / avg_kernel_s / 1e12
    result = {
        "metric": "predicted tokens/sec (GEMM+top-k+histogram), % of HBM/MFMA roofline",
        "value": wl.T * K / (total_ms / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": total_ms / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}-shaped prefill", "T": wl.T, "H": wl.H, "E": wl.E,
                   "k": wl.k,
                   "scoring": (f"{wl.kind}" + ("+bias" if wl.select_bias else "") +
                               (f", {wl.n_group} groups keep {wl.topk_group} (top-{wl.group_topn} sum)"
                                if wl.n_group > 1 else "")),
                   "ranks": wl.R, "slots_per_rank": wl.S, "swap_budget": wl.budget,
                   "split_mode": split_mode,
                   "step": "fb_predict_plan_packed on one batch (the prediction, then the swap "
                           "plan in its last workgroup); "
                           f"{args.streams} batches in flight on {args.streams} streams",
                   "router_packing": "once, before timing (fb_pack_router_weight)"},
        "clock_settle": {"ms": args.settle_ms, "steps": n_settle},
        "streams": args.streams,
        "ms_per_step_one_stream": one_stream_ms,
        "ms_per_step_repacking_router": unpacked_ms,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS,
                     "traffic": traffic_from_profile() if default else None,
                     "bytes_per_launch": nbytes, "kernel_ms": avg_kernel_s * 1e3,
                     "kernel_ms_from": "HIP events around K back-to-back predictor launches right "
                                       "after the timed steps",
                     "mfma": {"achieved": tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                              "frac": tflops / PEAK_BF16_TFLOPS}},
        "context": {"hipblaslt_router_gemm_ms": gemm_ms,
                    "what": "torch.matmul(hidden, router_w.T), bf16 in and out, same buffers and "
                            "stream, K back-to-back launches: the plain GEMM alone, without scores, "
                            "selection or histogram; compare with roofline.kernel_ms"},
        "extras": extras,
        "plan": {"swaps": len(host_plan.swaps), "kernel_ms": plan_ms,
                 "max_mean_before": float(out.max_mean.item()),
                 "max_mean_after": float(host_plan.rank_loads.max() * wl.R / host_plan.rank_loads.sum())},
        "cpu_baseline": cpu,
    }
    if args.layers > 0:
        result["sequence"] = measure_sequence(fb, torch, wl, x0, w, scoring, budget, e2r_t, slots_t,
                                              sb, args.layers, nbytes)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
