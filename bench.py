#!/usr/bin/env python3
"""Benchmark of one SPD pipeline step on one MI355X.

Workload (default): the 4B-class dense decoder (36 layers, d 2560, 32/8 heads of 128, FFN 9728,
vocab 151936, bf16 weights and KV), SPD width n = 4 (9 layers per stage), 1-layer PDM, a 2048-token
uniform-random prompt, synthetic N(0, 0.02) weights. A step is one spd_step: the PDM on its stream,
every stage's 9 layers, the exit LM head and verification.

Timed region: K back-to-back steps with drafts forced to the target's own greedy tokens (every step
accepts, so every step is a full-pipeline step), bracketed by device synchronisation. Reported:
us per step, algorithmic HBM bytes per step and GB/s against 8 TB/s, the dominant kernel's
roofline (HIP events around each launch of it when it runs alone), tokens/s at a Bernoulli(0.7)
acceptance pattern next to plain greedy decoding on the same GPU, the CPU oracle's time per step on
the host cores, and the 9B-class workloads (n = 4 at 4096 tokens; n = 8 with a two-layer PDM at 32768
tokens) with their step time, bandwidth and PDM hiding.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "µs per SPD pipeline step & achieved HBM GB/s (% roofline), 1 MI355X"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def prefill_with_progress(eng, prompt, label, every=20.0):
    """eng.spd_prefill(prompt) on a worker thread (the C call releases the interpreter lock), with a
    progress line every `every` seconds while it runs: a long prompt takes over a minute."""
    import threading
    out = {}

    def work():
        try:
            out["first"] = eng.spd_prefill(prompt)
        except BaseException as e:  # re-raised on the calling thread
            out["error"] = e

    t0 = time.time()
    th = threading.Thread(target=work, daemon=True)
    th.start()
    while True:
        th.join(every)
        if not th.is_alive():
            break
        log(f"[bench] {label}: prefill of {len(prompt)} tokens running, {time.time() - t0:.0f}s")
    if "error" in out:
        raise out["error"]
    return out["first"]


def pdm_kv_bytes(sh, ls, c, a, esz):
    """The draft module's keys and values in a step with c committed positions and a in-flight rows:
    its rows at positions c..c+a-1 attend over one shared cache, so each PDM layer's keys and values
    0..c+a-1 are read once, and the a rows are written."""
    kv_tok = 2 * sh.kv_dim * esz
    return ls * ((c + a) * kv_tok + a * kv_tok)


def step_bytes(sh, n, ls, c, esz, pdm_head=True):
    """Algorithmic HBM bytes of one full-pipeline step that starts with c committed positions:
    (target, PDM). pdm_head: the PDM streams its own pass over the LM head."""
    d, V, L = sh.d_model, sh.vocab, sh.n_layers
    kv_tok = 2 * sh.kv_dim * esz
    beta = [s * L // n for s in range(n + 1)]
    kv_read = 0
    for s in range(n):
        pos = c + n - 1 - s  # token of stage s attends to pos+1 keys of its own layers
        kv_read += (beta[s + 1] - beta[s]) * (pos + 1) * kv_tok
    target = L * layer_bytes(sh, esz) + kv_read + L * kv_tok + V * d * esz + d * esz
    pdm = d * n * d * esz + ls * layer_bytes(sh, esz) + pdm_kv_bytes(sh, ls, c, n, esz) + \
        (V * d * esz if pdm_head else 0)
    return target, pdm


def step_bytes_active(sh, n, ls, c, a, esz):
    """Algorithmic HBM bytes of a step (fused head) that starts with c committed positions and a
    in-flight tokens: stages 0..a-1 run (the token at depth s runs stage s), the two-row head pass
    runs every step, the PDM rewrites the a rows."""
    d, V, L = sh.d_model, sh.vocab, sh.n_layers
    kv_tok = 2 * sh.kv_dim * esz
    layer_w = layer_bytes(sh, esz)
    beta = [s * L // n for s in range(n + 1)]
    target = V * d * esz
    for s in range(a):
        pos = c + a - 1 - s
        nl = beta[s + 1] - beta[s]
        target += nl * (layer_w + (pos + 1) * kv_tok + kv_tok)
    return target + d * n * d * esz + ls * layer_w + pdm_kv_bytes(sh, ls, c, a, esz)


def layer_bytes(sh, esz):
    d, F, qd, kvd = sh.d_model, sh.ffn_dim, sh.q_dim, sh.kv_dim
    return (qd * d + 2 * kvd * d + d * qd + 3 * F * d) * esz + 2 * d * 4


def launch_bytes(sh, n, c, esz):
    """Algorithmic bytes of one steady-state launch of each stage-batched kernel class (all n stages
    active), starting the step with c committed positions: weights once, activations in and out."""
    d, F, qd, kvd, V = sh.d_model, sh.ffn_dim, sh.q_dim, sh.kv_dim, sh.vocab
    L = sh.n_layers
    beta = [s * L // n for s in range(n + 1)]
    # attention of slot 0 (every stage has a layer in slot 0): stage s reads c + n - s keys
    attn = sum((c + n - s) * 2 * kvd * esz + qd * 4 * 2 for s in range(n))
    return {
        "qkv": n * ((qd + 2 * kvd) * d * esz + 2 * d * 4 + qd * 4 + 2 * kvd * esz),
        "attn": attn,
        "oproj": n * (d * qd * esz + qd * 4 + 2 * d * 4),
        "gateup": n * (2 * F * d * esz + 2 * d * 4 + F * 4),
        "down": n * (d * F * esz + F * 4 + 2 * d * 4),
        "head": V * d * esz + 2 * d * 4,  # one pass; the fused form adds only a second activation row
        "_beta": beta,
    }


def default_attn_chunk(prompt_len):
    """Keys per attention split in the bench's workloads: about 16 splits over the prompt, in multiples
    of 64 keys (128 at the 2048-token headline size; 2048 at 32768 tokens, where fewer and longer
    splits share the GPU better with the other stage group than the library default's ~40)."""
    return max(64, (prompt_len // 16 + 63) // 64 * 64)


def timed_stages_per_launch(L, n, groups, first_slot):
    """Mean number of active stages in the stage launches of layer slots >= first_slot (the launches
    the kernel timing covers), with the stages spread over `groups` groups of consecutive stages. A
    stage with fewer layers than the longest is idle in the last slots (beta_{s+1} - beta_s < J), and a
    group launch with no active stage is not issued."""
    beta = [s * L // n for s in range(n + 1)]
    J = max(beta[s + 1] - beta[s] for s in range(n))
    counts = []
    for j in range(first_slot, J):
        for gi in range(groups):
            k = sum(1 for s in range(gi * n // groups, (gi + 1) * n // groups) if beta[s] + j < beta[s + 1])
            if k:
                counts.append(k)
    return sum(counts) / len(counts)


def cpu_baseline(sh, n, ctx, seed, budget_s=12.0):
    """Time the float64 CPU oracle on a bounded sample of the same step and scale it to one step.

    The sample: oracle.model.decoder_layer on one layer of the workload at context ctx (a stage layer
    and a PDM layer cost the same), oracle.model.lm_logits over the full vocabulary, and the PDM
    feature projection SPDOracle.feature on n anchors. A full-pipeline oracle step runs L target
    layers, n rows through each PDM layer, n feature projections and two LM heads."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import model as om
    from oracle import spd as osp

    rng = np.random.default_rng(0)
    model = om.Model(sh, seed)
    cache = om.LayerCache(sh.n_kv_heads, sh.head_dim, ctx + 8)
    cache.k[:ctx] = rng.standard_normal((ctx, sh.n_kv_heads, sh.head_dim))
    cache.v[:ctx] = rng.standard_normal((ctx, sh.n_kv_heads, sh.head_dim))
    cache.n = ctx
    lw = model.layer(0)
    h = rng.standard_normal(sh.d_model)

    def timed(fn, share):
        fn()  # warm (draws the weights)
        reps, t0 = 0, time.perf_counter()
        while True:
            fn()
            reps += 1
            el = time.perf_counter() - t0
            if el >= share * budget_s or reps >= 200:
                return el / reps, reps

    def one_layer():
        om.decoder_layer(sh, lw, h, ctx, cache)
        cache.truncate(ctx)

    t_layer, r_layer = timed(one_layer, 0.5)
    t_head, r_head = timed(lambda: om.lm_logits(model, h), 0.3)
    o = osp.SPDOracle.__new__(osp.SPDOracle)
    o.m, o.sh, o.n, o.L = model, sh, n, sh.n_layers
    o.anchor_layers = osp.stage_bounds(sh.n_layers, n)[:n]
    anchors = [rng.standard_normal(sh.d_model) for _ in range(n)]
    t_fc, r_fc = timed(lambda: o.feature(anchors, n), 0.2)
    step = (sh.n_layers + n * sh.pdm_layers) * t_layer + n * t_fc + 2 * t_head
    threads = 0
    for info in threadpool_info():
        if info.get("user_api") == "blas":
            threads = max(threads, int(info.get("num_threads", 0)))
    return {
        "value": round(1e6 * step, 1), "unit": "us/step", "cores": threads or len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": (f"extrapolated from timed oracle calls, not a timed oracle step: float64 decoder_layer of one "
                   f"{sh.name} layer at context {ctx} x{r_layer}, lm_logits over {sh.vocab} tokens x{r_head}, PDM "
                   f"feature projection ({n}*{sh.d_model} -> {sh.d_model}) x{r_fc}; one full-pipeline step = "
                   f"{sh.n_layers} target layers + {n} rows x {sh.pdm_layers} PDM layer(s) + {n} "
                   f"projections + 2 LM heads"),
        "cpu_model": cpu_model(),
        "per_layer_s": round(t_layer, 5), "head_s": round(t_head, 5), "fc_s": round(t_fc, 5),
    }


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="4b", choices=["tiny", "4b", "9b", "4b-sweep", "9b-long"])
    ap.add_argument("--n", type=int, default=None, help="SPD width (default: the workload's)")
    ap.add_argument("--prompt", type=int, default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="issue every launch instead of replaying the step graph")
    ap.add_argument("--separate-head", action="store_true",
                    help="the draft module runs its own LM-head pass on its stream instead of sharing the exit pass")
    ap.add_argument("--step-mode", type=int, default=2, choices=[0, 2],
                    help="stage compute: 0 five launches per layer slot covering all stages on one stream, "
                         "2 (default) stage groups, each on its own stream")
    ap.add_argument("--step-grid", type=int, default=0, help="workgroups of one stage launch (0: default)")
    ap.add_argument("--stage-groups", type=int, default=0, help="mode 2: stage streams (0: the library default)")
    ap.add_argument("--pdm-grid", type=int, default=0, help="workgroups per PDM GEMV launch (0: the default)")
    ap.add_argument("--pdm-place", type=int, default=0, choices=[0, 1, 2, 3],
                    help="PDM launches: own stream, main before the stages, first group before/after")
    ap.add_argument("--attn-chunk", type=int, default=0, help="keys per attention split (0: the workload's default)")
    ap.add_argument("--graph-steps", type=int, default=1, help="steps per replayed graph in batched runs")
    ap.add_argument("--extra-phases", choices=["auto", "on", "off"], default="auto",
                    help="the PDM's own head and sampled decoding, each on a handle of its own (auto: on "
                         "for prompts up to 4096 tokens; each needs its own prefill)")
    ap.add_argument("--extra-workloads", choices=["auto", "on", "off"], default="auto",
                    help="the 9B-class workloads (n = 4 at 4096 tokens; n = 8, two-layer PDM at 32768 tokens) after "
                         "the main one (auto: with the default 4B workload)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="profiling runs: a 1 GiB device copy (the known-size kernel for HBM counter scaling) "
                         "and marker dispatches around the measured phases")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the SPD step here is the single-GPU stage-batched "
              "form; multi-GPU sharding is not built", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2605_30852_amd import binding as B
    from paper_2605_30852_amd.engine import DeviceWeights, Engine

    wl = synth.WORKLOADS[args.workload]
    sh = wl["shape"]
    n = args.n or sh.n_stages
    sh = sh.with_(n_stages=n)
    P = args.prompt or wl["prompt_len"]
    K, W = args.steps, args.warmup
    esz = 2 if sh.dtype == "bf16" else 4
    K_GU, K_CLS, K_SPAN = 64, 16, 64
    # greedy reference long enough for every forced-accept phase below
    K_P50 = 64
    n_ref = W + K + K_GU + 6 * K_CLS + 4 * K_SPAN + K_P50 + 2 * n + 40
    # capacity and attention split size depend on the workload only (not on --steps), so that a
    # profiled run with fewer steps launches exactly the kernels the timed run launches
    max_tokens = P + max(1024, n_ref + 4 * n + 64)
    attn_chunk = args.attn_chunk or default_attn_chunk(P)

    if args.copy_calibration:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy calibration: 3 x 1 GiB device copies")
        del src, dst

    t0 = time.time()
    log(f"[bench] generating and uploading {sh.name} weights ({sh.param_bytes() / 1e9:.2f} GB)")
    weights = DeviceWeights(sh, args.seed, threads=16)
    torch.cuda.synchronize()
    log(f"[bench] weights ready in {time.time() - t0:.1f}s")
    prompt = synth.prompt(sh, args.seed, P)

    # plain greedy decoding (n = 1 through the same library): reference tokens and AR tokens/s
    t0 = time.time()
    fused = not args.separate_head
    mode = args.step_mode
    ar = Engine(weights, max_tokens=max_tokens, n=1, attn_chunk=attn_chunk, fused_head=fused)
    ar.spd_set_step_kernel(mode, args.step_grid, args.stage_groups if mode == 2 else -1)
    ar.spd_set_pdm_placement(args.pdm_place)
    # plain decoding needs no draft module: at n = 1 a step commits the target's token whatever the
    # draft, so the draft module's launches are left out of the reference and its tokens/s
    B.spd_set_pdm_enabled(ar.h, False)
    ar.spd_set_graph(not args.no_graph)
    first = ar.spd_prefill(prompt)
    log(f"[bench] AR prefill {P} tokens in {time.time() - t0:.1f}s")
    ar.spd_run_steps(1)  # the first step captures the step graph
    ar.spd_sync()
    torch.cuda.synchronize()
    ta = time.perf_counter()
    ar.spd_run_steps(n_ref - 1)
    ar.spd_sync()
    ar_s = time.perf_counter() - ta
    ar_tok_s = (n_ref - 1) / ar_s
    ref = ar.tokens()[P: P + n_ref + 1].astype(np.int64)
    assert ref[0] == first
    ar.close()
    log(f"[bench] AR: {n_ref} tokens, {1e6 * ar_s / n_ref:.1f} us/token")

    # SPD handle, all drafts forced to the greedy tokens: every step after the fill is a full step
    t0 = time.time()
    eng = Engine(weights, max_tokens=max_tokens, n=n, attn_chunk=attn_chunk, fused_head=fused)
    eng.spd_set_step_kernel(mode, args.step_grid, args.stage_groups if mode == 2 else -1)
    eng.spd_set_pdm_placement(args.pdm_place)
    eng.spd_set_pdm_grid(args.pdm_grid)
    eng.spd_set_graph(not args.no_graph)
    eng.spd_set_graph_steps(args.graph_steps)
    groups = B.spd_step_plan_info(eng.h)["stage_groups"]
    f2 = eng.spd_prefill(prompt)
    assert f2 == first
    log(f"[bench] SPD prefill {P} tokens in {time.time() - t0:.1f}s")
    eng.spd_set_forced_drafts(ref.astype(np.int32), P)
    eng.spd_run_steps(W)
    c0, a0, _, _ = eng.state()
    assert a0 == n, "pipeline not full after warm-up"
    phase_marker(args)  # phase 0: the steady-state timed run
    torch.cuda.synchronize()
    ts = time.perf_counter()
    eng.spd_run_steps(K)
    eng.spd_sync()
    torch.cuda.synchronize()
    el = time.perf_counter() - ts
    phase_marker(args)
    c1, a1, _, _ = eng.state()
    assert c1 - c0 == K and a1 == n, "forced-accept run left the steady state"
    toks = eng.tokens()[P: c1 + 1]
    assert np.array_equal(toks, ref[: len(toks)]), "SPD stream differs from greedy decoding"
    us_step = 1e6 * el / K
    c_mid = (c0 + c1) // 2
    tgt_b, pdm_b = step_bytes(sh, n, sh.pdm_layers, c_mid, esz, pdm_head=not fused)
    bytes_step = tgt_b + pdm_b
    gbs = bytes_step / (us_step * 1e-6) / 1e9
    log(f"[bench] SPD n={n}: {us_step:.1f} us/step, {bytes_step / 1e9:.3f} GB/step, {gbs:.0f} GB/s "
        f"({100 * gbs / PEAK_HBM_GBS:.1f}% of {PEAK_HBM_GBS:.0f})")
    # per-step durations: events on the handle's main stream between single-step replays (no host
    # synchronisation between the steps)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(K_P50 + 1)]
    evs[0].record(eng.main)
    for i in range(K_P50):
        eng.spd_run_steps(1)
        evs[i + 1].record(eng.main)
    eng.spd_sync()
    torch.cuda.synchronize()
    per_step = sorted(1e3 * evs[i].elapsed_time(evs[i + 1]) for i in range(K_P50))
    step_dist = {"steps": K_P50, "p50_us": round(per_step[K_P50 // 2], 1),
                 "p90_us": round(per_step[(9 * K_P50) // 10], 1), "min_us": round(per_step[0], 1),
                 "mean_us": round(sum(per_step) / K_P50, 1)}
    log(f"[bench] per-step durations: {step_dist}")

    # per-kernel HIP-event timing on the launching stream, steady state (every step accepts). Only the
    # slots after the draft module's span are timed, so that a kernel is timed without the side
    # stream sharing HBM.
    L_slots = max(sh.n_layers // n + (1 if sh.n_layers % n else 0), 1)
    first_slot = L_slots // 2

    def time_class(kid, steps):
        B.spd_set_kernel_timing(eng.h, kid, first_slot if kid != B.SPD_K_HEAD else 0)
        ca, _, _, _ = eng.state()
        eng.spd_run_steps(steps)
        eng.spd_sync()
        ms, nl = B.spd_kernel_timing(eng.h)
        B.spd_set_kernel_timing(eng.h, 0)
        cb, ab, _, _ = eng.state()
        assert cb - ca == steps and ab == n, "kernel timing left the steady state"
        assert nl > 0, "no launch of the timed class"
        return ms, nl, (ca + cb) // 2

    # Every sublayer class in the timed launch form. With stage groups a launch's events also hold the
    # time it waits for the compute units another group's launch occupies, so these are not kernel
    # durations; they show where the step's time goes.
    kernels = {}
    classes = (("qkv", B.SPD_K_QKV), ("attn", B.SPD_K_ATTN), ("oproj", B.SPD_K_OPROJ),
               ("gateup", B.SPD_K_GATEUP), ("down", B.SPD_K_DOWN), ("head", B.SPD_K_HEAD))
    stages_timed = timed_stages_per_launch(sh.n_layers, n, groups if mode == 2 else 1, first_slot)
    for kname, kid in classes:
        ms, nl, cm = time_class(kid, K_CLS)
        lb = launch_bytes(sh, n, cm, esz)[kname]
        if kname != "head":
            lb = lb / n * stages_timed  # per stage, times the stages a timed launch covers on average
        us = 1e3 * ms / max(1, nl)
        kernels[kname] = {"us_per_launch": round(us, 2), "timed_launches_per_step": nl / K_CLS,
                          "bytes_per_launch": int(lb), "GBps": round(lb / (us * 1e-6) / 1e9, 1)}
    log(f"[bench] kernels (concurrent launch form): {kernels}")
    # The dominant kernel (most bytes per step: the gate/up GEMV) with nothing beside it, so that its
    # event interval is its own execution: one stage group (every launch covers all n stages) and the
    # draft module's launches off (drafts are forced). The kernel trace of the same command times the
    # same launches (grid y = n).
    eng.spd_set_step_kernel(mode, args.step_grid, 1)
    B.spd_set_pdm_enabled(eng.h, False)
    eng.spd_run_steps(2)
    eng.spd_sync()
    phase_marker(args)  # phase 1: the dominant kernel alone
    ms, nl, cm = time_class(B.SPD_K_GATEUP, K_GU)
    phase_marker(args)
    lb = launch_bytes(sh, n, cm, esz)["gateup"] / n * timed_stages_per_launch(sh.n_layers, n, 1, first_slot)
    dom_us = 1e3 * ms / max(1, nl)
    dom = {"bytes_per_launch": int(lb), "us_per_launch": round(dom_us, 2), "launches": nl,
           "GBps": round(lb / (dom_us * 1e-6) / 1e9, 1)}
    B.spd_set_pdm_enabled(eng.h, True)
    eng.spd_set_step_kernel(mode, args.step_grid, args.stage_groups)
    eng.spd_run_steps(2)
    log(f"[bench] gate/up alone (one stage group, no PDM): {dom}")

    # PDM overlap: step start -> end of the stage compute (main) and -> end of the PDM (side stream)
    B.spd_set_kernel_timing(eng.h, B.SPD_K_SPANS)
    eng.spd_run_steps(K_SPAN)
    st_ms, pd_ms, late_ms, ns = B.spd_span_timing(eng.h)
    B.spd_set_kernel_timing(eng.h, 0)
    spans = {"stage_us": round(1e3 * st_ms / ns, 1), "pdm_us": round(1e3 * pd_ms / ns, 1),
             "verify_wait_us": round(1e3 * late_ms / ns, 2), "steps": ns,
             "pdm_hidden": late_ms == 0.0}
    # hidden fraction 1 - (T_with - T_without) / T_pdm: the step without the PDM's launches (drafts
    # are forced anyway), and the PDM alone (its launches on the main stream before the stages,
    # timed from the step start to their end)
    if True:
        B.spd_set_pdm_enabled(eng.h, False)
        eng.spd_run_steps(4)
        eng.spd_sync()
        torch.cuda.synchronize()
        ts = time.perf_counter()
        eng.spd_run_steps(K_SPAN)
        eng.spd_sync()
        t_without = 1e6 * (time.perf_counter() - ts) / K_SPAN
        B.spd_set_pdm_enabled(eng.h, True)
        B.spd_set_pdm_placement(eng.h, 1)
        B.spd_set_kernel_timing(eng.h, B.SPD_K_SPANS)
        eng.spd_run_steps(K_SPAN // 2)
        _, pd_alone_ms, _, na = B.spd_span_timing(eng.h)
        B.spd_set_kernel_timing(eng.h, 0)
        B.spd_set_pdm_placement(eng.h, args.pdm_place)
        t_pdm = 1e3 * pd_alone_ms / na
        spans.update({"step_us_without_pdm": round(t_without, 1), "pdm_alone_us": round(t_pdm, 1),
                      "hidden_fraction": round(1.0 - (us_step - t_without) / t_pdm, 3)})
        # the post-step schedule (the PDM after the stage compute, on deeper features): serial
        B.spd_set_pdm_schedule(eng.h, True)
        eng.spd_run_steps(4)
        eng.spd_sync()
        torch.cuda.synchronize()
        ts = time.perf_counter()
        eng.spd_run_steps(K_SPAN)
        eng.spd_sync()
        spans["post_step_us_per_step"] = round(1e6 * (time.perf_counter() - ts) / K_SPAN, 1)
        B.spd_set_pdm_schedule(eng.h, False)
        eng.spd_run_steps(2)  # captures the step graph again before the next timed run
        eng.spd_sync()
        ca, aa, _, _ = eng.state()
        assert aa == n, "PDM hiding measurement left the steady state"
    log(f"[bench] spans: {spans}")

    # tokens/s at a seeded Bernoulli acceptance pattern (rollback and refill exercised): one untimed
    # pass over the pattern, then the timed pass over the same steps
    p = wl.get("p_accept") or 0.7
    mask = synth.accept_mask(p, args.seed, max_tokens)
    table = np.full(len(ref), -1, dtype=np.int32)
    for i in range(1, len(ref)):
        q = P + i
        table[i] = ref[i] if mask[q] else (ref[i] + 1) % sh.vocab
    for timed_pass in (False, True):
        eng.spd_rollback(P, int(first))
        eng.spd_clear_forced_drafts()
        eng.spd_set_forced_drafts(table, P)
        torch.cuda.synchronize()
        ts = time.perf_counter()
        logp = eng.spd_run_steps(K, want_log=True)
        elp = time.perf_counter() - ts
        log(f"[bench] p-run ({'timed' if timed_pass else 'warm-up'}): {K} steps in {1e3 * elp:.2f} ms")
    committed = logp[-1]["committed_len"] - P
    spd_tok_s = committed / elp
    alpha = committed / K
    toks = eng.tokens()[P: logp[-1]["committed_len"] + 1]
    assert np.array_equal(toks, ref[: len(toks)]), "SPD stream differs from greedy decoding (p run)"
    for r in logp:
        if r["decision"] != B.SPD_NONE:
            assert r["decision"] == (B.SPD_ACCEPT if mask[r["verified_pos"]] else B.SPD_REJECT)
    # run mean over every step of the pattern (fill and refill steps stream only the active stages)
    run_bytes, c_pre, a_pre = 0, P, 1
    for r in logp:
        run_bytes += step_bytes_active(sh, n, sh.pdm_layers, c_pre, a_pre, esz)
        c_pre, a_pre = r["committed_len"], r["inflight"]
    run_mean = {"us_per_step": round(1e6 * elp / K, 1), "GB_per_step": round(run_bytes / K / 1e9, 3),
                "GBps": round(run_bytes / elp / 1e9, 1),
                "frac": round(run_bytes / elp / 1e9 / PEAK_HBM_GBS, 4)} if fused else None
    log(f"[bench] p={p}: alpha={alpha:.3f}, {spd_tok_s:.0f} tok/s (AR {ar_tok_s:.0f} tok/s); run mean {run_mean}")
    eng.close()

    extra = args.extra_phases == "on" or (args.extra_phases == "auto" and P <= 4096)
    if not extra:
        log(f"[bench] own-head and sampled phases skipped (--extra-phases {args.extra_phases}, prompt {P})")
    own_head = own_head_phase(args, weights, prompt, ref, max_tokens, attn_chunk, K, W, n, us_step) if extra else None

    sampled = None
    if fused and extra:
        sampled = sampled_phase(args, sh, weights, prompt, ref, first, mask, max_tokens, attn_chunk, K, W, n,
                                us_step, kernels.get("head"))

    # achievable HBM read bandwidth for context: a plain 16-byte non-temporal streaming read of 1 GiB
    # (past the 256 MB last-level cache), through the library's probe kernel
    pbuf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    psink = torch.empty(4096, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    pms = B.spd_probe_hbm_read(pbuf.data_ptr(), pbuf.numel(), psink.data_ptr(), 10,
                               torch.cuda.current_stream().cuda_stream)
    probe = {"GBps": round(pbuf.numel() / (pms * 1e-3) / 1e9, 1), "bytes": pbuf.numel(),
             "frac": round(pbuf.numel() / (pms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
             "kernel": "k_read_probe: 2048 workgroups, 16-byte non-temporal loads, 8 in flight per thread"}
    del pbuf, psink
    log(f"[bench] HBM read probe: {probe['GBps']} GB/s")
    del weights
    torch.cuda.empty_cache()

    workloads = None
    if args.extra_workloads == "on" or (args.extra_workloads == "auto" and args.workload == "4b"
                                        and args.prompt is None and args.n is None):
        t0 = time.time()
        log(f"[bench] generating and uploading 9b weights ({synth.B9.param_bytes() / 1e9:.2f} GB)")
        w9 = DeviceWeights(synth.B9, args.seed, threads=16)
        torch.cuda.synchronize()
        log(f"[bench] 9b weights ready in {time.time() - t0:.1f}s")
        workloads = {}
        workloads["9b_n4_4096"] = extra_workload("9b n=4, 4096-token prompt", w9, 4, 1, 4096, 0.7, args.seed)
        wl8 = w9.pdm_for_width(8, 2)
        workloads["9b_n8_32768"] = extra_workload("9b n=8, two-layer PDM, 32768-token prompt", wl8, 8, 2, 32768, 0.6,
                                                  args.seed)
        del wl8, w9
        torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.time()
        cpu = cpu_baseline(sh, n, P, args.seed)
        log(f"[bench] cpu baseline {cpu['value'] / 1e3:.1f} ms/step in {time.time() - t0:.1f}s")

    out = {
        "metric": METRIC,
        "value": round(us_step, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(us_step / 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": sh.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, uniform-random prompt, drafts forced to greedy tokens)",
        "config": {"workload": f"{sh.name}-class dense decoder ({sh.n_layers} layers, d {sh.d_model}, "
                               f"{sh.n_q_heads}/{sh.n_kv_heads} heads of {sh.head_dim}, FFN {sh.ffn_dim}, "
                               f"vocab {sh.vocab}), SPD width n={n}, {sh.pdm_layers}-layer PDM, "
                               f"{P}-token prompt, batch 1, steady-state full-pipeline steps",
                   "n": n, "prompt": P, "pdm_layers": sh.pdm_layers, "batch": 1,
                   "max_tokens": max_tokens, "attn_chunk": attn_chunk,
                   "lm_head": "one two-row pass shared by exit and draft" if fused else "separate passes",
                   "step_graph": not args.no_graph,
                   "stage_compute": {0: "five launches per layer slot covering all stages",
                                     2: f"{groups} stage groups on their own streams, five launches per layer slot "
                                        f"each covering the group's stages"}[mode],
                   "step_grid": args.step_grid or None,
                   "pdm_placement": {0: "own stream", 1: "main stream before the stages",
                                     2: "first stage group's stream, before its stages",
                                     3: "first stage group's stream, after its stages"}[args.pdm_place]},
        "bytes_per_step": int(bytes_step),
        "step_GBps": round(gbs, 1),
        "step_roofline_frac": round(gbs / PEAK_HBM_GBS, 4),
        "step_us_distribution": step_dist,
        "roofline": {"bound": "hbm", "achieved": dom["GBps"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(dom["GBps"] / PEAK_HBM_GBS, 4),
                     "traffic": traffic_from_profile("gateup_4b_n4_traffic.txt") if sh.name == "4b" and n == 4 else None,
                     "kernel": f"k_sgemv gate/up GEMV + SwiGLU, one launch over all {n} stages (grid y = {n}) with "
                               f"nothing beside it: one stage group, the PDM's launches off",
                     "bytes_per_launch": dom["bytes_per_launch"], "us_per_launch": dom["us_per_launch"],
                     "timing": f"dispatch-recorded HIP events on the launching stream, layer slots >= {first_slot} of "
                               f"{L_slots}, {K_GU} steady-state steps ({dom['launches']} launches)",
                     "concurrent": {"us_per_launch": kernels["gateup"]["us_per_launch"],
                                    "bytes_per_launch": kernels["gateup"]["bytes_per_launch"],
                                    "note": f"the timed launch form ({groups} stage groups): a launch's events also "
                                            f"hold its wait for the compute units the other group's launch occupies"}},
        "kernels": kernels,
        "pdm_overlap": spans,
        "hbm_read_probe": probe,
        "tokens_per_s": {"spd_forced_p": p, "alpha": round(alpha, 4), "spd": round(spd_tok_s, 1),
                         "ar_same_gpu": round(ar_tok_s, 1), "run_mean": run_mean,
                         "note": "context, not a target: on one GPU an SPD step streams about the bytes of one "
                                 "plain decoding step, and plain decoding through this library (n = 1, one "
                                 "chain of small launches per token) is launch-bound; neither figure is a "
                                 "property of the method"},
        "workloads": workloads,
        "pdm_own_head": own_head,
        "sampled": sampled,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def extra_workload(label, weights, n, ls, P, p, seed, steps=32, warmup=4, k_span=16, n_bern=96):
    """One more workload on one handle: prefill, the greedy reference from the handle's own decoding
    with the PDM's drafts (lossless, so its committed stream is greedy decoding), then steady-state
    steps with the drafts forced to it (us/step, algorithmic bytes, GB/s), the PDM's hiding (the
    step without the PDM's launches and the PDM alone), and a Bernoulli(p) draft pattern."""
    import numpy as np
    import torch

    import synth
    from paper_2605_30852_amd import binding as B
    from paper_2605_30852_amd.engine import Engine

    sh = weights.shape
    esz = 2 if sh.dtype == "bf16" else 4
    max_tokens = P + 2048
    prompt = synth.prompt(sh, seed, P)
    eng = Engine(weights, max_tokens=max_tokens, n=n, pdm_layers=ls, attn_chunk=default_attn_chunk(P))
    eng.spd_set_graph(True)
    t0 = time.time()
    log(f"[bench] {label}: prefill")
    first = prefill_with_progress(eng, prompt, label)
    log(f"[bench] {label}: prefill {P} tokens in {time.time() - t0:.1f}s")
    need = warmup + steps + 3 * k_span + 16 + 6 * n + 16
    while eng.state()[0] - P < need:
        eng.spd_run_steps(256)
        eng.spd_sync()
    c, _, _, _ = eng.state()
    ref = eng.tokens()[P: c + 1].astype(np.int64)
    log(f"[bench] {label}: {len(ref)} greedy reference tokens from the PDM's own drafts")
    eng.spd_rollback(P, int(first))
    eng.spd_set_forced_drafts(ref.astype(np.int32), P)
    eng.spd_run_steps(warmup + n)  # the pipeline fills in n - 1 steps
    c0, a0, _, _ = eng.state()
    assert a0 == n, f"{label}: pipeline not full after warm-up"
    torch.cuda.synchronize()
    ts = time.perf_counter()
    eng.spd_run_steps(steps)
    eng.spd_sync()
    us = 1e6 * (time.perf_counter() - ts) / steps
    c1, a1, _, _ = eng.state()
    assert c1 - c0 == steps and a1 == n
    tb, pb = step_bytes(sh, n, ls, (c0 + c1) // 2, esz, pdm_head=False)
    B.spd_set_kernel_timing(eng.h, B.SPD_K_SPANS)
    eng.spd_run_steps(k_span)
    st_ms, pd_ms, late_ms, ns = B.spd_span_timing(eng.h)
    B.spd_set_kernel_timing(eng.h, 0)
    B.spd_set_pdm_enabled(eng.h, False)
    eng.spd_run_steps(4)
    eng.spd_sync()
    ts = time.perf_counter()
    eng.spd_run_steps(k_span)
    eng.spd_sync()
    t_without = 1e6 * (time.perf_counter() - ts) / k_span
    B.spd_set_pdm_enabled(eng.h, True)
    B.spd_set_pdm_placement(eng.h, 1)
    B.spd_set_kernel_timing(eng.h, B.SPD_K_SPANS)
    eng.spd_run_steps(k_span)
    _, pd_alone_ms, _, na = B.spd_span_timing(eng.h)
    B.spd_set_kernel_timing(eng.h, 0)
    B.spd_set_pdm_placement(eng.h, 0)
    eng.spd_run_steps(2)  # captures the step graph again before the timed Bernoulli run
    eng.spd_sync()
    t_pdm = 1e3 * pd_alone_ms / na
    toks = eng.tokens()[P: eng.state()[0] + 1]
    assert np.array_equal(toks, ref[: len(toks)]), f"{label}: SPD stream differs from greedy decoding"
    # the Bernoulli(p) draft pattern: rollback, refill, tokens per second (an untimed pass over the
    # pattern, then the timed pass over the same steps)
    mask = synth.accept_mask(p, seed, max_tokens)
    table = np.array([ref[i] if mask[P + i] else (ref[i] + 1) % sh.vocab for i in range(len(ref))], dtype=np.int32)
    steps_b = min(n_bern, len(ref) - 2 * n)
    for _ in range(2):
        eng.spd_rollback(P, int(first))
        eng.spd_clear_forced_drafts()
        eng.spd_set_forced_drafts(table, P)
        torch.cuda.synchronize()
        ts = time.perf_counter()
        logp = eng.spd_run_steps(steps_b, want_log=True)
        elp = time.perf_counter() - ts
    committed = logp[-1]["committed_len"] - P
    exits = [r for r in logp if r["decision"] != B.SPD_NONE]
    agree = sum(1 for r in exits if r["decision"] == (B.SPD_ACCEPT if mask[r["verified_pos"]] else B.SPD_REJECT))
    toks = eng.tokens()[P: logp[-1]["committed_len"] + 1]
    assert np.array_equal(toks, ref[: len(toks)]), f"{label}: SPD stream differs from greedy decoding (p run)"
    eng.close()
    out = {"workload": f"{sh.name}-class dense decoder (d {sh.d_model}, FFN {sh.ffn_dim}), n={n}, {ls}-layer PDM, "
                       f"{P}-token prompt", "n": n, "pdm_layers": ls, "prompt": P, "steps": steps,
           "attn_chunk": default_attn_chunk(P),
           "us_per_step": round(us, 1), "bytes_per_step": int(tb + pb),
           "GBps": round((tb + pb) / (us * 1e-6) / 1e9, 1), "frac": round((tb + pb) / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
           "pdm": {"stage_us": round(1e3 * st_ms / ns, 1), "pdm_us": round(1e3 * pd_ms / ns, 1),
                   "verify_wait_us": round(1e3 * late_ms / ns, 2), "step_us_without_pdm": round(t_without, 1),
                   "pdm_alone_us": round(t_pdm, 1), "hidden_fraction": round(1.0 - (us - t_without) / t_pdm, 3)},
           "bernoulli": {"p": p, "steps": steps_b, "alpha": round(committed / steps_b, 4),
                         "tok_s": round(committed / elp, 1), "decisions_matching_mask": f"{agree}/{len(exits)}"}}
    log(f"[bench] {label}: {out}")
    return out


def own_head_phase(args, weights, prompt, ref, max_tokens, attn_chunk, K, W, n, shared_us, vocab=32768):
    """The PDM with its own LM head over a smaller vocabulary (initialised from the target's rows of
    that subset; at most half the target's): its head runs on the PDM's stream, the exit row alone on
    the main stream. Steady state with drafts forced to the greedy tokens (the stream is checked), and
    the PDM's span."""
    import numpy as np
    import torch

    from paper_2605_30852_amd import binding as B
    from paper_2605_30852_amd.engine import Engine

    P = len(prompt)
    vocab = min(vocab, weights.shape.vocab // 2)
    wv = weights.with_pdm_vocab(vocab)
    eng = Engine(wv, max_tokens=max_tokens, n=n, attn_chunk=attn_chunk)
    eng.spd_set_step_kernel(args.step_mode, args.step_grid, args.stage_groups if args.step_mode == 2 else -1)
    eng.spd_set_pdm_placement(args.pdm_place)
    eng.spd_set_pdm_grid(args.pdm_grid)
    eng.spd_set_graph(not args.no_graph)
    eng.spd_prefill(prompt)
    eng.spd_set_forced_drafts(ref.astype(np.int32), P)
    eng.spd_run_steps(W)
    c0, a0, _, _ = eng.state()
    assert a0 == n, "own-head pipeline not full after warm-up"
    torch.cuda.synchronize()
    ts = time.perf_counter()
    eng.spd_run_steps(K)
    eng.spd_sync()
    el = time.perf_counter() - ts
    c1, a1, _, _ = eng.state()
    assert c1 - c0 == K and a1 == n, "own-head forced-accept run left the steady state"
    toks = eng.tokens()[P: c1 + 1]
    assert np.array_equal(toks, ref[: len(toks)]), "own-head SPD stream differs from greedy decoding"
    B.spd_set_kernel_timing(eng.h, B.SPD_K_SPANS)
    eng.spd_run_steps(32)
    st_ms, pd_ms, late_ms, ns = B.spd_span_timing(eng.h)
    B.spd_set_kernel_timing(eng.h, 0)
    eng.close()
    del wv
    us = 1e6 * el / K
    out = {"pdm_vocab": vocab, "us_per_step": round(us, 1), "over_shared_fused_us": round(us - shared_us, 1),
           "stage_us": round(1e3 * st_ms / ns, 1), "pdm_us": round(1e3 * pd_ms / ns, 1),
           "verify_wait_us": round(1e3 * late_ms / ns, 2),
           "head_bytes": int(vocab * weights.shape.d_model * (2 if weights.shape.dtype == "bf16" else 4))}
    log(f"[bench] own PDM head ({vocab} tokens): {us:.1f} us/step ({us - shared_us:+.1f} over the shared fused "
        f"head), PDM span {out['pdm_us']} us, verify wait {out['verify_wait_us']} us")
    return out


def sampled_phase(args, sh, weights, prompt, ref, first, mask, max_tokens, attn_chunk, K, W, n, greedy_us,
                  greedy_head):
    """Sampled decoding at top-k 50, temperature 1 (the paper's sampling setting). With u_accept = 0 a
    judged draft is kept iff the target gives it mass, and with u_resample = 0 a draw takes the most
    likely token, so with the drafts forced to the greedy tokens every step keeps its draft and the
    stream is greedy decoding's while every step still runs the top-50 selection of both rows, the
    draws and the rejection-sampling verify. Then the Bernoulli(p) draft pattern: a wrong draft (a
    token outside the top 50) is rejected and the residual draw commits the greedy token."""
    import numpy as np
    import torch

    from paper_2605_30852_amd import binding as B
    from paper_2605_30852_amd.engine import Engine

    P = len(prompt)
    top_k, temp = 50, 1.0
    U = np.random.default_rng([args.seed, 4]).random((max_tokens, 3))
    U[:, 1] = 0.0
    U[:, 2] = 0.0
    sam = Engine(weights, max_tokens=max_tokens, n=n, attn_chunk=attn_chunk, fused_head=True)
    sam.spd_set_step_kernel(args.step_mode, args.step_grid, args.stage_groups if args.step_mode == 2 else -1)
    sam.spd_set_pdm_placement(args.pdm_place)
    sam.spd_set_pdm_grid(args.pdm_grid)
    sam.spd_set_sampling(top_k, temp, U)
    sam.spd_set_graph(not args.no_graph)
    assert sam.spd_prefill(prompt) == first, "the first sampled token at u = 0 is not the greedy token"
    sam.spd_set_forced_drafts(ref.astype(np.int32), P)
    sam.spd_run_steps(W)
    c0, a0, _, _ = sam.state()
    assert a0 == n, "sampled pipeline not full after warm-up"
    torch.cuda.synchronize()
    ts = time.perf_counter()
    sam.spd_run_steps(K)
    sam.spd_sync()
    el = time.perf_counter() - ts
    c1, a1, _, _ = sam.state()
    assert c1 - c0 == K and a1 == n, "sampled forced-accept run left the steady state"
    toks = sam.tokens()[P: c1 + 1]
    assert np.array_equal(toks, ref[: len(toks)]), "sampled stream at u = 0 differs from greedy decoding"
    us = 1e6 * el / K
    B.spd_set_kernel_timing(sam.h, B.SPD_K_HEAD, 0)
    sam.spd_run_steps(16)
    sam.spd_sync()
    ms, nl = B.spd_kernel_timing(sam.h)
    B.spd_set_kernel_timing(sam.h, 0)
    head_us = 1e3 * ms / max(1, nl)
    # Bernoulli(p) draft pattern
    sam.spd_rollback(P, int(first))
    table = np.full(len(ref), -1, dtype=np.int32)
    for i in range(1, len(ref)):
        table[i] = ref[i] if mask[P + i] else (ref[i] + 1) % sh.vocab
    sam.spd_clear_forced_drafts()
    sam.spd_set_forced_drafts(table, P)
    torch.cuda.synchronize()
    ts = time.perf_counter()
    logp = sam.spd_run_steps(K, want_log=True)
    elp = time.perf_counter() - ts
    committed = logp[-1]["committed_len"] - P
    agree = sum(1 for r in logp if r["decision"] != B.SPD_NONE
                and r["decision"] == (B.SPD_ACCEPT if mask[r["verified_pos"]] else B.SPD_REJECT))
    exits = sum(1 for r in logp if r["decision"] != B.SPD_NONE)
    sam.close()
    out = {"top_k": top_k, "temperature": temp, "us_per_step": round(us, 1),
           "over_greedy_us": round(us - greedy_us, 1),
           "head_verify_us_per_launch": round(head_us, 2),
           "greedy_head_verify_us_per_launch": greedy_head["us_per_launch"] if greedy_head else None,
           "p_run": {"alpha": round(committed / K, 4), "tok_s": round(committed / elp, 1),
                     "decisions_matching_mask": f"{agree}/{exits}"},
           "uniforms": "u_accept = u_resample = 0 (keep iff the target gives mass; draws take the most likely "
                       "token); u_draft seeded uniform"}
    log(f"[bench] sampled top-{top_k} T={temp}: {us:.1f} us/step ({us - greedy_us:+.1f} over greedy), "
        f"head+verify {head_us:.1f} us/launch; p-run alpha {committed / K:.3f}, {committed / elp:.0f} tok/s, "
        f"decisions matching the mask {agree}/{exits}")
    return out


def phase_marker(args):
    """Profiling runs (--copy-calibration): two dispatches of the library's read-probe kernel on a
    1 MiB buffer, with the GPU idle before and after, at the start and at the end of each measured
    phase. A counter file records kernel names and dispatch order but not grid shapes, so these
    markers are how its dispatches are assigned to phases (phase k between markers 2k and 2k+1;
    the probe kernel runs nowhere else before the closing bandwidth probe)."""
    if not args.copy_calibration:
        return
    import torch
    from paper_2605_30852_amd import binding as B
    torch.cuda.synchronize()
    buf = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    sink = torch.empty(4096, dtype=torch.float32, device="cuda")
    B.spd_probe_hbm_read(buf.data_ptr(), buf.numel(), sink.data_ptr(), 1, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()


def traffic_from_profile(name):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter summary
    profiles/<name>, or None when the counters were taken on other kernel sources (any .hip or .h file
    of csrc) than the ones built now."""
    from paper_2605_30852_amd.profsum import kernel_sources_digest
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    digest = kernel_sources_digest(os.path.join(ROOT, "paper_2605_30852_amd", "csrc"))
    if kv.get("kernels_sha256") != digest or "hbm_bytes_per_launch" not in kv:
        return None
    return int(float(kv["hbm_bytes_per_launch"]))


if __name__ == "__main__":
    main()
