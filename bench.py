#!/usr/bin/env python3
"""Benchmark of one SPD pipeline step on one MI355X.

Workload (default): the 4B-class dense decoder (36 layers, d 2560, 32/8 heads of 128, FFN 9728,
vocab 151936, bf16 weights and KV), SPD width n = 4 (9 layers per stage), 1-layer PDM, a 2048-token
uniform-random prompt, synthetic N(0, 0.02) weights. A step is one spd_step: the PDM on its stream,
every stage's 9 layers, the exit LM head and verification.

Timed region: K back-to-back steps with drafts forced to the target's own greedy tokens (every step
accepts, so every step is a full-pipeline step), bracketed by device synchronisation. Reported:
us per step, algorithmic HBM bytes per step and GB/s against 8 TB/s, the dominant kernel's
roofline (HIP events around each launch), tokens/s at a Bernoulli(0.7) acceptance pattern next to
plain greedy decoding on the same GPU, and the CPU oracle's time per step on the host cores.
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


def step_bytes(sh, n, ls, c, esz, pdm_head=True):
    """Algorithmic HBM bytes of one full-pipeline step that starts with c committed positions."""
    d, F, V, L = sh.d_model, sh.ffn_dim, sh.vocab, sh.n_layers
    qd, kvd = sh.q_dim, sh.kv_dim
    layer_w = (qd * d + 2 * kvd * d + d * qd + 3 * F * d) * esz + 2 * d * 4
    kv_tok = 2 * kvd * esz
    beta = [s * L // n for s in range(n + 1)]
    kv_read = 0
    for s in range(n):
        pos = c + n - 1 - s  # token of stage s attends to pos+1 keys
        kv_read += (beta[s + 1] - beta[s]) * (pos + 1) * kv_tok
    target = L * layer_w + kv_read + L * kv_tok + V * d * esz + d * esz
    pdm_kv = sum((c + i + 1) for i in range(n)) * ls * kv_tok + n * ls * kv_tok
    pdm = d * n * d * esz + ls * layer_w + pdm_kv + (V * d * esz if pdm_head else 0)
    return target, pdm


def cpu_baseline(sh, n, ctx, seed):
    """Time the float64 CPU oracle on a bounded sample of the same step and scale it to a step."""
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
    reps = 4
    om.decoder_layer(sh, lw, h, ctx, cache)  # warm
    cache.truncate(ctx)
    t0 = time.perf_counter()
    for _ in range(reps):
        om.decoder_layer(sh, lw, h, ctx, cache)
        cache.truncate(ctx)
    t_layer = (time.perf_counter() - t0) / reps
    model.w("lm_head")
    t0 = time.perf_counter()
    for _ in range(2):
        om.lm_logits(model, h)
    t_head = (time.perf_counter() - t0) / 2
    o = osp.SPDOracle.__new__(osp.SPDOracle)
    o.m, o.sh, o.n, o.L = model, sh, n, sh.n_layers
    o.anchor_layers = osp.stage_bounds(sh.n_layers, n)[:n]
    anchors = [rng.standard_normal(sh.d_model) for _ in range(n)]
    o.feature(anchors, n)  # draws W_in
    t0 = time.perf_counter()
    for _ in range(2):
        o.feature(anchors, n)
    t_fc = (time.perf_counter() - t0) / 2
    step = sh.n_layers * t_layer + sh.pdm_layers * n * t_layer / n + t_fc + 2 * t_head
    threads = 0
    for info in threadpool_info():
        if info.get("user_api") == "blas":
            threads = max(threads, int(info.get("num_threads", 0)))
    return {
        "value": 1e6 * step, "unit": "us/step", "cores": threads or len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": (f"float64 oracle: decoder_layer on one {sh.name} layer at context {ctx} x{reps}, "
                   f"LM head x2, PDM feature projection x2; scaled to {sh.n_layers} target layers + "
                   f"{sh.pdm_layers} PDM layer + projection + 2 LM heads per step"),
        "per_layer_s": t_layer, "head_s": t_head,
    }


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
    ap.add_argument("--no-ar", action="store_true", help="skip the plain greedy tokens/s line")
    ap.add_argument("--no-graph", action="store_true", help="issue every launch instead of replaying the step graph")
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
    max_tokens = P + W + 2 * K + 4 * n + 64

    t0 = time.time()
    log(f"[bench] generating and uploading {sh.name} weights ({sh.param_bytes() / 1e9:.2f} GB)")
    weights = DeviceWeights(sh, args.seed, threads=16)
    torch.cuda.synchronize()
    log(f"[bench] weights ready in {time.time() - t0:.1f}s")
    prompt = synth.prompt(sh, args.seed, P)

    # plain greedy decoding (n = 1 through the same library): reference tokens and AR tokens/s
    t0 = time.time()
    ar = Engine(weights, max_tokens=max_tokens, n=1)
    ar.spd_set_graph(not args.no_graph)
    first = ar.spd_prefill(prompt)
    log(f"[bench] AR prefill {P} tokens in {time.time() - t0:.1f}s")
    n_ref = W + 2 * K + 2 * n + 8
    torch.cuda.synchronize()
    ta = time.perf_counter()
    ar.spd_run_steps(n_ref)
    ar.spd_sync()
    ar_s = time.perf_counter() - ta
    ar_tok_s = n_ref / ar_s
    ref = ar.tokens()[P: P + n_ref + 1].astype(np.int64)
    assert ref[0] == first
    ar.close()
    log(f"[bench] AR: {n_ref} tokens, {1e6 * ar_s / n_ref:.1f} us/token")

    # SPD handle, all drafts forced to the greedy tokens: every step after the fill is a full step
    eng = Engine(weights, max_tokens=max_tokens, n=n)
    eng.spd_set_graph(not args.no_graph)
    f2 = eng.spd_prefill(prompt)
    assert f2 == first
    eng.spd_set_forced_drafts(ref.astype(np.int32), P)
    eng.spd_run_steps(W)
    c0, a0, _, _ = eng.state()
    assert a0 == n, "pipeline not full after warm-up"
    torch.cuda.synchronize()
    ts = time.perf_counter()
    eng.spd_run_steps(K)
    last = eng.spd_sync()
    torch.cuda.synchronize()
    el = time.perf_counter() - ts
    c1, a1, _, _ = eng.state()
    assert c1 - c0 == K and a1 == n, "forced-accept run left the steady state"
    toks = eng.tokens()[P: c1 + 1]
    assert np.array_equal(toks, ref[: len(toks)]), "SPD stream differs from greedy decoding"
    us_step = 1e6 * el / K
    tgt_b, pdm_b = step_bytes(sh, n, sh.pdm_layers, (c0 + c1) // 2, esz)
    bytes_step = tgt_b + pdm_b
    gbs = bytes_step / (us_step * 1e-6) / 1e9
    log(f"[bench] SPD n={n}: {us_step:.1f} us/step, {bytes_step / 1e9:.3f} GB/step, {gbs:.0f} GB/s")

    # dominant kernel: grouped gate/up + SwiGLU over the n stages, HIP events on the main stream
    B.spd_set_kernel_timing(eng.h, B.SPD_K_GATEUP)
    Kt = min(K, 64)
    eng.spd_run_steps(Kt)
    eng.spd_sync()
    ms, launches = B.spd_kernel_timing(eng.h)
    B.spd_set_kernel_timing(eng.h, 0)
    gu_bytes = n * (2 * sh.ffn_dim * sh.d_model * esz + sh.d_model * 4 + sh.ffn_dim * 4)
    gu_s = ms * 1e-3 / max(1, launches)
    gu_gbs = gu_bytes / gu_s / 1e9
    # all kernels' share for the log
    shares = {}
    for kname, kid in (("qkv", B.SPD_K_QKV), ("attn", B.SPD_K_ATTN), ("oproj", B.SPD_K_OPROJ),
                       ("down", B.SPD_K_DOWN), ("head", B.SPD_K_HEAD)):
        B.spd_set_kernel_timing(eng.h, kid)
        eng.spd_run_steps(8)
        eng.spd_sync()
        kms, kl = B.spd_kernel_timing(eng.h)
        shares[kname] = {"us_per_launch": 1e3 * kms / max(1, kl), "launches_per_step": kl / 8}
    B.spd_set_kernel_timing(eng.h, 0)
    shares["gateup"] = {"us_per_launch": 1e6 * gu_s, "launches_per_step": launches / Kt}
    log(f"[bench] gate/up: {1e6 * gu_s:.1f} us/launch, {gu_gbs:.0f} GB/s; kernels {shares}")

    # tokens/s at a seeded Bernoulli(0.7) acceptance pattern (rollback, refill exercised)
    p = wl.get("p_accept") or 0.7
    eng.spd_rollback(P, int(first))
    mask = synth.accept_mask(p, args.seed, max_tokens)
    table = np.full(len(ref), -1, dtype=np.int32)
    for i in range(1, len(ref)):
        q = P + i
        table[i] = ref[i] if mask[q] else (ref[i] + 1) % sh.vocab
    eng.spd_clear_forced_drafts()
    eng.spd_set_forced_drafts(table, P)
    Kp = K
    torch.cuda.synchronize()
    ts = time.perf_counter()
    logp = eng.spd_run_steps(Kp, want_log=True)
    elp = time.perf_counter() - ts
    committed = logp[-1]["committed_len"] - P
    spd_tok_s = committed / elp
    alpha = committed / Kp
    toks = eng.tokens()[P: logp[-1]["committed_len"] + 1]
    assert np.array_equal(toks, ref[: len(toks)]), "SPD stream differs from greedy decoding (p run)"
    log(f"[bench] p={p}: alpha={alpha:.3f}, {spd_tok_s:.0f} tok/s (AR {ar_tok_s:.0f} tok/s)")
    eng.close()

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
        "data": "synthetic (seeded N(0,0.02) weights, uniform-random prompt)",
        "graph": not args.no_graph,
        "config": {"workload": f"{sh.name}-class dense decoder, SPD width n={n}, PDM {sh.pdm_layers} layer, "
                               f"{P}-token prompt, steady-state full-pipeline steps",
                   "n": n, "layers": sh.n_layers, "d_model": sh.d_model, "prompt": P,
                   "pdm_layers": sh.pdm_layers, "global_batch": 1, "seq_len": P, "parallelism": "none"},
        "bytes_per_step": int(bytes_step),
        "step_GBps": round(gbs, 1),
        "step_roofline_frac": round(gbs / PEAK_HBM_GBS, 4),
        "roofline": {"bound": "hbm", "achieved": round(gu_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gu_gbs / PEAK_HBM_GBS, 4), "traffic": None,
                     "kernel": "k_gateup (grouped gate/up GEMV + SwiGLU over n stages)",
                     "bytes_per_launch": gu_bytes, "us_per_launch": round(1e6 * gu_s, 2)},
        "kernels": shares,
        "tokens_per_s": {"spd_forced_p": p, "alpha": round(alpha, 4), "spd": round(spd_tok_s, 1),
                         "ar_same_gpu": round(ar_tok_s, 1)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
