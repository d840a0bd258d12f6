"""GPU parity of the post-step PDM schedule (the ablation of Section 4.5) through the C ABI.

The PDM then runs after the step's stage compute and reads every in-flight token one stage deeper.
Lockstep against the oracle's post-step schedule (PDM rows, PDM logits, drafts, exit logits and
decisions, tolerances as for the pre-step schedule); at n = 1 the two schedules are bit-identical on
the GPU; and at the 4B-class size in the benchmark's launch form (stage groups, step graph) the
post-step stream with the PDM's own drafts is plain greedy decoding bit for bit."""
import sys

import numpy as np
import pytest

import synth
from oracle import model as om
from tests.lockstep import forced_table, run_lockstep

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 11


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def tiny_w():
    from paper_2605_30852_amd.engine import DeviceWeights
    return DeviceWeights(synth.TINY, SEED)


@pytest.fixture(scope="module")
def mid_w():
    from paper_2605_30852_amd.engine import DeviceWeights
    return DeviceWeights(synth.MID, SEED)


def _engine(w, n, max_tokens=160, **kw):
    from paper_2605_30852_amd.engine import Engine
    return Engine(w, max_tokens=max_tokens, n=n, page_seed=5, **kw)


@pytest.mark.parametrize("n,forced", [(2, False), (3, False), (4, False), (3, True)])
def test_tiny_post_step_lockstep(tiny_w, n, forced):
    _say(f"[post-step tiny lockstep n={n} forced={forced}]")
    sh = synth.TINY
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED, 23)
    draft_for = None
    if forced:
        ref = om.ar_greedy(model, prompt, 30)
        tab = forced_table(ref, synth.accept_mask(0.6, SEED + n, 200), len(prompt), sh.vocab)
        draft_for = tab.get
    eng = _engine(tiny_w, n)
    w = run_lockstep(eng, model, prompt, 20, draft_for=draft_for, schedule="post")
    eng.close()
    assert w["steps"] == 20, w
    assert w["hidden"] < 1e-4 and w["pdm_hidden"] < 1e-4  # fp32 weights and KV


@pytest.mark.parametrize("fused", [True, False])
def test_mid_bf16_post_step_lockstep(mid_w, fused):
    _say(f"[post-step mid lockstep fused_head={fused}]")
    sh = synth.MID
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED, 19)
    eng = _engine(mid_w, 3, fused_head=fused)
    w = run_lockstep(eng, model, prompt, 14, schedule="post")
    eng.close()
    assert w["steps"] == 14, w


def test_n1_post_step_bit_identical_to_pre_step(mid_w):
    prompt = synth.prompt(synth.MID, SEED, 17)
    logs = []
    for post in (False, True):
        eng = _engine(mid_w, 1)
        eng.spd_set_pdm_schedule(post)
        x = eng.spd_prefill(prompt)
        logs.append(([x] + [eng.spd_step().as_dict() for _ in range(16)], list(eng.tokens())))
        eng.close()
    assert logs[0] == logs[1]


def test_fullsize_4b_post_step_natural_drafts_lossless():
    """4B-class n = 4 with the PDM's own drafts under the post-step schedule, stage groups and the
    step graph: the committed stream equals greedy decoding (n = 1, same library) bit for bit, and the
    schedule changes the drafts (the pre-step run of the same prompt drafts differently somewhere)."""
    from paper_2605_30852_amd.engine import DeviceWeights, Engine

    sh = synth.B4
    P, rows = 24, 160
    prompt = synth.prompt(sh, 0, P)
    _say("[post-step 4b] uploading weights")
    W = DeviceWeights(sh, 0, threads=16)
    ar = Engine(W, max_tokens=rows, n=1)
    ar.spd_set_graph(True)
    ar.spd_prefill(prompt)
    ar.spd_run_steps(40)
    ar.spd_sync()
    ref = list(ar.tokens()[P: P + 41])
    ar.close()
    drafts = {}
    for post in (False, True):
        eng = Engine(W, max_tokens=rows, n=sh.n_stages)
        eng.spd_set_pdm_schedule(post)
        eng.spd_set_graph(True)
        eng.spd_prefill(prompt)
        log = eng.spd_run_steps(24, want_log=True)
        c = log[-1]["committed_len"]
        toks = list(eng.tokens()[P: c + 1])
        assert toks == ref[: len(toks)], f"post_step={post}: stream differs from greedy decoding"
        drafts[post] = [r["pdm_draft"] for r in log]
        eng.close()
    _say(f"[post-step 4b] drafts differ at {sum(a != b for a, b in zip(drafts[False], drafts[True]))} of 24 steps")
    assert drafts[False] != drafts[True]
