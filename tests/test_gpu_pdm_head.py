"""GPU parity of the PDM's own LM head over a smaller vocabulary (Section 4.1) through the C ABI.

Lockstep against the oracle's own-head PDM (its logits over the draft vocabulary, drafts mapped to
target tokens, and everything the pre-step lockstep checks), a 4B-class run in the benchmark's launch
form whose drafts are the mapped argmax of the HIP path's own PDM logits and whose stream is greedy
decoding bit for bit, and the argument checks at spd_init. (Sampled decoding with the own head is in
tests/test_gpu_sampling.py.)"""
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


@pytest.mark.parametrize("n,vd,forced", [(2, 300, False), (3, 300, True), (2, 1023, False)])
def test_tiny_own_head_lockstep(tiny_w, n, vd, forced):
    _say(f"[own PDM head tiny n={n} vocab={vd} forced={forced}]")
    w = tiny_w.with_pdm_vocab(vd)
    model = om.Model(w.shape, SEED)
    prompt = synth.prompt(w.shape, SEED, 21)
    draft_for = None
    if forced:
        ref = om.ar_greedy(model, prompt, 30)
        draft_for = forced_table(ref, synth.accept_mask(0.6, SEED + n, 200), len(prompt), w.shape.vocab).get
    eng = _engine(w, n)
    r = run_lockstep(eng, model, prompt, 18, draft_for=draft_for)
    eng.close()
    assert r["steps"] == 18, r
    assert r["hidden"] < 1e-4 and r["pdm_hidden"] < 1e-4


def test_mid_bf16_own_head_lockstep(mid_w):
    _say("[own PDM head mid n=3 vocab=1000]")
    w = mid_w.with_pdm_vocab(1000)
    model = om.Model(w.shape, SEED)
    prompt = synth.prompt(w.shape, SEED, 19)
    eng = _engine(w, 3)
    r = run_lockstep(eng, model, prompt, 14)
    eng.close()
    assert r["steps"] == 14, r


def test_own_head_argument_checks(tiny_w):
    from paper_2605_30852_amd.binding import SPDError
    w = tiny_w.with_pdm_vocab(300)
    with pytest.raises(SPDError):
        _engine(w, 2, fused_head=True)  # the two heads stream different weights
    bad = tiny_w.with_pdm_vocab(300)
    m = bad.t["pdm.vocab_map"].clone()
    m[7] = tiny_w.shape.vocab  # not a target token
    bad.t["pdm.vocab_map"] = m
    with pytest.raises(SPDError):
        _engine(bad, 2)


def test_fullsize_4b_own_head_drafts_and_lossless():
    """4B-class n = 4 with a 32768-token PDM vocabulary, stage groups and the step graph: each
    step's draft is the vocabulary map at the argmax (lowest draft id among equals) of the HIP path's
    own PDM logits, and the committed stream equals greedy decoding (n = 1) bit for bit."""
    from paper_2605_30852_amd.engine import DeviceWeights, Engine

    sh = synth.B4
    P, rows = 24, 160
    prompt = synth.prompt(sh, 0, P)
    _say("[own PDM head 4b] uploading weights")
    W = DeviceWeights(sh, 0, threads=16)
    ar = Engine(W, max_tokens=rows, n=1)
    ar.spd_set_graph(True)
    ar.spd_prefill(prompt)
    ar.spd_run_steps(40)
    ar.spd_sync()
    ref = list(ar.tokens()[P: P + 41])
    ar.close()
    Wv = W.with_pdm_vocab(32768)
    vmap = synth.pdm_vocab_map(Wv.shape, 0)
    eng = Engine(Wv, max_tokens=rows, n=sh.n_stages)
    eng.spd_set_graph(True)
    eng.spd_set_debug(True)
    eng.spd_prefill(prompt)
    for i in range(20):
        r = eng.spd_run_steps(1, want_log=True)[0]
        pl = eng.pdm_logits().astype(np.float32)
        assert pl.shape == (32768,)
        best = int(np.nonzero(pl == pl.max())[0][0])
        assert r["pdm_draft"] == int(vmap[best]), f"step {i}"
    c = eng.state()[0]
    toks = list(eng.tokens()[P: c + 1])
    assert toks == ref[: len(toks)]
    eng.close()
    _say(f"[own PDM head 4b] {len(toks)} tokens committed")
