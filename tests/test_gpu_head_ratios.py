"""GPU lockstep against the oracle at other query-head to KV-head ratios (bf16): eight query heads per
KV head (the stage attention's eight-slot split; a prefill chunk of 8 rows and a draft module of 5
rows are more queries than one matrix-core tile holds, so they take the one-token split per row) and
plain multi-head attention (one query head per KV head), with rejections and natural drafts."""
import sys

import pytest

import synth
from oracle import model as om
from tests.lockstep import forced_table, run_lockstep

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 41


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("shape,n,p,chunk", [
    (synth.GQA8, 4, 0.6, 16), (synth.GQA8, 5, 0.7, 32), (synth.GQA8, 2, None, 16),
    (synth.MHA, 3, 0.6, 16), (synth.MHA, 1, None, 32)])
def test_lockstep_head_ratios(shape, n, p, chunk):
    from paper_2605_30852_amd.engine import DeviceWeights, Engine
    _say(f"[head ratios {shape.name} n={n} p={p} chunk={chunk}]")
    sh = shape.with_(n_stages=n)
    model = om.Model(sh, SEED)
    w = DeviceWeights(sh, SEED)
    prompt = synth.prompt(sh, SEED + n, 45)  # 45 rows: five 8-row prefill chunks and a ragged tail
    draft_for = None
    if p is not None:
        ref = om.ar_greedy(model, prompt, 30)
        mask = synth.accept_mask(p, SEED + n, 400)
        tab = forced_table(ref, mask, len(prompt), sh.vocab)
        draft_for = tab.get
    eng = Engine(w, max_tokens=200, n=n, attn_chunk=chunk, page_seed=7)
    res = run_lockstep(eng, model, prompt, 20, draft_for=draft_for)
    eng.close()
    _say(f"  compared {res['steps']} steps, worst {res}")
    assert res["steps"] == 20, res
