"""GPU lockstep against the oracle for the shortest prompts: one token (the prefill is a single row,
its first token comes straight from that row, and every cache starts one position long), exactly one
and two full 8-row prefill chunks (no ragged tail), at n up to L (one layer per stage), on the fp32
and bf16 models, with Bernoulli rejections (rollbacks to the one-token prompt) and natural drafts;
and a one-row prefill chunk through the K-split row GEMV (an FFN of 2304)."""
import sys

import pytest

import synth
from oracle import model as om
from tests.lockstep import forced_table, run_lockstep

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 47


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("shape,P,n,p", [
    (synth.TINY, 1, 2, 0.6), (synth.TINY, 1, 4, 0.6), (synth.TINY, 8, 3, 0.6), (synth.TINY, 16, 4, None),
    (synth.MID, 1, 3, 0.7), (synth.MID, 1, 2, None), (synth.MID, 8, 3, None),
    (synth.TINY.with_(name="tiny-ffn2304", ffn_dim=2304), 1, 2, 0.6)])
def test_lockstep_short_prompts(shape, P, n, p):
    from paper_2605_30852_amd.engine import DeviceWeights, Engine
    _say(f"[short prompt {shape.name} P={P} n={n} p={p}]")
    sh = shape.with_(n_stages=n)
    model = om.Model(sh, SEED)
    w = DeviceWeights(sh, SEED)
    prompt = synth.prompt(sh, SEED + P, P)
    draft_for = None
    if p is not None:
        ref = om.ar_greedy(model, prompt, 30)
        mask = synth.accept_mask(p, SEED + n, 400)
        draft_for = forced_table(ref, mask, len(prompt), sh.vocab).get
    eng = Engine(w, max_tokens=120, n=n, page_seed=13)
    res = run_lockstep(eng, model, prompt, 20, draft_for=draft_for)
    eng.close()
    _say(f"  compared {res['steps']} steps, worst {res}")
    assert res["steps"] == 20, res
