"""GPU lockstep against the oracle for shapes whose prefill chunks take the K-split row GEMV: eight
prompt rows of the down projection's input (an FFN of 2304) do not fit the row GEMV's LDS budget at
full width, so each workgroup stages 1024-input chunks (here 1024, 1024 and a ragged 256) and the
column's last workgroup adds the chunks in order and runs the epilogue. Both weight types (fp32 and
bf16), a prompt of five full 8-row chunks and a ragged tail, rejections and natural drafts."""
import sys

import pytest

import synth
from oracle import model as om
from tests.lockstep import forced_table, run_lockstep

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 43
F32_WIDE_FFN = synth.TINY.with_(name="tiny-ffn2304", ffn_dim=2304)
BF16_WIDE_FFN = synth.MID.with_(name="mid-ffn2304", ffn_dim=2304)


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("shape,n,p", [(F32_WIDE_FFN, 2, 0.6), (F32_WIDE_FFN, 3, None),
                                       (BF16_WIDE_FFN, 3, 0.7), (BF16_WIDE_FFN, 2, None)])
def test_lockstep_with_k_split_prefill(shape, n, p):
    from paper_2605_30852_amd.engine import DeviceWeights, Engine
    _say(f"[K-split prefill {shape.name} n={n} p={p}]")
    sh = shape.with_(n_stages=n)
    model = om.Model(sh, SEED)
    w = DeviceWeights(sh, SEED)
    prompt = synth.prompt(sh, SEED + n, 45)
    draft_for = None
    if p is not None:
        ref = om.ar_greedy(model, prompt, 30)
        mask = synth.accept_mask(p, SEED + n, 400)
        draft_for = forced_table(ref, mask, len(prompt), sh.vocab).get
    eng = Engine(w, max_tokens=200, n=n, page_seed=9)
    res = run_lockstep(eng, model, prompt, 20, draft_for=draft_for)
    eng.close()
    _say(f"  compared {res['steps']} steps, worst {res}")
    assert res["steps"] == 20, res
