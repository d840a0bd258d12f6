"""The step log of spd_run_steps: the device keeps the last 4096 step results in a ring, and a call
that asks for its `count` results copies them out of the ring, also where they wrap past its end.
Checked against the same decoding logged in short calls that never wrap."""
import sys

import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 21
RING = 4096


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def test_log_across_the_ring_end():
    from paper_2605_30852_amd.engine import DeviceWeights, Engine
    w = DeviceWeights(synth.TINY, SEED)
    prompt = synth.prompt(synth.TINY, SEED, 20)
    pre, tail = RING - 96, 200  # the logged call covers steps RING - 95 .. RING + 104
    _say(f"[step log: {pre} steps, then {tail} logged across the ring end]")
    engs = [Engine(w, max_tokens=pre + tail + 64, n=2) for _ in range(2)]
    for e in engs:
        e.spd_prefill(prompt)
        e.spd_set_graph(True)
    a = engs[0]
    a.spd_run_steps(pre)
    log_a = a.spd_run_steps(tail, want_log=True)
    b = engs[1]
    log_b = []
    for _ in range((pre + tail) // 100):
        log_b += b.spd_run_steps(100, want_log=True)
    assert [r["step_index"] for r in log_a] == list(range(pre + 1, pre + tail + 1))
    assert log_a == log_b[pre:], "the wrapped log differs from the short calls' log"
    last = a.spd_sync()
    assert last.step_index == pre + tail and last.committed_len == log_a[-1]["committed_len"]
    assert np.array_equal(a.tokens(), b.tokens())
    for e in engs:
        e.close()
