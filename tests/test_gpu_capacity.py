"""Capacity limits on a live handle: spd_prefill, spd_step and spd_run_steps return SPD_E_CAPACITY when
the positions they would fill exceed max_tokens, and leave the handle as it was (device state, tokens,
in-flight rows), so that the caller can go on with a call that fits."""
import sys

import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 3


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def tiny_w():
    from paper_2605_30852_amd.engine import DeviceWeights
    return DeviceWeights(synth.TINY, SEED)


def _snapshot(eng):
    return eng.state(), eng.tokens().copy(), eng.resid().copy()


def _same(a, b):
    assert a[0] == b[0]
    assert np.array_equal(a[1], b[1])
    assert np.array_equal(a[2], b[2])


def test_prefill_over_capacity_leaves_the_handle_unchanged(tiny_w):
    from paper_2605_30852_amd import binding as B
    from paper_2605_30852_amd.engine import Engine
    _say("[capacity: prefill]")
    n, cap = 2, 40
    eng = Engine(tiny_w, max_tokens=cap, n=n)
    before = eng.state()
    # a prompt needs room for itself, the pipeline (n) and the first token
    with pytest.raises(B.SPDError) as e:
        eng.spd_prefill(synth.prompt(synth.TINY, SEED, cap - n))
    assert e.value.status == B.SPD_E_CAPACITY
    assert eng.state() == before
    first = eng.spd_prefill(synth.prompt(synth.TINY, SEED, cap - n - 1))  # the largest that fits
    assert 0 <= first < synth.TINY.vocab
    eng.close()


@pytest.mark.parametrize("n", [1, 3])
def test_step_and_run_steps_over_capacity(tiny_w, n):
    from paper_2605_30852_amd import binding as B
    from paper_2605_30852_amd.engine import Engine
    _say(f"[capacity: step / run_steps n={n}]")
    cap, P = 48, 20
    eng = Engine(tiny_w, max_tokens=cap, n=n)
    eng.spd_prefill(synth.prompt(synth.TINY, SEED + n, P))
    eng.spd_set_forced_drafts(np.full(cap, 5, dtype=np.int32), 0)  # every draft accepted or not, all fit
    # run_steps is refused when c + a could pass max_tokens within `count` steps
    c, a, _, _ = eng.state()
    room = cap - (c + a)
    snap = _snapshot(eng)
    with pytest.raises(B.SPDError) as e:
        eng.spd_run_steps(room + 1)
    assert e.value.status == B.SPD_E_CAPACITY
    _same(snap, _snapshot(eng))
    eng.spd_run_steps(room // 2)
    eng.spd_sync()
    # single steps until the next one would push past the last position
    steps = 0
    while True:
        c, a, _, _ = eng.state()
        snap = _snapshot(eng)
        if c + a >= cap:
            with pytest.raises(B.SPDError) as e:
                eng.spd_step()
            assert e.value.status == B.SPD_E_CAPACITY
            _same(snap, _snapshot(eng))
            break
        eng.spd_step()
        steps += 1
        assert steps < 4 * cap
    # a rollback frees positions and decoding goes on
    eng.spd_rollback(P + 1, 7)
    r = eng.spd_step()
    assert r.committed_len >= P + 1
    eng.close()
