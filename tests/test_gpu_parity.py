"""GPU parity: the HIP path through the C ABI against the CPU oracle, step by step, and the lossless
greedy invariant of the GPU path itself (SPD token ids and decisions bit-exact against the GPU's
plain greedy decode, i.e. the same library at n = 1)."""
import sys

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import spd as osp
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
    return Engine(w, max_tokens=max_tokens, n=n, page_seed=kw.pop("page_seed", 5), **kw)


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_tiny_fp32_lockstep_forced(tiny_w, n):
    _say(f"[tiny lockstep forced n={n}]")
    sh = synth.TINY
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED, 37)  # 37 rows: several 8-row prefill chunks and a ragged tail
    ref = om.ar_greedy(model, prompt, 30)
    mask = synth.accept_mask(0.7, SEED, 200)
    tab = forced_table(ref, mask, len(prompt), sh.vocab)
    eng = _engine(tiny_w, n)
    w = run_lockstep(eng, model, prompt, 24, draft_for=lambda q: tab.get(q))
    eng.close()
    assert w["steps"] == 24, w
    assert w["hidden"] < 1e-4  # fp32 weights and KV: only summation order differs


@pytest.mark.parametrize("n,fused", [(2, True), (2, False)])
def test_tiny_fp32_lockstep_natural_drafts(tiny_w, n, fused):
    _say(f"[tiny lockstep natural n={n} fused_head={fused}]")
    sh = synth.TINY
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED, 20)
    eng = _engine(tiny_w, n, fused_head=fused)
    w = run_lockstep(eng, model, prompt, 16)
    eng.close()
    assert w["steps"] == 16, w


@pytest.mark.parametrize("n,fused", [(1, True), (3, True), (3, False)])
def test_mid_bf16_lockstep(mid_w, n, fused):
    """bf16 weights and KV, ragged FFN (1000) and vocabulary (3001), chunked attention splits; the
    draft module's LM head fused with the exit pass or run as its own pass."""
    _say(f"[mid lockstep n={n} fused_head={fused}]")
    sh = synth.MID
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED, 75)
    ref = om.ar_greedy(model, prompt, 24)
    mask = synth.accept_mask(0.6, SEED + 1, 300)
    tab = forced_table(ref, mask, len(prompt), sh.vocab)
    eng = _engine(mid_w, n, max_tokens=200, attn_chunk=32, fused_head=fused)
    w = run_lockstep(eng, model, prompt, 20, draft_for=lambda q: tab.get(q))
    eng.close()
    assert w["steps"] == 20, w


def _gpu_stream(w, n, prompt, steps, table=None, max_tokens=400, **kw):
    eng = _engine(w, n, max_tokens=max_tokens, **kw)
    first = eng.spd_prefill(prompt)
    if table is not None:
        base = len(prompt)
        arr = np.full(len(table) + 8, -1, dtype=np.int32)
        for q, t in table.items():
            arr[q - base] = t
        eng.spd_set_forced_drafts(arr, base)
    res = [eng.spd_step().as_dict() for _ in range(steps)]
    toks = eng.tokens()
    c = res[-1]["committed_len"]
    eng.close()
    return first, list(toks[len(prompt): c + 1]), res


@pytest.mark.parametrize("which", ["tiny", "mid"])
@pytest.mark.parametrize("p", [None, 0.7, 1.0])
def test_lossless_gpu_spd_equals_gpu_greedy(tiny_w, mid_w, which, p):
    """Token ids and decisions of the GPU's own SPD run are bit-exact against the GPU's plain greedy
    decode (n = 1 through the same library), for natural and forced drafts."""
    w = tiny_w if which == "tiny" else mid_w
    sh = w.shape
    prompt = synth.prompt(sh, SEED + 3, 29)
    _say(f"[lossless {which} p={p}] AR reference")
    first, ar, _ = _gpu_stream(w, 1, prompt, 40, max_tokens=200)
    for n in (2, 3, 4):
        _say(f"[lossless {which} p={p}] n={n}")
        table = None
        mask = None
        if p is not None:
            mask = synth.accept_mask(p, SEED + n, 400)
            table = forced_table(ar, mask, len(prompt), sh.vocab)
        f2, toks, res = _gpu_stream(w, n, prompt, 40, table, max_tokens=200)
        assert f2 == first == ar[0]
        m = len(toks)
        assert m >= 2
        assert toks == ar[:m], f"n={n}: SPD stream differs from greedy"
        if p is not None:
            for r in res:
                if r["decision"] != 0:
                    assert r["decision"] == (1 if mask[r["verified_pos"]] else 2)
            K = osp.simulate_steps(n, m, lambda q: bool(mask[q]), len(prompt))
            assert len(res) >= K


def test_run_steps_matches_step_by_step(mid_w):
    _say("[run_steps]")
    sh = mid_w.shape
    prompt = synth.prompt(sh, SEED + 4, 40)
    first, ar, _ = _gpu_stream(mid_w, 1, prompt, 30, max_tokens=200)
    mask = synth.accept_mask(0.7, 99, 400)
    table = forced_table(ar, mask, len(prompt), sh.vocab)
    _, toks_a, res_a = _gpu_stream(mid_w, 3, prompt, 24, table, max_tokens=200)
    eng = _engine(mid_w, 3, max_tokens=200)
    eng.spd_prefill(prompt)
    arr = np.full(len(table) + 8, -1, dtype=np.int32)
    for q, t in table.items():
        arr[q - len(prompt)] = t
    eng.spd_set_forced_drafts(arr, len(prompt))
    log = eng.spd_run_steps(24, want_log=True)
    assert [r["decision"] for r in log] == [r["decision"] for r in res_a]
    assert [r["committed_len"] for r in log] == [r["committed_len"] for r in res_a]
    eng.close()


def test_rollback_api_and_state_errors(tiny_w):
    """spd_rollback to an earlier length continues like the oracle does after the same rollback;
    illegal call orders return SPD_E_STATE."""
    from paper_2605_30852_amd import binding as B
    sh = synth.TINY
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED + 5, 16)
    eng = _engine(tiny_w, 2, auto_rollback=False)
    with pytest.raises(B.SPDError) as e:
        eng.spd_step()
    assert e.value.status == B.SPD_E_STATE
    ora = osp.SPDOracle(model, n=2)
    assert eng.spd_prefill(prompt) == ora.prefill(prompt)
    with pytest.raises(B.SPDError) as e:
        eng.spd_prefill(prompt)
    assert e.value.status == B.SPD_E_STATE
    # natural drafts with random weights reject: the handle then waits for spd_rollback
    pending = False
    for _ in range(6):
        r = eng.spd_step()
        ro = ora.step()
        assert r.decision == ro.decision
        if r.decision == B.SPD_REJECT:
            pending = True
            with pytest.raises(B.SPDError) as e:
                eng.spd_step()
            assert e.value.status == B.SPD_E_STATE
            eng.spd_rollback(r.committed_len, r.target_argmax)
    assert pending
    # explicit rollback to an earlier length with another token
    keep = ora.c - 1
    with pytest.raises(B.SPDError):
        eng.spd_rollback(len(prompt) - 1, 3)  # below the prompt
    eng.spd_rollback(keep, 17)
    ora.rollback(keep, 17)
    eng.spd_set_debug(True)
    for _ in range(4):
        r = eng.spd_step()
        ro = ora.step()
        if r.decision == B.SPD_REJECT:
            eng.spd_rollback(r.committed_len, r.target_argmax)
        res = eng.resid()
        for q in range(ora.c, ora.c + ora.a):
            assert np.linalg.norm(res[q % 2] - ora.hidden[q]) <= 2e-2 * np.linalg.norm(ora.hidden[q])
    eng.close()


@pytest.mark.parametrize("mode,groups,place,post,graph_steps", [
    (2, -1, 0, False, 1), (2, -1, 0, False, 4), (2, 3, 0, False, 1), (2, 2, 1, False, 1), (2, 2, 2, False, 1),
    (2, 2, 3, False, 1), (0, -1, 0, False, 1), (0, -1, 1, False, 1), (2, -1, 0, True, 1)])
def test_graph_replay_matches_eager(mid_w, mode, groups, place, post, graph_steps):
    """Steps replayed from the captured step graph (graph_steps steps per graph, and the one-step
    graph for the remainder; the stage groups' and the draft module's streams as its branches,
    wherever the draft module is placed) give the same bits as launched steps, on every replay, with
    eager work and synchronisation between the replays; under the post-step schedule too."""
    _say(f"[graph replay mode={mode} groups={groups} pdm place={place} post_step={post} steps/graph={graph_steps}]")
    sh = mid_w.shape
    prompt = synth.prompt(sh, SEED + 6, 33)
    first, ar, _ = _gpu_stream(mid_w, 1, prompt, 30, max_tokens=200)
    mask = synth.accept_mask(0.7, 123, 400)
    table = forced_table(ar, mask, len(prompt), sh.vocab)
    arr = np.full(len(table) + 8, -1, dtype=np.int32)
    for q, t in table.items():
        arr[q - len(prompt)] = t
    engs = []
    for graph in (False, True):
        e = _engine(mid_w, 3, max_tokens=200)
        e.spd_set_step_kernel(mode, 0, groups if mode == 2 else -1)
        e.spd_set_pdm_placement(place)
        e.spd_set_pdm_schedule(post)
        assert e.spd_prefill(prompt) == first
        e.spd_set_forced_drafts(arr, len(prompt))
        e.spd_set_graph(graph)
        if graph:
            e.spd_set_graph_steps(graph_steps)
        engs.append(e)
    steps = 0
    for chunk in range(4):
        logs = [e.spd_run_steps(6, want_log=True) for e in engs]
        assert logs[0] == logs[1], f"replay chunk {chunk} differs"
        steps += 6
        r0, r1 = engs[0].resid(), engs[1].resid()
        assert np.array_equal(r0, r1)
        assert np.array_equal(engs[0].pdm_hidden(), engs[1].pdm_hidden())
        # one launched (non-graph) step on the graph engine in between replays
        if chunk == 1:
            for e in engs:
                e.spd_step(int(table.get(e.state()[0] + e.state()[1], 0)))
            steps += 1
    assert np.array_equal(engs[0].tokens(), engs[1].tokens())
    assert engs[0].state() == engs[1].state() and engs[0].state()[3] == steps
    for e in engs:
        e.close()


@pytest.mark.parametrize("which,n,groups,place", [
    ("mid", 3, -1, 0), ("tiny", 4, -1, 0), ("mid", 1, -1, 0), ("mid", 3, 3, 0), ("tiny", 4, 4, 0),
    ("tiny", 4, 3, 0), ("mid", 3, 1, 0), ("tiny", 4, 2, 1), ("mid", 3, 2, 2), ("tiny", 4, 4, 3)])
def test_stage_groups_bit_identical_to_sublayer_launches(tiny_w, mid_w, which, n, groups, place):
    """Stage groups on their own streams (mode 2 with `groups` groups; -1: the default) give the same
    bits as five launches per layer slot on one stream covering all stages (mode 0): decisions,
    tokens, in-flight residual streams and anchors after every step, with the draft module on its own
    stream, on main_stream before the stages, or on the first group's stream before or after its
    stages (place 0-3)."""
    _say(f"[stage groups vs one stream {which} n={n} groups={groups} pdm place={place}]")
    w = tiny_w if which == "tiny" else mid_w
    sh = w.shape
    prompt = synth.prompt(sh, SEED + 7, 41)
    first, ar, _ = _gpu_stream(w, 1, prompt, 30, max_tokens=200)
    mask = synth.accept_mask(0.6, 321 + n, 400)
    table = forced_table(ar, mask, len(prompt), sh.vocab)
    arr = np.full(len(table) + 8, -1, dtype=np.int32)
    for q, t in table.items():
        arr[q - len(prompt)] = t
    engs = []
    for m in (0, 2):
        e = _engine(w, n, max_tokens=200, attn_chunk=32)
        e.spd_set_step_kernel(m, 0, groups if m == 2 else -1)
        if m == 2:
            e.spd_set_pdm_placement(place)
        assert e.spd_prefill(prompt) == first
        e.spd_set_forced_drafts(arr, len(prompt))
        engs.append(e)
    for i in range(18):
        logs = [e.spd_run_steps(1, want_log=True) for e in engs]
        assert logs[0] == logs[1], f"step {i}: {logs}"
        c, a, _, _ = engs[0].state()
        assert engs[1].state()[:2] == (c, a)
        r0, r1 = engs[0].resid(), engs[1].resid()
        an0, an1 = engs[0].anchors(), engs[1].anchors()
        # only rows of in-flight tokens hold data (the rest of the workspace is uninitialised), and a
        # token at depth k has anchors 0..k
        for q in range(c, c + a):
            k = c + a - 1 - q
            assert np.array_equal(r0[q % n], r1[q % n]), f"step {i}: residual stream of position {q} differs"
            assert np.array_equal(an0[q % n, : min(k, n - 1) + 1], an1[q % n, : min(k, n - 1) + 1]), \
                f"step {i}: anchors of position {q} differ"
    assert np.array_equal(engs[0].tokens(), engs[1].tokens())
    for e in engs:
        e.close()


def test_pdm_disabled_with_forced_drafts_is_bit_identical(mid_w):
    """With every draft forced, skipping the PDM's launches (spd_set_pdm_enabled(0), used to measure
    how much of the PDM the stage compute hides) changes nothing on the target path: decisions,
    tokens, residual streams and anchors match a run with the PDM, bit for bit."""
    from paper_2605_30852_amd import binding as B
    sh = mid_w.shape
    prompt = synth.prompt(sh, SEED + 11, 29)
    first, ar, _ = _gpu_stream(mid_w, 1, prompt, 24, max_tokens=200)
    mask = synth.accept_mask(0.6, SEED + 12, 400)
    table = forced_table(ar, mask, len(prompt), sh.vocab)
    arr = np.full(len(table) + 8, -1, dtype=np.int32)
    for q, t in table.items():
        arr[q - len(prompt)] = t
    engs = []
    for on in (True, False):
        e = _engine(mid_w, 3, max_tokens=200, attn_chunk=32)
        B.spd_set_pdm_enabled(e.h, on)
        assert e.spd_prefill(prompt) == first
        e.spd_set_forced_drafts(arr, len(prompt))
        engs.append(e)
    for i in range(14):
        logs = [e.spd_run_steps(1, want_log=True)[0] for e in engs]
        for r in logs:
            r.pop("pdm_draft", None)
        assert logs[0] == logs[1], f"step {i}"
        c, a, _, _ = engs[0].state()
        for q in range(c, c + a):
            assert np.array_equal(engs[0].resid()[q % 3], engs[1].resid()[q % 3])
    assert np.array_equal(engs[0].tokens(), engs[1].tokens())
    for e in engs:
        e.close()


@pytest.mark.parametrize("chunk", [256, 384])
def test_multi_pass_attention_splits(mid_w, chunk):
    """Key splits longer than one 128-key pass (online softmax across passes inside a split, the
    next pass's keys loaded while the current one is computed): oracle parity and the lossless
    invariant against the GPU's plain greedy decode with the same split size."""
    _say(f"[multi-pass attention chunk={chunk}]")
    sh = synth.MID
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED + 8, 300)  # 300+ keys: splits of 2-3 passes and a ragged last split
    ref = om.ar_greedy(model, prompt, 16)
    mask = synth.accept_mask(0.6, SEED + 9, 600)
    tab = forced_table(ref, mask, len(prompt), sh.vocab)
    eng = _engine(mid_w, 3, max_tokens=400, attn_chunk=chunk)
    w = run_lockstep(eng, model, prompt, 12, draft_for=lambda q: tab.get(q))
    eng.close()
    assert w["steps"] == 12, w
    first, ar, _ = _gpu_stream(mid_w, 1, prompt, 20, max_tokens=400, attn_chunk=chunk)
    table = forced_table(ar, mask, len(prompt), sh.vocab)
    f2, toks, res = _gpu_stream(mid_w, 3, prompt, 20, table, max_tokens=400, attn_chunk=chunk)
    assert f2 == first
    assert toks == ar[: len(toks)], "SPD stream differs from greedy decoding"
