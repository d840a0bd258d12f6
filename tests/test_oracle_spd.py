"""Pins for the oracle's SPD step (CPU only).

The step's output stream has a plain definition (greedy SPD is lossless: Section 3.4), its internal
states have a brute-force definition (every in-flight state equals a no-cache forward of the same
prefix truncated at that depth), and its bookkeeping is fixed by the paper's equations (depth
staircase Eq. steady-g / Eq. warmup-g, anchor eligibility Eq. depth-to-type, the worked example of
Figure 1, rollback length t-n+1 of Section 3.4)."""
import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import spd as osp

SEED = 5
SH = synth.TINY
PROMPT = synth.prompt(SH, SEED, 12)


@pytest.fixture(scope="module")
def model():
    return om.Model(SH, SEED)


@pytest.fixture(scope="module")
def ar_ref(model):
    return om.ar_greedy(model, PROMPT, 24, return_logits=True)


def _forced(ref, p, seed, n_prompt):
    mask = synth.accept_mask(p, seed, n_prompt + len(ref) + 8)
    table = {n_prompt + i: (ref[i] if mask[n_prompt + i] else (ref[i] + 1) % SH.vocab) for i in range(len(ref))}
    return (lambda q: table.get(q)), mask


def test_n1_step_is_plain_greedy(model, ar_ref):
    ref, ref_logits = ar_ref
    o = osp.SPDOracle(model, n=1)
    assert o.prefill(PROMPT) == ref[0]
    for i in range(1, 12):
        r = o.step(want_logits=True)
        assert r.decision in (osp.ACCEPT, osp.REJECT)
        assert r.verified_token == ref[i]
        np.testing.assert_array_equal(r.exit_logits, ref_logits[i])  # bit-exact: same code path
    assert o.generated() == ref[:12]
    assert o.steps == 11 and o.verified == 12


@pytest.mark.parametrize("n", [2, 3, 4])
@pytest.mark.parametrize("p", [None, 0.0, 0.5, 0.7, 1.0])
def test_lossless_greedy(model, ar_ref, n, p):
    ref, _ = ar_ref
    draft_for = None
    if p is not None:
        draft_for, mask = _forced(ref, p, 100 + n, len(PROMPT))
    o, res = osp.run_spd(model, PROMPT, 16, n=n, draft_for=draft_for)
    assert o.generated() == ref[:16]
    if p is not None:
        # decisions at exit steps equal the mask bit of the position being verified
        for r in res:
            if r.decision != osp.NONE:
                assert r.decision == (osp.ACCEPT if mask[r.verified_pos] else osp.REJECT)
        # and the step count equals the pipeline timing simulator's
        assert len(res) == osp.simulate_steps(n, 16, lambda q: bool(mask[q]), len(PROMPT))
    if p == 1.0:
        assert all(r.decision in (osp.NONE, osp.ACCEPT) for r in res)
        assert len(res) == n - 1 + 15


@pytest.mark.parametrize("n", [2, 3, 4])
def test_inflight_states_equal_brute_force(model, ar_ref, n):
    """Every in-flight hidden state and every stored anchor equals the no-cache forward of the same
    prefix, truncated at the token's depth."""
    ref, _ = ar_ref
    draft_for, _ = _forced(ref, 0.6, 7 + n, len(PROMPT))
    o = osp.SPDOracle(model, n=n)
    o.prefill(PROMPT)
    beta = o.beta
    checked = 0
    for _ in range(10):
        o.step(forced_draft=draft_for(o.c + o.a))
        q_last = o.c + o.a - 1
        full = om.forward_full(model, o.toks[: q_last + 1])
        for q in range(o.c, o.c + o.a):
            k = o.depth(q)
            np.testing.assert_allclose(o.hidden[q], full[beta[k]][q], rtol=1e-9, atol=1e-11)
            for j, an in enumerate(o.anch[q]):
                np.testing.assert_allclose(an, full[beta[j]][q], rtol=1e-9, atol=1e-11)
            assert len(o.anch[q]) == min(k, n - 1) + 1
            checked += 1
    assert checked > 10


def test_ragged_stage_split():
    assert osp.stage_bounds(4, 3) == [0, 1, 2, 4]
    assert osp.stage_bounds(36, 8) == [0, 4, 9, 13, 18, 22, 27, 31, 36]
    assert osp.stage_bounds(36, 6) == [0, 6, 12, 18, 24, 30, 36]
    assert osp.stage_bounds(36, 4) == [0, 9, 18, 27, 36]


def test_anchor_eligibility_paper_anchors():
    """Eq. depth-to-type with the paper's own anchor set [0, 8, 16, 24, 31] for L = 32:
    l_max(k) = min(32, 32k/n); n = 4 gives l_max = 0, 8, 16, 24, 32 and so f = 0, 1, 2, 3, 4;
    n = 8 gives l_max = 0, 4, 8, ..., 32 and so f = 0, 0, 1, 1, 2, 2, 3, 3, 4."""
    B = [0, 8, 16, 24, 31]
    assert [osp.eligible_anchors(k, B, 32, 4) for k in range(5)] == [0, 1, 2, 3, 4]
    assert [osp.eligible_anchors(k, B, 32, 8) for k in range(9)] == [0, 0, 1, 1, 2, 2, 3, 3, 4]
    # with the stage inputs as anchors, a token at depth k sees min(k, n-1) + 1 anchors
    for L, n in [(4, 2), (4, 3), (36, 4), (36, 8), (32, 16)]:
        b = osp.stage_bounds(L, n)[:n]
        assert [osp.eligible_anchors(k, b, L, n) for k in range(n + 1)] == [min(k, n - 1) for k in range(n + 1)]


@pytest.mark.parametrize("n", [2, 4])
def test_depth_staircase(model, ar_ref, n):
    """Pre-step depths equal Eq. steady-g (a = n) and Eq. warmup-g (a < n), and agree with the
    structural mask of Appendix A.3 read from the newest token (query depth 0): the key at
    distance t-T has depth min(n, t-T) while t-T < fill, and the deepest depth otherwise."""
    ref, _ = ar_ref
    draft_for, _ = _forced(ref, 0.5, 3, len(PROMPT))
    o = osp.SPDOracle(model, n=n)
    o.prefill(PROMPT)
    seen_full = seen_warm = False
    for _ in range(14):
        a, c = o.a, o.c
        r = o.step(forced_draft=draft_for(c + a))
        t = c + a - 1
        dep = [r.depths[q] for q in range(t + 1)]
        expect = [n] * (t + 1 - a) + list(range(a - 1, -1, -1))
        assert dep == expect
        for T in range(t + 1):
            assert dep[T] == (min(n, t - T) if t - T < a else n)
        seen_full |= a == n
        seen_warm |= a < n
    assert seen_full and seen_warm


def test_kv_lengths_ragged_and_rollback(model, ar_ref):
    ref, _ = ar_ref
    n = 3
    draft_for, _ = _forced(ref, 0.7, 9, len(PROMPT))
    o = osp.SPDOracle(model, n=n)
    o.prefill(PROMPT)
    for _ in range(12):
        lens = o.kv_lengths()
        for s in range(n):
            for l in range(o.beta[s], o.beta[s + 1]):
                assert lens[l] == o.c + max(0, o.a - 1 - s)
        o.step(forced_draft=draft_for(o.c + o.a))
    keep = o.c - 2
    o.rollback(keep, 5)
    assert o.kv_lengths() == [keep] * SH.n_layers
    assert all(pc.n == keep for pc in o.pdm_caches)
    assert o.a == 1 and o.toks[keep] == 5 and len(o.toks) == keep + 1


def test_figure1_worked_indices(model, ar_ref):
    """n = 4, saturated cycle: in-flight x_{t-3}..x_t (1-indexed). x_{t-3} exits and its logits judge
    x_{t-2}; on accept the draft x_{t+1} enters stage 1; on reject the target KV keeps t-n+1 tokens."""
    ref, _ = ar_ref
    n = 4
    for accept in (True, False):
        o = osp.SPDOracle(model, n=n)
        o.prefill(PROMPT)
        for _ in range(n - 1):  # fill the pipeline with correct drafts
            o.step(forced_draft=ref[o.c + o.a - len(PROMPT)])
        assert o.a == n
        t = o.c + n  # 1-indexed position of the newest in-flight token
        q_draft = o.c + o.a
        fd = ref[q_draft - len(PROMPT)] if accept else (ref[q_draft - len(PROMPT)] + 1) % SH.vocab
        if not accept:  # make the token under verification (x_{t-2}) wrong instead
            o.toks[o.c + 1] = (o.toks[o.c + 1] + 1) % SH.vocab
        r = o.step(forced_draft=fd)
        assert r.exited_pos + 1 == t - 3 and r.verified_pos + 1 == t - 2
        if accept:
            assert r.decision == osp.ACCEPT and o.a == n and o.depth(t) == 0 and o.toks[t] == fd
        else:
            assert r.decision == osp.REJECT
            assert o.kv_lengths() == [t - n + 1] * SH.n_layers
            assert o.a == 1 and o.toks[t - n + 1] == r.target_argmax


def test_rollback_history_independence(model, ar_ref):
    """Rolling back to keep_len and continuing gives the same states, bit for bit, as a fresh
    prefill of the kept prefix followed by the same reseed."""
    ref, _ = ar_ref
    n = 3
    draft_for, _ = _forced(ref, 0.8, 21, len(PROMPT))
    o = osp.SPDOracle(model, n=n)
    o.prefill(PROMPT)
    for _ in range(9):
        o.step(forced_draft=draft_for(o.c + o.a))
    keep = o.c - 1
    o.rollback(keep, 77)
    f = osp.SPDOracle(model, n=n)
    f.prefill(o.toks[:keep])
    f.rollback(keep, 77)
    for _ in range(6):
        q = o.c + o.a
        ra, rb = o.step(forced_draft=draft_for(q)), f.step(forced_draft=draft_for(q))
        assert (ra.decision, ra.target_argmax, ra.pdm_draft) == (rb.decision, rb.target_argmax, rb.pdm_draft)
        assert o.toks == f.toks
        for q in o.hidden:
            np.testing.assert_array_equal(o.hidden[q], f.hidden[q])
        for i, (pa, pb) in enumerate(zip(o.pdm_caches, f.pdm_caches)):
            np.testing.assert_array_equal(pa.k[: pa.n], pb.k[: pb.n])


def test_pdm_closed_form_identity_path():
    """W_in = [I, 0, ...] and zero PDM W_o, W_d: the PDM passes the newest token's embedding
    through unchanged, so the draft is argmax W_lm . rmsnorm(E[x_newest])."""
    d, n = SH.d_model, 2
    ov = {"pdm.in": np.concatenate([np.eye(d), np.zeros((d, d))], axis=1),
          "pdm.layer.0.wo": np.zeros((d, SH.q_dim)), "pdm.layer.0.wd": np.zeros((d, SH.ffn_dim))}
    m = om.Model(SH, SEED, overrides=ov)
    o = osp.SPDOracle(m, n=n)
    o.prefill(PROMPT)
    E, W = m.w("embed"), m.w("lm_head")
    for _ in range(6):
        newest = o.toks[o.c + o.a - 1]
        x = E[newest]
        expect = int(np.argmax(W @ (x / np.sqrt(np.mean(x * x) + SH.rms_eps))))
        r = o.step()
        assert r.pdm_draft == expect


def test_pdm_anchor_selection_zero_fill():
    """W_in selecting only anchor 1 (and zero PDM W_o, W_d): a row sees H^{beta_1} if its depth is at
    least 1 and zero otherwise; the newest row is all zeros, so the draft is token 0."""
    d, n = SH.d_model, 2
    ov = {"pdm.in": np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1),
          "pdm.layer.0.wo": np.zeros((d, SH.q_dim)), "pdm.layer.0.wd": np.zeros((d, SH.ffn_dim))}
    m = om.Model(SH, SEED, overrides=ov)
    o = osp.SPDOracle(m, n=n)
    o.prefill(PROMPT)
    full_prompt = om.forward_full(m, PROMPT, layers_out=[o.beta[1]])
    np.testing.assert_allclose(o.pdm_caches[0].n, len(PROMPT))
    o.step()  # a = 1: only the newest row
    for _ in range(4):
        c, a = o.c, o.a
        anch = {q: [x.copy() for x in o.anch[q]] for q in range(c, c + a)}
        r = o.step()
        assert r.pdm_draft == 0
        for q in range(c, c + a):
            k = a - 1 - (q - c)
            expect = anch[q][1] if k >= 1 else np.zeros(d)
            np.testing.assert_allclose(r.pdm_hidden[q], expect, rtol=1e-12, atol=1e-14)
    assert full_prompt[o.beta[1]].shape[0] == len(PROMPT)


def test_target_closed_form_identity_layers():
    """All target W_o = W_d = 0: every H^l equals E[x], so greedy decoding is the iterated map
    x -> argmax W_lm . rmsnorm(E[x]), for plain decoding and for SPD alike."""
    ov = {}
    for l in range(SH.n_layers):
        ov[f"layer.{l}.wo"] = np.zeros((SH.d_model, SH.q_dim))
        ov[f"layer.{l}.wd"] = np.zeros((SH.d_model, SH.ffn_dim))
    m = om.Model(SH, SEED, overrides=ov)
    E, W = m.w("embed"), m.w("lm_head")

    def nxt(x):
        e = E[x]
        return int(np.argmax(W @ (e / np.sqrt(np.mean(e * e) + SH.rms_eps))))

    expect = [nxt(int(PROMPT[-1]))]
    for _ in range(9):
        expect.append(nxt(expect[-1]))
    assert om.ar_greedy(m, PROMPT, 10) == expect
    o, _ = osp.run_spd(m, PROMPT, 10, n=3)
    assert o.generated() == expect


def test_simulator_closed_form_alpha():
    """With iid acceptance p the expected steps per token are p + (1-p) n, so alpha -> 1/(p+(1-p)n)."""
    for n, p in [(4, 0.7), (8, 0.6), (2, 0.9)]:
        rng = np.random.default_rng(n)
        bits = rng.random(400000) < p
        N = 200000
        K = osp.simulate_steps(n, N, lambda q: bool(bits[q]), 0)
        assert abs(N / K - 1 / (p + (1 - p) * n)) < 0.01


@pytest.mark.parametrize("shape", [synth.TINY, synth.MID])
def test_batched_prefill_equals_token_by_token(shape):
    """The batched prefill (the whole prompt's causal forward as matrix products over its rows) and
    the token-by-token prefill fill the target and draft-module caches with the same keys and values,
    pick the same first token and continue identically (fp32 tiny, and the bf16 mid shape whose keys
    and values are rounded to bf16 as they are written)."""
    m = om.Model(shape, SEED)
    prompt = synth.prompt(shape, SEED, 23)
    a, b = osp.SPDOracle(m), osp.SPDOracle(m)
    assert a.prefill(prompt) == b.prefill(prompt, batched=True)
    for ca, cb in zip(a.caches + a.pdm_caches, b.caches + b.pdm_caches):
        assert ca.n == cb.n == len(prompt)
        np.testing.assert_allclose(cb.k[: cb.n], ca.k[: ca.n], rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(cb.v[: cb.n], ca.v[: ca.n], rtol=1e-9, atol=1e-12)
    for _ in range(8):
        ra, rb = a.step(want_logits=True), b.step(want_logits=True)
        assert (ra.decision, ra.target_argmax, ra.pdm_draft, ra.c, ra.a) == \
               (rb.decision, rb.target_argmax, rb.pdm_draft, rb.c, rb.a)
        np.testing.assert_allclose(rb.pdm_logits, ra.pdm_logits, rtol=1e-7, atol=1e-9)
    for q in range(a.c, a.c + a.a):
        np.testing.assert_allclose(b.hidden[q], a.hidden[q], rtol=1e-8, atol=1e-10)


def test_inflight_states_equal_brute_force_bf16():
    """The brute-force pin of in-flight states on the bf16 mid shape (keys and values rounded to bf16
    as the cache stores them, on both sides), with ragged stages (6 layers, n = 4)."""
    m = om.Model(synth.MID, SEED)
    prompt = synth.prompt(synth.MID, SEED, 17)
    ref = om.ar_greedy(m, prompt, 20)
    mask = synth.accept_mask(0.6, 19, 80)
    table = {len(prompt) + i: (t if mask[len(prompt) + i] else (t + 1) % synth.MID.vocab) for i, t in enumerate(ref)}
    o = osp.SPDOracle(m, n=4)
    o.prefill(prompt)
    beta = o.beta
    for _ in range(9):
        o.step(forced_draft=table.get(o.c + o.a))
        full = om.forward_full(m, o.toks[: o.c + o.a])
        for q in range(o.c, o.c + o.a):
            k = o.depth(q)
            np.testing.assert_allclose(o.hidden[q], full[beta[k]][q], rtol=1e-9, atol=1e-11)
            for j, an in enumerate(o.anch[q]):
                np.testing.assert_allclose(an, full[beta[j]][q], rtol=1e-9, atol=1e-11)
