"""Pins for the oracle's post-step schedule (CPU only).

Under the post-step schedule (the ablation of Section 4.5) the PDM reads the features left after the
step's stage compute, so every in-flight token is one stage deeper than under the pre-step schedule
of Section 3.3. What fixes it independently of the pipelined code: with W_in selecting one anchor
block and the PDM layers reduced to the identity, each PDM row must equal that anchor of its token as
the no-cache full forward of the same prefix computes it; at n = 1 the two schedules coincide (depth
0 and depth 1 both see anchor 0 only); and the schedule cannot change the verified stream (greedy
SPD is lossless, Section 3.4)."""
import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import spd as osp

SEED = 5
SH = synth.TINY
PROMPT = synth.prompt(SH, SEED, 12)


def _selector_model(n, j):
    """W_in passes anchor block j only; zero PDM W_o and W_d make the PDM layer the identity."""
    d = SH.d_model
    blocks = [np.eye(d) if i == j else np.zeros((d, d)) for i in range(n)]
    ov = {"pdm.in": np.concatenate(blocks, axis=1),
          "pdm.layer.0.wo": np.zeros((d, SH.q_dim)), "pdm.layer.0.wd": np.zeros((d, SH.ffn_dim))}
    return om.Model(SH, SEED, overrides=ov)


def _draft_of(m, h):
    """argmax of the shared head over rmsnorm(h) with the PDM's unit gain."""
    W = m.w("lm_head")
    return int(np.argmax(W @ (h / np.sqrt(np.mean(h * h) + SH.rms_eps))))


@pytest.mark.parametrize("n,j", [(2, 1), (3, 1), (3, 2)])
def test_post_step_rows_are_brute_force_anchors(n, j):
    """Post-step: row q at depth k (one more than pre-step) holds H^{beta_j}(x_0..x_q) from the
    no-cache forward when j <= f(k), else zeros; the draft is the head's argmax over the newest row."""
    m = _selector_model(n, j)
    o = osp.SPDOracle(m, n=n, schedule="post")
    o.prefill(PROMPT)
    layer = o.beta[j]
    checked = 0
    for _ in range(3 * n + 2):
        c, a = o.c, o.a
        toks = list(o.toks[: c + a])  # a reject rewrites the in-flight positions
        r = o.step()
        for i in range(a):
            q = c + i
            k = a - i  # post-step depth
            f = min(k, n - 1)
            if j <= f:
                expect = om.forward_full(m, toks[: q + 1], layers_out=[layer])[layer][-1]
                np.testing.assert_allclose(r.pdm_hidden[q], expect, rtol=1e-9, atol=1e-11)
                checked += 1
            else:
                np.testing.assert_array_equal(r.pdm_hidden[q], np.zeros(SH.d_model))
        newest = r.pdm_hidden[c + a - 1]
        assert r.pdm_draft == (_draft_of(m, newest) if np.any(newest) else 0)
    assert checked >= n


def test_pre_step_newest_row_sees_no_anchor_one():
    """The same selector under the pre-step schedule: the newest token is at depth 0, so its row is
    zero and the draft is token 0, while post-step it is the brute-force stage-0 output."""
    n = 2
    m = _selector_model(n, 1)
    pre, post = osp.SPDOracle(m, n=n), osp.SPDOracle(m, n=n, schedule="post")
    pre.prefill(PROMPT)
    post.prefill(PROMPT)
    rp, rq = pre.step(forced_draft=7), post.step(forced_draft=7)
    assert rp.pdm_draft == 0
    q = PROMPT.shape[0]
    h1 = om.forward_full(m, list(PROMPT) + [post.toks[q]], layers_out=[post.beta[1]])[post.beta[1]][-1]
    assert rq.pdm_draft == _draft_of(m, h1)


def test_n1_schedules_coincide():
    """n = 1: depth 0 and depth 1 both see anchor 0 only, so the two schedules give the same steps,
    bit for bit."""
    m = om.Model(SH, SEED)
    a, b = osp.SPDOracle(m, n=1), osp.SPDOracle(m, n=1, schedule="post")
    assert a.prefill(PROMPT) == b.prefill(PROMPT)
    for _ in range(8):
        ra, rb = a.step(), b.step()
        assert (ra.decision, ra.draft, ra.pdm_draft, ra.c, ra.a) == (rb.decision, rb.draft, rb.pdm_draft, rb.c, rb.a)
        for q in ra.pdm_hidden:
            np.testing.assert_array_equal(ra.pdm_hidden[q], rb.pdm_hidden[q])


@pytest.mark.parametrize("n,p", [(2, None), (3, 0.5), (4, 0.7)])
def test_post_step_is_lossless(n, p):
    """The verified stream is plain greedy decoding under either schedule, for natural drafts and
    for forced Bernoulli(p) drafts."""
    m = om.Model(SH, SEED)
    ref = om.ar_greedy(m, PROMPT, 14)
    draft_for = None
    if p is not None:
        mask = synth.accept_mask(p, SEED + n, len(PROMPT) + len(ref) + 8)
        P = len(PROMPT)
        table = {P + i: (ref[i] if mask[P + i] else (ref[i] + 1) % SH.vocab) for i in range(len(ref))}
        draft_for = table.get
    o, res = osp.run_spd(m, PROMPT, 14, n=n, draft_for=draft_for, schedule="post")
    assert o.generated()[:14] == ref
    if p is not None:
        for r in res:
            if r.decision != osp.NONE:
                assert r.decision == (osp.ACCEPT if mask[r.verified_pos] else osp.REJECT)
