"""Pins for the oracle's independent PDM head (CPU only).

Section 4.1: the PDM's LM head is initialised from the target's with a smaller vocabulary. With that
initialisation (the target's rows of the subset) the head's logits are the shared head's logits at
the subset's tokens, so the draft must be the shared head's argmax restricted to the subset and its
sampled distribution the top-k of those restricted logits; a subset holding every token is the
shared head; and the verified stream stays greedy decoding whatever the head drafts."""
import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import sampling as smp
from oracle import spd as osp

SEED = 5
SH = synth.TINY
PROMPT = synth.prompt(SH, SEED, 12)
VD = 300


def _pair(n, vd=VD, sampling=None):
    shared = osp.SPDOracle(om.Model(SH, SEED), n=n, sampling=sampling)
    own = osp.SPDOracle(om.Model(SH.with_(pdm_vocab=vd), SEED), n=n, sampling=sampling)
    return shared, own


@pytest.mark.parametrize("n", [2, 3])
def test_teacher_initialised_head_is_the_restricted_shared_head(n):
    shared, own = _pair(n)
    ids = synth.pdm_vocab_map(SH.with_(pdm_vocab=VD), SEED)
    ref = om.ar_greedy(om.Model(SH, SEED), PROMPT, 20)
    P = len(PROMPT)
    assert shared.prefill(PROMPT) == own.prefill(PROMPT)
    for i in range(14):
        q = shared.c + shared.a
        fd = int(ref[q - P]) if q - P < len(ref) else 0  # forced: both runs take the same path
        rs = shared.step(forced_draft=fd, want_logits=True)
        ro = own.step(forced_draft=fd, want_logits=True)
        for qq in rs.pdm_hidden:
            np.testing.assert_array_equal(rs.pdm_hidden[qq], ro.pdm_hidden[qq])
        restricted = rs.pdm_logits[ids]
        np.testing.assert_allclose(ro.pdm_logits, restricted, rtol=1e-12, atol=1e-14)
        best = ids[np.nonzero(restricted == restricted.max())[0][0]]  # lowest id among equals
        assert ro.pdm_draft == int(best)
        assert (rs.decision, rs.c, rs.a) == (ro.decision, ro.c, ro.a)


def test_full_subset_is_the_shared_head():
    shared, own = _pair(2, vd=SH.vocab)
    assert np.array_equal(synth.pdm_vocab_map(SH.with_(pdm_vocab=SH.vocab), SEED), np.arange(SH.vocab))
    shared.prefill(PROMPT)
    own.prefill(PROMPT)
    for _ in range(10):
        rs, ro = shared.step(want_logits=True), own.step(want_logits=True)
        assert rs.pdm_draft == ro.pdm_draft
        np.testing.assert_array_equal(rs.pdm_logits, ro.pdm_logits)


def test_sampled_draft_distribution_is_restricted_top_k():
    k, temp = 8, 0.7
    U = np.random.default_rng(3).random((96, 3))
    shared, own = _pair(2, sampling=smp.Sampling(k, temp, U))
    ids = synth.pdm_vocab_map(SH.with_(pdm_vocab=VD), SEED)
    shared.prefill(PROMPT)
    own.prefill(PROMPT)
    for _ in range(6):
        q = own.c + own.a
        rs = shared.step(forced_draft=7, want_logits=True)  # forced: both runs stay together
        ro = own.step(forced_draft=7, want_logits=True)
        lg = rs.pdm_logits[ids]
        order = np.lexsort((np.arange(len(ids)), -lg))[:k]
        z = lg[order] / temp
        w = np.exp(z - z[0])
        np.testing.assert_array_equal(ro.pdm_dist[0], ids[order])
        np.testing.assert_allclose(ro.pdm_dist[1], w / w.sum(), rtol=1e-12)
        assert ro.pdm_draft == smp.sample(ro.pdm_dist, U[q, smp.U_DRAFT])
        assert ro.pdm_draft in set(ids.tolist())


@pytest.mark.parametrize("n", [2, 4])
def test_own_head_is_lossless(n):
    m = om.Model(SH.with_(pdm_vocab=VD), SEED)
    ref = om.ar_greedy(om.Model(SH, SEED), PROMPT, 14)
    o, _ = osp.run_spd(m, PROMPT, 14, n=n)
    assert o.generated()[:14] == ref
