"""Pins for the oracle's sampled decoding (CPU only).

The rule has plain definitions to check against: a top-k, temperature-T distribution built from
logits whose probabilities are known by construction; the inverse-CDF draw, which on a stratified
grid of uniforms gives every index floor or ceil of N*p draws; the speculative-sampling theorem
(the token that rejection sampling emits follows the target distribution p exactly, whatever the
draft distribution q); top_k = 1, which reduces sampled SPD to greedy SPD; and the plain
autoregressive top-k distribution, which the first judged token of sampled SPD must follow."""
import numpy as np
import pytest
from scipy import stats

import synth
from oracle import model as om
from oracle import sampling as smp
from oracle import spd as osp

SEED = 5
SH = synth.TINY
PROMPT = synth.prompt(SH, SEED, 10)


def _known_logits(rng, v, ids, probs, floor=-60.0):
    """Logits whose top-len(ids) softmax is probs on ids (every other logit far below)."""
    lg = np.full(v, floor) + rng.uniform(-1.0, 0.0, size=v)
    lg[ids] = np.log(probs) + 3.0
    return lg


def test_top_k_dist_closed_form():
    rng = np.random.default_rng(1)
    v, k = 97, 7
    ids = rng.choice(v, size=k, replace=False)
    probs = rng.dirichlet(np.ones(k))
    lg = _known_logits(rng, v, ids, probs)
    got_ids, got_p = smp.top_k_dist(lg, k, 1.0)
    order = np.argsort(-probs, kind="stable")
    np.testing.assert_array_equal(got_ids, ids[order])
    np.testing.assert_allclose(got_p, probs[order], rtol=1e-12, atol=1e-15)
    # temperature T: p_i proportional to probs_i ** (1 / T)
    for t in (0.5, 2.0):
        _, pt = smp.top_k_dist(lg, k, t)
        w = probs[order] ** (1.0 / t)
        np.testing.assert_allclose(pt, w / w.sum(), rtol=1e-12)
    # a smaller k renormalises the k most probable
    _, p3 = smp.top_k_dist(lg, 3, 1.0)
    np.testing.assert_allclose(p3, probs[order][:3] / probs[order][:3].sum(), rtol=1e-12)
    # k above the vocabulary keeps everything
    assert len(smp.top_k_dist(lg, 1000, 1.0)[0]) == v


def test_top_k_dist_ties_take_lower_index_first():
    lg = np.zeros(10)
    lg[[7, 3, 5]] = 1.0
    ids, p = smp.top_k_dist(lg, 4, 1.0)
    np.testing.assert_array_equal(ids, [3, 5, 7, 0])
    assert p[0] == p[1] == p[2] > p[3]
    assert smp.top_k_dist(lg, 1, 1.0)[0][0] == om.argmax_first(lg)


def test_sample_index_stratified_counts():
    rng = np.random.default_rng(2)
    p = rng.dirichlet(np.ones(9) * 0.7)
    n = 4000
    counts = np.bincount([smp.sample_index(p, (j + 0.5) / n) for j in range(n)], minlength=len(p))
    assert np.all(np.abs(counts - n * p) <= 1.0 + 1e-9), (counts, n * p)
    # unnormalised weights draw the same way
    assert [smp.sample_index(3.0 * p, (j + 0.5) / 50) for j in range(50)] == \
           [smp.sample_index(p, (j + 0.5) / 50) for j in range(50)]
    assert smp.sample_index(p, 0.0) == 0
    assert smp.sample_index(p, np.nextafter(1.0, 0.0)) == len(p) - 1


def _emitted_distribution(p, q, vocab, na=120, nr=120):
    """Distribution of the emitted token: every draft x enumerated with weight q(x), the two uniforms
    on stratified grids (so the result is exact up to 1/na and 1/nr)."""
    out = np.zeros(vocab)
    for x, qx in zip(*q):
        for i in range(na):
            ua = (i + 0.5) / na
            for j in range(nr):
                _, tok = smp.rejection_verify(p, q, int(x), ua, (j + 0.5) / nr)
                out[tok] += qx / (na * nr)
    return out


@pytest.mark.parametrize("case", ["overlap", "disjoint", "same", "forced_in", "forced_out"])
def test_rejection_verify_emits_the_target_distribution(case):
    rng = np.random.default_rng(3)
    vocab = 12
    p_ids = rng.choice(vocab, size=6, replace=False)
    p = (p_ids, rng.dirichlet(np.ones(6)))
    if case == "overlap":
        q_ids = np.concatenate([p_ids[:3], [i for i in range(vocab) if i not in p_ids][:3]])
        q = (q_ids, rng.dirichlet(np.ones(6)))
    elif case == "disjoint":
        q_ids = np.array([i for i in range(vocab) if i not in p_ids][:4])
        q = (q_ids, rng.dirichlet(np.ones(4)))
    elif case == "same":
        q = p
    elif case == "forced_in":
        q = smp.point_mass(int(p_ids[2]))
    else:
        q = smp.point_mass(int([i for i in range(vocab) if i not in p_ids][0]))
    want = np.zeros(vocab)
    want[p[0]] = p[1]
    got = _emitted_distribution(p, q, vocab)
    np.testing.assert_allclose(got, want, atol=3.0 / 120)
    if case == "same":  # q = p: every draft is kept
        assert all(smp.rejection_verify(p, q, int(x), np.nextafter(1.0, 0.0), 0.5)[0] for x in p[0])


def test_rejection_verify_accept_probability_is_min_one_ratio():
    p = (np.array([4, 1, 7]), np.array([0.5, 0.3, 0.2]))
    q = (np.array([1, 7, 4]), np.array([0.6, 0.1, 0.3]))
    n = 1000
    for x, want in ((1, 0.3 / 0.6), (7, 1.0), (4, 1.0)):
        acc = sum(smp.rejection_verify(p, q, x, (j + 0.5) / n, 0.5)[0] for j in range(n))
        assert abs(acc / n - want) <= 1.0 / n + 1e-12
    # a reject draws only where p exceeds q: the residual here is {4: 0.2, 7: 0.1}
    toks = {smp.rejection_verify(p, q, 1, 0.99, (j + 0.5) / 30)[1] for j in range(30)}
    assert toks == {4, 7}


@pytest.fixture(scope="module")
def model():
    return om.Model(SH, SEED)


def _uniforms(seed, rows):
    return np.random.default_rng([seed, 11]).random((rows, 3))


@pytest.mark.parametrize("n,forced", [(1, False), (2, False), (2, True), (3, True)])
def test_top_k_one_is_greedy_spd(model, n, forced):
    ref = om.ar_greedy(model, PROMPT, 14)
    table = {len(PROMPT) + i: (ref[i] if i % 3 else (ref[i] + 1) % SH.vocab) for i in range(len(ref))}
    draft_for = (lambda q: table.get(q)) if forced else None
    g, rg = osp.run_spd(model, PROMPT, 8, n=n, draft_for=draft_for, max_steps=40)
    s, rs = osp.run_spd(model, PROMPT, 8, n=n, draft_for=draft_for, max_steps=40,
                        sampling=smp.Sampling(1, 1.0, _uniforms(n, 64)))
    assert [(r.decision, r.target_argmax, r.draft, r.pdm_draft) for r in rg] == \
           [(r.decision, r.target_argmax, r.draft, r.pdm_draft) for r in rs]
    assert g.generated() == s.generated()


def _chi2_pvalue(counts, probs):
    """Pearson chi-square with cells of expected count < 5 pooled."""
    exp = probs * counts.sum()
    big = exp >= 5.0
    obs_c = list(counts[big]) + [counts[~big].sum()]
    exp_c = list(exp[big]) + [exp[~big].sum()]
    if exp_c[-1] == 0.0:
        obs_c, exp_c = obs_c[:-1], exp_c[:-1]
    return stats.chisquare(obs_c, exp_c).pvalue


@pytest.mark.parametrize("forced", [False, True])
def test_first_judged_token_follows_ar_distribution(model, forced):
    """Sampled SPD, n = 2, top-k 8: with the prompt's first draw fixed, the token at the position
    judged by the first exit follows the plain autoregressive top-k distribution there."""
    k, runs, n = 8, 400, 2
    P = len(PROMPT)
    base_u = _uniforms(99, P + 8)
    o0 = osp.SPDOracle(model, n=n, sampling=smp.Sampling(k, 1.0, base_u))
    x_p = o0.prefill(PROMPT)
    last = om.forward_full(model, list(PROMPT) + [x_p], layers_out=[SH.n_layers])[SH.n_layers][-1]
    want_ids, want_p = smp.top_k_dist(om.lm_logits(model, last), k, 1.0)
    greedy_next = int(want_ids[0])
    probs = np.zeros(SH.vocab)
    probs[want_ids] = want_p
    counts = np.zeros(SH.vocab)
    rng = np.random.default_rng(1234 + forced)
    for _ in range(runs):
        u = base_u.copy()
        u[P + 1:] = rng.random((u.shape[0] - P - 1, 3))
        o = o0.clone()
        o.sampling = smp.Sampling(k, 1.0, u)
        while True:
            q = o.c + o.a
            r = o.step(forced_draft=greedy_next if (forced and q == P + 1) else None)
            if r.verified_pos == P + 1:
                counts[r.verified_token] += 1
                break
    assert counts[probs == 0.0].sum() == 0
    assert _chi2_pvalue(counts[want_ids], want_p) > 1e-3
    if forced:  # the forced token is kept with probability p(greedy_next): a residual slip shows here
        assert abs(counts[greedy_next] / runs - want_p[0]) < 4.0 * np.sqrt(want_p[0] * (1 - want_p[0]) / runs)
