"""Pins of the oracle to values the paper prints (fixtures in tests/golden/, each citing its source)."""
import os

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import spd as osp

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _kv(name):
    out = {}
    for line in open(os.path.join(GOLD, name)):
        line = line.split("#", 1)[0].strip()
        if "=" in line:
            k, v = line.split("=", 1)
            out[k.strip()] = v.strip()
    return out


def _rows(name):
    rows = []
    for line in open(os.path.join(GOLD, name)):
        line = line.split("#", 1)[0].strip()
        if line:
            rows.append(line.split())
    return rows


def test_figure1_indices_from_fixture():
    """Figure 1 (n = 4): the oldest in-flight token x_{t-3} exits and judges x_{t-2}; on accept the
    draft x_{t+1} enters stage 1; on reject (Section 3.4) the KV keeps t - n + 1 positions."""
    g = {k: int(v) for k, v in _kv("figure1_n4_indices.txt").items()}
    n = g["n"]
    sh = synth.TINY
    model = om.Model(sh, 5)
    prompt = synth.prompt(sh, 5, 10)
    ref = om.ar_greedy(model, prompt, 12)
    for accept in (True, False):
        o = osp.SPDOracle(model, n=n)
        o.prefill(prompt)
        while o.a < n:
            o.step(forced_draft=ref[o.c + o.a - len(prompt)])
        t = o.c + n  # 1-indexed position of the newest in-flight token
        assert [q + 1 for q in range(o.c, o.c + o.a)] == list(range(t + g["inflight_first"], t + g["inflight_last"] + 1))
        q_draft = o.c + o.a
        fd = ref[q_draft - len(prompt)]
        if not accept:
            fd = (fd + 1) % sh.vocab
            o.toks[o.c + 1] = (o.toks[o.c + 1] + 1) % sh.vocab  # the token under verification is wrong
        r = o.step(forced_draft=fd)
        assert r.exited_pos + 1 == t + g["exits"]
        assert r.verified_pos + 1 == t + g["verifies"]
        if accept:
            assert r.decision == osp.ACCEPT
            newest = o.c + o.a  # 1-indexed position of the token that entered stage 1
            assert newest == t + g["enters_on_accept"] and o.depth(newest - 1) == 0
        else:
            assert r.decision == osp.REJECT
            assert o.kv_lengths() == [t - n + g["kv_len_on_reject_minus_t_plus_n"]] * sh.n_layers


def test_paper_anchor_eligibility_from_fixture():
    """Eq. depth-to-type with the paper's anchors for L = 32: l_max(k) = min(L, kL/n); at n = 4 a
    token at depth k may use anchors 0..k (k <= 4); at n = 8 two depths share each anchor."""
    g = _kv("paper_anchors_L32.txt")
    L = int(g["L"])
    anchors = [int(x) for x in g["anchors"].split()]
    assert anchors[0] == 0
    for n in (4, 8, 16):
        f = [osp.eligible_anchors(k, anchors, L, n) for k in range(n + 1)]
        # brute force of the definition: the largest i with b_i <= min(L, kL/n)
        brute = [max(i for i, b in enumerate(anchors) if b <= min(L, k * L / n)) for k in range(n + 1)]
        assert f == brute
        assert f[0] == 0 and f[n] == len(anchors) - 1  # embedding only at k = 0, every anchor at k = n
        assert all(b >= a for a, b in zip(f, f[1:]))  # features grow richer with depth
    assert [osp.eligible_anchors(k, anchors, L, 4) for k in range(5)] == [0, 1, 2, 3, 4]


def test_table2_alpha_within_pipeline_bounds():
    """Table 2's step acceptance ratios: with greedy streaming verification every committed token costs
    between 1 step (accepted) and n steps (rejected, refill), so 1/n <= alpha <= 1; the oracle's step
    simulator reaches both ends and, for iid acceptance p, alpha = 1/(p + (1-p) n), which has a
    solution p in (0, 1) for every printed alpha."""
    for n, ls, a0, a1 in _rows("table2_alpha.txt"):
        n = int(n)
        for alpha in (float(a0), float(a1)):
            assert 1.0 / n < alpha < 1.0
            p = (1.0 / alpha - n) / (1.0 - n)
            assert 0.0 < p < 1.0
            assert abs(1.0 / (p + (1 - p) * n) - alpha) < 1e-12
    N = 2000
    for n in (4, 8):
        k_all = osp.simulate_steps(n, N, lambda q: True, 0)
        k_none = osp.simulate_steps(n, N, lambda q: False, 0)
        assert osp.step_acceptance(N, k_all) == pytest.approx(1.0, abs=2 * n / N)
        assert osp.step_acceptance(N, k_none) == pytest.approx(1.0 / n, rel=2 * n / N)


def test_table3_draft_cost_adjusted_speedup():
    """Table 3 (post-step features, L = 32): the draft-cost-adjusted speedup equals Eq. s-eagle's PPSD
    form S0 * L / (L_s * n + L), within the two-decimal rounding of both printed values."""
    for n, ls, tag, s0, sa in _rows("table3_post_step.txt"):
        n, ls, s0, sa = int(n), int(ls), float(s0), float(sa)
        f = 32 / (ls * n + 32)
        got = osp.speedup_serial_draft(s0, 32, ls, n)
        assert got == pytest.approx(s0 * f)
        assert abs(got - sa) <= 0.005 * f + 0.005 + 1e-9, (n, ls, tag)


def test_zero_cost_speedup_definition():
    """Eq. s0-spd: S0 = N / (K / n) = alpha * n; an SPD run with every draft correct approaches n."""
    sh = synth.TINY
    model = om.Model(sh, 5)
    prompt = synth.prompt(sh, 5, 8)
    ref = om.ar_greedy(model, prompt, 40)
    o, res = osp.run_spd(model, prompt, 40, n=2, draft_for=lambda q: ref[q - len(prompt)] if q - len(prompt) < 40 else None)
    N = o.verified - 1  # tokens generated by steps (the prefill's token came before any step)
    s0 = osp.speedup_zero_cost(osp.step_acceptance(N, len(res)), 2)
    assert s0 == pytest.approx(2 * N / len(res))
    assert 1.9 < s0 <= 2.0
