"""Pins for the oracle's Pipeline Draft Module pass with non-trivial PDM layers (CPU only).

The draft module runs its decoder layers causally over the feature sequence of Eq. input-seq: each
position q contributes one feature g_q, the projection of Eq. agg-main over the anchors its token has
reached. Before a step (Eq. steady-g, Eq. warmup-g) a committed position (q < c) has all n anchors,
and the in-flight token at position c+i has depth k = a-1-i and therefore anchors 0..min(k, n-1)
(Eq. depth-to-type with the stage inputs as anchors); under the post-step schedule every in-flight
token is one stage deeper. The oracle computes the draft module incrementally: its KV cache holds
the committed rows, and each step rewrites the a in-flight rows (Appendix A.1's refreshed rows).

The pin rebuilds every step from scratch: the anchors of every position from the target's no-cache
forward over the step's tokens, the feature sequence from the definitions above, and the draft
module's layers as a no-cache causal forward over that whole sequence, each row at its own position.
Every in-flight row, the draft logits and the draft must equal the oracle's to 1e-9. The draft module's
attention weights are scaled up so that its attention is far from uniform (a wrong position, span or
feature depth then moves the result by far more than the tolerance), and planted mistakes in a copy
of the oracle (wrong depth, wrong position, a stale committed row, no committed rows) must fail it.
A closed form checks the attention span on its own: with W_q = 0 every score is 0, so a row's
attention output is the plain mean of V over positions 0..q."""
import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import spd as osp

SEED = 9
PROMPT_LEN = 12


def _shape(n, ls):
    return synth.TINY.with_(n_stages=n, pdm_layers=ls)


def _model(n, ls, amplify=True, zero_wq=False):
    sh = _shape(n, ls)
    over = {}
    for l in range(ls):
        for k, f in (("wq", 6.0), ("wk", 6.0), ("wo", 4.0), ("wd", 4.0)):
            name = f"pdm.layer.{l}.{k}"
            w = synth.tensor(sh, SEED, name).astype(np.float64)
            if amplify:
                w = w * f
            if zero_wq and k == "wq":
                w = np.zeros_like(w)
            over[name] = w
    return om.Model(sh, SEED, overrides=over)


def _eligible(k, n):
    # stage inputs as anchors: beta_i = floor(i L / n) <= k L / n exactly when i <= k
    return min(k, n - 1)


def brute_force_pdm(model, tokens, c, a, schedule):
    """Rows 0..c+a-1 of the draft module's last layer for a step that starts with c committed
    positions and a in-flight tokens (tokens[q] for q < c + a), from scratch."""
    sh = model.shape
    n, L, d = sh.n_stages, sh.n_layers, sh.d_model
    beta = [s * L // n for s in range(n + 1)]
    T = c + a
    full = om.forward_full(model, tokens[:T], layers_out=beta[:n])
    w_in = model.w("pdm.in")
    G = np.zeros((T, d))
    for q in range(T):
        depth = n if q < c else (a - 1 - (q - c)) + (1 if schedule == "post" else 0)
        z = np.zeros(n * d)
        for j in range(_eligible(depth, n) + 1):
            z[j * d:(j + 1) * d] = full[beta[j]][q]
        G[q] = w_in @ z
    return om.forward_rows(model, G, "pdm.layer", sh.pdm_layers, layers_out=[sh.pdm_layers])[sh.pdm_layers]


def _drafts(model, p, seed):
    ref = om.ar_greedy(model, synth.prompt(model.shape, SEED, PROMPT_LEN), 40)
    mask = synth.accept_mask(p, seed, PROMPT_LEN + len(ref) + 8)
    table = {PROMPT_LEN + i: (ref[i] if mask[PROMPT_LEN + i] else (ref[i] + 1) % model.shape.vocab)
             for i in range(len(ref))}
    return table


def _check_run(model, n, schedule, steps, table, oracle_cls=osp.SPDOracle, tol=1e-9):
    """Lockstep of the oracle against the brute force; returns the kinds of steps covered."""
    o = oracle_cls(model, n=n, schedule=schedule)
    prompt = synth.prompt(model.shape, SEED, PROMPT_LEN)
    o.prefill(prompt)
    seen = {"warmup": 0, "steady": 0, "after_reject": 0}
    prev_reject = False
    for i in range(steps):
        c, a = o.c, o.a
        toks = list(o.toks)
        r = o.step(forced_draft=table.get(c + a), want_logits=True)
        H = brute_force_pdm(model, toks, c, a, schedule)
        for q in range(c, c + a):
            ref = H[q]
            got = r.pdm_hidden[q]
            err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
            assert err <= tol, f"step {i} (c={c} a={a} {schedule}): PDM row {q} rel err {err:.3e}"
        lg = model.w("lm_head") @ om.rms_norm(H[c + a - 1], model.w("pdm.norm"), model.shape.rms_eps)
        assert np.max(np.abs(lg - r.pdm_logits)) <= tol * max(1.0, np.max(np.abs(lg))), f"step {i}: draft logits"
        assert r.pdm_draft == int(np.argmax(lg)), f"step {i}: draft"
        if prev_reject:
            seen["after_reject"] += 1
        seen["steady" if a == n else "warmup"] += 1
        prev_reject = r.decision == osp.REJECT
    return seen


@pytest.mark.parametrize("schedule", ["pre", "post"])
@pytest.mark.parametrize("ls", [1, 2])
@pytest.mark.parametrize("n", [2, 3, 4])
def test_pdm_rows_equal_no_cache_forward_over_feature_sequence(n, ls, schedule):
    model = _model(n, ls)
    table = _drafts(model, 0.6, 31 + n)
    seen = _check_run(model, n, schedule, 16, table)
    # warm-up (a < n), steady state (a = n) and the step right after a rejection were all covered
    assert seen["warmup"] >= n - 1 and seen["steady"] >= 3 and seen["after_reject"] >= 1, seen


def test_pdm_pass_with_the_workload_weights():
    """The same pin with the seeded N(0, 0.02) draft-module weights of the workloads, unscaled."""
    model = _model(2, 1, amplify=False)
    _check_run(model, 2, "pre", 12, _drafts(model, 0.5, 77))


def test_uniform_attention_closed_form():
    """W_q = 0: every score is zero, so row q's attention output is the mean of V over rows 0..q of
    the draft module's cache: the committed prompt rows (full-depth features) and the in-flight rows
    up to q, each V from its own feature."""
    n = 3
    model = _model(n, 1, zero_wq=True)
    sh = model.shape
    o = osp.SPDOracle(model, n=n)
    o.prefill(synth.prompt(sh, SEED, PROMPT_LEN))
    table = _drafts(model, 0.7, 5)
    lw = model.layer(0, "pdm.layer")
    beta = [s * sh.n_layers // n for s in range(n + 1)]
    for i in range(8):
        c, a = o.c, o.a
        toks = list(o.toks)
        r = o.step(forced_draft=table.get(c + a))
        full = om.forward_full(model, toks[:c + a], layers_out=beta[:n])
        d = sh.d_model
        G = np.zeros((c + a, d))
        for q in range(c + a):
            k = n if q < c else a - 1 - (q - c)
            for j in range(min(k, n - 1) + 1):
                G[q] += model.w("pdm.in")[:, j * d:(j + 1) * d] @ full[beta[j]][q]
        U = om.rms_norm(G, lw["attn_norm"], sh.rms_eps)
        V = (U @ lw["wv"].T).reshape(c + a, sh.n_kv_heads, sh.head_dim)
        grp = sh.n_q_heads // sh.n_kv_heads
        for q in range(c, c + a):
            o_att = np.repeat(V[: q + 1].mean(axis=0), grp, axis=0).reshape(-1)
            h = G[q] + lw["wo"] @ o_att
            u = om.rms_norm(h, lw["mlp_norm"], sh.rms_eps)
            h = h + lw["wd"] @ (om.silu(lw["wg"] @ u) * (lw["wu"] @ u))
            err = np.linalg.norm(r.pdm_hidden[q] - h) / np.linalg.norm(h)
            assert err <= 1e-9, f"step {i}: row {q} rel err {err:.3e}"


# ----------------------------------------------------------------------------- planted mistakes
class _WrongDepth(osp.SPDOracle):
    """Every in-flight feature one anchor deeper than its depth allows."""

    def feature(self, anchors, k):
        return super().feature(anchors + [anchors[-1]] * self.n, min(k + 1, self.n))


class _WrongPosition(osp.SPDOracle):
    """Every in-flight row of the draft module rotated at the newest row's position (one position for
    the whole row block); prompt rows keep their own. (A uniform shift of every position would change
    nothing: rotary attention depends only on relative positions.)"""

    def pdm_row(self, g, pos):
        if self.a == 0 or pos < self.c:  # prefill: the prompt rows
            return super().pdm_row(g, pos)
        rot = self.c + self.a - 1
        h = g
        for i in range(self.ls):
            lw = self.m.layer(i, "pdm.layer")
            cache = self.pdm_caches[i]
            u = om.rms_norm(h, lw["attn_norm"], self.sh.rms_eps)
            q = om.rope((lw["wq"] @ u).reshape(self.sh.n_q_heads, -1), rot, self.sh.rope_base)
            k = om.rope((lw["wk"] @ u).reshape(self.sh.n_kv_heads, -1), rot, self.sh.rope_base)
            v = (lw["wv"] @ u).reshape(self.sh.n_kv_heads, -1)
            cache.append(pos, k, v)
            h = h + lw["wo"] @ om.attend(q, cache, pos)
            u = om.rms_norm(h, lw["mlp_norm"], self.sh.rms_eps)
            h = h + lw["wd"] @ (om.silu(lw["wg"] @ u) * (lw["wu"] @ u))
        return h


class _NoRefresh(osp.SPDOracle):
    """Committed rows keep the feature they had when first written (no rewrite of in-flight rows
    whose rows already exist)."""

    def step(self, forced_draft=None, want_logits=False):
        keep = [pc.n for pc in self.pdm_caches]
        saved = [(pc.k.copy(), pc.v.copy()) for pc in self.pdm_caches]
        r = super().step(forced_draft, want_logits)
        for pc, n0, (k, v) in zip(self.pdm_caches, keep, saved):
            m = min(n0, pc.n)
            pc.k[:m], pc.v[:m] = k[:m], v[:m]
        return r


class _NoPrefix(osp.SPDOracle):
    """The in-flight rows attend only to themselves (the committed rows' cache is dropped)."""

    def step(self, forced_draft=None, want_logits=False):
        for pc in self.pdm_caches:
            pc.k[: self.c] = 0.0
            pc.v[: self.c] = 0.0
        return super().step(forced_draft, want_logits)


@pytest.mark.parametrize("bad", [_WrongDepth, _WrongPosition, _NoRefresh, _NoPrefix])
def test_planted_mistakes_fail_the_pin(bad):
    n = 3
    model = _model(n, 2)
    table = _drafts(model, 0.6, 34)
    with pytest.raises(AssertionError):
        _check_run(model, n, "pre", 16, table, oracle_cls=bad, tol=1e-6)
