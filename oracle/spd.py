"""Oracle, part 2: one Speculative Pipeline Decoding step, in float64 on the CPU.

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

What it follows:
  * Token-level pipeline (Section 3.1): the L layers form n contiguous stages; each step advances
    every in-flight token of one sequence through one stage. Boundaries beta_s = floor(s*L/n)
    (the uniform split of Section 4.1 extended to n not dividing L).
  * Depth staircase (Eq. steady-g and Eq. warmup-g): a token at depth k has completed k stages.
    Pre-step, the a in-flight tokens at positions c..c+a-1 have depths a-1..0; positions < c are
    complete (depth n).
  * Multi-depth feature aggregation (Eq. depth-to-type and Eq. agg-main) with the anchor set
    B = (beta_0, ..., beta_{n-1}) (the stage inputs) and one projection W_in of width n*d:
    f(k) = min(k, n-1) anchors are eligible at depth k, and FC_{f(k)} is W_in applied to the
    concatenation of the eligible anchors with the ineligible blocks set to zero. No bias and no
    normalisation before the concatenation.
  * Pre-step schedule (Section 3.3): the PDM reads only features present before the step, so it
    runs concurrently with the stage compute; its L_s decoder layers run causally over the feature
    sequence; rows < c are final (their PDM KV rows persist), rows c..c+a-1 are recomputed each
    step. The draft is the argmax of the shared LM head over the PDM's last row after its own
    final RMSNorm (gain 1).
  * Streaming greedy verification and rollback (Section 3.4): when the pipeline is full (a = n)
    the oldest token exits; its logits judge the next in-flight token. Accept: the draft enters
    stage 1. Reject: caches keep the committed prefix only, in-flight work is dropped, and the
    target's own argmax is reseeded at depth 0. With n = 1 the judged token is this step's own
    draft, so the step is ordinary greedy decoding. While a < n (warm-up or refill) nothing exits
    and the draft is pushed unconditionally.
  * Sampled decoding (Section 3.4 under sampling, Section 4.1's top-k setting; oracle/sampling.py):
    the draft is drawn from the PDM's top-k distribution q with the draft position's u_draft, and q
    is kept with the in-flight token; the exit's top-k distribution p judges the successor by
    rejection sampling with the successor's u_accept / u_resample, and a reject reseeds the residual
    draw. A forced draft carries q = delta. The prompt's first token is drawn from p with u_resample.
  * The PDM's LM head (Section 4.1): shared with the target, or its own head over a smaller vocabulary
    (initialised from the target's rows of that subset); a draft id i then stands for target token
    map[i], map ascending, so ties still go to the lower target id.
  * Post-step schedule (the ablation of Section 4.5 against Section 3.3's pre-step choice): the PDM
    waits for the stage compute and reads the post-step features, every in-flight token one stage
    deeper (the newest contributes g^1 instead of g^0); drafting is then serial behind the step.
    Everything else (rows rewritten, the draft's position, verify) is as in the pre-step schedule.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

import synth
from .model import (LayerCache, Model, argmax_first, decoder_layer, embed, forward_rows, lm_logits, new_caches,
                    rms_norm)
from . import sampling as smp

NONE, ACCEPT, REJECT = 0, 1, 2


def stage_bounds(n_layers: int, n: int) -> List[int]:
    """beta_0 = 0 < beta_1 < ... < beta_n = L, with beta_s = floor(s * L / n)."""
    assert 1 <= n <= n_layers
    return [s * n_layers // n for s in range(n + 1)]


def l_max(k: int, n_layers: int, n: int) -> float:
    """Deepest layer available to a token that has completed k stages (Eq. before depth-to-type)."""
    return min(n_layers, k * n_layers / n)


def eligible_anchors(k: int, anchors: Sequence[int], n_layers: int, n: int) -> int:
    """f(k) = max{i : b_i <= l_max(k)} (Eq. depth-to-type)."""
    lm = l_max(k, n_layers, n)
    return max(i for i, b in enumerate(anchors) if b <= lm)


@dataclasses.dataclass
class StepResult:
    decision: int
    target_argmax: int  # y, the token committed at verified_pos (or -1 when nothing exited)
    draft: int  # the token the PDM proposed (after any forced override)
    pdm_draft: int  # the PDM's own argmax (sampled decoding: its own draw)
    exited_pos: int
    verified_pos: int
    verified_token: int
    c: int
    a: int
    exit_logits: Optional[np.ndarray] = None
    pdm_logits: Optional[np.ndarray] = None
    pdm_hidden: Optional[Dict[int, np.ndarray]] = None
    depths: Optional[Dict[int, int]] = None  # pre-step depth of every row the PDM read
    pdm_dist: Optional[smp.Dist] = None  # sampled decoding: the PDM's top-k distribution
    exit_dist: Optional[smp.Dist] = None  # sampled decoding: the exit's top-k distribution
    accepted_by_ratio: Optional[bool] = None  # sampled decoding: outcome of the acceptance test


class SPDOracle:
    """SPD state for one sequence: target KV per layer, PDM KV per PDM layer, in-flight tokens."""

    def __init__(self, model: Model, n: Optional[int] = None, pdm_layers: Optional[int] = None,
                 sampling: Optional[smp.Sampling] = None, schedule: str = "pre"):
        """schedule: "pre" (the PDM reads pre-step features, Section 3.3) or "post" (it reads the
        features after the step's stage compute)."""
        model = model.for_width(model.shape.n_stages if n is None else n, pdm_layers)
        sh = model.shape
        self.m = model
        self.sh = sh
        self.n = sh.n_stages
        self.ls = sh.pdm_layers
        self.L = sh.n_layers
        self.beta = stage_bounds(self.L, self.n)
        self.anchor_layers = self.beta[: self.n]  # B = stage inputs
        self.caches = new_caches(sh, self.L)
        self.pdm_caches = new_caches(sh, self.ls)
        self.toks: List[int] = []
        self.hidden: Dict[int, np.ndarray] = {}  # in-flight residual streams by position
        self.anch: Dict[int, List[np.ndarray]] = {}  # in-flight anchors by position
        self.c = 0
        self.a = 0
        self.prompt_len = 0
        self.steps = 0
        self.verified = 0  # N: prefill token + one per exit
        self.sampling = sampling
        self.qdist: Dict[int, smp.Dist] = {}  # sampled decoding: q of each in-flight token
        assert schedule in ("pre", "post")
        self.schedule = schedule
        # the PDM's own vocabulary (target ids of its draft ids), or None: the shared head
        self.pdm_ids = synth.pdm_vocab_map(sh, model.seed) if sh.pdm_vocab else None

    def clone(self) -> "SPDOracle":
        """An independent copy of the decoding state (the model is shared)."""
        o = object.__new__(SPDOracle)
        o.__dict__.update(self.__dict__)
        o.caches = [cc.clone() for cc in self.caches]
        o.pdm_caches = [cc.clone() for cc in self.pdm_caches]
        o.toks = list(self.toks)
        o.hidden = {q: h.copy() for q, h in self.hidden.items()}
        o.anch = {q: [x.copy() for x in v] for q, v in self.anch.items()}
        o.qdist = dict(self.qdist)
        return o

    def _target_dist(self, lg: np.ndarray) -> smp.Dist:
        return smp.top_k_dist(lg, self.sampling.top_k, self.sampling.temperature)

    # ------------------------------------------------------------------ PDM pieces
    def w_in(self) -> np.ndarray:
        w = self.m.w("pdm.in")
        assert w.shape == (self.sh.d_model, self.n * self.sh.d_model)
        return w

    def feature(self, anchors: List[np.ndarray], k: int) -> np.ndarray:
        """g^k = FC_{f(k)}(Concat(H^{b_0..b_f(k)})): W_in over the eligible anchors, zeros elsewhere."""
        d = self.sh.d_model
        f = eligible_anchors(k, self.anchor_layers, self.L, self.n)
        z = np.zeros(self.n * d)
        for j in range(f + 1):
            z[j * d:(j + 1) * d] = anchors[j]
        return self.w_in() @ z

    def pdm_logits(self, h: np.ndarray) -> np.ndarray:
        """The PDM's head over its last row: the shared W_lm, or its own head (draft ids)."""
        if self.pdm_ids is None:
            return lm_logits(self.m, h, "pdm.norm")
        return self.m.w("pdm.lm_head") @ rms_norm(h, self.m.w("pdm.norm"), self.sh.rms_eps)

    def pdm_token(self, i: int) -> int:
        return int(i) if self.pdm_ids is None else int(self.pdm_ids[int(i)])

    def pdm_row(self, g: np.ndarray, pos: int) -> np.ndarray:
        h = g
        for i in range(self.ls):
            h = decoder_layer(self.sh, self.m.layer(i, "pdm.layer"), h, pos, self.pdm_caches[i])
        return h

    # ------------------------------------------------------------------ prefill
    def prefill(self, prompt, batched: bool = False) -> int:
        """Process the prompt through the target (keeping the anchors), build the PDM KV over it
        with full-depth features, and place the target's first token in flight at depth 0.

        batched: the same causal forward over the whole prompt at once (every layer as one matrix
        product over the prompt's rows, causal attention over the row block), for long prompts; the
        caches receive the same keys and values a token-by-token pass appends."""
        prompt = [int(t) for t in prompt]
        P = len(prompt)
        assert P >= 1
        h = None
        if batched:
            H0 = self.m.w("embed")[np.asarray(prompt, dtype=np.int64)]
            full = forward_rows(self.m, H0, "layer", self.L, layers_out=sorted(set(self.anchor_layers) | {self.L}),
                                caches=self.caches)
            G = np.stack([self.feature([full[b][p] for b in self.anchor_layers], self.n) for p in range(P)])
            forward_rows(self.m, G, "pdm.layer", self.ls, layers_out=[], caches=self.pdm_caches)
            h = full[self.L][P - 1]
        else:
            for p, t in enumerate(prompt):
                h, kept = self._run_stage_range(embed(self.m, t), p, 0, self.n, capture=True)
                self.pdm_row(self.feature(kept, self.n), p)
        lg = lm_logits(self.m, h)
        x = argmax_first(lg) if self.sampling is None else smp.sample(
            self._target_dist(lg), self.sampling.u(P, smp.U_RESAMPLE))
        self.toks = prompt + [x]
        self.prompt_len = P
        self.c = P
        self._push(x, P)
        self.a = 1
        self.steps = 0
        self.verified = 1
        return x

    def _run_stage_range(self, h, pos, s0, s1, capture=False, anchors=None):
        """Run stages s0..s1-1 on one token; anchors[j] := H^{beta_j} as each stage completes."""
        kept = list(anchors) if anchors is not None else [h.copy()]
        for s in range(s0, s1):
            for l in range(self.beta[s], self.beta[s + 1]):
                h = decoder_layer(self.sh, self.m.layer(l), h, pos, self.caches[l])
            if s + 1 <= self.n - 1:
                if len(kept) == s + 1:
                    kept.append(h.copy())
                else:
                    kept[s + 1] = h.copy()
        return (h, kept) if capture else h

    def _push(self, tok: int, pos: int) -> None:
        e = embed(self.m, tok)
        self.hidden[pos] = e.copy()
        self.anch[pos] = [e.copy()]

    # ------------------------------------------------------------------ one step
    def depth(self, pos: int) -> int:
        return self.a - 1 - (pos - self.c) if pos >= self.c else self.n

    def step(self, forced_draft: Optional[int] = None, want_logits: bool = False) -> StepResult:
        c, a, n = self.c, self.a, self.n
        depths = {q: self.depth(q) for q in range(0, c + a)}

        def run_pdm(shift):
            # rows c..c+a-1 rewritten at depth (pre-step depth + shift), rows < c kept
            for pc in self.pdm_caches:
                pc.truncate(c)
            out = {}
            for i in range(a):
                q = c + i
                out[q] = self.pdm_row(self.feature(self.anch[q], a - 1 - i + shift), q)
            return out

        def run_target():
            # the token at depth s runs stage s
            for i in range(a):
                q = c + i
                s = a - 1 - i
                h, kept = self._run_stage_range(self.hidden[q], q, s, s + 1, capture=True, anchors=self.anch[q])
                self.hidden[q] = h
                self.anch[q] = kept

        if self.schedule == "pre":  # the PDM reads only pre-step features (Section 3.3)
            pdm_h = run_pdm(0)
            run_target()
        else:  # post-step: every in-flight token one stage deeper
            run_target()
            pdm_h = run_pdm(1)
        pdm_lg = self.pdm_logits(pdm_h[c + a - 1])
        dpos = c + a  # the draft's position
        if self.sampling is None:
            qd = None
            pdm_draft = self.pdm_token(argmax_first(pdm_lg))
        else:
            ids, probs = self._target_dist(pdm_lg)  # over draft ids, then as target tokens
            qd = (np.array([self.pdm_token(i) for i in ids], dtype=np.int64), probs)
            pdm_draft = smp.sample(qd, self.sampling.u(dpos, smp.U_DRAFT))
        draft = pdm_draft if forced_draft is None else int(forced_draft)
        q_draft = None if qd is None else (qd if forced_draft is None else smp.point_mass(draft))

        self.steps += 1
        res = StepResult(NONE, -1, draft, pdm_draft, -1, -1, -1, 0, 0, depths=depths,
                         pdm_hidden=pdm_h, pdm_dist=qd)
        if want_logits:
            res.pdm_logits = pdm_lg
        if q_draft is not None:
            self.qdist[dpos] = q_draft  # kept with the token while it is in flight
        if a == n:
            lg = lm_logits(self.m, self.hidden[c])
            succ = self.toks[c + 1] if n >= 2 else draft
            if self.sampling is None:
                y = argmax_first(lg)
            else:
                pd = self._target_dist(lg)
                ok, y = smp.rejection_verify(pd, self.qdist[c + 1], succ,
                                             self.sampling.u(c + 1, smp.U_ACCEPT),
                                             self.sampling.u(c + 1, smp.U_RESAMPLE))
                res.exit_dist, res.accepted_by_ratio = pd, ok
                del self.qdist[c + 1]  # judged once; committed from here on
            res.target_argmax, res.exited_pos, res.verified_pos, res.verified_token = y, c, c + 1, y
            if want_logits:
                res.exit_logits = lg
            del self.hidden[c], self.anch[c]
            self.c = c + 1
            self.verified += 1
            if succ == y:
                res.decision = ACCEPT
                q = c + a  # the draft's position
                self._set_tok(q, draft)
                self._push(draft, q)
            else:
                res.decision = REJECT
                self._truncate_to(self.c)
                self._set_tok(self.c, y)
                self._push(y, self.c)
                self.a = 1
        else:
            q = c + a
            self._set_tok(q, draft)
            self._push(draft, q)
            self.a = a + 1
        res.c, res.a = self.c, self.a
        return res

    def _set_tok(self, q: int, t: int) -> None:
        if q < len(self.toks):
            self.toks[q] = t
            del self.toks[q + 1:]
        else:
            assert q == len(self.toks)
            self.toks.append(t)

    def _truncate_to(self, keep: int) -> None:
        for cch in self.caches:
            cch.truncate(min(cch.n, keep))
        for pc in self.pdm_caches:
            pc.truncate(min(pc.n, keep))
        for q in [q for q in self.hidden if q >= keep]:
            del self.hidden[q], self.anch[q]
        for q in [q for q in self.qdist if q >= keep]:
            del self.qdist[q]
        del self.toks[keep:]

    def rollback(self, keep_len: int, reseed: int) -> None:
        """Keep positions < keep_len in every cache, drop in-flight work, reseed at keep_len."""
        assert self.prompt_len <= keep_len <= self.c
        self.c = keep_len
        self._truncate_to(keep_len)
        self._set_tok(keep_len, int(reseed))
        self._push(int(reseed), keep_len)
        self.a = 1

    # ------------------------------------------------------------------ views
    def generated(self) -> List[int]:
        """Verified tokens after the prompt: positions prompt_len..c (tok[c] is always verified)."""
        return self.toks[self.prompt_len: self.c + 1]

    def kv_lengths(self) -> List[int]:
        return [cc.n for cc in self.caches]

    def alpha(self) -> float:
        """Step acceptance ratio N/K (Section 4.2), N counting generated tokens."""
        return self.verified / max(1, self.steps)


def run_spd(model: Model, prompt, n_tokens: int, n: Optional[int] = None,
            draft_for: Optional[Callable[[int], Optional[int]]] = None, max_steps: int = 100000,
            sampling: Optional[smp.Sampling] = None, schedule: str = "pre"):
    """Run SPD until n_tokens generated tokens are verified. draft_for(position) may force drafts.

    Returns (oracle, list of StepResult)."""
    o = SPDOracle(model, n=n, sampling=sampling, schedule=schedule)
    o.prefill(prompt)
    results = []
    while o.verified < n_tokens and len(results) < max_steps:
        q = o.c + o.a
        fd = draft_for(q) if draft_for is not None else None
        results.append(o.step(forced_draft=fd))
    return o, results


def simulate_steps(n: int, n_tokens: int, accept_at: Callable[[int], bool], prompt_len: int) -> int:
    """Step count from the pipeline's timing alone: the first exit is n steps after prefill; after
    an exit verifying position q the next exit comes 1 step later if q was accepted, n if not."""
    if n_tokens <= 1:
        return 0
    t, verified, q = n, 2, prompt_len + 1  # the exit at step n verifies position prompt_len+1
    while verified < n_tokens:
        t += 1 if accept_at(q) else n
        q += 1
        verified += 1
    return t


# ----------------------------------------------------------------------------- accounting (Sec. 4.2)
def step_acceptance(n_tokens: int, n_steps: int) -> float:
    """alpha = N / K: generated tokens per executed pipeline step."""
    return n_tokens / n_steps


def speedup_zero_cost(alpha: float, n: int) -> float:
    """Eq. s0-spd: each step advances n stage tokens at 1/n of a full forward, so S0 = alpha * n."""
    return alpha * n


def speedup_serial_draft(s0: float, n_layers: int, draft_layers: int, draft_calls: int) -> float:
    """Eq. s-eagle: when drafting is not hidden, every step also pays draft_calls passes of an
    L_s-layer drafter, measured in target layers: S = S0 * L / (L_s * draft_calls + L). For PPSD and
    the post-step ablation draft_calls = n; for EAGLE-3 it is the draft length k."""
    return s0 * n_layers / (draft_layers * draft_calls + n_layers)

