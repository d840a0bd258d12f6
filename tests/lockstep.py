"""Run the HIP path (through the C ABI) and the CPU oracle side by side and compare every step.

Tolerances (float results): hidden states relative L2 <= 2e-2; logits max abs <= 5e-2; top-1 tokens
identical unless the oracle's top-2 margin is below 1e-2 (both choices are then correct). The last two
are read together: a row whose logits differ from the oracle's by e (at most 5e-2) can reorder any two
logits closer than 2e, so a top-1 difference is also accepted where the oracle's margin is below 2e,
the GPU's choice being a logit of the oracle's within 2e of its maximum; such cases are counted. Where such a
near tie makes the two runs choose different tokens, both are brought back to the same state with the
same rollback (keep the committed prefix, reseed the oracle's token at depth 0) and the comparison goes
on; a near tie of the draft module's argmax while the draft is forced changes nothing on the target
path and is only counted. Every step is compared: a run returns only after all n_steps were."""
import sys

import numpy as np

from oracle import model as om
from oracle import spd as osp

REL_HIDDEN = 2e-2
ABS_LOGIT = 5e-2
TIE_MARGIN = 1e-2


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def margin(logits) -> float:
    top = np.sort(np.asarray(logits))[-2:]
    return float(top[1] - top[0])


def top1_explained(oracle_logits, gpu_logits, gpu_choice) -> bool:
    """A top-1 difference both tolerances allow: the oracle's top-2 margin is below TIE_MARGIN, or the
    GPU's choice is within twice the row's measured logit error (<= ABS_LOGIT) of the oracle's maximum."""
    lo = np.asarray(oracle_logits, dtype=np.float64)
    e = float(np.max(np.abs(np.asarray(gpu_logits, dtype=np.float64) - lo)))
    gap = float(lo.max() - lo[int(gpu_choice)])
    return margin(lo) < TIE_MARGIN or (e <= ABS_LOGIT and gap <= 2.0 * e)


class NearTie(Exception):
    pass


def compare_state(eng, ora, tag, worst):
    """In-flight residual streams and anchors of every in-flight position."""
    res = eng.resid()
    anch = eng.anchors()
    n = ora.n
    for q in range(ora.c, ora.c + ora.a):
        r = rel_l2(res[q % n], ora.hidden[q])
        worst["hidden"] = max(worst["hidden"], r)
        assert r <= REL_HIDDEN, f"{tag}: hidden state of position {q} rel L2 {r:.3e}"
        for j, an in enumerate(ora.anch[q]):
            r = rel_l2(anch[q % n][j], an)
            worst["hidden"] = max(worst["hidden"], r)
            assert r <= REL_HIDDEN, f"{tag}: anchor {j} of position {q} rel L2 {r:.3e}"


def run_lockstep(eng, model, prompt, n_steps, draft_for=None, check_pdm=True, log=None, schedule="pre",
                 max_resyncs=None, batched_prefill=False):
    """eng: paper_2605_30852_amd.engine.Engine. Runs n_steps steps on both sides and compares each:
    the draft module's rows and logits, the exit logits, decisions, (c, a), positions and every
    in-flight residual stream and anchor. Returns the worst errors and the counts of compared steps,
    near ties and re-synchronisations (at most max_resyncs, default n_steps // 4). schedule: the
    PDM's ("pre" or "post"); the engine is set to the same one. batched_prefill: the oracle's
    prefill as one causal forward over the prompt (for long prompts)."""
    ora = osp.SPDOracle(model, n=eng.n, schedule=schedule)
    eng.spd_set_pdm_schedule(schedule == "post")
    worst = {"hidden": 0.0, "logit": 0.0, "pdm_hidden": 0.0, "pdm_logit": 0.0, "steps": 0, "near_tie": 0,
             "pdm_near_tie": 0, "resyncs": 0}
    max_resyncs = n_steps // 4 if max_resyncs is None else max_resyncs

    def resync(tag):
        # the same rollback on both sides: keep the committed prefix, reseed the oracle's token
        keep, tok = ora.c, ora.toks[ora.c]
        eng.spd_rollback(keep, tok)
        ora.rollback(keep, tok)
        worst["resyncs"] += 1
        assert worst["resyncs"] <= max_resyncs, f"{tag}: too many near ties to compare ({worst})"

    eng.spd_set_debug(True)
    xg = eng.spd_prefill(prompt)
    xo = ora.prefill(prompt, batched=batched_prefill)
    if xg != xo:
        lg = om.lm_logits(ora.m, _last_prompt_hidden(ora, model, prompt))
        assert margin(lg) < TIE_MARGIN, f"prefill token {xg} != oracle {xo}"
        worst["near_tie"] += 1
        resync("prefill")
    compare_state(eng, ora, "prefill", worst)
    for i in range(n_steps):
        q = ora.c + ora.a
        fd = draft_for(q) if draft_for is not None else None
        rg = eng.spd_step(fd)
        ro = ora.step(forced_draft=fd, want_logits=True)
        tag = f"step {i} (c={ro.c} a={ro.a})"
        diverged = False
        # PDM: hidden rows and logits
        if check_pdm:
            ph = eng.pdm_hidden()
            c0 = min(ro.pdm_hidden)
            for qq, h in ro.pdm_hidden.items():
                r = rel_l2(ph[qq - c0], h)
                worst["pdm_hidden"] = max(worst["pdm_hidden"], r)
                assert r <= REL_HIDDEN, f"{tag}: PDM row {qq} rel L2 {r:.3e}"
            pl = eng.pdm_logits()
            e = float(np.max(np.abs(pl - ro.pdm_logits)))
            worst["pdm_logit"] = max(worst["pdm_logit"], e)
            assert e <= ABS_LOGIT, f"{tag}: PDM logits max abs {e:.3e}"
            if rg.pdm_draft != ro.pdm_draft:
                assert top1_explained(ro.pdm_logits, pl, rg.pdm_draft), \
                    f"{tag}: PDM draft {rg.pdm_draft} != oracle {ro.pdm_draft} (margin {margin(ro.pdm_logits):.3e})"
                worst["pdm_near_tie"] += 1
                diverged = diverged or fd is None  # a forced draft replaces both drafts
        if ro.exit_logits is not None:
            el = eng.exit_logits()
            e = float(np.max(np.abs(el - ro.exit_logits)))
            worst["logit"] = max(worst["logit"], e)
            assert e <= ABS_LOGIT, f"{tag}: exit logits max abs {e:.3e}"
            if rg.target_argmax != ro.target_argmax:
                assert top1_explained(ro.exit_logits, el, rg.target_argmax), \
                    f"{tag}: target argmax {rg.target_argmax} != {ro.target_argmax} (margin {margin(ro.exit_logits):.3e})"
                worst["near_tie"] += 1
                diverged = True
        if not diverged:
            assert rg.decision == ro.decision, f"{tag}: decision {rg.decision} != {ro.decision}"
            assert (rg.committed_len, rg.inflight) == (ro.c, ro.a), f"{tag}: (c, a) differ"
            if ro.decision != osp.NONE:
                assert (rg.exited_pos, rg.exited_token, rg.verified_pos, rg.verified_token) == \
                       (ro.exited_pos, ora.toks[ro.exited_pos], ro.verified_pos, ro.verified_token), tag
            compare_state(eng, ora, tag, worst)
        else:
            assert rg.committed_len == ro.c, f"{tag}: committed lengths differ after a near tie"
            resync(tag)
            compare_state(eng, ora, tag + " after re-sync", worst)
        worst["steps"] += 1
        if log is not None:
            log.append((rg.as_dict(), ro.decision))
    toks = eng.tokens()
    assert list(toks[: ora.c + 1]) == ora.toks[: ora.c + 1], "token streams differ"
    print("lockstep worst:", worst, file=sys.stderr)
    assert worst["steps"] == n_steps, worst
    return worst


def _last_prompt_hidden(ora, model, prompt):
    full = om.forward_full(model, prompt, layers_out=[model.shape.n_layers])
    return full[model.shape.n_layers][-1]


def forced_table(ref, mask, prompt_len, vocab):
    """draft override by position: the reference token where the mask bit is set, a wrong one else."""
    table = {}
    for i, t in enumerate(ref):
        q = prompt_len + i
        table[q] = int(t) if mask[q] else int((t + 1) % vocab)
    return table
