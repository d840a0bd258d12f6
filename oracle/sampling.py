"""Oracle, part 3: sampled decoding for SPD, in float64 on the CPU.

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

What it follows:
  * Sampling setting of Section 4.1: temperature T, top-k filter, top-p 1.0 (no nucleus cut). A
    distribution over the vocabulary is the softmax of logits/T restricted to the k largest logits
    (order: value descending, lowest index first among equal values, as in greedy decoding).
  * Verification under sampling (Section 3.4: standard rejection sampling). Read as the
    speculative-sampling rule: a draft x drawn from the draft distribution q is kept with probability
    min(1, p(x)/q(x)), where p is the target's distribution at that position; otherwise the token is
    drawn from the residual max(0, p - q), normalised. The emitted token then follows p exactly. The
    reseed token of a reject is that residual draw (with greedy decoding it is the target's argmax).
  * Random numbers are inputs: each position owns three uniforms on [0, 1): u_draft (the draft module
    samples the token at that position), u_accept (the acceptance test of that position) and
    u_resample (the residual draw, or the plain draw of the prompt's first token).
  * A draw from (ids, probs) by inverse CDF in the listed order: the first i with u * S < cumsum_i,
    S the total mass (the last entry if rounding leaves none).
"""
from __future__ import annotations

import dataclasses
from typing import Tuple

import numpy as np

Dist = Tuple[np.ndarray, np.ndarray]  # (ids int64[m], probs float64[m]), value-descending order


@dataclasses.dataclass(frozen=True)
class Sampling:
    """top_k >= 1, temperature > 0, uniforms [positions, 3] on [0, 1): (u_draft, u_accept, u_resample)."""
    top_k: int
    temperature: float
    uniforms: np.ndarray

    def u(self, pos: int, which: int) -> float:
        return float(self.uniforms[pos, which])


U_DRAFT, U_ACCEPT, U_RESAMPLE = 0, 1, 2


def top_k_dist(logits: np.ndarray, k: int, temperature: float) -> Dist:
    """The top-k, temperature-T distribution: the k largest logits (ties: lower index first), their
    softmax at temperature T (max-subtracted), in that order."""
    logits = np.asarray(logits, dtype=np.float64)
    v = logits.shape[0]
    k = min(int(k), v)
    order = np.lexsort((np.arange(v), -logits))  # last key is primary: value descending, then index
    ids = order[:k].astype(np.int64)
    z = logits[ids] / float(temperature)
    w = np.exp(z - z[0])
    return ids, w / w.sum()


def point_mass(tok: int) -> Dist:
    """A draft that did not come from the draft module (a forced draft) has q = delta_tok."""
    return np.array([int(tok)], dtype=np.int64), np.array([1.0])


def sample_index(weights: np.ndarray, u: float) -> int:
    """Inverse CDF over nonnegative weights in their listed order: first i with u*S < cumsum_i."""
    cs = np.cumsum(np.asarray(weights, dtype=np.float64))
    hit = np.nonzero(u * cs[-1] < cs)[0]
    return int(hit[0]) if hit.size else len(cs) - 1


def sample(dist: Dist, u: float) -> int:
    ids, probs = dist
    return int(ids[sample_index(probs, u)])


def prob_of(dist: Dist, tok: int) -> float:
    ids, probs = dist
    hit = np.nonzero(ids == int(tok))[0]
    return float(probs[hit[0]]) if hit.size else 0.0


def rejection_verify(p: Dist, q: Dist, x: int, u_accept: float, u_resample: float) -> Tuple[bool, int]:
    """Keep x with probability min(1, p(x)/q(x)) (accept iff u*q(x) < p(x)); otherwise draw from
    max(0, p - q) normalised, over p's support in p's order (from p itself if that mass is zero).

    Returns (accepted, emitted token)."""
    px, qx = prob_of(p, x), prob_of(q, x)
    if u_accept * qx < px:
        return True, int(x)
    ids, probs = p
    resid = np.array([max(0.0, probs[i] - prob_of(q, ids[i])) for i in range(len(ids))])
    w = resid if resid.sum() > 0.0 else probs
    return False, int(ids[sample_index(w, u_resample)])
