"""GPU parity of sampled decoding (top-k, temperature, rejection-sampling verify) through the C ABI.

Random numbers are inputs (three uniforms per position), so the HIP path and the oracle make the same
draws. The oracle and the kernels compute logits in different precisions, so every uniform is first
moved, by the oracle alone, at least TOL_U away from every decision boundary it meets (the CDF
boundaries of each draw and the acceptance ratio p(x)/q(x)), staying inside the interval it was in,
so the oracle's run is unchanged; after that the HIP path must make every decision the oracle makes:
draft, acceptance, committed token, pipeline state, step by step. The draft distributions the HIP path
keeps with the in-flight tokens must hold the oracle's top-k ids (the last place may differ when the
oracle's k-th and (k+1)-th logits are closer than TIE), each with its probability to PROB_ABS, in the
oracle's order except between entries whose logits lie within twice the measured logit error.
At any size: top_k = 1 is greedy decoding, bit for bit; and at the 4B-class size the kept
distribution is exactly the top-50 of the HIP path's own logits with their softmax."""
import sys

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import sampling as smp
from oracle import spd as osp

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 11
TOL_U = 5e-3
TIE = 1e-3
PROB_ABS = 1e-4


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


def _engine(w, n, max_tokens, **kw):
    from paper_2605_30852_amd.engine import Engine
    return Engine(w, max_tokens=max_tokens, n=n, page_seed=5, **kw)


def _intervals(weights):
    w = np.asarray(weights, dtype=np.float64)
    cs = np.cumsum(w) / w.sum()
    return np.concatenate([[0.0], cs[:-1]]), np.concatenate([cs[:-1], [1.0]])


def _settle(u, uses, tol_u=TOL_U):
    """A float32 value for one uniform that lies at least TOL_U inside its interval in every
    inverse-CDF draw it takes part in (uses: (weights, avoid_last) each; avoid_last: never the last
    entry, whose top-k membership is a near tie). The draws the current u makes are kept when some
    value allows that (the nearest such value), else the value with the widest clearance is taken
    (the run then changes, and the caller runs again)."""
    grid = (np.arange(20000) + 0.5) / 20000.0
    keep = np.ones_like(grid, dtype=bool)
    margin = np.full_like(grid, np.inf)
    ok_now = True
    for w, avoid_last in uses:
        lo, hi = _intervals(w)
        i = smp.sample_index(w, u)
        if not (lo[i] + tol_u <= u < hi[i] - tol_u) or (avoid_last and i == len(lo) - 1):
            ok_now = False
        keep &= (grid >= lo[i] + 1.5 * tol_u) & (grid < hi[i] - 1.5 * tol_u)
        if avoid_last and i == len(lo) - 1:
            keep[:] = False
        j = np.searchsorted(hi, grid, side="right").clip(max=len(lo) - 1)
        m = np.minimum(grid - lo[j], hi[j] - grid)
        if avoid_last:
            m = np.where(j == len(lo) - 1, -1.0, m)
        margin = np.minimum(margin, m)
    if ok_now:
        return u
    if keep.any():
        cand = grid[keep]
        v = cand[np.argmin(np.abs(cand - u))]
    else:
        v = grid[np.argmax(margin)]
    return float(np.float32(v))


def _oracle_run(model, prompt, n, k, temp, U, steps, draft_for, nudge, schedule="pre", tol_u=TOL_U):
    """One oracle run; with nudge, every uniform the run draws with is settled clear of its decision
    boundaries (in place; see _settle). Returns (results, near-tie positions, moved?)."""
    ora = osp.SPDOracle(model, n=n, sampling=smp.Sampling(k, temp, U), schedule=schedule)
    ties = set()
    uses = {}
    P = len(prompt)
    ora.prefill(prompt)
    lg = om.lm_logits(model, om.forward_full(model, prompt, layers_out=[model.shape.n_layers])[model.shape.n_layers][-1])
    uses.setdefault((P, smp.U_RESAMPLE), []).append((smp.top_k_dist(lg, k, temp)[1], _kth_gap(lg, k) < TIE))
    out = []
    for _ in range(steps):
        c, a = ora.c, ora.a
        dpos = c + a
        fd = draft_for(dpos) if draft_for else None
        q_succ = ora.qdist.get(c + 1)
        succ = ora.toks[c + 1] if (a == n and n >= 2) else None
        r = ora.step(forced_draft=fd, want_logits=True)
        out.append(r)
        tie = fd is None and _kth_gap(r.pdm_logits, k) < TIE
        if tie:
            ties.add(dpos)
        if fd is None:  # a position is drafted again after a reject, with the same u_draft
            uses.setdefault((dpos, smp.U_DRAFT), []).append((r.pdm_dist[1], tie))
        if a == n:
            if n == 1:
                succ = r.draft
                q_succ = r.pdm_dist if fd is None else smp.point_mass(fd)
            p = r.exit_dist
            ratio = smp.prob_of(p, succ) / smp.prob_of(q_succ, succ)
            if ratio < 1.0:  # accept iff u < ratio
                uses.setdefault((c + 1, smp.U_ACCEPT), []).append(([ratio, 1.0 - ratio], False))
            if not r.accepted_by_ratio:
                res = np.array([max(0.0, p[1][i] - smp.prob_of(q_succ, p[0][i])) for i in range(len(p[0]))])
                w = res if res.sum() > 0.0 else p[1]
                uses.setdefault((c + 1, smp.U_RESAMPLE), []).append((w, _kth_gap(r.exit_logits, k) < TIE))
    moved = False
    if nudge:
        for (pos, j), us in uses.items():
            v = _settle(float(U[pos, j]), us, tol_u)
            if v != U[pos, j]:
                U[pos, j] = v
                moved = True
    return out, ties, moved


def _check_kept(gi, gp, ids, probs, tie, swap, p_tol, tag):
    """The kept top-k list of one position against the oracle's. The verify reads it only as a map
    from ids to probabilities (q(x) and max(0, p - q) per id), so each id's probability is compared
    by id. The order must be the oracle's except between entries whose oracle log-probabilities lie
    within `swap` of each other (logits off by e can reorder any two closer than 2e); where the
    oracle's k-th and (k+1)-th logits nearly tie, one id may be the oracle's (k+1)-th instead."""
    where = {int(t): j for j, t in enumerate(ids)}
    pos = [where.get(int(t), -1) for t in gi]
    assert sum(j < 0 for j in pos) <= (1 if tie else 0), f"{tag}: ids {list(gi)} vs {list(ids)}"
    assert len(set(pos)) == len(pos), f"{tag}: repeated ids {list(gi)}"
    lp = np.log(np.asarray(probs, dtype=np.float64))
    mine = [(j, lp[i]) for j, i in enumerate(pos) if i >= 0]
    lowest = np.inf  # oracle log-probabilities must not rise along the kept order beyond `swap`
    for j, v in mine:
        assert v <= lowest + swap, f"{tag}: place {j} (id {gi[j]}) out of order beyond {swap:.2e}"
        lowest = min(lowest, v)
    got = np.array([gp[j] for j, _ in mine])
    want = np.array([probs[pos[j]] for j, _ in mine])
    np.testing.assert_allclose(got, want, atol=p_tol, err_msg=tag)


def _clear_uniforms(model, prompt, n, k, temp, rows, steps, draft_for, seed, schedule="pre", tol_u=TOL_U):
    U = np.random.default_rng([seed, 3]).random((rows, 3)).astype(np.float32).astype(np.float64)
    for _ in range(20):
        _, _, moved = _oracle_run(model, prompt, n, k, temp, U, steps, draft_for, nudge=True, schedule=schedule,
                                  tol_u=tol_u)
        U = U.astype(np.float32).astype(np.float64)  # the values the GPU sees
        U[U >= 1.0] = float(np.nextafter(np.float32(1.0), np.float32(0.0)))
        if not moved:
            return U
    raise AssertionError("uniforms did not settle away from the decision boundaries")


def _kth_gap(logits, k):
    s = np.sort(np.asarray(logits, dtype=np.float64))[::-1]
    return s[k - 1] - s[k] if k < len(s) else np.inf


@pytest.mark.parametrize("which,n,k,temp,forced,schedule,head", [
    ("tiny", 1, 8, 1.0, False, "pre", "fused"), ("tiny", 2, 8, 0.5, True, "pre", "fused"),
    ("tiny", 2, 64, 1.0, False, "pre", "fused"), ("tiny", 3, 16, 0.2, True, "pre", "fused"),
    ("tiny", 4, 50, 0.7, False, "pre", "fused"), ("tiny", 3, 16, 0.5, False, "post", "fused"),
    ("tiny", 2, 16, 0.5, False, "pre", "unfused"), ("tiny", 2, 16, 0.5, False, "pre", "own"),
    ("tiny", 3, 8, 0.3, True, "post", "own"),
    ("mid", 3, 50, 1.0, False, "pre", "fused"), ("mid", 2, 16, 0.7, True, "pre", "fused"),
    ("mid", 3, 50, 1.0, False, "pre", "unfused")])
def test_sampled_lockstep_matches_oracle(tiny_w, mid_w, which, n, k, temp, forced, schedule, head):
    """head: the two-row pass ("fused"), the PDM's own pass over the shared head ("unfused") or over
    its own 300-token head ("own"); the last two select q in the PDM's pass and p in the exit row's.
    which: the fp32 tiny model, or the bf16 mid model (the kernels' sampled head in its bf16 form),
    whose logits differ from the oracle's by more: its uniforms are kept 1e-2 clear of every decision
    boundary, and the kept probabilities may differ by what the measured logit error allows
    (p * (exp(2 e / T) - 1) <= exp(2 e / T) - 1 for a logit error e)."""
    _say(f"[sampled lockstep {which} n={n} k={k} T={temp} forced={forced} schedule={schedule} head={head}]")
    base = tiny_w if which == "tiny" else mid_w
    w = base.with_pdm_vocab(300) if head == "own" else base
    tol_u = TOL_U if which == "tiny" else 1e-2
    sh = w.shape
    model = om.Model(sh, SEED)
    prompt = synth.prompt(sh, SEED, 21)
    P, steps, rows = len(prompt), 28, 96
    draft_for = None
    if forced:
        ref = om.ar_greedy(model, prompt, 40)
        mask = synth.accept_mask(0.7, SEED + n, rows + 8)
        table = {P + i: (int(t) if mask[P + i] else int((t + 1) % sh.vocab)) for i, t in enumerate(ref)}
        draft_for = table.get
    U = _clear_uniforms(model, prompt, n, k, temp, rows, steps, draft_for, seed=100 * n + k, schedule=schedule,
                        tol_u=tol_u)
    _, ties, _ = _oracle_run(model, prompt, n, k, temp, U, steps, draft_for, nudge=False, schedule=schedule,
                             tol_u=tol_u)
    ora = osp.SPDOracle(model, n=n, sampling=smp.Sampling(k, temp, U), schedule=schedule)
    eng = _engine(w, n, rows, fused_head=head == "fused")
    eng.spd_set_pdm_schedule(schedule == "post")
    eng.spd_set_sampling(k, temp, U)
    eng.spd_set_debug(True)
    assert eng.spd_prefill(prompt) == ora.prefill(prompt)
    accepts = rejects = 0
    lg_err = 0.0  # the largest logit error seen so far (PDM and exit rows)
    for i in range(steps):
        dpos = ora.c + ora.a
        fd = draft_for(dpos) if draft_for else None
        ro = ora.step(forced_draft=fd, want_logits=True)
        rg = eng.spd_step(fd)
        tag = f"step {i} (c={ro.c} a={ro.a})"
        lg_err = max(lg_err, float(np.max(np.abs(eng.pdm_logits() - ro.pdm_logits))))
        if ro.exit_logits is not None:
            lg_err = max(lg_err, float(np.max(np.abs(eng.exit_logits() - ro.exit_logits))))
        assert lg_err <= 5e-2, f"{tag}: logits max abs {lg_err:.3e}"
        p_tol = PROB_ABS if which == "tiny" else PROB_ABS + float(np.expm1(2.0 * lg_err / temp))
        assert rg.decision == ro.decision, tag
        # the library reports no pushed draft on a reject (the in-flight tokens are dropped)
        assert (rg.draft, rg.pdm_draft) == (-1 if ro.decision == osp.REJECT else ro.draft, ro.pdm_draft), tag
        assert (rg.committed_len, rg.inflight) == (ro.c, ro.a), tag
        if ro.decision != osp.NONE:
            assert (rg.exited_pos, rg.verified_pos, rg.verified_token) == \
                   (ro.exited_pos, ro.verified_pos, ro.verified_token), tag
            accepts += ro.decision == osp.ACCEPT
            rejects += ro.decision == osp.REJECT
        for q, (ids, probs) in ora.qdist.items():
            gi, gp = eng.qdist(q)
            assert len(gi) == len(ids), f"{tag}: q of position {q} has {len(gi)} entries, oracle {len(ids)}"
            _check_kept(gi, gp, ids, probs, q in ties, 2.0 * lg_err / temp, p_tol, f"{tag}: q of position {q}")
    toks = eng.tokens()
    assert list(toks[: ora.c + 1]) == ora.toks[: ora.c + 1]
    eng.close()
    _say(f"  {accepts} accepts, {rejects} rejects, c={ora.c}, worst logit error {lg_err:.2e}")
    assert accepts + rejects >= steps // n  # after a reject the pipeline refills for n - 1 steps
    if forced:
        assert accepts >= 1


@pytest.mark.parametrize("n,forced", [(2, False), (3, True)])
def test_top_k_one_is_greedy_bit_exact(tiny_w, n, forced):
    _say(f"[top_k=1 vs greedy n={n} forced={forced}]")
    sh = synth.TINY
    prompt = synth.prompt(sh, SEED, 19)
    rows = 80
    U = np.random.default_rng(7).random((rows, 3))
    logs = []
    for k in (0, 1):
        eng = _engine(tiny_w, n, rows)
        if k:
            eng.spd_set_sampling(1, 1.0, U)
        x = eng.spd_prefill(prompt)
        if forced:
            ref = om.ar_greedy(om.Model(sh, SEED), prompt, 30)
            eng.spd_set_forced_drafts(np.array([t if i % 4 else (t + 3) % sh.vocab for i, t in enumerate(ref)],
                                               dtype=np.int32), len(prompt))
        log = [x] + [eng.spd_step().as_dict() for _ in range(30)]
        logs.append((log, list(eng.tokens())))
        eng.close()
    assert logs[0] == logs[1]


def test_sampling_setter_rules(tiny_w):
    from paper_2605_30852_amd.binding import SPDError
    rows = 64
    U = np.random.default_rng(1).random((rows, 3))
    eng = _engine(tiny_w, 2, rows)
    with pytest.raises(SPDError):
        eng.spd_set_sampling(65, 1.0, U)  # top_k above 64
    with pytest.raises(SPDError):
        eng.spd_set_sampling(8, 0.0, U)  # temperature 0
    with pytest.raises(SPDError):
        eng.spd_set_sampling(8, 1.0, U[:-1])  # not max_tokens rows
    bad = U.copy()
    bad[5, 1] = 1.0
    with pytest.raises(SPDError):
        eng.spd_set_sampling(8, 1.0, bad)  # outside [0, 1)
    eng.spd_set_sampling(8, 1.0, U)
    eng.spd_prefill(synth.prompt(synth.TINY, SEED, 9))
    with pytest.raises(SPDError):
        eng.spd_set_sampling(0)  # only before prefill
    eng.close()


def test_fullsize_4b_sampled_step_selection():
    """4B-class n = 4 with top-k 50 at T = 1 in the benchmark's launch form (stage groups, step
    graph): after every step the kept draft distribution of the newest token is the top-50 of the
    HIP path's own PDM logits (value descending) with their softmax, and every committed token lies in
    the top-50 of the exit logits; top_k = 1 reproduces greedy decoding bit for bit."""
    from paper_2605_30852_amd.engine import DeviceWeights, Engine

    sh = synth.B4
    n, P, seed, rows = sh.n_stages, 20, 0, 96
    prompt = synth.prompt(sh, seed, P)
    _say("[fullsize 4b sampled] uploading weights")
    W = DeviceWeights(sh, seed, threads=16)
    U = np.random.default_rng(5).random((rows, 3))
    logs = []
    for k in (0, 1):
        eng = Engine(W, max_tokens=rows, n=n)
        if k:
            eng.spd_set_sampling(1, 1.0, U)
        eng.spd_set_graph(True)
        x = eng.spd_prefill(prompt)
        logs.append([x] + [r for r in eng.spd_run_steps(10, want_log=True)])
        eng.close()
    assert logs[0] == logs[1]
    _say("[fullsize 4b sampled] top_k=1 equals greedy; top-50 selection")
    eng = Engine(W, max_tokens=rows, n=n)
    eng.spd_set_sampling(50, 1.0, U)
    eng.spd_set_graph(True)
    eng.spd_set_debug(True)
    eng.spd_prefill(prompt)
    exits = 0
    for i in range(10):
        r = eng.spd_run_steps(1, want_log=True)[0]
        c, a, _, _ = eng.state()
        if r["decision"] == osp.REJECT:
            continue
        pl = eng.pdm_logits().astype(np.float32)
        order = np.lexsort((np.arange(len(pl)), -pl))[:50]
        ids, probs = eng.qdist(c + a - 1)
        np.testing.assert_array_equal(ids, order, err_msg=f"step {i}")
        z = pl[order].astype(np.float64)
        w = np.exp(z - z[0])
        np.testing.assert_allclose(probs, w / w.sum(), rtol=1e-4, atol=1e-7, err_msg=f"step {i}")
        if r["decision"] != osp.NONE:
            exits += 1
            el = eng.exit_logits().astype(np.float32)
            top = set(np.lexsort((np.arange(len(el)), -el))[:50].tolist())
            assert r["verified_token"] in top
    eng.close()
    _say(f"[fullsize 4b sampled] {exits} exits checked")


def _pit(ids, probs, tok, w):
    """A point w of the way through token tok's interval of the inverse CDF in the listed order; U(0, 1)
    over draws when tok follows (ids, probs) and w is an independent uniform."""
    probs = np.asarray(probs, dtype=np.float64)
    probs = probs / probs.sum()
    hit = np.nonzero(np.asarray(ids) == tok)[0]
    assert hit.size == 1, f"token {tok} outside the distribution"
    j = int(hit[0])
    return float(probs[:j].sum() + w * probs[j])


def test_fullsize_4b_sampled_tokens_follow_their_distributions():
    """Any size: under sampled decoding (top-50, T = 1) with the PDM's own draws, each committed
    token follows the exit's top-50 distribution p (the rejection-sampling guarantee) and each draw of
    the PDM follows its q. With p and q built from the HIP path's own logits, the randomised
    probability-integral transform of every committed token and every draft is uniform (KS test),
    at the 4B-class size in the benchmark's launch form (stage groups, step graph)."""
    from scipy import stats

    from paper_2605_30852_amd.engine import DeviceWeights, Engine

    sh = synth.B4
    n, P, rows, steps = 2, 24, 400, 300
    prompt = synth.prompt(sh, 0, P)
    _say("[fullsize 4b PIT] uploading weights")
    W = DeviceWeights(sh, 0, threads=16)
    U = np.random.default_rng(9).random((rows, 3))
    eng = Engine(W, max_tokens=rows, n=n)
    eng.spd_set_sampling(50, 1.0, U)
    eng.spd_set_graph(True)
    eng.spd_set_debug(True)
    eng.spd_prefill(prompt)
    rng = np.random.default_rng(21)
    pit_p, pit_q, accepts = [], [], 0
    for i in range(steps):
        r = eng.spd_run_steps(1, want_log=True)[0]
        if r["decision"] != osp.NONE:
            el = eng.exit_logits().astype(np.float64)
            order = np.lexsort((np.arange(len(el)), -el))[:50]
            z = el[order]
            pit_p.append(_pit(order, np.exp(z - z[0]), r["verified_token"], rng.random()))
            accepts += r["decision"] == osp.ACCEPT
        if r["decision"] != osp.REJECT:  # the newest token is the PDM's draw, kept with its q
            c, a, _, _ = eng.state()
            ids, probs = eng.qdist(c + a - 1)
            pit_q.append(_pit(ids, probs, r["pdm_draft"], rng.random()))
    eng.close()
    ks_p = stats.kstest(pit_p, "uniform")
    ks_q = stats.kstest(pit_q, "uniform")
    _say(f"[fullsize 4b PIT] {len(pit_p)} exits ({accepts} accepts), KS p = {ks_p.pvalue:.3f}; "
         f"{len(pit_q)} drafts, KS p = {ks_q.pvalue:.3f}")
    assert len(pit_p) >= 100 and len(pit_q) >= 100
    assert ks_p.pvalue > 1e-3 and ks_q.pvalue > 1e-3
