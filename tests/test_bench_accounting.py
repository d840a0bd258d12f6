"""The benchmark's byte accounting (CPU only): the algorithmic bytes the roofline figures divide by.

A full-pipeline step (a = n) streams every layer's weights once, reads each stage token's keys, writes
one K/V row per layer, makes one two-row pass over the LM head and runs the PDM over n rows; a step
with a < n in-flight tokens streams only stages 0..a-1. The PDM's rows share one cache, so its keys
and values are read once per step (through the newest row's position), not once per row. These are checked against sums written out
here from the shapes, independently of how bench.py arranges them."""
import pytest

import bench
import synth


def _layer(sh, esz):
    d, F = sh.d_model, sh.ffn_dim
    return (sh.q_dim * d + 2 * sh.kv_dim * d + d * sh.q_dim + 3 * F * d) * esz + 2 * d * 4


@pytest.mark.parametrize("sh,n,c", [(synth.B4, 4, 2300), (synth.B9, 4, 4200), (synth.B4, 8, 8300)])
def test_full_step_bytes_agree(sh, n, c):
    esz = 2
    tgt, pdm = bench.step_bytes(sh, n, sh.pdm_layers, c, esz, pdm_head=False)
    active = bench.step_bytes_active(sh, n, sh.pdm_layers, c, n, esz)
    assert abs((tgt + pdm) - active) <= sh.d_model * esz  # step_bytes also counts the exit row itself


def test_one_token_step_is_stage_zero_plus_head_and_pdm():
    sh, n, c, esz = synth.B4, 4, 2048, 2
    kv_tok = 2 * sh.kv_dim * esz
    stage0 = sh.n_layers // n  # beta_1 = floor(L / n)
    expect = stage0 * (_layer(sh, esz) + (c + 1) * kv_tok + kv_tok)  # keys 0..c read, one row written
    expect += sh.vocab * sh.d_model * esz  # the two-row head pass runs every step
    expect += sh.d_model * n * sh.d_model * esz + sh.pdm_layers * _layer(sh, esz)  # PDM projection, layer
    expect += sh.pdm_layers * ((c + 1) * kv_tok + kv_tok)  # PDM KV of its one row
    assert bench.step_bytes_active(sh, n, sh.pdm_layers, c, 1, esz) == expect


def test_steady_step_bytes_at_the_headline_size():
    """4B-class n = 4 at 2300 committed positions: 7.267 GB of layer weights, 0.778 GB of LM head,
    about 0.37 GB of keys and values, 0.26 GB for the PDM."""
    sh, esz = synth.B4, 2
    total = bench.step_bytes_active(sh, 4, 1, 2300, 4, esz)
    assert 8.6e9 < total < 8.75e9
    assert abs(sh.n_layers * _layer(sh, esz) - 7.267e9) < 5e6


@pytest.mark.parametrize("n,ls,c", [(4, 1, 2048), (8, 2, 32768)])
def test_pdm_kv_is_read_once_per_step(n, ls, c):
    """The a = n rows at positions c..c+n-1 all read one shared cache: keys and values 0..c+n-1 of each
    PDM layer once, plus the n rows written; the PDM's other bytes are its weights."""
    sh, esz = synth.B9, 2
    kv_tok = 2 * sh.kv_dim * esz
    _, pdm = bench.step_bytes(sh, n, ls, c, esz, pdm_head=False)
    weights = sh.d_model * n * sh.d_model * esz + ls * _layer(sh, esz)
    assert pdm - weights == ls * (c + n) * kv_tok + ls * n * kv_tok
    # a per-row count would have read sum_i (c + i + 1) keys per layer instead
    assert pdm - weights < ls * sum(c + i + 1 for i in range(n)) * kv_tok


@pytest.mark.parametrize("L,n,groups,first_slot,expect", [
    (36, 4, 2, 4, 2.0),            # 9 layers per stage: every timed launch covers its group's 2 stages
    (36, 4, 1, 4, 4.0),
    (36, 8, 1, 2, (8 + 8 + 4) / 3),  # stages of 4 or 5 layers: slot 4 has only the four 5-layer stages
    (36, 8, 2, 2, 10 / 3),         # per group (4 stages): 4, 4, 2 in slots 2, 3, 4
    (36, 6, 2, 3, 3.0),
])
def test_timed_stage_launches_count_only_active_stages(L, n, groups, first_slot, expect):
    """The per-launch bytes of the kernel timing divide by launches of layer slots >= first_slot; a
    stage shorter than the longest is idle in the last slot and moves nothing there."""
    assert bench.timed_stages_per_launch(L, n, groups, first_slot) == pytest.approx(expect)


class _SlowPrefill:
    def __init__(self, secs, fail=False):
        self.secs, self.fail = secs, fail

    def spd_prefill(self, prompt):
        import time
        time.sleep(self.secs)
        if self.fail:
            raise RuntimeError("prefill refused")
        return int(prompt[-1])


def test_prefill_progress_lines_and_result(capsys):
    """The bench's long prefills run on a worker thread: progress lines while it runs, then the first
    token; an error on the worker is raised on the caller."""
    assert bench.prefill_with_progress(_SlowPrefill(0.35), [3, 9, 5], "w", every=0.1) == 5
    assert "prefill of 3 tokens running" in capsys.readouterr().err
    with pytest.raises(RuntimeError, match="refused"):
        bench.prefill_with_progress(_SlowPrefill(0.05, fail=True), [1], "w", every=0.1)
