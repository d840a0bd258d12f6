"""CPU oracle for one Speculative Pipeline Decoding step (float64, numpy).

TEST INFRASTRUCTURE ONLY: only tests/, the smoke check and the benchmark's CPU-baseline leg may
import it. It shares no code with the GPU path; both draw their inputs from the `synth` module.

Pins (what ties each function to something other than itself) are in tests/test_oracle_*.py:
  model.rms_norm, model.silu, model.attend   -> torch.nn.functional routines, closed forms
  model.rope                                 -> complex-rotation form, norm and relative-position
                                                invariants
  model.decoder_layer / ar_greedy            -> the transformers Llama implementation of the same
                                                architecture; brute-force forward_full
  spd.SPDOracle.step                         -> n=1 equals plain greedy decode; brute-force
                                                recomputation of every in-flight state; lossless
                                                greedy stream; staircase of Eq. steady-g/warmup-g;
                                                worked indices of Figure 1; closed forms for
                                                special weights
  sampling.top_k_dist / sample_index         -> closed-form distributions built from known
                                                probabilities; exact counts on stratified uniforms
  sampling.rejection_verify                  -> the emitted token follows p exactly (enumerated
                                                drafts, stratified uniforms), for PDM and forced q
  spd.SPDOracle (sampled decoding)           -> top_k = 1 equals greedy SPD step for step; the
                                                token after the first exit follows the plain AR
                                                top-k distribution (chi-square over seeded runs)
  spd.simulate_steps                         -> exact step counts of the oracle under forced masks
  spd.speedup_*                              -> Table 3's printed speedups (tests/golden/)
Parity unpinned: the PDM's draft quality (it has random weights); only its definition is pinned.
"""
from .model import (LayerCache, Model, ar_greedy, argmax_first, attend, decoder_layer, embed,
                    forward_full, forward_rows, lm_logits, rms_norm, rope, rope_angles, round_bf16, silu)
from .sampling import (Sampling, point_mass, prob_of, rejection_verify, sample, sample_index,
                       top_k_dist)
from .spd import (ACCEPT, NONE, REJECT, SPDOracle, StepResult, eligible_anchors, l_max, run_spd,
                  simulate_steps, speedup_serial_draft, speedup_zero_cost, stage_bounds,
                  step_acceptance)
