"""CPU oracle for StepPrune's inference-time selection path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 NumPy
statement of what the selector computes, written from the paper (Section
"Conditional Sequential Pointer Policy", Eq. 2 and Eq. 4, and Algorithm 1)
so that the HIP library can be checked against it.  Only the test suite,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it; the library and its Python binding never do, and it shares no code
with them (its inputs come from the seeded generator, which holds none of the
method's arithmetic).

Modules
  rounding     round-to-nearest-even to bfloat16 / float32 storage
  projection   Algorithm 1 step 1: projected keys/queries/values, text context
  selection    Algorithm 1 steps 2-4: the pointer recurrence with STOP (Eq. 4)
  trajectory   the trajectory sums of the training surrogate (Eqs. 5-7)
  compaction   Algorithm 1 step 5: gather of kept tokens ahead of the prompt
  denoise      the training pathway's noise gate (Eq. 9) and masked denoiser
  encoder      the cross-modal input encoder (Eq. 3)
  calibration  the STOP bias that gives a target mean retained count

Every function states the passage it follows.  Readings of points the paper
leaves open are listed in the module that takes them.
"""
from .rounding import round_bf16, round_f32, round_to
from .projection import project, text_context, layer_norm
from .selection import (StepRecord, EpisodeResult, SelectResult, run_episode,
                        select, STOP)
from .trajectory import TrajectoryResult, step_distribution, aggregate, run_trajectory
from .compaction import compact
from .calibration import stop_thresholds, choose_stop_bias
from .denoise import DenoiserParams, vp_gate, denoise, gate_denoise
from .encoder import EncoderBlock, text_projection, encode

__all__ = [
    "round_bf16", "round_f32", "round_to", "project", "text_context", "layer_norm",
    "StepRecord", "EpisodeResult", "SelectResult", "run_episode", "select", "STOP",
    "compact", "stop_thresholds", "choose_stop_bias",
    "TrajectoryResult", "step_distribution", "aggregate", "run_trajectory",
    "DenoiserParams", "vp_gate", "denoise", "gate_denoise",
    "EncoderBlock", "text_projection", "encode",
]
