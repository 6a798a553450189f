"""Seeded synthetic inputs for the DART policy-update hot path.

This package is shared by the HIP path's tests/bench and by the float64 oracle's
tests. It holds NO arithmetic of the method itself (no softmax, entropy, ratio,
clip or selection): only a counter-based random generator, the shapes of the
workloads, and the recipe that turns random draws into logits, targets, step
lengths, advantages and the offsets that perturb log-probabilities.

Three implementations of the same generator exist and are tested bit-exact
against each other:

* ``synth.gen``      numpy, the readable definition;
* ``synth.host``     C + OpenMP (``csrc/synth_host.c``) for full-size host rows;
* ``synth.device``   HIP (``csrc/synth_dev.hip``) that fills device buffers.
"""

from .gen import (  # noqa: F401
    Workload,
    WORKLOADS,
    make_workload,
    custom_workload,
    normal_table,
    counter_hash,
    draw_normal,
    draw_uniform,
    logits_rows_numpy,
    perturbed_logprobs,
    reference_logprobs,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    gaussian_bits,
    lmhead_problem,
    lmhead_custom,
    LmHeadProblem,
)
