"""Seeded synthetic inputs for the Archer cached-prompt decoding path.

This package is the only code shared by the CPU oracle (``oracle/``) and the
HIP path's tests and benchmark.  It holds workload shapes and random-number
generation only -- none of the method's arithmetic (no norms, attention,
projections, decisions or refresh logic).

* :mod:`synth.workloads` -- the model / decoding shapes of the five synthetic
  workloads (a tiny bidirectional DLM, an LLaDA-8B-shaped model at three
  prompt regimes, and a Dream-7B-shaped GQA model).
* :mod:`synth.gen` -- seeded generators for weights, prompts and ragged prompt
  lengths.
"""

from .workloads import ModelShape, DecodeShape, Workload, WORKLOADS, get_workload  # noqa: F401
from .gen import (  # noqa: F401
    normal_tensor,
    model_weights,
    prompts,
    prompt_lengths,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
)
