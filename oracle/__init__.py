"""CPU oracle (fp64) of the action-expert denoiser (and its π0-style variant),
the VLM prefill and the future correction module.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``, never by the GPU path.
"""
from .actionexpert import (Expert, ada_rms_norm, attention_bruteforce, denoise, gelu_tanh,
                           integrate, modulation, prefix_self_attention, rms_normalize, rope,
                           softmax_rows, step_times, swish, time_conditioning,
                           timestep_embedding, velocity, widen)
from .vlm import prefill as vlm_prefill
from . import correction, pi0

__all__ = ["Expert", "ada_rms_norm", "attention_bruteforce", "denoise", "gelu_tanh", "integrate",
           "modulation", "prefix_self_attention", "rms_normalize", "rope", "softmax_rows",
           "step_times", "swish", "time_conditioning", "timestep_embedding", "velocity", "widen", "vlm_prefill", "correction", "pi0"]
