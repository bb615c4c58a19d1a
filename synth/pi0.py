"""Seeded synthetic inputs of the π0-style action-expert variant: its weight
names and shapes and the robot-state vectors.  Like the rest of ``synth`` it
holds no arithmetic of the method: only the generator (``synth.normal_f32``),
bf16 rounding and shapes.  Prefix KV and noise come from ``synth`` itself.
"""
from __future__ import annotations

import numpy as np

from . import WEIGHT_STD, Dims, Workload, f32_to_bf16_bits, normal_f32

STATE_DIM = 32   # robot-state values per rollout (the action width of the pi0.5-shape expert)


def pi0_weight_specs(d: Dims, state_dim: int = STATE_DIM):
    """(name, shape, is_matrix) for every tensor of the π0-style expert."""
    W, F, A, Dh, nH = d.width, d.mlp_dim, d.action_dim, d.head_dim, d.n_heads
    specs = [("action_in.w", (W, A), True), ("action_in.b", (W,), False),
             ("action_time_mlp_in.w", (W, 2 * W), True), ("action_time_mlp_in.b", (W,), False),
             ("action_time_mlp_out.w", (W, W), True), ("action_time_mlp_out.b", (W,), False),
             ("state_proj.w", (W, state_dim), True), ("state_proj.b", (W,), False)]
    for l in range(d.n_layers):
        p = "layers.%d." % l
        specs += [(p + "attn_norm.w", (W,), False), (p + "q.w", (nH * Dh, W), True), (p + "k.w", (Dh, W), True),
                  (p + "v.w", (Dh, W), True), (p + "o.w", (W, nH * Dh), True), (p + "mlp_norm.w", (W,), False),
                  (p + "gate.w", (F, W), True), (p + "up.w", (F, W), True), (p + "down.w", (W, F), True)]
    specs += [("final_norm.w", (W,), False), ("action_out.w", (A, W), True), ("action_out.b", (A,), False)]
    return specs


def make_pi0_weights(wl: Workload, std: float = WEIGHT_STD, state_dim: int = STATE_DIM):
    """name -> array (matrices bf16 bit patterns on the bf16 path, fp32 otherwise;
    vectors fp32), all std * N(0,1); generator keys carry a ``pi0.`` prefix."""
    out = {}
    for name, shape, is_mat in pi0_weight_specs(wl.dims, state_dim):
        a = normal_f32(wl.seed, "pi0." + name, std, shape)
        out[name] = f32_to_bf16_bits(a) if is_mat and wl.dtype == "bf16" else a
    return out


def make_state(wl: Workload, rollouts=None, state_dim: int = STATE_DIM):
    """Robot state [B][state_dim] (fp32), N(0,1)."""
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    return np.stack([normal_f32(wl.seed, "pi0.state.b%d" % b, 1.0, (state_dim,)) for b in rollouts])
