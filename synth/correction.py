"""Seeded synthetic inputs of the future correction module: shapes, weights,
committed actions, VLM final-layer states and hidden-state buffer contents.
Like the rest of ``synth`` it holds no arithmetic of the method: only the
generator (``synth.normal_f32``), bf16 rounding and shapes.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

from . import DEFAULT_SEED, WEIGHT_STD, f32_to_bf16_bits, normal_f32


@dataclass(frozen=True)
class CorrDims:
    width: int        # d_AE: the action expert's width (tokens of the correction item)
    n_heads: int
    head_dim: int
    mlp_dim: int
    action_dim: int
    vlm_width: int    # d_VLM: width of the VLM final-layer state
    n_query: int      # T': compressed tokens (4 in the paper)


@dataclass(frozen=True)
class CorrWorkload:
    name: str
    dims: CorrDims
    batch: int
    n_actions: int    # committed actions handed to the module (Delta or Delta_ae)
    vlm_tokens: int   # T: tokens of the VLM final-layer state
    seed: int = DEFAULT_SEED

    def with_(self, **kw) -> "CorrWorkload":
        return replace(self, **kw)


CORR_TINY = CorrDims(width=256, n_heads=4, head_dim=64, mlp_dim=512, action_dim=7, vlm_width=256, n_query=4)
# d_AE = 1024 and d_VLM = 2048 are the pi0.5 expert and LLM widths; the
# block sizes give the module about 40M parameters
CORR_40M = CorrDims(width=1024, n_heads=8, head_dim=128, mlp_dim=2048, action_dim=32, vlm_width=2048, n_query=4)

CORR_WORKLOADS = {
    "corr-tiny": CorrWorkload("corr-tiny", CORR_TINY, batch=2, n_actions=5, vlm_tokens=40),
    "corr40m-p816": CorrWorkload("corr40m-p816", CORR_40M, batch=1, n_actions=10, vlm_tokens=816),
}

BLOCKS = ("qformer", "action_block", "blocks.0", "blocks.1")


def corr_weight_specs(d: CorrDims):
    """(name, shape, is_matrix) for every tensor of the module; biases, norm
    weights and the learned queries are fp32 vectors."""
    W, F, Dh, nH, A, V, T = d.width, d.mlp_dim, d.head_dim, d.n_heads, d.action_dim, d.vlm_width, d.n_query
    specs = [("qformer.query", (T, W), False), ("qformer.xk.w", (Dh, V), True), ("qformer.xv.w", (Dh, V), True),
             ("action_mlp.0.w", (W, A), True), ("action_mlp.0.b", (W,), False),
             ("action_mlp.1.w", (W, W), True), ("action_mlp.1.b", (W,), False),
             ("fuse.w", (W, 2 * W), True), ("fuse.b", (W,), False)]
    for p in BLOCKS:
        p += "."
        specs += [(p + "attn_norm.w", (W,), False), (p + "q.w", (nH * Dh, W), True), (p + "k.w", (Dh, W), True),
                  (p + "v.w", (Dh, W), True), (p + "o.w", (W, nH * Dh), True), (p + "mlp_norm.w", (W,), False),
                  (p + "gate.w", (F, W), True), (p + "up.w", (F, W), True), (p + "down.w", (W, F), True)]
    specs += [("final_norm.w", (W,), False), ("corr_head.w", (W, W), True), ("corr_head.b", (W,), False),
              ("conf_head.w", (1, W), True), ("conf_head.b", (1,), False)]
    return specs


def make_corr_weights(wl: CorrWorkload, std: float = WEIGHT_STD):
    """name -> array (matrices as bf16 bit patterns, vectors fp32), all std * N(0,1),
    except the learned queries, which are N(0,1) like token embeddings."""
    out = {}
    for name, shape, is_mat in corr_weight_specs(wl.dims):
        a = normal_f32(wl.seed, "corr." + name, 1.0 if name == "qformer.query" else std, shape)
        out[name] = f32_to_bf16_bits(a) if is_mat else a
    return out


def make_vlm_state(wl: CorrWorkload, rollouts=None):
    """VLM final-layer state [B][T][d_VLM] as bf16 bit patterns, N(0,1) (a
    normalised hidden state has unit RMS)."""
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    return np.stack([f32_to_bf16_bits(normal_f32(wl.seed, "corr.vlm_state.b%d" % b, 1.0,
                                                 (wl.vlm_tokens, wl.dims.vlm_width))) for b in rollouts])


def make_actions(wl: CorrWorkload, rollouts=None):
    """Committed actions [B][n_actions][A] (fp32), N(0,1)."""
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    return np.stack([normal_f32(wl.seed, "corr.actions.b%d" % b, 1.0, (wl.n_actions, wl.dims.action_dim))
                     for b in rollouts])


def make_state(wl: CorrWorkload, rollouts=None):
    """Hidden-state buffer contents [B][T'][W] (fp32), N(0,1)."""
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    return np.stack([normal_f32(wl.seed, "corr.state.b%d" % b, 1.0, (wl.dims.n_query, wl.dims.width))
                     for b in rollouts])


def make_item(seed: int, batch: int, n_corr: int, width: int, rollouts=None):
    """Correction item handed to the action expert [B][n_corr][W] (fp32), N(0,1)."""
    rollouts = list(range(batch)) if rollouts is None else list(rollouts)
    return np.stack([normal_f32(seed, "corr.item.b%d" % b, 1.0, (n_corr, width)) for b in rollouts])
