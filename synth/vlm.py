"""Seeded synthetic inputs of the VLM prefill (the LLM pass that produces the
action expert's prefix KV): shapes, weights and token embeddings.  Like the
rest of ``synth`` it holds no arithmetic of the method: only the generator
(``synth.normal_f32``), bf16 rounding and shapes.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

from . import DEFAULT_SEED, WEIGHT_STD, f32_to_bf16_bits, normal_f32

@dataclass(frozen=True)
class VlmDims:
    n_layers: int
    width: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    mlp_dim: int


@dataclass(frozen=True)
class VlmWorkload:
    name: str
    dims: VlmDims
    prefix: int          # prefix tokens per rollout (image + instruction embeddings)
    batch: int
    seed: int = DEFAULT_SEED

    def with_(self, **kw) -> "VlmWorkload":
        return replace(self, **kw)


VLM_TINY = VlmDims(n_layers=2, width=256, n_heads=4, n_kv_heads=1, head_dim=64, mlp_dim=1024)
GEMMA_2B = VlmDims(n_layers=18, width=2048, n_heads=8, n_kv_heads=1, head_dim=256, mlp_dim=16384)

VLM_WORKLOADS = {
    "vlm-tiny": VlmWorkload("vlm-tiny", VLM_TINY, prefix=64, batch=1),
    "gemma2b-p816": VlmWorkload("gemma2b-p816", GEMMA_2B, prefix=816, batch=1),
}


def vlm_weight_specs(d: VlmDims):
    """(name, shape, is_matrix) for every LLM tensor; norm weights are vectors."""
    W, F, Dh, nH = d.width, d.mlp_dim, d.head_dim, d.n_heads
    kvd = d.n_kv_heads * Dh
    specs = []
    for l in range(d.n_layers):
        p = "layers.%d." % l
        specs += [(p + "attn_norm.w", (W,), False), (p + "q.w", (nH * Dh, W), True), (p + "k.w", (kvd, W), True),
                  (p + "v.w", (kvd, W), True), (p + "o.w", (W, nH * Dh), True), (p + "mlp_norm.w", (W,), False),
                  (p + "gate.w", (F, W), True), (p + "up.w", (F, W), True), (p + "down.w", (W, F), True)]
    specs.append(("final_norm.w", (W,), False))
    return specs


def make_vlm_weights(wl: VlmWorkload, std: float = WEIGHT_STD, n_layers=None):
    """name -> array (matrices as bf16 bit patterns, norm weights fp32), all std * N(0,1).
    Tensor keys carry a ``vlm.`` prefix so they never coincide with the expert's.
    ``n_layers`` truncates the stack (the first layers of the full model)."""
    d = wl.dims if n_layers is None else replace(wl.dims, n_layers=n_layers)
    out = {}
    for name, shape, is_mat in vlm_weight_specs(d):
        a = normal_f32(wl.seed, "vlm." + name, std, shape)
        out[name] = f32_to_bf16_bits(a) if is_mat else a
    return out


def make_embeddings(wl: VlmWorkload, rollouts=None):
    """Input token embeddings [B][P][W] (fp32), N(0,1)."""
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    return np.stack([normal_f32(wl.seed, "vlm.emb.b%d" % b, 1.0, (wl.prefix, wl.dims.width)) for b in rollouts])
