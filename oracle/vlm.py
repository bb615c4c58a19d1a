"""CPU oracle (fp64) of the VLM prefill that produces the action expert's
prefix KV.  TEST INFRASTRUCTURE ONLY (same rules as ``actionexpert.py``).

The LLM of the π-series models (Table "pi_architecture": 18 layers, width
2048, 8 heads of dimension 256, one KV head; Appendix: its per-layer KV
cache conditions the action expert) is a Gemma decoder.  Readings where the
paper is silent:

V1  Pre-norm decoder layer: y = rms(h) * (1 + w_attn); q, k, v = y W^T with
    one shared KV head; RoPE on q and k at positions 0 .. P-1 (base 1e4,
    half-split pairs, as the expert's reading R6); attention over the whole
    prefix with no causal mask (image and instruction tokens form one
    prefix that attends to itself); h += o W_o^T; y = rms(h) * (1 + w_mlp);
    h += (gelu_tanh(y W_g^T) * (y W_u^T)) W_d^T.  No biases.
V2  MLP width 16384 (the table does not list it).
V3  The cache holds K after RoPE and V as projected (the expert's R7 takes
    the prefix K as already rotated).
V4  The input is the token embeddings (ViT + projector and text embeddings
    are outside the path).  The final-layer hidden state is rms(h) * (1 + w_final).
"""
from __future__ import annotations

import numpy as np

from .actionexpert import RMS_EPS, gelu_tanh, rms_normalize, rope, softmax_rows, widen


def prefill(dims, weights: dict, emb):
    """emb: [P][W] for one rollout.  Returns (K [L][P][Dh] rotated, V [L][P][Dh],
    hidden [P][W]) in fp64."""
    w = {k: widen(v) for k, v in weights.items()}
    L, W, nH, Dh = dims.n_layers, dims.width, dims.n_heads, dims.head_dim
    if dims.n_kv_heads != 1:
        raise ValueError("one shared KV head")
    h = widen(emb).copy()
    P = h.shape[0]
    pos = np.arange(P)
    Ks, Vs = [], []
    for l in range(L):
        p = "layers.%d." % l
        y = rms_normalize(h, RMS_EPS) * (1.0 + w[p + "attn_norm.w"])
        q = (y @ w[p + "q.w"].T).reshape(P, nH, Dh).transpose(1, 0, 2)   # [nH][P][Dh]
        k = y @ w[p + "k.w"].T                                             # [P][Dh]
        v = y @ w[p + "v.w"].T
        q = rope(q, pos)
        k = rope(k, pos)
        Ks.append(k)
        Vs.append(v)
        o = np.empty((nH, P, Dh))
        for n in range(nH):
            o[n] = softmax_rows(q[n] @ k.T / np.sqrt(Dh)) @ v
        h = h + o.transpose(1, 0, 2).reshape(P, nH * Dh) @ w[p + "o.w"].T
        y = rms_normalize(h, RMS_EPS) * (1.0 + w[p + "mlp_norm.w"])
        h = h + (gelu_tanh(y @ w[p + "gate.w"].T) * (y @ w[p + "up.w"].T)) @ w[p + "down.w"].T
    hidden = rms_normalize(h, RMS_EPS) * (1.0 + w["final_norm.w"])
    return np.stack(Ks), np.stack(Vs), hidden
