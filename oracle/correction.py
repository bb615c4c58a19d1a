"""CPU oracle (fp64) of the future correction module.  TEST INFRASTRUCTURE
ONLY (same rules as ``actionexpert.py``).

What the paper fixes (Section "Foresight-Aligned Asynchronous Correction";
Appendix "Architecture of Future Correction Module" and its figure;
Algorithm 1):

* Inputs: the actions committed for execution during the inference window
  and the VLM final-layer state at time t.
* The action sequence goes through an MLP and then a Transformer block; the
  last token of the block's output is kept.
* The VLM final-layer state is compressed by a Q-Former block to T' = 4
  tokens of the expert's width.
* The two branches are concatenated, projected and passed through two
  Transformer blocks; a correction head gives the compressed state at
  t + Delta (the correction item handed to the expert) and a confidence head
  a scalar confidence.
* The module has about 40M parameters.
* Algorithm 1 feeds the hidden-state buffer back: after a skipped VLM the
  module starts from its own previous prediction instead of a fresh
  compression.

Readings where the paper is silent:

C1  Every Transformer block is the VLM's pre-norm decoder layer (reading V1 of
    ``vlm.py``) at the expert's width: y = rms(h) (1 + w_attn), one shared KV
    head, h += o W_o^T, y = rms(h) (1 + w_mlp), tanh-GeGLU MLP with residual,
    no biases.  Sizes 8 heads x 128, MLP 2048 (about 40M parameters in all).
C2  Q-Former: T' learned queries (the residual stream's start) attend jointly
    to the VLM tokens' keys and values, projected from d_VLM by their own two
    matrices, and to their own; no positional rotation anywhere in it.  The
    compressed state c is the block's residual output [T'][W].
C3  Action branch: u_i = W2 gelu_tanh(W1 a_i + b1) + b2 for each committed
    action; one block over them with RoPE at positions 0 .. n-1 and no mask;
    s is the last token's residual output.
C4  Concatenation is along features, with s repeated for every compressed
    token: z_j = W_f [c_j ; s] + b_f.  Two blocks over the T' tokens follow,
    no positional rotation.
C5  Heads: y = rms(z) (1 + w_final); the correction item is
    h_j = W_c y_j + b_c; the confidence is w_conf . mean_j(y_j) + b_conf,
    unbounded (Algorithm 1 compares it with a threshold theta < 0).
C6  The hidden-state buffer holds c-space tokens: c = Q-Former(h_t) after a
    VLM refresh, else the previous correction item.
"""
from __future__ import annotations

import math

import numpy as np

from .actionexpert import RMS_EPS, gelu_tanh, rms_normalize, rope, softmax_rows, widen

BLOCKS = ("qformer", "action_block", "blocks.0", "blocks.1")


def block(w, p: str, nH: int, h, kx=None, vx=None, pos=None):
    """One decoder block (reading C1) over the rows of h [n][W].

    kx, vx: [T][Dh] extra keys and values the rows also attend to (the
    Q-Former's VLM tokens, reading C2); pos: RoPE positions of the rows or
    None for no rotation.  Returns the new residual stream [n][W].
    """
    n = h.shape[0]
    Dh = w[p + "k.w"].shape[0]
    y = rms_normalize(h, RMS_EPS) * (1.0 + w[p + "attn_norm.w"])
    q = (y @ w[p + "q.w"].T).reshape(n, nH, Dh).transpose(1, 0, 2)      # [nH][n][Dh]
    k = y @ w[p + "k.w"].T
    v = y @ w[p + "v.w"].T
    if pos is not None:
        q = rope(q, pos)
        k = rope(k, pos)
    if kx is not None:
        k = np.concatenate([kx, k], axis=0)
        v = np.concatenate([vx, v], axis=0)
    o = np.empty((nH, n, Dh))
    for i in range(nH):
        o[i] = softmax_rows(q[i] @ k.T / math.sqrt(Dh)) @ v
    h = h + o.transpose(1, 0, 2).reshape(n, nH * Dh) @ w[p + "o.w"].T
    y = rms_normalize(h, RMS_EPS) * (1.0 + w[p + "mlp_norm.w"])
    return h + (gelu_tanh(y @ w[p + "gate.w"].T) * (y @ w[p + "up.w"].T)) @ w[p + "down.w"].T


def compress(dims, weights: dict, vlm_state):
    """Q-Former (reading C2): vlm_state [T][d_VLM] -> c [T'][W] for one rollout."""
    w = {k: widen(v) for k, v in weights.items()}
    x = widen(vlm_state)
    kx = x @ w["qformer.xk.w"].T
    vx = x @ w["qformer.xv.w"].T
    return block(w, "qformer.", dims.n_heads, w["qformer.query"].copy(), kx, vx)


def action_summary(dims, weights: dict, actions):
    """Action branch (reading C3): actions [n][A] -> s [W] for one rollout."""
    w = {k: widen(v) for k, v in weights.items()}
    a = np.asarray(actions, dtype=np.float64)
    u = gelu_tanh(a @ w["action_mlp.0.w"].T + w["action_mlp.0.b"]) @ w["action_mlp.1.w"].T + w["action_mlp.1.b"]
    return block(w, "action_block.", dims.n_heads, u, pos=np.arange(a.shape[0]))[-1]


def correct(dims, weights: dict, c, actions):
    """Fusion, two blocks and both heads (readings C4, C5) for one rollout.

    c: [T'][W] compressed state; actions: [n][A].  Returns (correction item
    [T'][W], confidence)."""
    w = {k: widen(v) for k, v in weights.items()}
    s = action_summary(dims, weights, actions)
    c = np.asarray(c, dtype=np.float64)
    cat = np.concatenate([c, np.broadcast_to(s, c.shape)], axis=1)         # [T'][2W]: c_j then s
    z = cat @ w["fuse.w"].T + w["fuse.b"]
    for p in ("blocks.0.", "blocks.1."):
        z = block(w, p, dims.n_heads, z)
    y = rms_normalize(z, RMS_EPS) * (1.0 + w["final_norm.w"])
    item = y @ w["corr_head.w"].T + w["corr_head.b"]
    conf = float(w["conf_head.w"][0] @ y.mean(axis=0) + w["conf_head.b"][0])
    return item, conf


def forward(dims, weights: dict, actions, vlm_state=None, state=None):
    """f_corr for a batch (reading C6): from the VLM final-layer state
    vlm_state [B][T][d_VLM] (fresh compression) or from the hidden-state
    buffer state [B][T'][W].  actions: [B][n][A].  Returns (items [B][T'][W],
    confidences [B])."""
    if (vlm_state is None) == (state is None):
        raise ValueError("give exactly one of vlm_state and state")
    B = len(actions)
    items, confs = [], []
    for b in range(B):
        c = compress(dims, weights, vlm_state[b]) if vlm_state is not None else state[b]
        it, cf = correct(dims, weights, c, actions[b])
        items.append(it)
        confs.append(cf)
    return np.stack(items), np.array(confs)
