"""CPU oracle (fp64) of the π0-style action expert, a variant of the expert
in ``actionexpert.py``.  TEST INFRASTRUCTURE ONLY (same rules).

The paper runs both π0 and π0.5 (Table "pi_architecture" lists one action
expert for the π series; Table 1 times both) and describes their expert only
as a DiT over action noise that attends to the LLM's per-layer KV.  The
π0-style variant differs from the default expert in how time and the robot
state enter.  Readings (the paper is silent on all of them):

P1  Layers: the pre-norm decoder layer without time modulation --
    y = rms(h) (1 + w_norm), plain residual (gate 1, shift 0) -- with the
    expert's projections, RoPE, one KV head and tanh-GeGLU; final norm
    rms(h) (1 + w_final) before the action-out projection.
P2  Time enters through the action tokens only: an action-time MLP,
    h_i = W_o swish(W_i [W_a a_i + b_a ; e(t)] + b_i) + b_o, with the
    sinusoidal embedding e(t) of reading R3.
P3  The robot state s (a vector of state_dim values) enters as one suffix
    token s' = W_s s + b_s ahead of the action tokens: RoPE position
    prefix_len for it and prefix_len + 1 + i for action token i.  It attends
    to the prefix and to itself only (block-causal); the action tokens
    attend to the prefix, the state token and each other.
P4  Flow, grid, committed rows and Euler update as readings R1 and R9.
"""
from __future__ import annotations

import numpy as np

from .actionexpert import (RMS_EPS, gelu_tanh, integrate, prefix_self_attention, rms_normalize, rope, swish,
                           timestep_embedding, widen)


def _w(weights):
    """fp64 weights (arrays already in fp64 are taken as they are)."""
    return {k: v if isinstance(v, np.ndarray) and v.dtype == np.float64 else widen(v) for k, v in weights.items()}


def velocity(dims, weights: dict, x, t: float, Kp, Vp, prefix_len, state):
    """v(x, t) for a batch of rollouts.  x: [B][H][A]; Kp, Vp: [L][B][P][Dh];
    prefix_len: [B]; state: [B][state_dim].  Returns [B][H][A]."""
    w = _w(weights)
    B, H, A = x.shape
    W, nH, Dh, L = dims.width, dims.n_heads, dims.head_dim, dims.n_layers
    e = timestep_embedding(t, W)
    a = np.asarray(x, np.float64).reshape(B * H, A) @ w["action_in.w"].T + w["action_in.b"]
    cat = np.concatenate([a, np.broadcast_to(e, a.shape)], axis=1)                     # reading P2
    act = swish(cat @ w["action_time_mlp_in.w"].T + w["action_time_mlp_in.b"]) @ w["action_time_mlp_out.w"].T \
        + w["action_time_mlp_out.b"]
    st = np.asarray(state, np.float64) @ w["state_proj.w"].T + w["state_proj.b"]       # reading P3
    S = H + 1
    h = np.concatenate([st[:, None, :], act.reshape(B, H, W)], axis=1).reshape(B * S, W)
    for l in range(L):
        p = "layers.%d." % l
        y = rms_normalize(h, RMS_EPS) * (1.0 + w[p + "attn_norm.w"])                   # reading P1
        q = (y @ w[p + "q.w"].T).reshape(B, S, nH, Dh)
        ks = (y @ w[p + "k.w"].T).reshape(B, S, Dh)
        vs = (y @ w[p + "v.w"].T).reshape(B, S, Dh)
        o = np.empty((B, S, nH * Dh))
        for b in range(B):
            pl = int(prefix_len[b])
            pos = pl + np.arange(S)
            qb = rope(np.transpose(q[b], (1, 0, 2)), pos)                              # [nH][S][Dh]
            kb = rope(ks[b], pos)
            Kb, Vb = widen(Kp[l, b]), widen(Vp[l, b])
            # the state token sees the prefix and itself; the actions see everything
            o_s = prefix_self_attention(qb[:, :1], Kb, Vb, pl, kb[:1], vs[b][:1])
            o_a = prefix_self_attention(qb[:, 1:], Kb, Vb, pl, kb, vs[b])
            ob = np.concatenate([o_s, o_a], axis=1)
            o[b] = np.transpose(ob, (1, 0, 2)).reshape(S, nH * Dh)
        h = h + o.reshape(B * S, nH * Dh) @ w[p + "o.w"].T
        y = rms_normalize(h, RMS_EPS) * (1.0 + w[p + "mlp_norm.w"])
        h = h + (gelu_tanh(y @ w[p + "gate.w"].T) * (y @ w[p + "up.w"].T)) @ w[p + "down.w"].T
    h = h.reshape(B, S, W)[:, 1:, :].reshape(B * H, W)
    v = (rms_normalize(h, RMS_EPS) * (1.0 + w["final_norm.w"])) @ w["action_out.w"].T + w["action_out.b"]
    return v.reshape(B, H, A)


def denoise(dims, weights: dict, noise, Kp, Vp, prefix_len, n_steps: int, state, committed=None, n_fixed: int = 0):
    """Action chunk from noise by N Euler steps of the π0-style velocity."""
    x = np.array(noise, dtype=np.float64)
    if n_fixed:
        x[:, :n_fixed, :] = np.asarray(committed, dtype=np.float64)
    w = _w(weights)  # widened once for all steps
    return integrate(x, n_fixed, n_steps, lambda xx, t: velocity(dims, w, xx, t, Kp, Vp, prefix_len, state))
