"""CPU oracle of the flow-matching action-expert denoiser (fp64, numpy).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares
no code with the GPU path (``paper_2607_12659_amd``) and must never be used
as a fallback for it.

What it computes (the paper's π-series action expert, Appendix "Model
Architecture of π series Models", and the flow-matching description in the
Background section):

* The action expert is a DiT whose input is random action noise.  At every
  layer the action tokens attend with queries from themselves and keys/values
  formed by concatenating the KV cache of the matching LLM layer with the
  action tokens' own keys/values.
* Starting from noise, a fixed number of flow-matching denoising steps
  (10 in Table "pi_architecture") progressively refines the chunk.
* Shapes of the π0.5 expert: 18 layers, width 1024, 8 attention heads of
  head dimension 256 (Table "pi_architecture").

Where the paper is silent the following readings are used (each one is a
choice, written out at the function that applies it):

R1  Flow runs from noise at t=1 to actions at t=0 on the uniform grid
    t_k = 1 - k/N, explicit Euler with dt = -1/N, velocity at the start of
    each step: x <- x + dt * v(x, t_k).
R3  Time embedding: [cos(1000 t f_j) | sin(1000 t f_j)], f_j = 10^(-4 j/(W/2)).
R4  Time MLP: two W->W linear layers with bias, each followed by swish.
R5  adaRMSNorm: y = h / sqrt(mean(h^2) + 1e-6) * (1 + scale) + shift, with
    (scale, shift, gate) = Linear(cond); residual h += gate * sublayer(y)
    (DiT adaLN-Zero form).  The final norm has scale and shift only.
R6  Gemma-family details: no biases in q/k/v/o/gate/up/down, tanh-GELU,
    logits scaled by 1/sqrt(Dh), no soft-cap, RoPE base 1e4 with half-split
    pairs (j, j + Dh/2).
R7  Suffix token i sits at RoPE position prefix_len + i; the prefix K is
    taken as already rotated; V is never rotated.
R8  Each action query sees prefix keys j < prefix_len and all H action keys;
    masked prefix slots are never read.
R9  Committed rows (i < n_fixed) are ordinary tokens that share the global t
    and are never Euler-updated.
R9b Variant (not the default): committed rows carry flow time t = 0 -- they
    are clean actions -- while the other rows carry the step's t_k, so the
    adaRMSNorm modulation (scale, shift, gate) is chosen per row.  The
    correction tokens keep the step's t.
R10 The correction item (T' tokens already in the expert's width, Section
    "Foresight-Aligned Asynchronous Correction") enters as T' extra suffix
    tokens placed ahead of the action tokens: correction token j sits at RoPE
    position prefix_len + j and action token i at prefix_len + T' + i.  The
    correction tokens skip the action in-projection, go through every layer
    with the step's modulation, attend to and are attended by all suffix
    tokens, restart from the given values at every step, and give no
    velocity (only action tokens are Euler-updated).
R13 Rollouts are independent (own prefix KV, own prefix_len).

All arithmetic is fp64.  bf16 inputs arrive as bit patterns and are widened
exactly.  Matrix products use numpy's matmul as a library primitive.
"""
from __future__ import annotations

import math

import numpy as np

RMS_EPS = 1e-6
ROPE_BASE = 1.0e4
TIME_SCALE = 1000.0
TIME_MAX_PERIOD = 1.0e4


# ---------------------------------------------------------------------------
# input widening
# ---------------------------------------------------------------------------
def widen(a: np.ndarray) -> np.ndarray:
    """fp64 copy of an input array; uint16 arrays are bf16 bit patterns."""
    a = np.asarray(a)
    out = np.empty(a.shape, dtype=np.float64)
    if a.dtype == np.uint16:
        bits = a.astype(np.uint32)
        np.left_shift(bits, 16, out=bits)
        out[...] = bits.view(np.float32)
    else:
        out[...] = a
    return out


class Expert:
    """The expert's tensors, widened to fp64, plus its shape parameters."""

    def __init__(self, dims, weights: dict):
        self.L = dims.n_layers
        self.W = dims.width
        self.nH = dims.n_heads
        self.nKV = dims.n_kv_heads
        self.Dh = dims.head_dim
        self.F = dims.mlp_dim
        self.A = dims.action_dim
        self.H = dims.horizon
        if self.nKV != 1:
            raise ValueError("the oracle implements one shared KV head (GQA with 1 KV head)")
        self.w = {k: widen(v) for k, v in weights.items()}


# ---------------------------------------------------------------------------
# elementary functions (each a textbook definition)
# ---------------------------------------------------------------------------
def swish(z):
    """z * sigmoid(z)."""
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z):
    """tanh approximation of GELU (Hendrycks & Gimpel 2016)."""
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))


def rms_normalize(h, eps=RMS_EPS):
    """h / sqrt(mean over the last axis of h^2 + eps)."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def ada_rms_norm(h, scale, shift, eps=RMS_EPS):
    """Reading R5: rms(h) * (1 + scale) + shift."""
    return rms_normalize(h, eps) * (1.0 + scale) + shift


def rope(x, pos, base=ROPE_BASE):
    """Rotary position embedding (Su et al. 2021), half-split pairing (reading R6).

    x: [..., T, D], pos: [T].  Pair (j, j + D/2) is rotated by pos * base^(-2j/D).
    """
    D = x.shape[-1]
    half = D // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def timestep_embedding(t: float, W: int):
    """Reading R3: sinusoidal embedding of 1000 t, [cos | sin] halves of width W."""
    half = W // 2
    f = np.exp(-math.log(TIME_MAX_PERIOD) * np.arange(half, dtype=np.float64) / half)
    arg = TIME_SCALE * t * f
    return np.concatenate([np.cos(arg), np.sin(arg)])


# ---------------------------------------------------------------------------
# attention (Appendix "Model Architecture of π series Models")
# ---------------------------------------------------------------------------
def softmax_rows(s):
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def prefix_self_attention(q, Kp, Vp, prefix_len, ks, vs):
    """Queries from the action tokens; keys/values are the LLM layer's KV
    concatenated with the action tokens' own (reading R8 for the mask).

    q: [nH][H][Dh] (already rotated), Kp/Vp: [P][Dh] (only the first
    ``prefix_len`` rows are read), ks/vs: [H][Dh].  One KV head is shared by
    all query heads.  Returns [nH][H][Dh].
    """
    Dh = q.shape[-1]
    K = np.concatenate([Kp[:prefix_len], ks], axis=0)
    V = np.concatenate([Vp[:prefix_len], vs], axis=0)
    s = (q @ K.T) / math.sqrt(Dh)
    return softmax_rows(s) @ V


def attention_bruteforce(q, Kp, Vp, prefix_len, ks, vs):
    """Independent formulation used to pin ``prefix_self_attention``: every
    score over all P + H key slots is materialised, masked slots get -inf, and
    each output row is an explicit weighted sum over keys.  Finite inputs only.
    """
    nH, H, Dh = q.shape
    P = Kp.shape[0]
    keys = list(Kp) + list(ks)
    vals = list(Vp) + list(vs)
    out = np.zeros((nH, H, Dh))
    for n in range(nH):
        for i in range(H):
            scores = []
            for j in range(P + H):
                if j < P and j >= prefix_len:
                    scores.append(-math.inf)
                else:
                    scores.append(float(np.dot(q[n, i], keys[j])) / math.sqrt(Dh))
            mx = max(scores)
            wts = [math.exp(s - mx) if s != -math.inf else 0.0 for s in scores]
            tot = sum(wts)
            acc = np.zeros(Dh)
            for j in range(P + H):
                if wts[j] != 0.0:
                    acc += (wts[j] / tot) * vals[j]
            out[n, i] = acc
    return out


# ---------------------------------------------------------------------------
# the velocity field v_theta(x, t | prefix KV)
# ---------------------------------------------------------------------------
def time_conditioning(ex: Expert, t: float):
    """Reading R4: cond = swish(T2 swish(T1 e + b1) + b2)."""
    w = ex.w
    e = timestep_embedding(t, ex.W)
    c = swish(w["time_mlp.0.w"] @ e + w["time_mlp.0.b"])
    return swish(w["time_mlp.1.w"] @ c + w["time_mlp.1.b"])


def modulation(ex: Expert, name: str, cond):
    """Split Linear(cond) into (scale, shift[, gate]) chunks of width W."""
    m = ex.w[name + ".w"] @ cond + ex.w[name + ".b"]
    return tuple(m[i * ex.W:(i + 1) * ex.W] for i in range(m.shape[0] // ex.W))


def velocity(ex: Expert, x, t: float, Kp, Vp, prefix_len, corr=None, n_t0: int = 0):
    """v(x, t) for a batch of independent rollouts.

    x: [B][H][A]; Kp, Vp: [L][B][P][Dh] (any dtype, widened here);
    prefix_len: [B]; corr: [B][T'][W] correction tokens or None (reading
    R10); n_t0: leading action rows that carry t = 0 instead of t (reading
    R9b).  Returns v [B][H][A].
    """
    w = ex.w
    B, H, A = x.shape
    W, nH, Dh, L = ex.W, ex.nH, ex.Dh, ex.L
    C = 0 if corr is None else np.asarray(corr).shape[1]
    S = C + H                                                                  # suffix tokens per rollout
    cond = time_conditioning(ex, t)
    cond0 = time_conditioning(ex, 0.0) if n_t0 else cond
    zero_t = np.zeros((B, S, 1), dtype=bool)
    zero_t[:, C:C + n_t0] = True                                               # reading R9b
    zero_t = zero_t.reshape(B * S, 1)

    def mod(name):
        """Per-row (scale, shift[, gate]): the t = 0 chunks on rows in zero_t."""
        return tuple(np.where(zero_t, m0, mt) for m0, mt in zip(modulation(ex, name, cond0),
                                                                 modulation(ex, name, cond)))

    act = x.reshape(B, H, A) @ w["action_in.w"].T + w["action_in.b"]           # [B][H][W]
    if C:
        act = np.concatenate([widen(corr).reshape(B, C, W), act], axis=1)      # reading R10
    h = act.reshape(B * S, W)
    for l in range(L):
        p = "layers.%d." % l
        scale, shift, gate = mod(p + "attn_mod")
        y = ada_rms_norm(h, scale, shift)
        q = (y @ w[p + "q.w"].T).reshape(B, S, nH, Dh)
        ks = (y @ w[p + "k.w"].T).reshape(B, S, Dh)
        vs = (y @ w[p + "v.w"].T).reshape(B, S, Dh)
        o = np.empty((B, S, nH * Dh))
        for b in range(B):
            pl = int(prefix_len[b])
            pos = pl + np.arange(S)                                            # readings R7, R10
            qb = rope(np.transpose(q[b], (1, 0, 2)), pos)                      # [nH][S][Dh]
            kb = rope(ks[b], pos)
            ob = prefix_self_attention(qb, widen(Kp[l, b]), widen(Vp[l, b]), pl, kb, vs[b])
            o[b] = np.transpose(ob, (1, 0, 2)).reshape(S, nH * Dh)
        h = h + gate * (o.reshape(B * S, nH * Dh) @ w[p + "o.w"].T)
        scale, shift, gate = mod(p + "mlp_mod")
        y = ada_rms_norm(h, scale, shift)
        z = gelu_tanh(y @ w[p + "gate.w"].T) * (y @ w[p + "up.w"].T)
        h = h + gate * (z @ w[p + "down.w"].T)
    scale, shift = (m.reshape(B, S, W)[:, C:, :].reshape(B * H, W) for m in mod("final_mod"))
    h = h.reshape(B, S, W)[:, C:, :].reshape(B * H, W)                          # action tokens only
    v = ada_rms_norm(h, scale, shift) @ w["action_out.w"].T + w["action_out.b"]
    return v.reshape(B, H, A)


# ---------------------------------------------------------------------------
# flow-matching integration (Background section; reading R1, R9)
# ---------------------------------------------------------------------------
def step_times(n_steps: int):
    """t_k = 1 - k/N for k = 0..N-1, each computed directly (no accumulation)."""
    return [1.0 - k / n_steps for k in range(n_steps)]


def integrate(x1, n_fixed: int, n_steps: int, vel_fn):
    """Explicit Euler from t=1 to t=0: x <- x + dt * vel_fn(x, t_k), dt = -1/N.

    x1: [B][H][A] (rows < n_fixed already hold the committed values).  Rows
    i < n_fixed are never updated.  ``vel_fn(x, t)`` returns [B][H][A].
    """
    if n_steps < 1:
        raise ValueError("n_steps must be >= 1")
    x = np.array(x1, dtype=np.float64)
    dt = -1.0 / n_steps
    for t in step_times(n_steps):
        v = vel_fn(x, t)
        x[:, n_fixed:, :] = x[:, n_fixed:, :] + dt * v[:, n_fixed:, :]
    return x


def denoise(ex: Expert, noise, Kp, Vp, prefix_len, n_steps: int, committed=None, n_fixed: int = 0,
            corr=None, committed_t0: bool = False):
    """The whole hot path: action chunk from noise by N Euler steps.

    noise: [B][H][A]; committed: [B][n_fixed][A] or None; corr: [B][T'][W]
    correction tokens or None (reading R10); committed_t0: the committed rows
    carry t = 0 (reading R9b).  Returns fp64 [B][H][A].
    """
    x = np.array(noise, dtype=np.float64)
    if n_fixed:
        x[:, :n_fixed, :] = np.asarray(committed, dtype=np.float64)
    return integrate(x, n_fixed, n_steps,
                     lambda xx, t: velocity(ex, xx, t, Kp, Vp, prefix_len, corr,
                                            n_fixed if committed_t0 else 0))
