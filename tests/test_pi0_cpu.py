"""Pins of the π0-style expert oracle (CPU only): independent scalar loops,
the two-stage form the GPU uses (the state token's keys and values computed
once and appended to the prefix), identity layers in closed form, and time
entering only through the action-time MLP."""
import math

import numpy as np
import pytest

import oracle
import synth
from oracle import pi0 as op
from synth import pi0 as sp

SMALL = synth.Dims(n_layers=2, width=16, n_heads=2, n_kv_heads=1, head_dim=8, mlp_dim=24, action_dim=3, horizon=4)
SD = 5


def _case(seed=31, P=6, B=2, dtype="f32", std=0.3):
    wl = synth.Workload("pi0-small", SMALL, prefix=P, batch=B, n_steps=3, n_fixed=0, dtype=dtype, seed=seed)
    w = sp.make_pi0_weights(wl, std=std, state_dim=SD)
    K, V = synth.make_prefix(wl)
    return wl, w, K, V, synth.make_noise(wl), sp.make_state(wl, state_dim=SD)


def _scalar_velocity(w, d, x, t, Kp, Vp, pl, st):
    """One rollout with explicit loops: token 0 is the state, 1.. the actions."""
    W, H, nH, Dh = d.width, d.horizon, d.n_heads, d.head_dim
    g = {k: np.asarray(synth.bf16_bits_to_f32(v) if v.dtype == np.uint16 else v, np.float64) for k, v in w.items()}

    def lin(name, vec, bias=None):
        M = g[name]
        out = [sum(M[o, i] * vec[i] for i in range(M.shape[1])) for o in range(M.shape[0])]
        return [out[o] + g[bias][o] for o in range(len(out))] if bias else out

    def norm(r, wn):
        s = math.sqrt(sum(v * v for v in r) / len(r) + 1e-6)
        return [r[i] / s * (1 + wn[i]) for i in range(len(r))]

    def rot(v, p):
        hd = len(v) // 2
        o = list(v)
        for j in range(hd):
            a = p * 10000 ** (-2 * j / len(v))
            o[j] = v[j] * math.cos(a) - v[j + hd] * math.sin(a)
            o[j + hd] = v[j] * math.sin(a) + v[j + hd] * math.cos(a)
        return o

    sw = lambda z: z / (1 + math.exp(-z))
    half = W // 2
    e = [math.cos(1000 * t * 10000 ** (-j / half)) for j in range(half)] + \
        [math.sin(1000 * t * 10000 ** (-j / half)) for j in range(half)]
    h = [lin("state_proj.w", st, "state_proj.b")]
    for i in range(H):
        a = lin("action_in.w", x[i], "action_in.b")
        m = [sw(z) for z in lin("action_time_mlp_in.w", a + e, "action_time_mlp_in.b")]
        h.append(lin("action_time_mlp_out.w", m, "action_time_mlp_out.b"))
    S = H + 1
    for l in range(d.n_layers):
        p = "layers.%d." % l
        y = [norm(h[i], g[p + "attn_norm.w"]) for i in range(S)]
        ks = [rot(lin(p + "k.w", y[i]), pl + i) for i in range(S)]
        vs = [lin(p + "v.w", y[i]) for i in range(S)]
        new = []
        for i in range(S):
            n_own = 1 if i == 0 else S          # the state token does not see the actions
            keys = [list(Kp[l][j]) for j in range(pl)] + ks[:n_own]
            vals = [list(Vp[l][j]) for j in range(pl)] + vs[:n_own]
            qi = lin(p + "q.w", y[i])
            att = []
            for hn in range(nH):
                q = rot(qi[hn * Dh:(hn + 1) * Dh], pl + i)
                sc = [sum(q[c] * k[c] for c in range(Dh)) / math.sqrt(Dh) for k in keys]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                att += [sum(ex[j] * vals[j][c] for j in range(len(keys))) / sum(ex) for c in range(Dh)]
            ao = lin(p + "o.w", att)
            new.append([h[i][c] + ao[c] for c in range(W)])
        h = new
        for i in range(S):
            yi = norm(h[i], g[p + "mlp_norm.w"])
            gg, uu = lin(p + "gate.w", yi), lin(p + "up.w", yi)
            z = [0.5 * gg[f] * (1 + math.tanh(math.sqrt(2 / math.pi) * (gg[f] + 0.044715 * gg[f] ** 3))) * uu[f]
                 for f in range(len(gg))]
            dn = lin(p + "down.w", z)
            h[i] = [h[i][c] + dn[c] for c in range(W)]
    return np.array([lin("action_out.w", norm(h[i], g["final_norm.w"]), "action_out.b") for i in range(1, S)])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pi0_velocity_matches_scalar_loops(dtype):
    wl, w, K, V, noise, st = _case(dtype=dtype)
    plens = [6, 2]
    v = op.velocity(SMALL, w, noise, 0.45, K, V, plens, st)
    for b in range(2):
        ref = _scalar_velocity(w, SMALL, noise[b].astype(np.float64), 0.45, oracle.widen(K[:, b]),
                               oracle.widen(V[:, b]), plens[b], st[b])
        np.testing.assert_allclose(v[b], ref, rtol=1e-10, atol=1e-12)


def test_pi0_state_token_as_extra_prefix_keys():
    """Block-causal: the state token's keys and values never depend on the
    actions or on t, so they can be computed once (a pass over the state
    token alone, with the prefix as context) and appended to the prefix; the
    action tokens at positions prefix_len + 1 + i then give the same velocity."""
    wl, w, K, V, noise, st = _case()
    g = {k: oracle.widen(v) for k, v in w.items()}
    plens = [6, 3]
    L, Dh = SMALL.n_layers, SMALL.head_dim
    K2 = np.zeros((L, 2, 7, Dh))
    V2 = np.zeros_like(K2)
    for b in range(2):
        pl = plens[b]
        hs = st[b].astype(np.float64) @ g["state_proj.w"].T + g["state_proj.b"]
        for l in range(L):
            p = "layers.%d." % l
            y = oracle.rms_normalize(hs[None, :]) * (1 + g[p + "attn_norm.w"])
            q = oracle.rope((y @ g[p + "q.w"].T).reshape(1, SMALL.n_heads, Dh).transpose(1, 0, 2), np.array([pl]))
            k = oracle.rope(y @ g[p + "k.w"].T, np.array([pl]))
            v = y @ g[p + "v.w"].T
            K2[l, b, :pl], V2[l, b, :pl] = K[l, b, :pl], V[l, b, :pl]
            K2[l, b, pl], V2[l, b, pl] = k[0], v[0]
            o = oracle.prefix_self_attention(q, K[l, b], V[l, b], pl, k, v)
            hs = hs + o.transpose(1, 0, 2).reshape(1, -1)[0] @ g[p + "o.w"].T
            y = oracle.rms_normalize(hs[None, :]) * (1 + g[p + "mlp_norm.w"])
            hs = hs + ((oracle.gelu_tanh(y @ g[p + "gate.w"].T) * (y @ g[p + "up.w"].T)) @ g[p + "down.w"].T)[0]
    # the action tokens alone over the extended prefix
    t = 0.7
    B, H, A, W = 2, SMALL.horizon, SMALL.action_dim, SMALL.width
    e = oracle.timestep_embedding(t, W)
    a = noise.reshape(B * H, A).astype(np.float64) @ g["action_in.w"].T + g["action_in.b"]
    h = oracle.swish(np.concatenate([a, np.broadcast_to(e, a.shape)], 1) @ g["action_time_mlp_in.w"].T
                     + g["action_time_mlp_in.b"]) @ g["action_time_mlp_out.w"].T + g["action_time_mlp_out.b"]
    for l in range(L):
        p = "layers.%d." % l
        y = oracle.rms_normalize(h) * (1 + g[p + "attn_norm.w"])
        q = (y @ g[p + "q.w"].T).reshape(B, H, SMALL.n_heads, Dh)
        k = (y @ g[p + "k.w"].T).reshape(B, H, Dh)
        v = (y @ g[p + "v.w"].T).reshape(B, H, Dh)
        o = np.empty((B, H, SMALL.n_heads * Dh))
        for b in range(B):
            pos = plens[b] + 1 + np.arange(H)
            ob = oracle.prefix_self_attention(oracle.rope(q[b].transpose(1, 0, 2), pos), K2[l, b], V2[l, b],
                                              plens[b] + 1, oracle.rope(k[b], pos), v[b])
            o[b] = ob.transpose(1, 0, 2).reshape(H, -1)
        h = h + o.reshape(B * H, -1) @ g[p + "o.w"].T
        y = oracle.rms_normalize(h) * (1 + g[p + "mlp_norm.w"])
        h = h + (oracle.gelu_tanh(y @ g[p + "gate.w"].T) * (y @ g[p + "up.w"].T)) @ g[p + "down.w"].T
    ref = (oracle.rms_normalize(h) * (1 + g["final_norm.w"])) @ g["action_out.w"].T + g["action_out.b"]
    got = op.velocity(SMALL, w, noise, t, K, V, plens, st)
    np.testing.assert_allclose(got.reshape(B * H, A), ref, rtol=1e-11, atol=1e-12)


def test_pi0_identity_layers_closed_form_and_time_only_through_the_mlp():
    wl, w, K, V, noise, st = _case()
    for l in range(SMALL.n_layers):
        w["layers.%d.o.w" % l][:] = 0.0
        w["layers.%d.down.w" % l][:] = 0.0
    t = 0.3
    v = op.velocity(SMALL, w, noise, t, K, V, [6, 6], st)
    g = {k: oracle.widen(x) for k, x in w.items()}
    W = SMALL.width
    half = W // 2
    f = 10000.0 ** (-np.arange(half) / half)
    e = np.concatenate([np.cos(1000 * t * f), np.sin(1000 * t * f)])
    a = noise.reshape(-1, 3).astype(np.float64) @ g["action_in.w"].T + g["action_in.b"]
    z = a @ g["action_time_mlp_in.w"][:, :W].T + g["action_time_mlp_in.w"][:, W:] @ e + g["action_time_mlp_in.b"]
    h = (z / (1 + np.exp(-z))) @ g["action_time_mlp_out.w"].T + g["action_time_mlp_out.b"]
    y = h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + 1e-6) * (1 + g["final_norm.w"])
    np.testing.assert_allclose(v.reshape(-1, 3), y @ g["action_out.w"].T + g["action_out.b"], rtol=1e-11, atol=1e-12)
    # the prefix and the state matter once the layers do
    wl, w, K, V, noise, st = _case()
    base = op.velocity(SMALL, w, noise, t, K, V, [6, 6], st)
    assert np.abs(op.velocity(SMALL, w, noise, t, K, V, [6, 6], st * 2) - base).max() > 1e-4
    assert np.abs(op.velocity(SMALL, w, noise, t, K, V * 2, [6, 6], st) - base).max() > 1e-4
    # time columns of the action-time MLP zeroed: t has no effect at all
    w["action_time_mlp_in.w"][:, W:] = 0.0
    assert np.array_equal(op.velocity(SMALL, w, noise, 0.1, K, V, [6, 6], st),
                          op.velocity(SMALL, w, noise, 0.9, K, V, [6, 6], st))


def test_pi0_denoise_committed_rows_and_constant_field():
    wl, w, K, V, noise, st = _case()
    com = np.random.default_rng(2).normal(size=(2, 1, 3))
    out = op.denoise(SMALL, w, noise, K, V, [6, 4], 3, st, committed=com, n_fixed=1)
    assert np.array_equal(out[:, :1], com) and np.abs(out[:, 1:] - noise[:, 1:]).max() > 1e-3
    w["action_out.w"][:] = 0.0
    c = np.array([0.5, 1.0, -2.0], np.float32)
    w["action_out.b"][:] = c
    out = op.denoise(SMALL, w, noise, K, V, [6, 4], 4, st)
    np.testing.assert_allclose(out, noise - c.astype(np.float64), rtol=0, atol=1e-12)
