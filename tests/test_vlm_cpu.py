"""CPU checks of the VLM prefill: the oracle against an independent
scalar-loop implementation and closed-form special cases, and the C ABI's
host-side argument checks (no GPU needed).

Readings pinned here (oracle/vlm.py V1-V4): RMSNorm with (1 + w), RoPE from
position 0, attention over the whole prefix (a later token changes an earlier
token's keys at the next layer; a causal mask would not), K cached after RoPE.
"""
import math

import numpy as np
import pytest

import oracle
import synth
import synth.vlm as synth_vlm


def _dims(L=2, W=8, nH=2, Dh=4, F=8):
    return synth_vlm.VlmDims(n_layers=L, width=W, n_heads=nH, n_kv_heads=1, head_dim=Dh, mlp_dim=F)


def _weights(d, seed=3, std=0.3):
    rng = np.random.default_rng(seed)
    w = {}
    for name, shape, is_mat in synth_vlm.vlm_weight_specs(d):
        w[name] = rng.normal(size=shape) * std
    return w


def _bruteforce(d, w, emb):
    """Independent scalar loops: [out][in] matrices, explicit RoPE pairs and softmax."""
    P, W, nH, Dh, F = emb.shape[0], d.width, d.n_heads, d.head_dim, d.mlp_dim
    h = [list(map(float, row)) for row in emb]

    def norm(x, g):
        ms = sum(v * v for v in x) / len(x)
        r = 1.0 / math.sqrt(ms + 1e-6)
        return [x[i] * r * (1.0 + g[i]) for i in range(len(x))]

    def mat(m, x):
        return [sum(m[o][i] * x[i] for i in range(len(x))) for o in range(len(m))]

    def rot(v, pos):
        half = len(v) // 2
        out = list(v)
        for j in range(half):
            ang = pos * 10000.0 ** (-2.0 * j / len(v))
            c, s = math.cos(ang), math.sin(ang)
            out[j] = v[j] * c - v[j + half] * s
            out[j + half] = v[j] * s + v[j + half] * c
        return out

    Ks, Vs = [], []
    for l in range(d.n_layers):
        p = "layers.%d." % l
        ys = [norm(h[t], w[p + "attn_norm.w"]) for t in range(P)]
        qs = [mat(w[p + "q.w"], y) for y in ys]
        ks = [rot(mat(w[p + "k.w"], y), t) for t, y in enumerate(ys)]
        vs = [mat(w[p + "v.w"], y) for y in ys]
        Ks.append(ks)
        Vs.append(vs)
        for t in range(P):
            att = []
            for n in range(nH):
                qn = rot(qs[t][n * Dh:(n + 1) * Dh], t)
                logits = [sum(qn[e] * ks[u][e] for e in range(Dh)) / math.sqrt(Dh) for u in range(P)]
                m = max(logits)
                ex = [math.exp(x - m) for x in logits]
                s = sum(ex)
                att += [sum(ex[u] * vs[u][e] for u in range(P)) / s for e in range(Dh)]
            o = mat(w[p + "o.w"], att)
            h[t] = [h[t][i] + o[i] for i in range(W)]
        for t in range(P):
            y = norm(h[t], w[p + "mlp_norm.w"])
            g, u = mat(w[p + "gate.w"], y), mat(w[p + "up.w"], y)
            z = [0.5 * g[i] * (1 + math.tanh(math.sqrt(2 / math.pi) * (g[i] + 0.044715 * g[i] ** 3))) * u[i]
                 for i in range(F)]
            dn = mat(w[p + "down.w"], z)
            h[t] = [h[t][i] + dn[i] for i in range(W)]
    hidden = [norm(h[t], w["final_norm.w"]) for t in range(P)]
    return np.array(Ks), np.array(Vs), np.array(hidden)


def test_oracle_matches_scalar_loops():
    d = _dims()
    w = _weights(d)
    emb = np.random.default_rng(4).normal(size=(6, d.width))
    K, V, hid = oracle.vlm_prefill(d, w, emb)
    Kb, Vb, hb = _bruteforce(d, w, emb)
    np.testing.assert_allclose(K, Kb, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(V, Vb, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(hid, hb, rtol=1e-11, atol=1e-12)


def test_zero_norm_gain_makes_layers_identities():
    # (1 + w) = 0 zeroes every sublayer input: K = V = 0 and the hidden state is
    # the final norm of the embeddings
    d = _dims(L=3)
    w = _weights(d)
    for l in range(d.n_layers):
        w["layers.%d.attn_norm.w" % l][:] = -1.0
        w["layers.%d.mlp_norm.w" % l][:] = -1.0
    emb = np.random.default_rng(5).normal(size=(7, d.width))
    K, V, hid = oracle.vlm_prefill(d, w, emb)
    assert np.all(K == 0) and np.all(V == 0)
    ref = emb / np.sqrt((emb ** 2).mean(-1, keepdims=True) + 1e-6) * (1 + w["final_norm.w"])
    np.testing.assert_allclose(hid, ref, rtol=1e-13)


def test_first_layer_keys_start_at_position_zero():
    d = _dims(L=1)
    w = _weights(d)
    emb = np.random.default_rng(6).normal(size=(5, d.width))
    K, _, _ = oracle.vlm_prefill(d, w, emb)
    y0 = emb[0] / np.sqrt((emb[0] ** 2).mean() + 1e-6) * (1 + w["layers.0.attn_norm.w"])
    np.testing.assert_allclose(K[0, 0], w["layers.0.k.w"] @ y0, rtol=1e-12)   # RoPE at 0 is the identity


def test_no_causal_mask():
    # changing the last token changes the first token's layer-1 keys
    d = _dims(L=2)
    w = _weights(d)
    emb = np.random.default_rng(7).normal(size=(5, d.width))
    K1, _, _ = oracle.vlm_prefill(d, w, emb)
    emb2 = emb.copy()
    emb2[-1] += 1.0
    K2, _, _ = oracle.vlm_prefill(d, w, emb2)
    assert np.abs(K1[1, 0] - K2[1, 0]).max() > 1e-3
    assert np.array_equal(K1[0, 0], K2[0, 0])   # layer 0 keys are per token


def test_vlm_create_rejects_bad_config_on_the_host():
    from paper_2607_12659_amd import jpi
    base = dict(n_layers=2, width=256, n_heads=4, n_kv_heads=1, head_dim=64, mlp_dim=1024, max_batch=1,
                max_prefix=64, dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
    for bad in (dict(n_layers=0), dict(width=100), dict(n_kv_heads=2), dict(head_dim=48), dict(mlp_dim=1000),
                dict(max_batch=0), dict(max_prefix=0), dict(rms_eps=0.0), dict(width=8192)):
        st, _ = jpi.jpi_vlm_create(jpi.jpi_vlm_config(**{**base, **bad}))
        assert st == jpi.JPI_ERR_ARG, bad
    st, _ = jpi.jpi_vlm_create(jpi.jpi_vlm_config(**{**base, "dtype": jpi.JPI_F32}))
    assert st == jpi.JPI_ERR_UNSUPPORTED
    assert jpi.jpi_vlm_destroy(None) == jpi.JPI_OK
