"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests re-calls the oracle routine it checks as its own
expectation: each compares against a closed form, a brute-force
formulation, a library routine (scipy / complex arithmetic), a value the
paper prints, or an invariant of the definition.
"""
import json
import math
import os

import numpy as np
import pytest
from scipy import special

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Euler driver: closed forms (flow from noise at t=1 to actions at t=0)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N", [1, 2, 3, 10])
def test_euler_constant_velocity(N):
    rng = np.random.default_rng(0)
    x1 = rng.normal(size=(2, 5, 3))
    c = rng.normal(size=(2, 5, 3))
    x0 = oracle.integrate(x1, 0, N, lambda x, t: c)
    np.testing.assert_allclose(x0, x1 - c, rtol=0, atol=1e-12)


@pytest.mark.parametrize("N", [1, 4, 10])
@pytest.mark.parametrize("a", [0.5, -1.3])
def test_euler_linear_in_x(N, a):
    x1 = np.random.default_rng(1).normal(size=(1, 4, 2))
    x0 = oracle.integrate(x1, 0, N, lambda x, t: a * x)
    np.testing.assert_allclose(x0, (1 - a / N) ** N * x1, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("N", [2, 7])
def test_euler_affine_in_x(N):
    a, b = 0.7, -0.4
    x1 = np.random.default_rng(2).normal(size=(1, 3, 2))
    xs = -b / a
    x0 = oracle.integrate(x1, 0, N, lambda x, t: a * x + b)
    np.testing.assert_allclose(x0, xs + (1 - a / N) ** N * (x1 - xs), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("N", [1, 3, 10])
def test_euler_linear_in_t(N):
    alpha, beta = 1.7, -0.3
    x1 = np.random.default_rng(3).normal(size=(1, 3, 2))
    x0 = oracle.integrate(x1, 0, N, lambda x, t: np.full_like(x, alpha * t + beta))
    np.testing.assert_allclose(x0, x1 - beta - alpha * (N + 1) / (2 * N), rtol=0, atol=1e-12)


def test_euler_step_times_are_the_uniform_grid():
    seen = []
    oracle.integrate(np.zeros((1, 1, 1)), 0, 4, lambda x, t: (seen.append(t), np.zeros_like(x))[1])
    assert seen == [1.0, 0.75, 0.5, 0.25]


def test_euler_committed_rows_untouched():
    x1 = np.random.default_rng(4).normal(size=(2, 6, 3))
    x0 = oracle.integrate(x1, 2, 5, lambda x, t: np.ones_like(x))
    assert np.array_equal(x0[:, :2], x1[:, :2])
    np.testing.assert_allclose(x0[:, 2:], x1[:, 2:] - 1.0, atol=1e-12)


def test_euler_rejects_zero_steps():
    with pytest.raises(ValueError):
        oracle.integrate(np.zeros((1, 1, 1)), 0, 0, lambda x, t: x)


# ---------------------------------------------------------------------------
# elementary functions vs library routines / closed forms
# ---------------------------------------------------------------------------
def test_gelu_tanh_against_erf_gelu_and_odd_part():
    z = np.linspace(-6, 6, 1001)
    g = oracle.gelu_tanh(z)
    exact = 0.5 * z * (1 + special.erf(z / math.sqrt(2)))
    assert np.max(np.abs(g - exact)) < 5e-4          # known accuracy of the tanh form
    np.testing.assert_allclose(g - oracle.gelu_tanh(-z), z, atol=1e-12)
    assert oracle.gelu_tanh(np.array([0.0]))[0] == 0.0


def test_swish_against_expit():
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(oracle.swish(z), z * special.expit(z), rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(oracle.swish(z) - oracle.swish(-z), z, atol=1e-12)


def test_rms_normalize_special_cases():
    h = np.random.default_rng(5).normal(size=(4, 64)) * 3.0
    y = oracle.rms_normalize(h)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-6)
    c = np.full((1, 8), -2.5)
    np.testing.assert_allclose(oracle.rms_normalize(c), -1.0 / math.sqrt(1 + 1e-6 / 6.25), rtol=1e-14)
    # (1 + scale), + shift: scale = -1 leaves exactly the shift
    sh = np.arange(64.0)
    np.testing.assert_allclose(oracle.ada_rms_norm(h, -np.ones(64), sh), np.broadcast_to(sh, h.shape))


def test_rope_against_complex_rotation():
    rng = np.random.default_rng(6)
    D, T = 8, 5
    x = rng.normal(size=(T, D))
    pos = np.array([0, 1, 7, 100, 816])
    got = oracle.rope(x, pos)
    half = D // 2
    for t in range(T):
        for j in range(half):
            z = complex(x[t, j], x[t, j + half]) * np.exp(1j * pos[t] * 1e4 ** (-2 * j / D))
            assert abs(got[t, j] - z.real) < 1e-12 and abs(got[t, j + half] - z.imag) < 1e-12


def test_rope_invariants():
    rng = np.random.default_rng(7)
    q, k = rng.normal(size=(1, 16)), rng.normal(size=(1, 16))
    np.testing.assert_array_equal(oracle.rope(q, [0]), q)
    np.testing.assert_allclose(np.linalg.norm(oracle.rope(q, [123])), np.linalg.norm(q), rtol=1e-13)
    d1 = (oracle.rope(q, [10]) @ oracle.rope(k, [3]).T).item()
    d2 = (oracle.rope(q, [57]) @ oracle.rope(k, [50]).T).item()
    assert abs(d1 - d2) < 1e-11


def test_timestep_embedding_values():
    e = oracle.timestep_embedding(0.0, 8)
    np.testing.assert_array_equal(e, [1, 1, 1, 1, 0, 0, 0, 0])
    t = 0.3
    e = oracle.timestep_embedding(t, 4)
    # frequencies 10^(-4 j / 2) for j = 0, 1 -> 1 and 1e-2; argument scaled by 1000
    np.testing.assert_allclose(e, [math.cos(300.0), math.cos(3.0), math.sin(300.0), math.sin(3.0)],
                               rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# attention: brute force and closed forms
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("plen", [0, 1, 5, 9])
def test_attention_matches_bruteforce(plen):
    rng = np.random.default_rng(10 + plen)
    nH, H, Dh, P = 3, 4, 8, 9
    q = rng.normal(size=(nH, H, Dh))
    Kp, Vp = rng.normal(size=(P, Dh)), rng.normal(size=(P, Dh))
    ks, vs = rng.normal(size=(H, Dh)), rng.normal(size=(H, Dh))
    got = oracle.prefix_self_attention(q, Kp, Vp, plen, ks, vs)
    ref = oracle.attention_bruteforce(q, Kp, Vp, plen, ks, vs)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_attention_zero_query_is_mean_of_valid_values():
    rng = np.random.default_rng(11)
    P, H, Dh, plen = 12, 3, 4, 7
    Kp, Vp = rng.normal(size=(P, Dh)), rng.normal(size=(P, Dh))
    ks, vs = rng.normal(size=(H, Dh)), rng.normal(size=(H, Dh))
    out = oracle.prefix_self_attention(np.zeros((2, H, Dh)), Kp, Vp, plen, ks, vs)
    mean = np.concatenate([Vp[:plen], vs]).mean(axis=0)
    np.testing.assert_allclose(out, np.broadcast_to(mean, out.shape), rtol=1e-13)


def test_attention_single_key_and_dominant_logit():
    rng = np.random.default_rng(12)
    Dh = 4
    vs = rng.normal(size=(1, Dh))
    out = oracle.prefix_self_attention(rng.normal(size=(1, 1, Dh)), np.zeros((3, Dh)),
                                       np.zeros((3, Dh)), 0, rng.normal(size=(1, Dh)), vs)
    np.testing.assert_allclose(out[0, 0], vs[0], rtol=1e-15)
    Kp = np.zeros((5, Dh))
    Kp[3] = [1e3, 0, 0, 0]
    Vp = rng.normal(size=(5, Dh))
    q = np.array([[[1.0, 0, 0, 0]]]) * math.sqrt(Dh)
    out = oracle.prefix_self_attention(q, Kp, Vp, 5, np.zeros((1, Dh)), np.zeros((1, Dh)))
    np.testing.assert_allclose(out[0, 0], Vp[3], rtol=1e-12)


def test_attention_never_reads_masked_slots():
    rng = np.random.default_rng(13)
    P, H, Dh, plen = 10, 2, 4, 6
    Kp, Vp = rng.normal(size=(P, Dh)), rng.normal(size=(P, Dh))
    args = (rng.normal(size=(2, H, Dh)), rng.normal(size=(H, Dh)), rng.normal(size=(H, Dh)))
    a = oracle.prefix_self_attention(args[0], Kp, Vp, plen, args[1], args[2])
    Kp[plen:] = np.nan
    Vp[plen:] = np.inf
    b = oracle.prefix_self_attention(args[0], Kp, Vp, plen, args[1], args[2])
    assert np.array_equal(a, b)


# ---------------------------------------------------------------------------
# whole network: special cases and invariants on a small expert
# ---------------------------------------------------------------------------
SMALL = synth.Dims(n_layers=2, width=16, n_heads=2, n_kv_heads=1, head_dim=8, mlp_dim=24,
                   action_dim=3, horizon=4)


def _small(seed=99, P=6, B=2, dtype="f32"):
    wl = synth.Workload("small", SMALL, prefix=P, batch=B, n_steps=3, n_fixed=0, dtype=dtype,
                        seed=seed)
    w = synth.make_weights(wl, std=0.3)
    K, V = synth.make_prefix(wl)
    return wl, w, K, V, synth.make_noise(wl)


def _bruteforce_velocity(w, d, x, t, Kp, Vp, plen, corr=(), n_t0=0):
    """Scalar-loop velocity for one rollout, written from the same readings
    with explicit [out][in] indexing (a second, independent formulation).
    ``corr`` holds correction tokens, which occupy the first suffix slots;
    the first ``n_t0`` action tokens are conditioned on t = 0."""
    W, H, A, nH, Dh, F = d.width, d.horizon, d.action_dim, d.n_heads, d.head_dim, d.mlp_dim
    g = {k: np.asarray(synth.bf16_bits_to_f32(v) if v.dtype == np.uint16 else v, dtype=np.float64)
         for k, v in w.items()}

    def lin(name, vec, bias=None):
        M = g[name]
        out = [sum(M[o, i] * vec[i] for i in range(M.shape[1])) for o in range(M.shape[0])]
        if bias is not None:
            out = [out[o] + g[bias][o] for o in range(M.shape[0])]
        return out

    sig = lambda z: 1.0 / (1.0 + math.exp(-z))
    half = W // 2

    def conditioning(tt):
        emb = [math.cos(1000 * tt * 10000 ** (-j / half)) for j in range(half)] + \
              [math.sin(1000 * tt * 10000 ** (-j / half)) for j in range(half)]
        c = [z * sig(z) for z in lin("time_mlp.0.w", emb, "time_mlp.0.b")]
        return [z * sig(z) for z in lin("time_mlp.1.w", c, "time_mlp.1.b")]

    conds = [conditioning(t), conditioning(0.0)]

    def norm(row, s, b):
        r = math.sqrt(sum(v * v for v in row) / len(row) + 1e-6)
        return [row[i] / r * (1 + s[i]) + b[i] for i in range(len(row))]

    def rot(vec, pos):
        hd = len(vec) // 2
        out = list(vec)
        for j in range(hd):
            a = pos * 10000 ** (-2 * j / len(vec))
            out[j] = vec[j] * math.cos(a) - vec[j + hd] * math.sin(a)
            out[j + hd] = vec[j] * math.sin(a) + vec[j + hd] * math.cos(a)
        return out

    C = len(corr)
    h = [list(map(float, corr[j])) for j in range(C)] + [lin("action_in.w", x[i], "action_in.b") for i in range(H)]
    H = C + d.horizon                       # every suffix token goes through the layers
    which = [1 if C <= i < C + n_t0 else 0 for i in range(H)]   # conditioning of each token

    def mods(name):
        return [lin(name + ".w", cnd, name + ".b") for cnd in conds]

    for l in range(d.n_layers):
        p = "layers.%d." % l
        mm2 = mods(p + "attn_mod")
        y = [norm(h[i], mm2[which[i]][:W], mm2[which[i]][W:2 * W]) for i in range(H)]
        q = [lin(p + "q.w", y[i]) for i in range(H)]
        ks = [rot(lin(p + "k.w", y[i]), plen + i) for i in range(H)]
        vs = [lin(p + "v.w", y[i]) for i in range(H)]
        keys = [list(Kp[l][j]) for j in range(plen)] + ks
        vals = [list(Vp[l][j]) for j in range(plen)] + vs
        o = [[0.0] * (nH * Dh) for _ in range(H)]
        for i in range(H):
            for n in range(nH):
                qn = rot(q[i][n * Dh:(n + 1) * Dh], plen + i)
                sc = [sum(qn[e] * kk[e] for e in range(Dh)) / math.sqrt(Dh) for kk in keys]
                mx = max(sc)
                ex = [math.exp(v - mx) for v in sc]
                tot = sum(ex)
                for e in range(Dh):
                    o[i][n * Dh + e] = sum(ex[j] * vals[j][e] for j in range(len(keys))) / tot
        for i in range(H):
            ao = lin(p + "o.w", o[i])
            gt = mm2[which[i]][2 * W:]
            h[i] = [h[i][c_] + gt[c_] * ao[c_] for c_ in range(W)]
        mm2 = mods(p + "mlp_mod")
        for i in range(H):
            s, sh, gt = mm2[which[i]][:W], mm2[which[i]][W:2 * W], mm2[which[i]][2 * W:]
            yi = norm(h[i], s, sh)
            gg, uu = lin(p + "gate.w", yi), lin(p + "up.w", yi)
            z = [0.5 * gg[f] * (1 + math.tanh(math.sqrt(2 / math.pi) * (gg[f] + 0.044715 * gg[f] ** 3))) * uu[f]
                 for f in range(F)]
            dn = lin(p + "down.w", z)
            h[i] = [h[i][c_] + gt[c_] * dn[c_] for c_ in range(W)]
    fm = mods("final_mod")
    return np.array([lin("action_out.w", norm(h[i], fm[which[i]][:W], fm[which[i]][W:]), "action_out.b")
                     for i in range(C, H)])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_velocity_matches_scalar_bruteforce(dtype):
    wl, w, K, V, noise = _small(dtype=dtype)
    ex = oracle.Expert(SMALL, w)
    plens = [6, 3]
    v = oracle.velocity(ex, noise, 0.7, K, V, plens)
    for b in range(2):
        Kb = oracle.widen(K[:, b])
        Vb = oracle.widen(V[:, b])
        ref = _bruteforce_velocity(w, SMALL, noise[b].astype(np.float64), 0.7, Kb, Vb, plens[b])
        np.testing.assert_allclose(v[b], ref, rtol=1e-10, atol=1e-12)


def test_n_steps_1_is_noise_minus_velocity_at_t1():
    wl, w, K, V, noise = _small()
    ex = oracle.Expert(SMALL, w)
    out = oracle.denoise(ex, noise, K, V, [6, 6], 1)
    v = _bruteforce_velocity(w, SMALL, noise[0].astype(np.float64), 1.0, oracle.widen(K[:, 0]),
                             oracle.widen(V[:, 0]), 6)
    np.testing.assert_allclose(out[0], noise[0] - v, rtol=1e-10, atol=1e-12)


def test_zero_gates_make_layers_identity():
    wl, w, K, V, noise = _small()
    W = SMALL.width
    for l in range(SMALL.n_layers):
        for mod in ("attn_mod", "mlp_mod"):
            w["layers.%d.%s.w" % (l, mod)][:] = 0.0
            w["layers.%d.%s.b" % (l, mod)][2 * W:] = 0.0          # gate chunk
    ex = oracle.Expert(SMALL, w)
    t = 0.4
    v = oracle.velocity(ex, noise, t, K, V, [6, 6])
    # hand form: v = (rms(h0) (1 + s_f) + b_f) W_out^T + b_out, h0 = x W_in^T + b_in
    cond = oracle.time_conditioning(ex, t)
    fm = w["final_mod.w"].astype(np.float64) @ cond + w["final_mod.b"]
    h0 = noise.reshape(-1, 3).astype(np.float64) @ w["action_in.w"].T.astype(np.float64) + w["action_in.b"]
    rms = np.linalg.norm(h0, axis=1, keepdims=True) / math.sqrt(W)
    y = h0 / np.sqrt(rms ** 2 + 1e-6) * (1 + fm[:W]) + fm[W:]
    ref = y @ w["action_out.w"].T.astype(np.float64) + w["action_out.b"]
    np.testing.assert_allclose(v.reshape(-1, 3), ref, rtol=1e-11, atol=1e-12)


def test_constant_field_through_the_network():
    wl, w, K, V, noise = _small()
    w["action_out.w"][:] = 0.0
    c = np.array([0.25, -1.5, 2.0], np.float32)
    w["action_out.b"][:] = c
    ex = oracle.Expert(SMALL, w)
    out = oracle.denoise(ex, noise, K, V, [6, 6], 5)
    np.testing.assert_allclose(out, noise - c.astype(np.float64), rtol=0, atol=1e-12)


def test_invariants_rollouts_permutation_masking_committed():
    wl, w, K, V, noise = _small(P=8)
    ex = oracle.Expert(SMALL, w)
    plens = [8, 5]
    ref = oracle.denoise(ex, noise, K, V, plens, 3)
    # rollout independence
    solo = oracle.denoise(ex, noise[1:], K[:, 1:], V[:, 1:], plens[1:], 3)
    np.testing.assert_allclose(solo[0], ref[1], rtol=1e-13, atol=1e-14)
    # prefix-token permutation within the valid range
    perm = np.random.default_rng(3).permutation(5)
    K2, V2 = K.copy(), V.copy()
    K2[:, 1, :5] = K[:, 1, perm]
    V2[:, 1, :5] = V[:, 1, perm]
    np.testing.assert_allclose(oracle.denoise(ex, noise, K2, V2, plens, 3), ref, rtol=1e-12, atol=1e-13)
    # garbage in masked slots
    K3, V3 = K.copy(), V.copy()
    K3[:, 1, 5:] = np.nan
    V3[:, 1, 5:] = np.nan
    assert np.array_equal(oracle.denoise(ex, noise, K3, V3, plens, 3), ref)
    # committed rows are returned exactly and the others still move
    com = np.random.default_rng(4).normal(size=(2, 2, 3))
    out = oracle.denoise(ex, noise, K, V, plens, 3, committed=com, n_fixed=2)
    assert np.array_equal(out[:, :2], com)
    assert np.abs(out[:, 2:] - noise[:, 2:]).max() > 1e-3


def test_prefix_kv_matters():
    wl, w, K, V, noise = _small(P=8)
    ex = oracle.Expert(SMALL, w)
    a = oracle.denoise(ex, noise, K, V, [8, 8], 3)
    b = oracle.denoise(ex, noise, K, V * 1.5, [8, 8], 3)
    assert np.abs(a - b).max() > 1e-3


# ---------------------------------------------------------------------------
# correction tokens in the expert (reading R10)
# ---------------------------------------------------------------------------
def _corr(B=2, C=3, seed=21):
    return np.random.default_rng(seed).normal(size=(B, C, SMALL.width))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_velocity_with_correction_matches_scalar_bruteforce(dtype):
    wl, w, K, V, noise = _small(dtype=dtype)
    ex = oracle.Expert(SMALL, w)
    corr = _corr()
    plens = [6, 2]
    v = oracle.velocity(ex, noise, 0.3, K, V, plens, corr)
    for b in range(2):
        ref = _bruteforce_velocity(w, SMALL, noise[b].astype(np.float64), 0.3, oracle.widen(K[:, b]),
                                   oracle.widen(V[:, b]), plens[b], corr[b])
        np.testing.assert_allclose(v[b], ref, rtol=1e-10, atol=1e-12)


def test_one_layer_correction_tokens_act_as_extra_prefix_keys():
    """With one layer the correction tokens reach the action tokens only
    through their layer-0 keys and values, so the velocity equals the one
    without them over a prefix extended by those keys (rotated at the slots
    prefix_len + j) and values, with the action tokens at the same positions."""
    d1 = synth.Dims(n_layers=1, width=16, n_heads=2, n_kv_heads=1, head_dim=8, mlp_dim=24,
                    action_dim=3, horizon=4)
    wl = synth.Workload("one", d1, prefix=6, batch=2, n_steps=3, n_fixed=0, dtype="f32", seed=5)
    w = synth.make_weights(wl, std=0.3)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    ex = oracle.Expert(d1, w)
    corr = _corr()
    C, t, plens = corr.shape[1], 0.55, [6, 4]
    v = oracle.velocity(ex, noise, t, K, V, plens, corr)
    cond = oracle.time_conditioning(ex, t)
    g = {k: np.asarray(val, np.float64) for k, val in w.items()}
    m = g["layers.0.attn_mod.w"] @ cond + g["layers.0.attn_mod.b"]
    W = d1.width
    K2 = np.zeros((1, 2, 6 + C, d1.head_dim))
    V2 = np.zeros_like(K2)
    for b in range(2):
        pl = plens[b]
        rms = np.sqrt(np.mean(corr[b] ** 2, axis=1, keepdims=True) + 1e-6)
        y = corr[b] / rms * (1 + m[:W]) + m[W:2 * W]
        kc = y @ g["layers.0.k.w"].T
        ang = (pl + np.arange(C))[:, None] * 1e4 ** (-np.arange(4) / 4.0)[None, :]
        kr = np.concatenate([kc[:, :4] * np.cos(ang) - kc[:, 4:] * np.sin(ang),
                             kc[:, :4] * np.sin(ang) + kc[:, 4:] * np.cos(ang)], axis=1)
        K2[0, b, :pl] = K[0, b, :pl]
        V2[0, b, :pl] = V[0, b, :pl]
        K2[0, b, pl:pl + C] = kr
        V2[0, b, pl:pl + C] = y @ g["layers.0.v.w"].T
    ref = oracle.velocity(ex, noise, t, K2, V2, [p + C for p in plens])
    np.testing.assert_allclose(v, ref, rtol=1e-11, atol=1e-12)


def test_correction_tokens_constant_field_committed_and_influence():
    wl, w, K, V, noise = _small()
    corr = _corr()
    ex = oracle.Expert(SMALL, w)
    com = np.random.default_rng(8).normal(size=(2, 1, 3))
    a = oracle.denoise(ex, noise, K, V, [6, 6], 3, committed=com, n_fixed=1, corr=corr)
    assert np.array_equal(a[:, :1], com)
    b = oracle.denoise(ex, noise, K, V, [6, 6], 3, committed=com, n_fixed=1, corr=corr * 1.5)
    assert np.abs(a - b).max() > 1e-3
    # no correction tokens at all is the expert without them
    e = oracle.denoise(ex, noise, K, V, [6, 6], 3, corr=np.zeros((2, 0, SMALL.width)))
    assert np.array_equal(e, oracle.denoise(ex, noise, K, V, [6, 6], 3))
    # the velocity is read from action tokens only: a constant field stays exact
    w["action_out.w"][:] = 0.0
    c = np.array([0.5, -0.25, 1.0], np.float32)
    w["action_out.b"][:] = c
    ex = oracle.Expert(SMALL, w)
    out = oracle.denoise(ex, noise, K, V, [6, 6], 4, corr=corr)
    np.testing.assert_allclose(out, noise - c.astype(np.float64), rtol=0, atol=1e-12)


def test_workload_shapes_match_paper_table():
    with open(os.path.join(GOLDEN, "pi_architecture.json")) as f:
        arch = json.load(f)["action_expert"]
    for name in ("pi05-b1", "pi05-b1-committed10", "pi05-b8", "pi05-b64-p1600"):
        wl = synth.WORKLOADS[name]
        assert wl.dims.n_layers == arch["layers"]
        assert wl.dims.width == arch["embedding_dim"]
        assert wl.dims.n_heads == arch["attention_heads"]
        assert wl.dims.head_dim == arch["head_dim"]
        assert wl.n_steps == arch["denoising_steps"]


def test_synth_c_matches_numpy_twin():
    for name, shape, std in (("layers.3.q.w", (64, 33), 0.02), ("noise.b0", (50, 32), 1.0)):
        a = synth.normal_f32(1234, name, std, shape)
        b = synth.normal_f32_numpy(1234, name, std, shape)
        assert np.array_equal(a, b)
    z = synth.normal_f32(7, "stats", 1.0, (200000,)).astype(np.float64)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01


def test_bf16_rounding_is_rne():
    a = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.4e38], np.float32)
    bits = synth.f32_to_bf16_bits(a)
    assert [int(b) for b in bits] == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x7F80]
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(bits)[:4], [1.0, 1.0, 1.0 + 2 ** -6, -2.5])


# ---------------------------------------------------------------------------
# committed rows at t = 0 (reading R9b)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("with_corr", [False, True])
def test_velocity_with_committed_rows_at_t0_matches_scalar_bruteforce(with_corr):
    wl, w, K, V, noise = _small()
    ex = oracle.Expert(SMALL, w)
    corr = _corr(C=2) if with_corr else None
    plens = [6, 3]
    v = oracle.velocity(ex, noise, 0.6, K, V, plens, corr, n_t0=2)
    for b in range(2):
        ref = _bruteforce_velocity(w, SMALL, noise[b].astype(np.float64), 0.6, oracle.widen(K[:, b]),
                                   oracle.widen(V[:, b]), plens[b], () if corr is None else corr[b], n_t0=2)
        np.testing.assert_allclose(v[b], ref, rtol=1e-10, atol=1e-12)


def test_committed_t0_matters_only_through_time():
    wl, w, K, V, noise = _small()
    com = np.random.default_rng(6).normal(size=(2, 2, 3))
    ex = oracle.Expert(SMALL, w)
    a = oracle.denoise(ex, noise, K, V, [6, 6], 3, committed=com, n_fixed=2, committed_t0=True)
    b = oracle.denoise(ex, noise, K, V, [6, 6], 3, committed=com, n_fixed=2)
    assert np.array_equal(a[:, :2], com)
    assert np.abs(a - b).max() > 1e-3
    # no committed rows: the variant is the default exactly
    assert np.array_equal(oracle.denoise(ex, noise, K, V, [6, 6], 3, committed_t0=True),
                          oracle.denoise(ex, noise, K, V, [6, 6], 3))
    # conditioning that ignores t: both readings agree bit for bit
    w["time_mlp.0.w"][:] = 0.0
    ex = oracle.Expert(SMALL, w)
    a = oracle.denoise(ex, noise, K, V, [6, 6], 3, committed=com, n_fixed=2, committed_t0=True)
    b = oracle.denoise(ex, noise, K, V, [6, 6], 3, committed=com, n_fixed=2)
    assert np.array_equal(a, b)
