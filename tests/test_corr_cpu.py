"""Pins of the future-correction-module oracle (CPU only): a scalar-loop
block, closed forms of the heads and the concatenation order, the Q-Former's
invariance to the order of the VLM tokens, and the parameter count the paper
states."""
import math

import numpy as np
import pytest

import oracle
import synth
from oracle import correction as oc
from synth import correction as sc

MINI = sc.CorrDims(width=8, n_heads=2, head_dim=4, mlp_dim=6, action_dim=3, vlm_width=5, n_query=2)


def _wl(d=MINI, n=4, T=6, B=2, seed=77):
    return sc.CorrWorkload("mini", d, batch=B, n_actions=n, vlm_tokens=T, seed=seed)


def _w(wl, std=0.4):
    return {k: oracle.widen(v) for k, v in sc.make_corr_weights(wl, std=std).items()}


def _block_scalar(w, p, nH, h, kx=(), vx=(), pos=None):
    """Scalar-loop decoder block written from reading C1 with explicit indexing."""
    n, W = len(h), len(h[0])
    Dh = w[p + "k.w"].shape[0]

    def mv(M, x):
        return [sum(M[o][i] * x[i] for i in range(len(x))) for o in range(len(M))]

    def norm(r, g):
        s = math.sqrt(sum(v * v for v in r) / len(r) + 1e-6)
        return [r[i] / s * (1 + g[i]) for i in range(len(r))]

    def rot(x, ps):
        if pos is None:
            return list(x)
        hd = len(x) // 2
        out = list(x)
        for j in range(hd):
            a = ps * 10000 ** (-2 * j / len(x))
            out[j] = x[j] * math.cos(a) - x[j + hd] * math.sin(a)
            out[j + hd] = x[j] * math.sin(a) + x[j + hd] * math.cos(a)
        return out

    h = [list(r) for r in h]
    y = [norm(r, w[p + "attn_norm.w"]) for r in h]
    keys = [list(k) for k in kx] + [rot(mv(w[p + "k.w"], y[i]), pos[i] if pos is not None else 0) for i in range(n)]
    vals = [list(v) for v in vx] + [mv(w[p + "v.w"], y[i]) for i in range(n)]
    att = []
    for i in range(n):
        qi = mv(w[p + "q.w"], y[i])
        row = []
        for hd in range(nH):
            q = rot(qi[hd * Dh:(hd + 1) * Dh], pos[i] if pos is not None else 0)
            sc_ = [sum(q[e] * k[e] for e in range(Dh)) / math.sqrt(Dh) for k in keys]
            mx = max(sc_)
            ex = [math.exp(s - mx) for s in sc_]
            row += [sum(ex[j] * vals[j][e] for j in range(len(keys))) / sum(ex) for e in range(Dh)]
        att.append(row)
    for i in range(n):
        ao = mv(w[p + "o.w"], att[i])
        h[i] = [h[i][c] + ao[c] for c in range(W)]
        yi = norm(h[i], w[p + "mlp_norm.w"])
        g, u = mv(w[p + "gate.w"], yi), mv(w[p + "up.w"], yi)
        z = [0.5 * g[f] * (1 + math.tanh(math.sqrt(2 / math.pi) * (g[f] + 0.044715 * g[f] ** 3))) * u[f]
             for f in range(len(g))]
        dn = mv(w[p + "down.w"], z)
        h[i] = [h[i][c] + dn[c] for c in range(W)]
    return np.array(h)


@pytest.mark.parametrize("mode", ["plain", "extra_keys", "rope"])
def test_block_matches_scalar_loops(mode):
    wl = _wl()
    w = _w(wl)
    rng = np.random.default_rng(1)
    h = rng.normal(size=(3, MINI.width))
    kx = rng.normal(size=(4, MINI.head_dim)) if mode == "extra_keys" else None
    vx = rng.normal(size=(4, MINI.head_dim)) if mode == "extra_keys" else None
    pos = np.arange(3) + 2 if mode == "rope" else None
    got = oc.block(w, "blocks.1.", MINI.n_heads, h, kx, vx, pos)
    ref = _block_scalar(w, "blocks.1.", MINI.n_heads, h, () if kx is None else kx, () if vx is None else vx,
                        None if pos is None else list(pos))
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def _identity_blocks(w):
    for p in sc.BLOCKS:
        w[p + ".o.w"][:] = 0.0
        w[p + ".down.w"][:] = 0.0


def test_heads_and_concat_order_closed_form():
    """Identity blocks, W_f = [I | 0], plain final norm and an identity
    correction head: the item is the normalised compressed state."""
    wl = _wl()
    w = _w(wl)
    _identity_blocks(w)
    W = MINI.width
    w["fuse.w"][:] = np.concatenate([np.eye(W), np.zeros((W, W))], axis=1)
    w["fuse.b"][:] = 0.0
    w["final_norm.w"][:] = 0.0
    w["corr_head.w"][:] = np.eye(W)
    w["corr_head.b"][:] = 0.0
    vs = synth.f32_to_bf16_bits(np.random.default_rng(2).normal(size=(2, 6, MINI.vlm_width)).astype(np.float32))
    acts = sc.make_actions(wl)
    items, confs = oc.forward(MINI, w, acts, vlm_state=vs)
    Q = w["qformer.query"]
    want = Q / np.sqrt(np.mean(Q * Q, axis=1, keepdims=True) + 1e-6)
    for b in range(2):
        np.testing.assert_allclose(items[b], want, rtol=1e-13, atol=1e-14)
        assert abs(confs[b] - (w["conf_head.w"][0] @ want.mean(axis=0) + w["conf_head.b"][0])) < 1e-13


def test_action_branch_keeps_the_last_token():
    """Identity blocks and W_f = [0 | I]: every item token is the normalised
    MLP output of the last committed action."""
    wl = _wl(n=5)
    w = _w(wl)
    _identity_blocks(w)
    W = MINI.width
    w["fuse.w"][:] = np.concatenate([np.zeros((W, W)), np.eye(W)], axis=1)
    w["fuse.b"][:] = 0.0
    w["final_norm.w"][:] = 0.0
    w["corr_head.w"][:] = np.eye(W)
    w["corr_head.b"][:] = 0.0
    acts = sc.make_actions(wl)
    items, _ = oc.forward(MINI, w, acts, state=sc.make_state(wl))
    for b in range(2):
        a = acts[b, -1].astype(np.float64)
        pre = w["action_mlp.0.w"] @ a + w["action_mlp.0.b"]
        g = 0.5 * pre * (1 + np.tanh(math.sqrt(2 / math.pi) * (pre + 0.044715 * pre ** 3)))
        s = w["action_mlp.1.w"] @ g + w["action_mlp.1.b"]
        want = s / math.sqrt(np.mean(s * s) + 1e-6)
        for j in range(MINI.n_query):
            np.testing.assert_allclose(items[b, j], want, rtol=1e-12, atol=1e-13)


def test_qformer_zero_queries_average_all_values():
    """With W_q = 0 every query attends uniformly to the T VLM tokens and the
    T' queries, so the attention output is the mean of all their values."""
    wl = _wl()
    w = _w(wl)
    w["qformer.q.w"][:] = 0.0
    w["qformer.down.w"][:] = 0.0
    rng = np.random.default_rng(3)
    x = rng.normal(size=(6, MINI.vlm_width))
    c = oc.compress(MINI, w, x)
    Q = w["qformer.query"]
    y = Q / np.sqrt(np.mean(Q * Q, axis=1, keepdims=True) + 1e-6) * (1 + w["qformer.attn_norm.w"])
    vals = np.concatenate([x @ w["qformer.xv.w"].T, y @ w["qformer.v.w"].T], axis=0)
    mean = vals.mean(axis=0)
    want = Q + np.tile(mean, MINI.n_heads) @ w["qformer.o.w"].T
    np.testing.assert_allclose(c, np.broadcast_to(want, c.shape), rtol=1e-12, atol=1e-13)


def test_qformer_ignores_token_order_and_actions_do_not():
    wl = _wl(n=4)
    w = _w(wl)
    rng = np.random.default_rng(4)
    x = rng.normal(size=(6, MINI.vlm_width))
    c = oc.compress(MINI, w, x)
    np.testing.assert_allclose(oc.compress(MINI, w, x[rng.permutation(6)]), c, rtol=1e-12, atol=1e-13)
    acts = sc.make_actions(wl)[0]
    it, cf = oc.correct(MINI, w, c, acts)
    it2, cf2 = oc.correct(MINI, w, c, acts[[1, 0, 2, 3]])
    assert np.abs(it - it2).max() > 1e-6          # the action block is order-aware (RoPE)
    it3, _ = oc.correct(MINI, w, c * 1.3, acts)
    assert np.abs(it - it3).max() > 1e-6


def test_state_and_fresh_compression_agree_and_delta_varies():
    wl = _wl(n=3)
    w = _w(wl)
    vs = synth.f32_to_bf16_bits(np.random.default_rng(5).normal(size=(2, 6, MINI.vlm_width)).astype(np.float32))
    acts = sc.make_actions(wl)
    a, ca = oc.forward(MINI, w, acts, vlm_state=vs)
    st = np.stack([oc.compress(MINI, w, vs[b]) for b in range(2)])
    b_, cb = oc.forward(MINI, w, acts, state=st)
    assert np.array_equal(a, b_) and np.array_equal(ca, cb)
    for n in (1, 2, 7):
        acts_n = np.random.default_rng(n).normal(size=(2, n, MINI.action_dim))
        it, cf = oc.forward(MINI, w, acts_n, state=st)
        assert it.shape == (2, MINI.n_query, MINI.width) and np.all(np.isfinite(cf))
    with pytest.raises(ValueError):
        oc.forward(MINI, w, acts)


def test_module_size_is_about_40m():
    n = sum(int(np.prod(s)) for _, s, _ in sc.corr_weight_specs(sc.CORR_40M))
    assert 38e6 <= n <= 42e6
