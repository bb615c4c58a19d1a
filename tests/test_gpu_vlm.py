"""VLM prefill on the GPU against the fp64 oracle, and the in-place hand-off
of its KV cache to the action expert.

Bars: bf16 path, relative L2 <= 2e-2 (per layer for K, per rollout for the
hidden state and the actions), as for the expert.
"""
import ctypes

import numpy as np
import pytest

import oracle
import synth
import synth.vlm as synth_vlm
from gpu_util import (Vlm, bf16_bits_to_f64, device_view_i16, make_expert, rel_l2_per_rollout, run, torch_cuda)

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def _expert_for(vd, horizon, action_dim, mlp_dim, width, n_heads, max_prefix):
    d = synth.Dims(n_layers=vd.n_layers, width=width, n_heads=n_heads, n_kv_heads=1, head_dim=vd.head_dim,
                   mlp_dim=mlp_dim, action_dim=action_dim, horizon=horizon)
    wl = synth.Workload("expert", d, prefix=max_prefix, batch=1, n_steps=3, n_fixed=0, dtype="bf16")
    w = synth.make_weights(wl)
    return wl, w, make_expert(wl, w, max_batch=1, max_prefix=max_prefix)


def _kp_layers(ae, L, Pmax, Dh, prefix):
    from paper_2607_12659_amd import jpi
    st, k_ptr, _ = ae_prefix_ptrs(ae)
    kv = device_view_i16(k_ptr, (L, 1, Pmax, Dh)).cpu().numpy()
    return bf16_bits_to_f64(kv[:, 0, :prefix])


def _vt_layers(ae, L, Dh, _unused=None):
    """The expert's transposed prefix V of rollout 0, [L][Dh][ld] as fp64."""
    from paper_2607_12659_amd import jpi
    st, vt_ptr, ld = jpi.jpi_debug_prefix_vt(ae.ctx)
    assert st == jpi.JPI_OK
    raw = device_view_i16(vt_ptr, (L, ae.max_batch, Dh, ld)).cpu().numpy()
    return bf16_bits_to_f64(raw[:, 0])


def ae_prefix_ptrs(ae):
    from paper_2607_12659_amd import jpi
    k = ctypes.c_void_p()
    v = ctypes.c_void_p()
    st = jpi._lib.jpi_prefix_buffers(ae.ctx, ctypes.byref(k), ctypes.byref(v))
    return st, k.value, v.value


def _check_prefill(vwl, n_layers=None, denoise=True):
    torch = torch_cuda()
    from paper_2607_12659_amd.expert import to_device
    vd = vwl.dims if n_layers is None else vwl.dims.__class__(**{**vwl.dims.__dict__, "n_layers": n_layers})
    print("case %s layers %d prefix %d" % (vwl.name, vd.n_layers, vwl.prefix), flush=True)
    vw = synth_vlm.make_vlm_weights(vwl, n_layers=vd.n_layers)
    emb = synth_vlm.make_embeddings(vwl)
    K_o, V_o, hid_o = oracle.vlm_prefill(vd, vw, emb[0])
    vlm = Vlm(vd, vw, 1, vwl.prefix)
    # an action expert with the same layer count and head_dim (its own width)
    aw = 256 if vd.width <= 256 else 1024
    ewl, ew, ae = _expert_for(vd, horizon=10, action_dim=7, mlp_dim=4 * aw, width=aw, n_heads=4, max_prefix=vwl.prefix)
    try:
        hidden = torch.empty((1, vwl.prefix, vd.width), dtype=torch.int16, device="cuda")
        vlm.prefill(to_device(np.ascontiguousarray(emb, np.float32)), 1, vwl.prefix, ae, hidden)
        torch.cuda.synchronize()
        K_g = _kp_layers(ae, vd.n_layers, vwl.prefix, vd.head_dim, vwl.prefix)
        for l in range(vd.n_layers):
            r = _rel(K_g[l], K_o[l])
            print("  K layer %d rel-L2 %.3e" % (l, r), flush=True)
            assert r <= TOL
        h_g = bf16_bits_to_f64(hidden.cpu().numpy())[0]
        rh = _rel(h_g, hid_o)
        print("  hidden rel-L2 %.3e" % rh, flush=True)
        assert rh <= TOL
        if denoise:
            # the expert runs on the KV the prefill left in its buffers; the
            # oracle runs on the oracle's KV rounded to bf16
            noise = synth.make_noise(ewl)
            from paper_2607_12659_amd.expert import to_device as td
            out = ae.denoise(td(np.ascontiguousarray(noise, np.float32)), ewl.n_steps)
            ae.sync()
            got = out.cpu().numpy().astype(np.float64)
            rb = lambda a: synth.f32_to_bf16_bits(a.astype(np.float32))
            Kb = rb(K_o)[:, None]
            Vb = rb(V_o)[:, None]
            ex = oracle.Expert(ewl.dims, ew)
            ref = oracle.denoise(ex, noise, Kb, Vb, [vwl.prefix], ewl.n_steps)
            ra = rel_l2_per_rollout(got, ref)
            # the check has teeth: the oracle on another prefix (V negated)
            # differs from the GPU output by far more than the GPU error
            ref2 = oracle.denoise(ex, noise, Kb, Vb ^ np.uint16(0x8000), [vwl.prefix], ewl.n_steps)
            effect = rel_l2_per_rollout(got, ref2)
            print("  actions after the hand-off rel-L2 %.3e (negated prefix V: %.3e)" % (ra, effect), flush=True)
            assert ra <= TOL
            assert effect > 20 * ra
    finally:
        ae.close()
        vlm.close()


def test_vlm_tiny_prefill_and_handoff():
    _check_prefill(synth_vlm.VLM_WORKLOADS["vlm-tiny"])


def test_vlm_gemma_width_two_layers():
    # full Gemma-2B width, MLP and head shape, the first two layers, 816 tokens
    _check_prefill(synth_vlm.VLM_WORKLOADS["gemma2b-p816"], n_layers=2, denoise=False)


def test_vlm_full_gemma_into_pi05_expert():
    """All 18 layers at full size (816 tokens) into the pi0.5 expert: K and V
    of every layer and the final hidden state against the stored oracle run
    (tests/golden/gemma2b-p816-l18: 32 evenly spaced token positions), then
    the expert's actions on that KV repeat exactly across two prefills."""
    torch = torch_cuda()
    from paper_2607_12659_amd.expert import to_device
    from gpu_util import GOLDEN, assert_bf16
    import json
    import os
    vwl = synth_vlm.VLM_WORKLOADS["gemma2b-p816"]
    g = np.load(os.path.join(GOLDEN, "gemma2b-p816-l18.npz"), allow_pickle=False)
    with open(os.path.join(GOLDEN, "gemma2b-p816-l18.json")) as f:
        meta = json.load(f)
    assert meta["n_layers"] == vwl.dims.n_layers == 18 and meta["prefix"] == vwl.prefix
    tok = g["tokens"]
    print("case gemma2b-p816 full (18 layers) into pi05 expert", flush=True)
    vlm = Vlm(vwl.dims, synth_vlm.make_vlm_weights(vwl), 1, vwl.prefix)
    ewl = synth.WORKLOADS["pi05-b1"]
    ae = make_expert(ewl, synth.make_weights(ewl), max_batch=1, max_prefix=vwl.prefix)
    try:
        emb = to_device(np.ascontiguousarray(synth_vlm.make_embeddings(vwl), np.float32))
        noise = to_device(np.ascontiguousarray(synth.make_noise(ewl), np.float32))
        hidden = torch.empty((1, vwl.prefix, vwl.dims.width), dtype=torch.int16, device="cuda")
        outs, ks = [], []
        for rep in range(2):
            vlm.prefill(emb, 1, vwl.prefix, ae, hidden if rep == 0 else None)
            out = ae.denoise(noise, ewl.n_steps)
            ae.sync()
            outs.append(out.cpu().numpy())
            _, k_ptr, v_ptr = ae_prefix_ptrs(ae)
            ks.append(device_view_i16(k_ptr, (vwl.dims.n_layers, 1, vwl.prefix, vwl.dims.head_dim)).cpu().numpy())
            if rep == 0:
                # the prefill writes V transposed ([L][max_batch][Dh][ld]), the
                # attention kernels' operand
                vt = _vt_layers(ae, vwl.dims.n_layers, vwl.dims.head_dim)
        Kg = bf16_bits_to_f64(ks[0][:, 0][:, tok])
        Vg = vt[:, :, tok].transpose(0, 2, 1)
        for l in range(vwl.dims.n_layers):
            assert_bf16(Kg[l][None], g["K"][l][None].astype(np.float64), "K layer %d" % l)
            assert_bf16(Vg[l][None], g["V"][l][None].astype(np.float64), "V layer %d" % l)
        hg = bf16_bits_to_f64(hidden.cpu().numpy())[0][tok]
        assert_bf16(hg[None], g["hidden"][None].astype(np.float64), "final hidden state")
        assert np.isfinite(outs[0]).all()
        assert np.array_equal(outs[0], outs[1]) and np.array_equal(ks[0], ks[1])
    finally:
        ae.close()
        vlm.close()
