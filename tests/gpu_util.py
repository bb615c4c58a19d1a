"""Helpers shared by the GPU tests: run a workload through the C ABI."""
from __future__ import annotations

import json
import os

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


class Inputs:
    """Seeded inputs of a workload (host arrays)."""

    def __init__(self, wl, rollouts=None):
        self.wl = wl
        self.rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
        self.weights = synth.make_weights(wl)
        self.K, self.V = synth.make_prefix(wl, self.rollouts)
        self.noise = synth.make_noise(wl, self.rollouts)
        self.committed = synth.make_committed(wl, self.rollouts) if wl.n_fixed else None
        self.prefix_len = [wl.valid_lengths()[b] for b in self.rollouts]


def make_expert(wl, weights, max_batch=None, max_prefix=None, max_corr=0):
    from paper_2607_12659_amd.expert import ActionExpert
    ae = ActionExpert(wl.dims, wl.dtype, max_batch or wl.batch, max_prefix if max_prefix is not None else wl.prefix,
                      max_corr=max_corr)
    ae.load_weights(weights)
    return ae


def run(ae, K, V, noise, n_steps, prefix_len=None, committed=None, n_fixed=0, corr=None):
    """Bind and denoise; returns fp64 host actions.  corr: host [B][n_corr][W] correction tokens."""
    torch = torch_cuda()
    from paper_2607_12659_amd.expert import to_device
    ae.bind_prefix(to_device(K), to_device(V), prefix_len)
    ae.bind_state(None if committed is None else to_device(np.ascontiguousarray(committed, np.float32)), n_fixed,
                  None if corr is None else to_device(np.ascontiguousarray(corr, np.float32)))
    out = ae.denoise(to_device(np.ascontiguousarray(noise, np.float32)), n_steps)
    ae.sync()
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def run_env(ae, env, *args, **kw):
    """run() with JPI_PERSIST set to env ("0" forces the multi-kernel path, None the default choice)."""
    old = os.environ.get("JPI_PERSIST")
    if env is None:
        os.environ.pop("JPI_PERSIST", None)
    else:
        os.environ["JPI_PERSIST"] = env
    try:
        return run(ae, *args, **kw)
    finally:
        if old is None:
            os.environ.pop("JPI_PERSIST", None)
        else:
            os.environ["JPI_PERSIST"] = old


def load_golden(name):
    with open(os.path.join(GOLDEN, name + ".json")) as f:
        meta = json.load(f)
    return np.load(os.path.join(GOLDEN, name + ".npy"), allow_pickle=False), meta


def rel_l2_per_rollout(got, ref):
    """max over rollouts of ||got_b - ref_b||_2 / ||ref_b||_2."""
    num = np.sqrt(((got - ref) ** 2).reshape(got.shape[0], -1).sum(1))
    den = np.sqrt((ref ** 2).reshape(ref.shape[0], -1).sum(1))
    return float((num / den).max())


class Vlm:
    """A jpi_vlm context loaded with synthetic weights (bf16)."""

    def __init__(self, vd, weights, max_batch, max_prefix):
        torch = torch_cuda()
        from paper_2607_12659_amd import jpi
        self.jpi = jpi
        cfg = jpi.jpi_vlm_config(n_layers=vd.n_layers, width=vd.width, n_heads=vd.n_heads, n_kv_heads=vd.n_kv_heads,
                                 head_dim=vd.head_dim, mlp_dim=vd.mlp_dim, max_batch=max_batch,
                                 max_prefix=max_prefix, dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
        st, self.ctx = jpi.jpi_vlm_create(cfg)
        assert st == jpi.JPI_OK, st
        for name, arr in weights.items():
            arr = np.ascontiguousarray(arr)
            dt = jpi.JPI_BF16 if arr.dtype == np.uint16 else jpi.JPI_F32
            st = jpi.jpi_vlm_set_weight(self.ctx, name, arr, arr.size, dt, 0)
            assert st == jpi.JPI_OK, (name, jpi.jpi_vlm_last_error(self.ctx))
        assert jpi.jpi_vlm_finalize_weights(self.ctx) == jpi.JPI_OK, jpi.jpi_vlm_last_error(self.ctx)
        self.torch = torch

    def prefill(self, emb_dev, batch, prefix, ae, hidden=None):
        st = self.jpi.jpi_vlm_prefill(self.ctx, emb_dev, batch, prefix, ae.ctx, hidden)
        assert st == self.jpi.JPI_OK, self.jpi.jpi_vlm_last_error(self.ctx)

    def close(self):
        self.jpi.jpi_vlm_destroy(self.ctx)


class Corr:
    """A jpi_corr module loaded with synthetic weights (bf16)."""

    def __init__(self, d, weights, max_batch, max_actions, max_vlm_tokens):
        torch = torch_cuda()
        from paper_2607_12659_amd import jpi
        self.jpi, self.torch, self.d = jpi, torch, d
        cfg = jpi.jpi_corr_config(width=d.width, n_heads=d.n_heads, n_kv_heads=1, head_dim=d.head_dim,
                                  mlp_dim=d.mlp_dim, action_dim=d.action_dim, vlm_width=d.vlm_width,
                                  n_query=d.n_query, max_batch=max_batch, max_actions=max_actions,
                                  max_vlm_tokens=max_vlm_tokens, dtype=jpi.JPI_BF16, rms_eps=1e-6, rope_base=1e4)
        st, self.ctx = jpi.jpi_corr_create(cfg)
        assert st == jpi.JPI_OK, st
        for name, arr in weights.items():
            arr = np.ascontiguousarray(arr)
            dt = jpi.JPI_BF16 if arr.dtype == np.uint16 else jpi.JPI_F32
            st = jpi.jpi_corr_set_weight(self.ctx, name, arr, arr.size, dt, 0)
            assert st == jpi.JPI_OK, (name, jpi.jpi_corr_last_error(self.ctx))
        assert jpi.jpi_corr_finalize_weights(self.ctx) == jpi.JPI_OK, jpi.jpi_corr_last_error(self.ctx)

    def compress(self, vlm_state_dev, batch, n_tokens, out=None):
        out = out if out is not None else self.torch.empty((batch, self.d.n_query, self.d.width), device="cuda")
        st = self.jpi.jpi_corr_compress(self.ctx, vlm_state_dev, batch, n_tokens, out)
        assert st == self.jpi.JPI_OK, self.jpi.jpi_corr_last_error(self.ctx)
        return out

    def predict(self, state_dev, actions_dev, batch, n_actions, item=None, conf=None):
        torch = self.torch
        item = item if item is not None else torch.empty((batch, self.d.n_query, self.d.width), device="cuda")
        conf = conf if conf is not None else torch.empty((batch,), device="cuda")
        st = self.jpi.jpi_corr_predict(self.ctx, state_dev, actions_dev, batch, n_actions, item, conf)
        assert st == self.jpi.JPI_OK, self.jpi.jpi_corr_last_error(self.ctx)
        return item, conf

    def close(self):
        self.jpi.jpi_corr_destroy(self.ctx)


def device_view_i16(ptr, shape):
    """torch int16 view of device memory at ptr (zero-copy, read through the array interface)."""
    import torch

    class _A:
        __cuda_array_interface__ = {"shape": tuple(shape), "typestr": "<i2", "data": (int(ptr), False), "version": 2}

    return torch.as_tensor(_A(), device="cuda")


def bf16_bits_to_f64(bits):
    return (np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# bf16-path bars.  The spec bar is a per-rollout relative L2 error of
# 2e-2; a norm over a whole chunk can hide one badly wrong element, so every
# bf16 comparison also bounds each element by 2e-2 of its rollout's largest
# reference magnitude.
BF16_REL = 2e-2
BF16_ELEM = 2e-2


def elem_err_per_rollout(got, ref):
    """max over rollouts of max|got_b - ref_b| / max|ref_b|."""
    B = got.shape[0]
    num = np.abs(got - ref).reshape(B, -1).max(1)
    den = np.abs(ref).reshape(B, -1).max(1)
    return float((num / den).max())


def assert_bf16(got, ref, label="", reg_rel=None, reg_abs=None):
    """Assert the bf16 bars (relative L2 and element-wise) per rollout, plus
    optional regression bars (tighter than the contract: a relative L2 and a
    max-abs well above the measured error).  Returns (rel, max_abs)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.ndim == 1:
        got, ref = got[None], ref[None]
    rel = rel_l2_per_rollout(got, ref)
    elem = elem_err_per_rollout(got, ref)
    mabs = float(np.abs(got - ref).max())
    if label:
        print("%s: rel-L2 %.3e elem %.3e max-abs %.3e" % (label, rel, elem, mabs), flush=True)
    assert np.isfinite(got).all(), label
    assert rel <= BF16_REL, (label, rel)
    assert elem <= BF16_ELEM, (label, elem)
    if reg_rel is not None:
        assert rel <= reg_rel, (label, rel, reg_rel)
    if reg_abs is not None:
        assert mabs <= reg_abs, (label, mabs, reg_abs)
    return rel, mabs
