"""Convenience wrapper over the libjpi C ABI for Python callers.

PyTorch provides device memory and streams only; every step of the denoise
runs inside libjpi.  Weights arrive as host arrays (numpy: fp32, or uint16
bf16 bit patterns) keyed by the tensor names of include/jpi.h.
"""
from __future__ import annotations

import numpy as np
import torch

from . import jpi as _j


def _dt(dtype: str) -> int:
    return {"f32": _j.JPI_F32, "bf16": _j.JPI_BF16}[dtype]


def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    """Host array -> device tensor with identical bytes (uint16 bf16 patterns become int16)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


class ActionExpert:
    """One libjpi context on one GPU."""

    def __init__(self, dims, dtype: str, max_batch: int, max_prefix: int, device: int = 0,
                 rms_eps: float = 1e-6, rope_base: float = 1e4, max_corr: int = 0, variant: int = 0,
                 state_dim: int = 0):
        """variant: jpi.JPI_VARIANT_ADARMS (0) or JPI_VARIANT_ACTION_TIME (1, with state_dim)."""
        self.dims, self.dtype, self.device = dims, dtype, device
        self.max_batch, self.max_prefix = max_batch, max_prefix
        cfg = _j.jpi_config(dims.n_layers, dims.width, dims.n_heads, dims.n_kv_heads, dims.head_dim,
                            dims.mlp_dim, dims.action_dim, dims.horizon, max_batch, max_prefix, _dt(dtype),
                            rms_eps, rope_base, max_corr, variant, state_dim)
        st, ctx = _j.jpi_create(cfg, device)
        _j.check(st, None)
        self.ctx = ctx
        self.batch = 0

    def close(self):
        if self.ctx:
            _j.jpi_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _chk(self, st):
        _j.check(st, self.ctx)

    def load_weights(self, weights: dict, stream=None):
        for name, arr in weights.items():
            arr = np.ascontiguousarray(arr)
            dt = _j.JPI_BF16 if arr.dtype == np.uint16 else _j.JPI_F32
            self._chk(_j.jpi_set_weight(self.ctx, name, arr, arr.size, dt, 0, stream))
        self._chk(_j.jpi_finalize_weights(self.ctx, stream))

    def bind_prefix(self, K: torch.Tensor, V: torch.Tensor, prefix_len=None, stream=None):
        """K, V: device tensors [L][B][P][Dh] (fp32 or int16-viewed bf16)."""
        L, B, P, Dh = K.shape
        self._chk(_j.jpi_bind_prefix(self.ctx, K, V, prefix_len, B, P, stream))
        self.batch = B

    def bind_state(self, committed: torch.Tensor | None, n_fixed: int, corr: torch.Tensor | None = None,
                   stream=None):
        """committed: device [B][n_fixed][A] fp32; corr: device [B][n_corr][W] fp32 correction tokens."""
        n_corr = 0 if corr is None else int(corr.shape[1])
        self._chk(_j.jpi_bind_state(self.ctx, committed, n_fixed, corr, n_corr, stream))

    def bind_robot_state(self, state: torch.Tensor, stream=None):
        """state: device [B][state_dim] fp32 (action-time variant)."""
        self._chk(_j.jpi_bind_robot_state(self.ctx, state, stream))

    def set_committed_t0(self, enable: bool):
        """Committed rows at flow time t = 0 (True) or at the step's t (False, the default)."""
        self._chk(_j.jpi_set_committed_t0(self.ctx, int(bool(enable))))

    def denoise(self, noise: torch.Tensor, n_steps: int, out: torch.Tensor | None = None, stream=None):
        if out is None:
            out = torch.empty_like(noise)
        self._chk(_j.jpi_denoise(self.ctx, noise, n_steps, out, stream))
        return out

    def sync(self, stream=None):
        self._chk(_j.jpi_sync(self.ctx, stream))
