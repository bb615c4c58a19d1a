"""Seeded synthetic inputs for the action-expert denoiser.

This package is shared by the CPU oracle and by the GPU path's tests and
benchmark.  It holds no arithmetic of the method itself: only the
counter-based normal generator (SplitMix64 + Box-Muller, see ``synth.c``),
bf16 rounding of the generated values, and the shapes of the five named
workloads.  Every tensor is keyed by a name that does not depend on the
batch size, so the batch-1 and batch-8 workloads share weights, rollout-0
prefix KV and rollout-0 noise.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libjpisynth.so")
_lib = None

DEFAULT_SEED = 1234
WEIGHT_STD = 0.02


def build_lib(force: bool = False) -> str:
    """Compile ``synth.c`` into ``libjpisynth.so`` (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp",
                               "-fno-fast-math", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build_lib()
        lib = ctypes.CDLL(_LIB)
        lib.jpi_synth_key.restype = ctypes.c_uint64
        lib.jpi_synth_key.argtypes = [ctypes.c_char_p]
        lib.jpi_synth_normal_f32.restype = None
        lib.jpi_synth_normal_f32.argtypes = [ctypes.c_uint64, ctypes.c_char_p, ctypes.c_double,
                                             ctypes.c_void_p, ctypes.c_int64]
        lib.jpi_synth_f32_to_bf16.restype = None
        lib.jpi_synth_f32_to_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        _lib = lib
    return _lib


def key(name: str) -> int:
    return int(_load().jpi_synth_key(name.encode()))


def normal_f32(seed: int, name: str, std: float, shape) -> np.ndarray:
    """fp32 array of ``std * N(0,1)`` deviates for tensor ``name``."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.float32)
    if n:
        _load().jpi_synth_normal_f32(seed & 0xFFFFFFFFFFFFFFFF, name.encode(), float(std),
                                     out.ctypes.data, n)
    return out.reshape(shape)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest even); returns the bf16 bit patterns as uint16."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    if a.size:
        _load().jpi_synth_f32_to_bf16(a.ctypes.data, out.ctypes.data, a.size)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# numpy twin of the C generator (slow; used to cross-check the C library)
# ---------------------------------------------------------------------------
_M64 = np.uint64(0xFFFFFFFFFFFFFFFF)


def _fnv1a64_py(name: str) -> int:
    h = 0xCBF29CE484222325
    for b in name.encode():
        h ^= b
        h = (h * 0x100000001B3) & 0xFFFFFFFFFFFFFFFF
    return h


def _splitmix64_np(x: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = x + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def normal_f32_numpy(seed: int, name: str, std: float, shape) -> np.ndarray:
    n = int(np.prod(shape)) if len(shape) else 1
    base = np.uint64((seed + _fnv1a64_py(name)) & 0xFFFFFFFFFFFFFFFF)
    j = np.arange(n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        c = base + np.uint64(2) * j
        u1 = ((_splitmix64_np(c) >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * 2.0 ** -53
        u2 = ((_splitmix64_np(c + np.uint64(1)) >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * 2.0 ** -53
    z = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)
    return (std * z).astype(np.float32).reshape(shape)


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class Dims:
    n_layers: int
    width: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    mlp_dim: int
    action_dim: int
    horizon: int


@dataclass(frozen=True)
class Workload:
    name: str
    dims: Dims
    prefix: int          # prefix tokens per rollout (all valid unless prefix_len says otherwise)
    batch: int
    n_steps: int
    n_fixed: int         # committed action rows (never Euler-updated)
    dtype: str           # "f32" or "bf16": storage type of matrices and prefix KV
    seed: int = DEFAULT_SEED
    prefix_len: tuple = field(default=())   # per-rollout valid prefix length; () = all `prefix`
    mod_gain: float = 1.0  # power of two multiplying every layer's modulation matrix and bias

    def valid_lengths(self):
        return list(self.prefix_len) if self.prefix_len else [self.prefix] * self.batch

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = Dims(n_layers=2, width=256, n_heads=4, n_kv_heads=1, head_dim=64, mlp_dim=1024,
            action_dim=7, horizon=10)
PI05 = Dims(n_layers=18, width=1024, n_heads=8, n_kv_heads=1, head_dim=256, mlp_dim=4096,
            action_dim=32, horizon=50)

WORKLOADS = {
    "tiny-fp32": Workload("tiny-fp32", TINY, prefix=64, batch=1, n_steps=4, n_fixed=0, dtype="f32"),
    "pi05-b1": Workload("pi05-b1", PI05, prefix=816, batch=1, n_steps=10, n_fixed=0, dtype="bf16"),
    "pi05-b1-committed10": Workload("pi05-b1-committed10", PI05, prefix=816, batch=1, n_steps=10,
                                    n_fixed=10, dtype="bf16"),
    "pi05-b8": Workload("pi05-b8", PI05, prefix=816, batch=8, n_steps=10, n_fixed=0, dtype="bf16"),
    "pi05-b64-p1600": Workload("pi05-b64-p1600", PI05, prefix=1600, batch=64, n_steps=10, n_fixed=0,
                               dtype="bf16"),
}


def weight_specs(d: Dims):
    """(name, shape, is_matrix) for every expert tensor, in a fixed order.

    Matrices are row-major [out][in] (y = x W^T); biases are vectors.
    """
    W, F, A, Dh, nH = d.width, d.mlp_dim, d.action_dim, d.head_dim, d.n_heads
    kvd = d.n_kv_heads * Dh
    specs = [("action_in.w", (W, A), True), ("action_in.b", (W,), False),
             ("time_mlp.0.w", (W, W), True), ("time_mlp.0.b", (W,), False),
             ("time_mlp.1.w", (W, W), True), ("time_mlp.1.b", (W,), False)]
    for l in range(d.n_layers):
        p = "layers.%d." % l
        specs += [(p + "attn_mod.w", (3 * W, W), True), (p + "attn_mod.b", (3 * W,), False),
                  (p + "q.w", (nH * Dh, W), True), (p + "k.w", (kvd, W), True),
                  (p + "v.w", (kvd, W), True), (p + "o.w", (W, nH * Dh), True),
                  (p + "mlp_mod.w", (3 * W, W), True), (p + "mlp_mod.b", (3 * W,), False),
                  (p + "gate.w", (F, W), True), (p + "up.w", (F, W), True),
                  (p + "down.w", (W, F), True)]
    specs += [("final_mod.w", (2 * W, W), True), ("final_mod.b", (2 * W,), False),
              ("action_out.w", (A, W), True), ("action_out.b", (A,), False)]
    return specs


def make_weights(wl: Workload, std: float = WEIGHT_STD):
    """name -> array.  Matrices are fp32 on the fp32 path and bf16 bit patterns
    (uint16) on the bf16 path; biases are always fp32.

    ``wl.mod_gain`` (a power of two, so that the bf16 rounding of the scaled
    values is the scaled rounding) multiplies the layers' attention and MLP
    modulation tensors: with N(0, 0.02) weights the adaRMSNorm gates are about
    0.06, which damps every sublayer; a gain of 8 makes each sublayer move the
    residual stream by tens of percent."""
    g = float(wl.mod_gain)
    m, e = np.frexp(g)
    if g <= 0 or m != 0.5:
        raise ValueError("mod_gain must be a power of two")
    out = {}
    for name, shape, is_mat in weight_specs(wl.dims):
        a = normal_f32(wl.seed, name, std, shape)
        if g != 1.0 and ("attn_mod" in name or "mlp_mod" in name):
            a = a * np.float32(g)
        if is_mat and wl.dtype == "bf16":
            a = f32_to_bf16_bits(a)
        out[name] = a
    return out


def make_prefix(wl: Workload, rollouts=None):
    """Prefix K and V, each [L][len(rollouts)][P][Dh] (fp32, or bf16 bits), N(0,1)."""
    d = wl.dims
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    kvd = d.n_kv_heads * d.head_dim
    dt = np.uint16 if wl.dtype == "bf16" else np.float32
    K = np.empty((d.n_layers, len(rollouts), wl.prefix, kvd), dtype=dt)
    V = np.empty_like(K)
    for l in range(d.n_layers):
        for i, b in enumerate(rollouts):
            for arr, tag in ((K, "k"), (V, "v")):
                a = normal_f32(wl.seed, "prefix.%s.l%d.b%d" % (tag, l, b), 1.0, (wl.prefix, kvd))
                arr[l, i] = f32_to_bf16_bits(a) if wl.dtype == "bf16" else a
    return K, V


def make_noise(wl: Workload, rollouts=None):
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    d = wl.dims
    return np.stack([normal_f32(wl.seed, "noise.b%d" % b, 1.0, (d.horizon, d.action_dim))
                     for b in rollouts])


def make_committed(wl: Workload, rollouts=None):
    """Committed (already executed) action rows [B][n_fixed][A], N(0,1)."""
    rollouts = list(range(wl.batch)) if rollouts is None else list(rollouts)
    d = wl.dims
    return np.stack([normal_f32(wl.seed, "committed.b%d" % b, 1.0, (d.horizon, d.action_dim))[:wl.n_fixed]
                     for b in rollouts]).reshape(len(rollouts), wl.n_fixed, d.action_dim)
