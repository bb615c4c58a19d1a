"""ctypes binding of libjpi (include/jpi.h).

Argument marshalling only: every function here has the name of the C entry
point it calls and forwards plain pointers and sizes.  Tensors may be given
as torch tensors (device memory), numpy arrays (host memory) or raw integer
addresses; streams as torch.cuda.Stream objects, raw hipStream_t integers or
None (the null stream).  There is no fallback: if libjpi.so is missing the
import of this module fails.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# JPI_LIB selects another build of the same library (the trace build of
# trace_links.py); the default is the in-tree libjpi.so
LIB_PATH = os.environ.get("JPI_LIB") or os.path.join(_HERE, "libjpi.so")

JPI_OK, JPI_ERR_ARG, JPI_ERR_SHAPE, JPI_ERR_DTYPE, JPI_ERR_STATE, JPI_ERR_OOM, JPI_ERR_HIP, JPI_ERR_UNSUPPORTED = range(8)
JPI_F32, JPI_BF16 = 0, 1
JPI_VARIANT_ADARMS, JPI_VARIANT_ACTION_TIME = 0, 1

EXPORTED = ["jpi_abi_version", "jpi_status_str", "jpi_last_error", "jpi_create", "jpi_destroy", "jpi_set_weight",
            "jpi_finalize_weights", "jpi_prefix_buffers", "jpi_debug_prefix_vt", "jpi_debug_persist_trace",
            "jpi_bind_prefix", "jpi_bind_state", "jpi_denoise",
            "jpi_sync", "jpi_debug_gemm", "jpi_gemm_noalloc", "jpi_gemm_noalloc_scratch_bytes",
            "jpi_gemm_noalloc_last_error", "jpi_debug_attention", "jpi_debug_time_kernel", "jpi_debug_kernel_time",
            "jpi_debug_set_spin_limit",
            "jpi_sched_run", "jpi_sched_sim_hooks", "jpi_vlm_create", "jpi_vlm_destroy", "jpi_vlm_set_weight",
            "jpi_vlm_finalize_weights", "jpi_vlm_prefill", "jpi_vlm_last_error", "jpi_set_committed_t0", "jpi_bind_robot_state", "jpi_corr_create",
            "jpi_corr_destroy", "jpi_corr_set_weight", "jpi_corr_finalize_weights", "jpi_corr_compress",
            "jpi_corr_predict", "jpi_corr_last_error"]
JPI_KERNEL_NONE, JPI_KERNEL_QKV, JPI_KERNEL_ATTENTION, JPI_KERNEL_OPROJ, JPI_KERNEL_GATEUP, JPI_KERNEL_DOWN, \
    JPI_KERNEL_PERSISTENT = range(-1, 6)


class jpi_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("width", ctypes.c_int), ("n_heads", ctypes.c_int),
                ("n_kv_heads", ctypes.c_int), ("head_dim", ctypes.c_int), ("mlp_dim", ctypes.c_int),
                ("action_dim", ctypes.c_int), ("horizon", ctypes.c_int), ("max_batch", ctypes.c_int),
                ("max_prefix", ctypes.c_int), ("dtype", ctypes.c_int), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("max_corr", ctypes.c_int), ("variant", ctypes.c_int),
                ("state_dim", ctypes.c_int)]


# include/jpi_vlm.h
class jpi_vlm_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("width", ctypes.c_int), ("n_heads", ctypes.c_int),
                ("n_kv_heads", ctypes.c_int), ("head_dim", ctypes.c_int), ("mlp_dim", ctypes.c_int),
                ("max_batch", ctypes.c_int), ("max_prefix", ctypes.c_int), ("dtype", ctypes.c_int),
                ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float)]


# include/jpi_corr.h
class jpi_corr_config(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int), ("n_heads", ctypes.c_int), ("n_kv_heads", ctypes.c_int),
                ("head_dim", ctypes.c_int), ("mlp_dim", ctypes.c_int), ("action_dim", ctypes.c_int),
                ("vlm_width", ctypes.c_int), ("n_query", ctypes.c_int), ("max_batch", ctypes.c_int),
                ("max_actions", ctypes.c_int), ("max_vlm_tokens", ctypes.c_int), ("dtype", ctypes.c_int),
                ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float)]


# include/jpi_sched.h
class jpi_sched_config(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_double), ("delta", ctypes.c_int), ("delta_ae", ctypes.c_int),
                ("chunk_len", ctypes.c_int), ("action_ms", ctypes.c_double), ("iterations", ctypes.c_int64)]


SCHED_VLM_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(ctypes.c_double))
SCHED_CORR_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                 ctypes.c_int64, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double))
SCHED_ACT_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int64,
                                ctypes.POINTER(ctypes.c_double))


class jpi_sched_hooks(ctypes.Structure):
    _fields_ = [("vlm", SCHED_VLM_FN), ("corr", SCHED_CORR_FN), ("act", SCHED_ACT_FN), ("user", ctypes.c_void_p)]


class jpi_sched_event(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int64), ("vlm", ctypes.c_int), ("n_committed", ctypes.c_int),
                ("conf_in", ctypes.c_double), ("conf_out", ctypes.c_double), ("ms", ctypes.c_double),
                ("executed", ctypes.c_int64), ("starved", ctypes.c_int64)]


class jpi_sched_stats(ctypes.Structure):
    _fields_ = [("iterations", ctypes.c_int64), ("vlm_calls", ctypes.c_int64), ("startup_ms", ctypes.c_double),
                ("total_ms", ctypes.c_double), ("reaction_ms", ctypes.c_double), ("control_hz", ctypes.c_double),
                ("vlm_fraction", ctypes.c_double), ("actions_executed", ctypes.c_int64),
                ("actions_starved", ctypes.c_int64)]


class jpi_sched_sim(ctypes.Structure):
    _fields_ = [("vit_ms", ctypes.c_double), ("llm_ms", ctypes.c_double), ("corr_ms", ctypes.c_double),
                ("ae_ms", ctypes.c_double), ("conf", ctypes.POINTER(ctypes.c_double)), ("n_conf", ctypes.c_int64),
                ("corr_calls", ctypes.c_int64), ("vlm_calls", ctypes.c_int64), ("act_calls", ctypes.c_int64)]


if not os.path.exists(LIB_PATH):
    raise ImportError("libjpi.so is not built (run paper_2607_12659_amd/build.py); there is no fallback path")
# PyTorch-ROCm bundles its own HIP runtime (SONAME libamdhip64.so.7).  Map it
# before libjpi so that libjpi's dependency resolves to that same copy: two
# HIP runtimes in one process do not share devices, memory or streams.
try:
    import torch  # noqa: F401
except ImportError:
    pass
_lib = ctypes.CDLL(LIB_PATH)

_vp, _i, _i64, _f = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
_sig = {
    "jpi_abi_version": (_i, []),
    "jpi_status_str": (ctypes.c_char_p, [_i]),
    "jpi_last_error": (ctypes.c_char_p, [_vp]),
    "jpi_create": (_i, [ctypes.POINTER(jpi_config), _i, ctypes.POINTER(_vp)]),
    "jpi_destroy": (_i, [_vp]),
    "jpi_set_weight": (_i, [_vp, ctypes.c_char_p, _vp, _i64, _i, _i, _vp]),
    "jpi_finalize_weights": (_i, [_vp, _vp]),
    "jpi_prefix_buffers": (_i, [_vp, ctypes.POINTER(_vp), ctypes.POINTER(_vp)]),
    "jpi_debug_prefix_vt": (_i, [_vp, ctypes.POINTER(_vp), ctypes.POINTER(_i)]),
    "jpi_debug_persist_trace": (_i, [_vp, _vp, _i64, ctypes.POINTER(_i), ctypes.POINTER(_i),
                                     ctypes.POINTER(ctypes.c_double)]),
    "jpi_bind_prefix": (_i, [_vp, _vp, _vp, _vp, _i, _i, _vp]),
    "jpi_bind_state": (_i, [_vp, _vp, _i, _vp, _i, _vp]),
    "jpi_denoise": (_i, [_vp, _vp, _i, _vp, _vp]),
    "jpi_sync": (_i, [_vp, _vp]),
    "jpi_debug_gemm": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "jpi_gemm_noalloc": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "jpi_gemm_noalloc_scratch_bytes": (ctypes.c_size_t, []),
    "jpi_gemm_noalloc_last_error": (ctypes.c_char_p, []),
    "jpi_debug_attention": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp]),
    "jpi_debug_time_kernel": (_i, [_vp, _i]),
    "jpi_debug_set_spin_limit": (_i, [_vp, ctypes.c_uint32]),
    "jpi_debug_kernel_time": (_i, [_vp, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(_i)]),
    "jpi_sched_run": (_i, [ctypes.POINTER(jpi_sched_config), ctypes.POINTER(jpi_sched_hooks),
                           ctypes.POINTER(jpi_sched_stats), ctypes.POINTER(jpi_sched_event), _i64]),
    "jpi_sched_sim_hooks": (_i, [ctypes.POINTER(jpi_sched_sim), ctypes.POINTER(jpi_sched_hooks)]),
    "jpi_vlm_create": (_i, [ctypes.POINTER(jpi_vlm_config), _i, ctypes.POINTER(_vp)]),
    "jpi_vlm_destroy": (_i, [_vp]),
    "jpi_vlm_set_weight": (_i, [_vp, ctypes.c_char_p, _vp, _i64, _i, _i, _vp]),
    "jpi_vlm_finalize_weights": (_i, [_vp, _vp]),
    "jpi_vlm_prefill": (_i, [_vp, _vp, _i, _i, _vp, _vp, _vp]),
    "jpi_vlm_last_error": (ctypes.c_char_p, [_vp]),
    "jpi_set_committed_t0": (_i, [_vp, _i]),
    "jpi_bind_robot_state": (_i, [_vp, _vp, _vp]),
    "jpi_corr_create": (_i, [ctypes.POINTER(jpi_corr_config), _i, ctypes.POINTER(_vp)]),
    "jpi_corr_destroy": (_i, [_vp]),
    "jpi_corr_set_weight": (_i, [_vp, ctypes.c_char_p, _vp, _i64, _i, _i, _vp]),
    "jpi_corr_finalize_weights": (_i, [_vp, _vp]),
    "jpi_corr_compress": (_i, [_vp, _vp, _i, _i, _vp, _vp]),
    "jpi_corr_predict": (_i, [_vp, _vp, _vp, _i, _i, _vp, _vp, _vp]),
    "jpi_corr_last_error": (ctypes.c_char_p, [_vp]),
}
for _name, (_res, _args) in _sig.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


def addr(t) -> int | None:
    """Address of a torch tensor / numpy array / int / None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if hasattr(t, "data_ptr"):
        return t.data_ptr()
    if hasattr(t, "ctypes"):
        return t.ctypes.data
    raise TypeError("cannot take the address of %r" % type(t))


def stream_handle(s) -> int | None:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _i32_host(a):
    if a is None:
        return None
    import numpy as np
    arr = np.ascontiguousarray(a, dtype=np.int32)
    return arr


# ---------------------------------------------------------------------------
# same-named wrappers (return the jpi_status, plus outputs where the C call has them)
# ---------------------------------------------------------------------------
def jpi_abi_version() -> int:
    return _lib.jpi_abi_version()


def jpi_status_str(status: int) -> str:
    return _lib.jpi_status_str(status).decode()


def jpi_last_error(ctx) -> str:
    return _lib.jpi_last_error(ctx).decode()


def jpi_create(cfg: jpi_config, device: int = 0):
    out = _vp()
    st = _lib.jpi_create(ctypes.byref(cfg), device, ctypes.byref(out))
    return st, out.value


def jpi_destroy(ctx) -> int:
    return _lib.jpi_destroy(ctx)


def jpi_set_weight(ctx, name: str, data, n_elems: int, dtype: int, is_device: int, stream=None) -> int:
    return _lib.jpi_set_weight(ctx, name.encode(), addr(data), n_elems, dtype, is_device, stream_handle(stream))


def jpi_finalize_weights(ctx, stream=None) -> int:
    return _lib.jpi_finalize_weights(ctx, stream_handle(stream))


def jpi_prefix_buffers(ctx):
    k, v = _vp(), _vp()
    st = _lib.jpi_prefix_buffers(ctx, ctypes.byref(k), ctypes.byref(v))
    return st, k.value, v.value


def jpi_debug_persist_trace(ctx):
    """(status, stamps [workgroups][slots] uint64 or None, ticks per microsecond)."""
    import numpy as np
    nw, ns, tpu = _i(), _i(), ctypes.c_double()
    st = _lib.jpi_debug_persist_trace(ctx, None, 0, ctypes.byref(nw), ctypes.byref(ns), ctypes.byref(tpu))
    if st != JPI_OK:
        return st, None, 0.0
    out = np.zeros((nw.value, ns.value), dtype=np.uint64)
    st = _lib.jpi_debug_persist_trace(ctx, out.ctypes.data, out.size, ctypes.byref(nw), ctypes.byref(ns),
                                      ctypes.byref(tpu))
    return st, out, tpu.value


def jpi_debug_prefix_vt(ctx):
    vt, ld = _vp(), _i()
    st = _lib.jpi_debug_prefix_vt(ctx, ctypes.byref(vt), ctypes.byref(ld))
    return st, vt.value, ld.value


def jpi_bind_prefix(ctx, k, v, prefix_len_host, batch: int, prefix: int, stream=None) -> int:
    lens = _i32_host(prefix_len_host)
    return _lib.jpi_bind_prefix(ctx, addr(k), addr(v), None if lens is None else lens.ctypes.data, batch, prefix,
                                stream_handle(stream))


def jpi_bind_state(ctx, committed_dev, n_fixed: int, corr_tokens=None, n_corr: int = 0, stream=None) -> int:
    return _lib.jpi_bind_state(ctx, addr(committed_dev), n_fixed, addr(corr_tokens), n_corr, stream_handle(stream))


def jpi_denoise(ctx, noise_dev, n_steps: int, actions_dev, stream=None) -> int:
    return _lib.jpi_denoise(ctx, addr(noise_dev), n_steps, addr(actions_dev), stream_handle(stream))


def jpi_sync(ctx, stream=None) -> int:
    return _lib.jpi_sync(ctx, stream_handle(stream))


def jpi_debug_gemm(A, W, C, M: int, N: int, K: int, dtype: int, splitk: int = 1, stream=None) -> int:
    return _lib.jpi_debug_gemm(addr(A), addr(W), addr(C), M, N, K, dtype, splitk, stream_handle(stream))


def jpi_gemm_noalloc(A, W, C, M: int, N: int, K: int, dtype: int, splitk: int = 1, stream=None) -> int:
    return _lib.jpi_gemm_noalloc(addr(A), addr(W), addr(C), M, N, K, dtype, splitk, stream_handle(stream))


def jpi_gemm_noalloc_scratch_bytes() -> int:
    return _lib.jpi_gemm_noalloc_scratch_bytes()


def jpi_gemm_noalloc_last_error() -> str:
    return (_lib.jpi_gemm_noalloc_last_error() or b"").decode()


def jpi_debug_attention(q, ks, vs, kp, vp, prefix_len_host, batch, n_heads, H, P, Dh, dtype, out, stream=None) -> int:
    lens = _i32_host(prefix_len_host)
    return _lib.jpi_debug_attention(addr(q), addr(ks), addr(vs), addr(kp), addr(vp), lens.ctypes.data, batch, n_heads,
                                    H, P, Dh, dtype, addr(out), stream_handle(stream))


def jpi_debug_set_spin_limit(ctx, polls: int) -> int:
    """Bound of the single-launch kernel's waits in polls (0: the default); a test hook for its failure path."""
    return _lib.jpi_debug_set_spin_limit(ctx, polls)


def jpi_debug_time_kernel(ctx, kind: int) -> int:
    return _lib.jpi_debug_time_kernel(ctx, kind)


def jpi_debug_kernel_time(ctx):
    ms, n = ctypes.c_float(), _i()
    st = _lib.jpi_debug_kernel_time(ctx, ctypes.byref(ms), ctypes.byref(n))
    return st, ms.value, n.value


def jpi_sched_run(cfg: jpi_sched_config, hooks: jpi_sched_hooks, trace_cap: int = 0):
    """Returns (status, stats, events); events holds the first trace_cap iterations."""
    stats = jpi_sched_stats()
    trace = (jpi_sched_event * trace_cap)() if trace_cap > 0 else None
    st = _lib.jpi_sched_run(ctypes.byref(cfg), ctypes.byref(hooks), ctypes.byref(stats), trace, trace_cap)
    return st, stats, (list(trace) if trace is not None else [])


def jpi_sched_sim_hooks(sim: jpi_sched_sim, hooks: jpi_sched_hooks) -> int:
    return _lib.jpi_sched_sim_hooks(ctypes.byref(sim), ctypes.byref(hooks))


def jpi_vlm_create(cfg: jpi_vlm_config, device: int = 0):
    out = ctypes.c_void_p()
    st = _lib.jpi_vlm_create(ctypes.byref(cfg), device, ctypes.byref(out))
    return st, out


def jpi_vlm_destroy(vlm) -> int:
    return _lib.jpi_vlm_destroy(vlm)


def jpi_vlm_set_weight(vlm, name: str, data, n_elems: int, dtype: int, is_device: int, stream=None) -> int:
    return _lib.jpi_vlm_set_weight(vlm, name.encode(), addr(data), n_elems, dtype, is_device, stream_handle(stream))


def jpi_vlm_finalize_weights(vlm, stream=None) -> int:
    return _lib.jpi_vlm_finalize_weights(vlm, stream_handle(stream))


def jpi_vlm_prefill(vlm, emb, batch: int, prefix: int, ae_ctx, hidden_out=None, stream=None) -> int:
    return _lib.jpi_vlm_prefill(vlm, addr(emb), batch, prefix, ae_ctx, addr(hidden_out), stream_handle(stream))


def jpi_vlm_last_error(vlm) -> str:
    return _lib.jpi_vlm_last_error(vlm).decode()


def jpi_set_committed_t0(ctx, enable: int) -> int:
    return _lib.jpi_set_committed_t0(ctx, enable)


def jpi_bind_robot_state(ctx, state_dev, stream=None) -> int:
    return _lib.jpi_bind_robot_state(ctx, addr(state_dev), stream_handle(stream))


def jpi_corr_create(cfg: jpi_corr_config, device: int = 0):
    out = _vp()
    st = _lib.jpi_corr_create(ctypes.byref(cfg), device, ctypes.byref(out))
    return st, out


def jpi_corr_destroy(m) -> int:
    return _lib.jpi_corr_destroy(m)


def jpi_corr_set_weight(m, name: str, data, n_elems: int, dtype: int, is_device: int, stream=None) -> int:
    return _lib.jpi_corr_set_weight(m, name.encode(), addr(data), n_elems, dtype, is_device, stream_handle(stream))


def jpi_corr_finalize_weights(m, stream=None) -> int:
    return _lib.jpi_corr_finalize_weights(m, stream_handle(stream))


def jpi_corr_compress(m, vlm_state, batch: int, n_tokens: int, state_out, stream=None) -> int:
    return _lib.jpi_corr_compress(m, addr(vlm_state), batch, n_tokens, addr(state_out), stream_handle(stream))


def jpi_corr_predict(m, state, actions, batch: int, n_actions: int, item_out, conf_out, stream=None) -> int:
    return _lib.jpi_corr_predict(m, addr(state), addr(actions), batch, n_actions, addr(item_out), addr(conf_out),
                                 stream_handle(stream))


def jpi_corr_last_error(m) -> str:
    return _lib.jpi_corr_last_error(m).decode()


class JpiError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (jpi_status_str(status), msg))
        self.status = status


def check(status: int, ctx=None):
    if status != JPI_OK:
        raise JpiError(status, jpi_last_error(ctx))
