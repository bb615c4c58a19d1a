"""C-ABI checks that need no GPU: the library loads, exports every entry point
include/jpi.h declares, and rejects bad arguments on the host before any
device work."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    from paper_2607_12659_amd import jpi
    return jpi


def declared_entry_points():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            with open(os.path.join(ROOT, "include", h)) as f:
                text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
            names |= set(re.findall(r"\b(jpi_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


def test_header_declares_the_boundary():
    names = declared_entry_points()
    for must in ("jpi_create", "jpi_destroy", "jpi_set_weight", "jpi_finalize_weights", "jpi_prefix_buffers",
                 "jpi_bind_prefix", "jpi_bind_state", "jpi_denoise", "jpi_sync", "jpi_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol():
    j = _lib()
    lib = ctypes.CDLL(j.LIB_PATH)
    for name in declared_entry_points():
        assert hasattr(lib, name), name
    assert set(declared_entry_points()) == set(j.EXPORTED)


def test_abi_version_and_status_strings():
    j = _lib()
    assert j.jpi_abi_version() == 4
    for st in range(8):
        assert j.jpi_status_str(st)
    assert j.jpi_status_str(99) == "unknown status"


def _cfg(**kw):
    j = _lib()
    base = dict(n_layers=2, width=256, n_heads=4, n_kv_heads=1, head_dim=64, mlp_dim=1024, action_dim=7, horizon=10,
                max_batch=1, max_prefix=64, dtype=j.JPI_F32, rms_eps=1e-6, rope_base=1e4)
    base.update(kw)
    return j.jpi_config(**base)


@pytest.mark.parametrize("bad", [dict(n_layers=0), dict(width=-1), dict(n_kv_heads=2), dict(head_dim=48),
                                 dict(width=100), dict(mlp_dim=1000), dict(max_batch=0), dict(horizon=0),
                                 dict(dtype=7), dict(rms_eps=0.0), dict(rope_base=1.0), dict(action_dim=0),
                                 dict(max_prefix=-1)])
def test_create_rejects_bad_config_before_touching_the_device(bad):
    j = _lib()
    st, ctx = j.jpi_create(_cfg(**bad), 0)
    assert st == j.JPI_ERR_ARG and not ctx
    assert j.jpi_last_error(None)


def test_null_arguments():
    j = _lib()
    assert j._lib.jpi_create(None, 0, None) == j.JPI_ERR_ARG
    assert j.jpi_destroy(None) == j.JPI_OK
    assert j.jpi_set_weight(None, "action_in.w", 1, 1, j.JPI_F32, 0) == j.JPI_ERR_ARG
    assert j.jpi_finalize_weights(None) == j.JPI_ERR_ARG
    assert j.jpi_bind_prefix(None, 1, 1, None, 1, 1) == j.JPI_ERR_ARG
    assert j.jpi_bind_state(None, None, 0) == j.JPI_ERR_ARG
    assert j.jpi_denoise(None, 1, 1, 1) == j.JPI_ERR_ARG
    assert j.jpi_sync(None) == j.JPI_ERR_ARG
    assert j.jpi_set_committed_t0(None, 1) == j.JPI_ERR_ARG
    assert j.jpi_bind_robot_state(None, 1) == j.JPI_ERR_ARG
    assert j.jpi_corr_destroy(None) == j.JPI_OK
    assert j.jpi_corr_set_weight(None, "fuse.w", 1, 1, j.JPI_BF16, 0) == j.JPI_ERR_ARG
    assert j.jpi_corr_finalize_weights(None) == j.JPI_ERR_ARG
    assert j.jpi_corr_compress(None, 1, 1, 1, 1) == j.JPI_ERR_ARG
    assert j.jpi_corr_predict(None, 1, 1, 1, 1, 1, 1) == j.JPI_ERR_ARG
    assert j.jpi_corr_last_error(None)
    assert j.jpi_vlm_destroy(None) == j.JPI_OK
    assert j.jpi_vlm_prefill(None, 1, 1, 1, None) == j.JPI_ERR_ARG
    assert j.jpi_debug_gemm(None, 1, 1, 4, 4, 64, j.JPI_BF16) == j.JPI_ERR_ARG
    assert j.jpi_debug_gemm(1, 1, 1, 4, 4, 65, j.JPI_BF16) == j.JPI_ERR_ARG      # K not a multiple of 64
    assert j.jpi_debug_gemm(1, 1, 1, 0, 4, 64, j.JPI_BF16) == j.JPI_ERR_ARG
    assert j.jpi_debug_gemm(1, 1, 1, 4, 4, 64, j.JPI_BF16, splitk=2) == j.JPI_ERR_ARG
    import numpy as np
    assert j.jpi_debug_attention(1, 1, 1, 1, 1, np.array([5]), 1, 1, 4, 4, 64, j.JPI_F32, 1) == j.JPI_ERR_ARG
    assert j.jpi_debug_attention(1, 1, 1, 1, 1, np.array([2]), 1, 1, 4, 4, 48, j.JPI_F32, 1) == j.JPI_ERR_ARG


@pytest.mark.parametrize("bad", [dict(max_corr=-1), dict(max_corr=65), dict(variant=2), dict(state_dim=3),
                                 dict(variant=1), dict(variant=1, state_dim=8, max_corr=2),
                                 dict(variant=1, state_dim=8, max_prefix=0)])
def test_create_rejects_bad_variant_or_correction_config(bad):
    j = _lib()
    st, ctx = j.jpi_create(_cfg(**bad), 0)
    assert st == j.JPI_ERR_ARG and not ctx


def test_corr_create_rejects_bad_config_before_touching_the_device():
    j = _lib()
    good = dict(width=256, n_heads=4, n_kv_heads=1, head_dim=64, mlp_dim=512, action_dim=7, vlm_width=256,
                n_query=4, max_batch=1, max_actions=5, max_vlm_tokens=40, dtype=j.JPI_BF16, rms_eps=1e-6,
                rope_base=1e4)
    for bad in (dict(width=100), dict(n_kv_heads=2), dict(head_dim=48), dict(vlm_width=200), dict(n_query=0),
                dict(max_actions=0), dict(action_dim=300), dict(rms_eps=0.0)):
        st, m = j.jpi_corr_create(j.jpi_corr_config(**{**good, **bad}))
        assert st == j.JPI_ERR_ARG and not m, bad
    st, m = j.jpi_corr_create(j.jpi_corr_config(**{**good, "dtype": j.JPI_F32}))
    assert st == j.JPI_ERR_UNSUPPORTED and not m


def test_build_entry_compiles_everything():
    """__graft_entry__.build() must produce the library and the generator."""
    import importlib
    ge = importlib.import_module("__graft_entry__")
    assert callable(ge.build) and callable(ge.smoke)


def test_noalloc_gemm_rejects_bad_arguments_on_the_host():
    """jpi_gemm_noalloc checks every argument, including the static scratch
    limit, before touching a device (no GPU here; the pointers are never
    dereferenced)."""
    j = _lib()
    fake = 0x1000
    assert j.jpi_gemm_noalloc_scratch_bytes() == 16 << 20
    assert j.jpi_gemm_noalloc(None, fake, fake, 50, 1024, 1024, j.JPI_BF16, 1) == j.JPI_ERR_ARG
    assert j.jpi_gemm_noalloc(fake, fake, fake, 0, 1024, 1024, j.JPI_BF16, 1) == j.JPI_ERR_ARG
    assert j.jpi_gemm_noalloc(fake, fake, fake, 50, 1024, 1000, j.JPI_BF16, 1) == j.JPI_ERR_ARG
    assert "multiple of" in j.jpi_gemm_noalloc_last_error()
    # 16 slices of 64 x 8192 fp32 = 32 MiB > 16 MiB
    assert j.jpi_gemm_noalloc(fake, fake, fake, 64, 8192, 4096, j.JPI_BF16, 16) == j.JPI_ERR_ARG
    assert "exceeds the static scratch" in j.jpi_gemm_noalloc_last_error()
