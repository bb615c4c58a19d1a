"""Kernel-level parity of the GEMM and attention kernels (through the C ABI)
against fp64 references computed from the same input values."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import torch_cuda

pytestmark = pytest.mark.gpu


def _bf16(a):
    return synth.f32_to_bf16_bits(np.asarray(a, np.float32))


def _dev(a):
    from paper_2607_12659_amd.expert import to_device
    return to_device(a)


def _runtime_maps():
    import os
    with open("/proc/self/maps") as f:
        m = f.read()
    libs = sorted(set(l.split()[-1] for l in m.splitlines() if "amdhip" in l or "hsa-runtime" in l))
    return "mapped HIP runtimes: %s" % libs


def _gemm(A, W, M, N, K, dt, splitk):
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    st = jpi.jpi_debug_gemm(_dev(A), _dev(W), C, M, N, K, dt, splitk)
    assert st == jpi.JPI_OK, jpi.jpi_last_error(None) + " | " + _runtime_maps()
    torch.cuda.synchronize()
    return C.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("M", [1, 10, 50, 64, 65, 130, 400])
@pytest.mark.parametrize("N,K", [(2560, 1024), (1024, 2048), (8192, 1024), (1024, 4096), (96, 128)])
@pytest.mark.parametrize("splitk", [1, 2])
def test_gemm_bf16(M, N, K, splitk):
    from paper_2607_12659_amd import jpi
    quantum = 256 if M <= 64 else 64        # K granularity of one split (skinny: 8 waves x 32)
    if K % (quantum * splitk):
        pytest.skip("K=%d cannot be split %d ways" % (K, splitk))
    rng = np.random.default_rng(M * 7 + N + K + splitk)
    A = _bf16(rng.normal(size=(M, K)))
    W = _bf16(rng.normal(size=(N, K)) * 0.02)
    got = _gemm(A, W, M, N, K, jpi.JPI_BF16, splitk)
    a, w = oracle.widen(A), oracle.widen(W)
    ref = a @ w.T
    bound = np.abs(a) @ np.abs(w).T
    assert np.all(np.abs(got - ref) <= 1e-5 * bound + 1e-6), np.abs(got - ref).max()


@pytest.mark.parametrize("M,N,K,splitk", [(50, 1024, 4096, 16), (50, 2560, 1024, 4), (3200, 8192, 1024, 1),
                                          (200, 200, 192, 3), (3200, 2560, 1024, 1), (3200, 1024, 4096, 2),
                                          (816, 2048, 2048, 4), (816, 2560, 2048, 1), (700, 1536, 1024, 1),
                                          (400, 8192, 1024, 1), (400, 1024, 4096, 8), (450, 8100, 320, 1),
                                          (2900, 8000, 512, 1), (3000, 2400, 1024, 1)])
def test_gemm_bf16_more_shapes(M, N, K, splitk):
    from paper_2607_12659_amd import jpi
    rng = np.random.default_rng(M + N + K)
    A = _bf16(rng.normal(size=(M, K)))
    W = _bf16(rng.normal(size=(N, K)) * 0.02)
    got = _gemm(A, W, M, N, K, jpi.JPI_BF16, splitk)
    a, w = oracle.widen(A), oracle.widen(W)
    assert np.all(np.abs(got - a @ w.T) <= 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-6)


@pytest.mark.parametrize("M,N,K,splitk", [(10, 384, 256, 1), (10, 2048, 256, 4), (50, 1024, 2048, 8),
                                          (77, 130, 96, 1)])
def test_gemm_f32(M, N, K, splitk):
    from paper_2607_12659_amd import jpi
    rng = np.random.default_rng(M + N)
    A = rng.normal(size=(M, K)).astype(np.float32)
    W = (rng.normal(size=(N, K)) * 0.02).astype(np.float32)
    got = _gemm(A, W, M, N, K, jpi.JPI_F32, splitk)
    a, w = A.astype(np.float64), W.astype(np.float64)
    assert np.all(np.abs(got - a @ w.T) <= 1e-5 * (np.abs(a) @ np.abs(w).T) + 1e-6)


def test_gemm_splitk_is_deterministic():
    from paper_2607_12659_amd import jpi
    rng = np.random.default_rng(5)
    A = _bf16(rng.normal(size=(50, 4096)))
    W = _bf16(rng.normal(size=(1024, 4096)) * 0.02)
    r1 = _gemm(A, W, 50, 1024, 4096, jpi.JPI_BF16, 16)
    r2 = _gemm(A, W, 50, 1024, 4096, jpi.JPI_BF16, 16)
    assert np.array_equal(r1, r2)


def _attention(dt, B, nH, H, P, Dh, lens, seed=0, nan_masked=False, zero_q=False, loud_key=None):
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(B, nH, H, Dh)) * (0.0 if zero_q else 1.0)
    ks, vs = rng.normal(size=(B, H, Dh)), rng.normal(size=(B, H, Dh))
    kp, vp = rng.normal(size=(B, P, Dh)), rng.normal(size=(B, P, Dh))
    if loud_key is not None:
        kp[:, loud_key] *= 200.0  # scores of about +-200 against ~ +-3 for the other keys
    if nan_masked:
        for b in range(B):
            kp[b, lens[b]:] = np.nan
            vp[b, lens[b]:] = np.nan
    conv = _bf16 if dt == jpi.JPI_BF16 else (lambda a: np.asarray(a, np.float32))
    arrs = [conv(a) for a in (q, ks, vs, kp, vp)]
    out = torch.full((B * H, nH * Dh), float("nan"), dtype=torch.float32, device="cuda")
    st = jpi.jpi_debug_attention(*[_dev(a) for a in arrs], np.array(lens, np.int32), B, nH, H, P, Dh, dt, out)
    assert st == jpi.JPI_OK, jpi.jpi_last_error(None)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64).reshape(B, H, nH, Dh)
    ref = np.empty_like(got)
    w = [oracle.widen(a) for a in arrs]
    for b in range(B):
        r = oracle.prefix_self_attention(w[0][b], w[3][b], w[4][b], lens[b], w[1][b], w[2][b])
        ref[b] = np.transpose(r, (1, 0, 2))
    return got, ref, w


@pytest.mark.parametrize("B,nH,H,P,Dh,lens", [(2, 8, 50, 816, 256, [816, 301]), (1, 8, 50, 1600, 256, [1600]),
                                              (3, 4, 10, 64, 64, [64, 0, 17]), (1, 2, 70, 130, 128, [129]),
                                              (5, 8, 37, 300, 256, [300, 1, 0, 63, 64]),
                                              (16, 8, 50, 816, 256, [816] * 15 + [5]),
                                              (64, 8, 50, 1600, 256, [1600] * 63 + [777])])
def test_attention_bf16(B, nH, H, P, Dh, lens):
    # covers one and several key ranges per query tile, action blocks with a
    # ragged tail (H = 37, 70), empty and one-key prefixes, and the batch-64 shape
    from paper_2607_12659_amd import jpi
    got, ref, _ = _attention(jpi.JPI_BF16, B, nH, H, P, Dh, lens)
    # probabilities enter the PV product rounded to bf16 (relative 2^-9 each)
    assert np.abs(got - ref).max() < 1e-2, np.abs(got - ref).max()
    assert np.sqrt(((got - ref) ** 2).mean()) < 2e-3


@pytest.mark.parametrize("B", [1, 16, 64])
def test_attention_bf16_late_dominant_key(B):
    # one prefix key far into the sequence scores hundreds of nats above the
    # keys seen before it: the rows where it wins must come out as its value
    # row (the kernel's probability reference has to move up for them)
    from paper_2607_12659_amd import jpi
    got, ref, _ = _attention(jpi.JPI_BF16, B, 8, 50, 816, 256, [816] * B, seed=5, loud_key=700)
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() < 1e-2, np.abs(got - ref).max()


@pytest.mark.parametrize("B,nH,H,P,Dh,lens", [(2, 8, 50, 816, 256, [816, 301]), (1, 4, 10, 64, 64, [64]),
                                              (2, 4, 10, 64, 64, [0, 33])])
def test_attention_f32(B, nH, H, P, Dh, lens):
    from paper_2607_12659_amd import jpi
    got, ref, _ = _attention(jpi.JPI_F32, B, nH, H, P, Dh, lens)
    assert np.abs(got - ref).max() < 2e-5, np.abs(got - ref).max()


@pytest.mark.parametrize("dt_name", ["bf16", "f32"])
def test_attention_masked_slots_never_read(dt_name):
    from paper_2607_12659_amd import jpi
    dt = jpi.JPI_BF16 if dt_name == "bf16" else jpi.JPI_F32
    lens = [100, 7]
    a, _, _ = _attention(dt, 2, 8, 50, 816, 256, lens, seed=3)
    b, _, _ = _attention(dt, 2, 8, 50, 816, 256, lens, seed=3, nan_masked=True)
    assert not np.isnan(b).any()
    assert np.array_equal(a, b)


def test_attention_zero_query_averages_valid_values():
    from paper_2607_12659_amd import jpi
    got, _, w = _attention(jpi.JPI_F32, 1, 2, 10, 64, 64, [40], zero_q=True)
    mean = np.concatenate([w[4][0][:40], w[2][0]]).mean(axis=0)
    np.testing.assert_allclose(got[0], np.broadcast_to(mean, got[0].shape), atol=2e-6)
