"""End-to-end parity of jpi_denoise with the fp64 oracle, plus invariants of
the GPU path.

Bars: fp32 path max-abs <= 1e-4 on every output element; bf16 path (bf16
weights and prefix KV, fp32 accumulation) per-rollout relative L2 error
<= 2e-2 on the final actions and every element within 2e-2 of its
rollout's largest reference magnitude.  The pi0.5-shape cases also carry
regression bars (relative L2 <= 2e-3, max-abs <= 1e-2; measured about
3.5e-4 and 1.8e-3), so that a kernel change that loses accuracy fails long
before the contract bar.  Large workloads compare with oracle outputs
stored by tests/golden/make_golden.py (oracle + generator only).
"""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import (Inputs, assert_bf16, load_golden, make_expert, rel_l2_per_rollout, run, run_env,
                      torch_cuda)

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4
REG_REL = 2e-3   # regression bars of the pi0.5-shape bf16 cases
REG_ABS = 1e-2


@pytest.fixture(scope="module")
def tiny():
    wl = synth.WORKLOADS["tiny-fp32"]
    inp = Inputs(wl)
    ae = make_expert(wl, inp.weights, max_batch=4, max_prefix=wl.prefix)
    yield wl, inp, ae
    ae.close()


def _oracle(wl, inp, n_steps=None, lens=None, noise=None, committed=None, n_fixed=0, K=None, V=None):
    ex = oracle.Expert(wl.dims, inp.weights)
    return oracle.denoise(ex, inp.noise if noise is None else noise, inp.K if K is None else K,
                          inp.V if V is None else V, inp.prefix_len if lens is None else lens,
                          n_steps or wl.n_steps, committed=committed, n_fixed=n_fixed)


def test_tiny_fp32_matches_oracle(tiny):
    wl, inp, ae = tiny
    print("case tiny-fp32", flush=True)
    got = run(ae, inp.K, inp.V, inp.noise, wl.n_steps)
    ref = _oracle(wl, inp)
    err = np.abs(got - ref).max()
    print("tiny-fp32 max-abs %.3e" % err)
    assert err <= F32_TOL


@pytest.mark.parametrize("n_steps", [1, 2, 7])
def test_tiny_fp32_step_counts(tiny, n_steps):
    wl, inp, ae = tiny
    got = run(ae, inp.K, inp.V, inp.noise, n_steps)
    assert np.abs(got - _oracle(wl, inp, n_steps=n_steps)).max() <= F32_TOL


def test_tiny_n_steps_1_is_noise_minus_velocity(tiny):
    wl, inp, ae = tiny
    got = run(ae, inp.K, inp.V, inp.noise, 1)
    v = oracle.velocity(oracle.Expert(wl.dims, inp.weights), inp.noise.astype(np.float64), 1.0, inp.K, inp.V,
                        inp.prefix_len)
    assert np.abs(got - (inp.noise - v)).max() <= F32_TOL


def test_tiny_batched_ragged_prefix_and_committed(tiny):
    wl, inp, ae = tiny
    wl4 = wl.with_(batch=3, n_fixed=3, prefix_len=(64, 0, 23))
    i4 = Inputs(wl4)
    got = run(ae, i4.K, i4.V, i4.noise, wl.n_steps, prefix_len=i4.prefix_len, committed=i4.committed, n_fixed=3)
    ref = _oracle(wl4, i4, committed=i4.committed, n_fixed=3)
    assert np.abs(got - ref).max() <= F32_TOL
    assert np.array_equal(got[:, :3].astype(np.float32), i4.committed.astype(np.float32))


def test_tiny_masked_garbage_invariance(tiny):
    wl, inp, ae = tiny
    lens = [40]
    a = run(ae, inp.K, inp.V, inp.noise, wl.n_steps, prefix_len=lens)
    K, V = inp.K.copy(), inp.V.copy()
    K[:, 0, 40:] = np.nan
    V[:, 0, 40:] = np.inf
    b = run(ae, K, V, inp.noise, wl.n_steps, prefix_len=lens)
    assert not np.isnan(b).any() and np.array_equal(a, b)
    assert np.abs(a - _oracle(wl, inp, lens=lens)).max() <= F32_TOL


def test_tiny_prefix_permutation_invariance(tiny):
    wl, inp, ae = tiny
    a = run(ae, inp.K, inp.V, inp.noise, wl.n_steps)
    perm = np.random.default_rng(0).permutation(wl.prefix)
    b = run(ae, inp.K[:, :, perm], inp.V[:, :, perm], inp.noise, wl.n_steps)
    assert np.abs(a - b).max() <= 1e-5


def test_tiny_graph_replay_matches_eager_bitwise(tiny):
    wl, inp, ae = tiny
    os.environ.pop("JPI_EAGER", None)
    g1 = run(ae, inp.K, inp.V, inp.noise, wl.n_steps)
    g2 = run(ae, inp.K, inp.V, inp.noise, wl.n_steps)
    os.environ["JPI_EAGER"] = "1"
    try:
        e = run(ae, inp.K, inp.V, inp.noise, wl.n_steps)
    finally:
        os.environ.pop("JPI_EAGER", None)
    assert np.array_equal(g1, g2) and np.array_equal(g1, e)


def test_tiny_constant_velocity_field():
    wl = synth.WORKLOADS["tiny-fp32"]
    inp = Inputs(wl)
    w = dict(inp.weights)
    w["action_out.w"] = np.zeros_like(w["action_out.w"])
    c = np.linspace(-1, 1, wl.dims.action_dim).astype(np.float32)
    w["action_out.b"] = c
    ae = make_expert(wl, w)
    try:
        got = run(ae, inp.K, inp.V, inp.noise, 5)
    finally:
        ae.close()
    np.testing.assert_allclose(got, inp.noise - c.astype(np.float64), atol=2e-6, rtol=0)


# ---------------------------------------------------------------------------
# pi0.5-shape workloads against stored oracle outputs
# ---------------------------------------------------------------------------
@pytest.fixture(scope="module")
def pi05():
    torch_cuda()
    wl = synth.WORKLOADS["pi05-b8"]
    print("generating pi0.5 weights", flush=True)
    w = synth.make_weights(wl)
    ae = make_expert(wl, w, max_batch=8, max_prefix=816)
    yield w, ae
    ae.close()


def _check_bf16(name, got, label=None):
    ref, meta = load_golden(name)
    assert_bf16(got, ref, label or name, reg_rel=REG_REL, reg_abs=REG_ABS)
    return ref


def test_pi05_b1(pi05):
    w, ae = pi05
    wl = synth.WORKLOADS["pi05-b1"]
    print("case pi05-b1", flush=True)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    got = run(ae, K, V, noise, wl.n_steps)
    _check_bf16("pi05-b1", got)
    # replay determinism
    assert np.array_equal(got, run(ae, K, V, noise, wl.n_steps))


@pytest.mark.parametrize("path", [None, "0"], ids=["single-launch", "multi-kernel"])
def test_pi05_b1_amplified_gates(path):
    """The pi0.5 shape with every layer's modulation tensors x 8 (gates near
    0.5): each sublayer, attention included, now moves the actions by far more
    than the bf16 bar.  The oracle's own output with the prefix V negated
    differs from the stored output by the recorded amount (0.18, nine times
    the bar); the GPU output with the negated V must differ from the stored
    output by about as much."""
    torch_cuda()
    ref, meta = load_golden("pi05-b1-amp8")
    wl = synth.WORKLOADS["pi05-b1"].with_(mod_gain=8.0, name="pi05-b1-amp8")
    print("case pi05-b1-amp8 path %s" % ("default" if path is None else "multi-kernel"), flush=True)
    inp = Inputs(wl)
    ae = make_expert(wl, inp.weights)
    try:
        got = run_env(ae, path, inp.K, inp.V, inp.noise, wl.n_steps)
        flipped = run_env(ae, path, inp.K, inp.V ^ np.uint16(0x8000), inp.noise, wl.n_steps)
    finally:
        ae.close()
    rel, _ = assert_bf16(got, ref, "pi05-b1-amp8", reg_rel=REG_REL * 2, reg_abs=REG_ABS * 4)
    moved = rel_l2_per_rollout(flipped, ref)
    print("pi05-b1-amp8: negating the prefix V moves the actions by %.3e (oracle %.3e), bar %.0e"
          % (moved, meta["prefix_v_negated_rel_l2"], BF16_TOL), flush=True)
    assert meta["prefix_v_negated_rel_l2"] > 5 * BF16_TOL
    assert moved > 5 * BF16_TOL and moved > 0.5 * meta["prefix_v_negated_rel_l2"]


def test_pi05_b1_committed10(pi05):
    w, ae = pi05
    wl = synth.WORKLOADS["pi05-b1-committed10"]
    print("case pi05-b1-committed10", flush=True)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    com = synth.make_committed(wl)
    got = run(ae, K, V, noise, wl.n_steps, committed=com, n_fixed=wl.n_fixed)
    _check_bf16("pi05-b1-committed10", got)
    assert np.array_equal(got[:, :10].astype(np.float32), com)


def test_pi05_b8_and_rollout_independence(pi05):
    w, ae = pi05
    wl = synth.WORKLOADS["pi05-b8"]
    print("case pi05-b8", flush=True)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    got = run(ae, K, V, noise, wl.n_steps)
    _check_bf16("pi05-b8", got)
    ref1, _ = load_golden("pi05-b1")
    # rollout 0 of the batch-8 workload is the batch-1 workload (shared seeds)
    assert_bf16(got[:1], ref1, "pi05-b8 rollout 0 vs pi05-b1", reg_rel=REG_REL, reg_abs=REG_ABS)


def test_pi05_ragged_prefix(pi05):
    w, ae = pi05
    ref, meta = load_golden("pi05-b2-ragged")
    wl = synth.WORKLOADS["pi05-b8"].with_(batch=2, prefix_len=tuple(meta["prefix_len"]))
    print("case pi05-b2-ragged", flush=True)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    got = run(ae, K, V, noise, wl.n_steps, prefix_len=meta["prefix_len"])
    _check_bf16("pi05-b2-ragged", got)


def test_pi05_b64_p1600_all_rollouts():
    torch_cuda()
    ref, meta = load_golden("pi05-b64-p1600")
    wl = synth.WORKLOADS["pi05-b64-p1600"]
    assert meta["rollouts"] == list(range(wl.batch))
    print("case pi05-b64-p1600 (all %d rollouts)" % wl.batch, flush=True)
    w = synth.make_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    ae = make_expert(wl, w)
    try:
        got = run(ae, K, V, noise, wl.n_steps)
    finally:
        ae.close()
    _check_bf16("pi05-b64-p1600", got)


def test_pi05_fp32_shape_at_1e4():
    torch_cuda()
    ref, meta = load_golden("pi05-f32-b1")
    wl = synth.WORKLOADS["pi05-b1"].with_(dtype="f32", name="pi05-f32-b1")
    print("case pi05-f32-b1", flush=True)
    inp = Inputs(wl)
    ae = make_expert(wl, inp.weights)
    try:
        got = run(ae, inp.K, inp.V, inp.noise, wl.n_steps)
    finally:
        ae.close()
    err = np.abs(got - ref).max()
    print("pi05-f32-b1 max-abs %.3e" % err, flush=True)
    assert err <= F32_TOL


# ---------------------------------------------------------------------------
# single-launch (persistent) path: batch * horizon <= 64 with bf16 weights
# ---------------------------------------------------------------------------
def test_persistent_tiny_bf16_batched_ragged_committed():
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", batch=3, n_fixed=2, prefix_len=(64, 5, 41),
                                            name="tiny-bf16-b3")
    inp = Inputs(wl)
    ae = make_expert(wl, inp.weights)
    try:
        got = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, prefix_len=inp.prefix_len,
                       committed=inp.committed, n_fixed=2)
        multi = run_env(ae, "0", inp.K, inp.V, inp.noise, wl.n_steps, prefix_len=inp.prefix_len,
                         committed=inp.committed, n_fixed=2)
    finally:
        ae.close()
    ref = _oracle(wl, inp, committed=inp.committed, n_fixed=2)
    print("tiny-bf16-b3 persistent vs multi-kernel path %.3e" % rel_l2_per_rollout(got, multi))
    assert_bf16(got, ref, "tiny-bf16-b3 persistent", reg_rel=2e-3)
    assert_bf16(multi, ref, "tiny-bf16-b3 multi-kernel", reg_rel=2e-3)
    assert rel_l2_per_rollout(got, multi) <= 5e-3
    assert np.array_equal(got[:, :2].astype(np.float32), inp.committed.astype(np.float32))


def test_persistent_matches_multikernel_pi05(pi05):
    w, ae = pi05
    wl = synth.WORKLOADS["pi05-b1"]
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    a = run_env(ae, None, K, V, noise, 2)
    b = run_env(ae, "0", K, V, noise, 2)
    print("pi05 2-step: persistent vs multi-kernel rel-L2 %.3e" % rel_l2_per_rollout(a, b))
    assert rel_l2_per_rollout(a, b) <= 5e-3
    # graph replay determinism of the single-launch kernel
    assert np.array_equal(a, run_env(ae, None, K, V, noise, 2))


def test_persistent_repeated_calls_bitwise(pi05):
    """The single-launch kernel orders its phases with per-workgroup completion
    flags (each consumer waits only for its producers).  A missing dependency
    would show as run-to-run variation, so repeated calls on two alternating
    inputs must reproduce their first results bit for bit."""
    from paper_2607_12659_amd.expert import to_device
    torch = torch_cuda()
    w, ae = pi05
    wl = synth.WORKLOADS["pi05-b1"]
    K, V = synth.make_prefix(wl)
    n1 = synth.make_noise(wl)
    n2 = np.ascontiguousarray(-n1[:, ::-1])
    ref1 = run(ae, K, V, n1, wl.n_steps)
    ref2 = run(ae, K, V, n2, wl.n_steps)
    assert not np.array_equal(ref1, ref2)
    d1 = to_device(np.ascontiguousarray(n1, np.float32))
    d2 = to_device(np.ascontiguousarray(n2, np.float32))
    print("case pi05-b1 x 24 alternating calls", flush=True)
    for i in range(12):
        for d, ref in ((d1, ref1), (d2, ref2)):
            out = ae.denoise(d, wl.n_steps)
            ae.sync()
            torch.cuda.synchronize()
            assert np.array_equal(out.cpu().numpy().astype(np.float64), ref), "call %d differs" % i


def test_persistent_tiny_bf16_repeated_calls_bitwise():
    """Ragged batch of three with committed rows: many short calls in a row."""
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", batch=3, n_fixed=2, prefix_len=(64, 5, 41),
                                            name="tiny-bf16-b3")
    inp = Inputs(wl)
    ae = make_expert(wl, inp.weights)
    try:
        ref = run(ae, inp.K, inp.V, inp.noise, wl.n_steps, prefix_len=inp.prefix_len,
                  committed=inp.committed, n_fixed=2)
        from paper_2607_12659_amd.expert import to_device
        d = to_device(np.ascontiguousarray(inp.noise, np.float32))
        print("case tiny-bf16-b3 x 40 calls", flush=True)
        for i in range(40):
            out = ae.denoise(d, wl.n_steps)
            ae.sync()
            torch.cuda.synchronize()
            assert np.array_equal(out.cpu().numpy().astype(np.float64), ref), "call %d differs" % i
    finally:
        ae.close()


def test_persistent_wait_timeout_is_reported_and_recovers():
    """Failure path of the single-launch kernel, forced from the host: with a
    bound of one poll its waits give up at once (the producers cannot have
    finished), the launch still ends, jpi_sync reports the timeout, and with
    the default bound restored the next call is exact again."""
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import to_device
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype="bf16", batch=3, n_fixed=2, prefix_len=(64, 5, 41),
                                            name="tiny-bf16-b3")
    inp = Inputs(wl)
    ae = make_expert(wl, inp.weights)
    try:
        ref = run(ae, inp.K, inp.V, inp.noise, wl.n_steps, prefix_len=inp.prefix_len,
                  committed=inp.committed, n_fixed=2)
        d = to_device(np.ascontiguousarray(inp.noise, np.float32))
        print("case tiny-bf16-b3 with a one-poll wait bound", flush=True)
        assert jpi.jpi_debug_set_spin_limit(ae.ctx, 1) == jpi.JPI_OK
        ae.denoise(d, wl.n_steps)
        with pytest.raises(jpi.JpiError, match="timed out"):
            ae.sync()
        torch.cuda.synchronize()
        assert jpi.jpi_debug_set_spin_limit(ae.ctx, 0) == jpi.JPI_OK
        out = ae.denoise(d, wl.n_steps)
        ae.sync()
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().astype(np.float64), ref)
    finally:
        ae.close()
