"""The committed-rows-at-t=0 variant (jpi_set_committed_t0) against the fp64
oracle, on both denoise paths.  Same bars as the denoise parity."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import Inputs, assert_bf16, load_golden, make_expert, rel_l2_per_rollout, run_env, torch_cuda
from synth import correction as sc

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4


@pytest.mark.parametrize("dtype,n_corr", [("f32", 0), ("f32", 3), ("bf16", 0), ("bf16", 3)])
def test_tiny_committed_rows_at_t0(dtype, n_corr):
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype=dtype, batch=2, n_fixed=3, prefix_len=(64, 9),
                                            name="tiny-t0-%s" % dtype)
    inp = Inputs(wl)
    # a time MLP ten times stronger than the N(0, 0.02) default, so that the
    # flow time of the committed rows moves the result well above the error bars
    for k in ("time_mlp.0.w", "time_mlp.1.w"):
        a = inp.weights[k]
        inp.weights[k] = (synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(a) * np.float32(10)) if a.dtype == np.uint16
                          else (a * np.float32(10)).astype(np.float32))
    corr = sc.make_item(wl.seed, 2, n_corr, wl.dims.width) if n_corr else None
    print("case tiny %s committed rows at t=0, %d correction tokens" % (dtype, n_corr), flush=True)
    ae = make_expert(wl, inp.weights, max_corr=4)
    kw = dict(prefix_len=inp.prefix_len, committed=inp.committed, n_fixed=3, corr=corr)
    try:
        base = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, **kw)
        ae.set_committed_t0(True)
        got = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, **kw)
        multi = run_env(ae, "0", inp.K, inp.V, inp.noise, wl.n_steps, **kw)
        ae.set_committed_t0(False)
        back = run_env(ae, None, inp.K, inp.V, inp.noise, wl.n_steps, **kw)
    finally:
        ae.close()
    ex = oracle.Expert(wl.dims, inp.weights)
    ref = oracle.denoise(ex, inp.noise, inp.K, inp.V, inp.prefix_len, wl.n_steps, committed=inp.committed, n_fixed=3,
                         corr=corr, committed_t0=True)
    ref0 = oracle.denoise(ex, inp.noise, inp.K, inp.V, inp.prefix_len, wl.n_steps, committed=inp.committed,
                          n_fixed=3, corr=corr)
    err, rel = np.abs(got - ref).max(), rel_l2_per_rollout(got, ref)
    print("max-abs %.3e rel-L2 %.3e; multi-kernel vs oracle %.3e; the variant moves the actions by %.3e"
          % (err, rel, rel_l2_per_rollout(multi, ref), np.abs(ref - ref0).max()), flush=True)
    if dtype == "f32":
        assert err <= F32_TOL
    else:
        assert_bf16(got, ref, "single-launch")
        assert_bf16(multi, ref, "multi-kernel")
        assert rel_l2_per_rollout(got, multi) <= 5e-3
    assert np.abs(ref - ref0).max() > 20 * max(err, 1e-6)  # the variant is far outside the error
    assert np.array_equal(got[:, :3].astype(np.float32), inp.committed.astype(np.float32))
    assert np.array_equal(base, back)


def test_pi05_committed10_at_t0():
    """pi0.5, one rollout, 10 committed rows at t = 0, against the stored
    oracle output on the single-launch and the multi-kernel path.  (With the
    N(0, 0.02) time MLP the variant moves these actions by only ~6e-4, so the
    tiny tests carry the discrimination.)"""
    torch_cuda()
    wl = synth.WORKLOADS["pi05-b1-committed10"]
    print("case pi05-b1-committed10-t0", flush=True)
    w = synth.make_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    com = synth.make_committed(wl)
    ae = make_expert(wl, w, max_batch=1, max_prefix=816)
    try:
        ae.set_committed_t0(True)
        got = run_env(ae, None, K, V, noise, wl.n_steps, committed=com, n_fixed=10)
        multi = run_env(ae, "0", K, V, noise, wl.n_steps, committed=com, n_fixed=10)
        again = run_env(ae, None, K, V, noise, wl.n_steps, committed=com, n_fixed=10)
    finally:
        ae.close()
    ref, meta = load_golden("pi05-b1-committed10-t0")
    assert meta["committed_t0"] is True
    plain, _ = load_golden("pi05-b1-committed10")
    effect = rel_l2_per_rollout(plain, ref)
    for label, out in (("single-launch", got), ("multi-kernel", multi)):
        rel = rel_l2_per_rollout(out, ref)
        print("%s: rel-L2 %.3e max-abs %.3e; the variant moves the actions by %.3e"
              % (label, rel, np.abs(out - ref).max(), effect), flush=True)
        assert_bf16(out, ref, label, reg_rel=2e-3, reg_abs=1e-2)
        assert np.array_equal(out[:, :10].astype(np.float32), com)
    assert np.array_equal(got, again)


# ---------------------------------------------------------------------------
# the action-time (pi0-style) expert
# ---------------------------------------------------------------------------
from oracle import pi0 as opi0  # noqa: E402
from synth import pi0 as spi0  # noqa: E402


def _pi0_expert(wl, w, max_batch, max_prefix, state_dim=spi0.STATE_DIM):
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import ActionExpert
    ae = ActionExpert(wl.dims, wl.dtype, max_batch, max_prefix, variant=jpi.JPI_VARIANT_ACTION_TIME,
                      state_dim=state_dim)
    ae.load_weights(w)
    return ae


def _pi0_run(ae, K, V, noise, n_steps, lens, state, committed=None, n_fixed=0, persist=None):
    """persist: None (default path choice) or "0" (force the multi-kernel path)."""
    import os
    from paper_2607_12659_amd.expert import to_device
    torch = torch_cuda()
    old = os.environ.pop("JPI_PERSIST", None)
    if persist is not None:
        os.environ["JPI_PERSIST"] = persist
    try:
        return _pi0_run_now(ae, K, V, noise, n_steps, lens, state, committed, n_fixed, to_device, torch)
    finally:
        os.environ.pop("JPI_PERSIST", None)
        if old is not None:
            os.environ["JPI_PERSIST"] = old


def _pi0_run_now(ae, K, V, noise, n_steps, lens, state, committed, n_fixed, to_device, torch):
    ae.bind_prefix(to_device(K), to_device(V), lens)
    ae.bind_state(None if committed is None else to_device(np.ascontiguousarray(committed, np.float32)), n_fixed)
    ae.bind_robot_state(to_device(np.ascontiguousarray(state, np.float32)))
    out = ae.denoise(to_device(np.ascontiguousarray(noise, np.float32)), n_steps)
    ae.sync()
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_action_time_variant(dtype):
    torch_cuda()
    wl = synth.WORKLOADS["tiny-fp32"].with_(dtype=dtype, batch=2, n_fixed=2, prefix_len=(64, 9),
                                            name="tiny-pi0-%s" % dtype)
    print("case tiny action-time variant %s, prefix_len %s" % (dtype, wl.prefix_len), flush=True)
    w = spi0.make_pi0_weights(wl, std=0.1)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    com = synth.make_committed(wl)
    st = spi0.make_state(wl)
    lens = list(wl.prefix_len)
    ae = _pi0_expert(wl, w, 2, wl.prefix + 1)
    try:
        got = _pi0_run(ae, K, V, noise, wl.n_steps, lens, st, com, 2)
        again = _pi0_run(ae, K, V, noise, wl.n_steps, lens, st, com, 2)
        moved = _pi0_run(ae, K, V, noise, wl.n_steps, lens, st * 3.0, com, 2)
        multi = _pi0_run(ae, K, V, noise, wl.n_steps, lens, st, com, 2, persist="0")
    finally:
        ae.close()
    ref = opi0.denoise(wl.dims, w, noise, K, V, lens, wl.n_steps, st, committed=com, n_fixed=2)
    ref3 = opi0.denoise(wl.dims, w, noise, K, V, lens, wl.n_steps, st * 3.0, committed=com, n_fixed=2)
    err, rel = np.abs(got - ref).max(), rel_l2_per_rollout(got, ref)
    effect = np.abs(ref3 - ref).max()
    print("max-abs %.3e rel-L2 %.3e; tripling the state moves the actions by %.3e (GPU: %.3e)"
          % (err, rel, effect, np.abs(moved - got).max()), flush=True)
    if dtype == "f32":
        assert err <= F32_TOL
        assert np.abs(moved - ref3).max() <= F32_TOL
    else:
        # bf16 with 2 x 10 rows runs the single-launch kernel once per step
        assert_bf16(got, ref, "single-launch steps")
        assert_bf16(moved, ref3, "single-launch steps, state x 3")
        # with these N(0, 0.1) weights each path is ~6e-3 from the oracle in bf16, so the
        # two paths are held to the same bar against each other as against the oracle
        print("single-launch steps vs multi-kernel rel-L2 %.3e; multi-kernel vs oracle %.3e"
              % (rel_l2_per_rollout(got, multi), rel_l2_per_rollout(multi, ref)), flush=True)
        assert_bf16(multi, ref, "multi-kernel")
        assert rel_l2_per_rollout(got, multi) <= BF16_TOL
    assert effect > 20 * max(err, 1e-6)
    assert np.array_equal(got, again)
    assert np.array_equal(got[:, :2].astype(np.float32), com.astype(np.float32))


def test_action_time_variant_rejects_a_full_prefix_and_needs_the_state():
    torch = torch_cuda()
    from paper_2607_12659_amd import jpi
    from paper_2607_12659_amd.expert import to_device
    wl = synth.WORKLOADS["tiny-fp32"]
    w = spi0.make_pi0_weights(wl)
    K, V = synth.make_prefix(wl)
    ae = _pi0_expert(wl, w, 1, wl.prefix)
    try:
        # every prefix slot taken: no room for the state token
        assert jpi.jpi_bind_prefix(ae.ctx, to_device(K), to_device(V), None, 1, wl.prefix, None) == jpi.JPI_ERR_SHAPE
        assert jpi.jpi_bind_prefix(ae.ctx, to_device(K), to_device(V), [wl.prefix - 1], 1, wl.prefix, None) == jpi.JPI_OK
        noise = to_device(synth.make_noise(wl).astype(np.float32))
        assert jpi.jpi_denoise(ae.ctx, noise, 2, noise, None) == jpi.JPI_ERR_STATE   # no robot state yet
        assert jpi.jpi_set_weight(ae.ctx, "time_mlp.0.w", np.zeros(wl.dims.width ** 2, np.float32),
                                  wl.dims.width ** 2, jpi.JPI_F32, 0, None) == jpi.JPI_ERR_ARG
        torch.cuda.synchronize()
    finally:
        ae.close()


def test_pi0_shape_action_time_variant():
    """The pi0-style expert at the pi0.5 shape (18 layers, width 1024, 8 x 256,
    816-token prefix slots with 815 valid, 10 committed rows) against the
    stored oracle output."""
    torch_cuda()
    ref, meta = load_golden("pi0-b1")
    assert meta["variant"] == "action_time"
    wl = synth.WORKLOADS["pi05-b1-committed10"].with_(name="pi0-b1", prefix_len=(815,))
    print("case pi0-b1", flush=True)
    w = spi0.make_pi0_weights(wl)
    K, V = synth.make_prefix(wl)
    noise = synth.make_noise(wl)
    ae = _pi0_expert(wl, w, 1, 816)
    try:
        got = _pi0_run(ae, K, V, noise, wl.n_steps, [815], spi0.make_state(wl), synth.make_committed(wl), 10)
        multi = _pi0_run(ae, K, V, noise, wl.n_steps, [815], spi0.make_state(wl), synth.make_committed(wl), 10,
                         persist="0")
    finally:
        ae.close()
    for label, out in (("single-launch steps", got), ("multi-kernel", multi)):
        rel = rel_l2_per_rollout(out, ref)
        print("%s: rel-L2 %.3e max-abs %.3e" % (label, rel, np.abs(out - ref).max()), flush=True)
        assert_bf16(out, ref, label, reg_rel=1e-2, reg_abs=5e-2)
