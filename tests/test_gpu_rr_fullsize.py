"""Residual Rescaling at the mid (B = 4, T = 2306) and large (T = 10176)
shapes, and on a short sequence whose projections split K over blocks,
against the oracle, teacher-forced on the device's own hidden states.

Step 0 runs with the layer state empty: every layer is computed and the
state is established, p_a = h_s - h_q and R_a = h_e - h_s (Eq. crr-reference).
Step 1 takes the device's latent after step 0 with reuse forced.

* Gate (Eq. crr-alpha, crr-gate): the device's alpha, cos and relative fit
  per sample and branch against the oracle's formulas applied to the same
  float32 tensors, the device's h_q and h_s at both steps read back with
  wam_hidden (the same kernels in the same order as inside the Residual
  Rescaling step, so the same bits).  Both sides sum in float64, in
  different orders: 1e-9.
* Injection (Eq. residual-injection): the device's velocity with reuse forced
  minus its velocity with the middle computed, against the oracle's tail
  layers [e, L) and final layer run in float64 from h_s + alpha R_a and from
  the device's h_e at step 1; bf16 tolerance 2e-2 of the largest change.  At
  the mid shape the same oracle quantity with R_a dropped is checked to move
  by at least ten times that tolerance, so the check would catch a broken
  injection.
"""
import time

import numpy as np
import pytest

from oracle import dit as OD, method as OM
from synth import get_workload, make_initial_noise, make_observations, make_weights
from gpu_common import device, to_dev, rel_err, f32_sigmas, model_for, rr_of

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
STAT_TOL = 1e-9


@pytest.fixture(scope="module")
def dev():
    return device()


def _say(name, t0, what):
    print(f"[{name} {time.time() - t0:6.1f} s] {what}", flush=True)


def _model(name, dev):
    """The workload's cached model, or for "small_short" the small model on
    a 64-token sequence with two samples: its 128 rows make the attention
    output and MLP-down projections split K over blocks, so the head's h_q
    is stored by the split reduce pass rather than the tile epilogue."""
    if name != "small_short":
        return model_for(name, dev)
    from paper_2609_34608_amd import runtime as R
    spec = get_workload("small").replace(B=2, Nv=24, No=8)
    W = make_weights(spec)
    return spec, W, R.WamModel(R.config_of(spec), W, device=dev)


@pytest.mark.parametrize("name", ["small_short", "mid", "large"])
def test_full_size_rr_gate_and_injection(dev, name):
    from paper_2609_34608_amd import _lib as L
    t0 = time.time()
    spec, W, m = _model(name, dev)
    q, s, e = spec.rr_bounds
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    skip_g, skip_o = rr_of(spec, L.WAM_RR_FORCE_SKIP)
    full_g, _ = rr_of(spec, L.WAM_RR_FORCE_FULL)
    cd = to_dev(make_observations(spec, 0)[0], dev)
    x = to_dev(make_initial_noise(spec), dev)

    def hid(k, n):
        return m.hidden(k, x, cd, n).cpu().numpy()

    hq0, hs0, he0 = hid(0, q), hid(0, s), hid(0, e)
    m.reset_layer_state()
    m.denoise_step(0, x, cd, rr=skip_g)  # establishes (p_a, R_a); x becomes the step-1 latent
    hq1, hs1, he1 = hid(1, q), hid(1, s), hid(1, e)
    v_skip, info = m.velocity(1, x, cd, rr=skip_g)
    assert info.attempted and info.accepted
    v_full, _ = m.velocity(1, x, cd, rr=full_g)
    dv = v_skip.cpu().numpy().astype(np.float64) - v_full.cpu().numpy()
    _say(name, t0, "device done")

    # gate statistics on the device's float32 tensors
    p_a_all = hs0 - hq0  # float32, as the device forms it
    p_i_all = hs1 - hq1
    R_a = (he0 - hs0).astype(np.float64)
    alpha = np.zeros((spec.B, 2))
    worst = 0.0
    for b in range(spec.B):
        for j, rows in enumerate(OM.branch_rows(spec)):
            a, c, f, _ = OM.rr_branch_stats(p_i_all[b, rows], p_a_all[b, rows], skip_o)
            alpha[b, j] = a
            for got, ref in ((info.alpha[b, j], a), (info.cos[b, j], c), (info.fit[b, j], f)):
                worst = max(worst, abs(got - ref) / max(abs(ref), 1e-30))
    print(f"{name}: gate statistics max rel diff {worst:.2e}; alpha {info.alpha.ravel()}, "
          f"cos {info.cos.ravel()}, fit {info.fit.ravel()}")
    assert worst <= STAT_TOL, worst

    # injection: oracle tail from h_s + alpha R_a against the tail from h_e
    threads = OD.ATTENTION_THREADS
    OD.ATTENTION_THREADS = 8  # bit-identical to the serial head loop
    try:
        c1 = OD.cond_vector(W, sig[1])
        h_inj = hs1.astype(np.float64)
        for j, rows in enumerate(OM.branch_rows(spec)):
            h_inj[:, rows] += alpha[:, j][:, None, None] * R_a[:, rows]

        def tail(h):
            return OD.final_layer(W, spec, OD.run_layers(W, spec, h, c1, e, spec.L), c1)

        v_full_ref = tail(he1.astype(np.float64))
        _say(name, t0, "oracle tail from h_e done")
        ref = tail(h_inj) - v_full_ref
        _say(name, t0, "oracle tail from the injected state done")
        err = rel_err(dv, ref)
        print(f"{name}: injection velocity change rel err {err:.3e} (max |change| {np.max(np.abs(ref)):.3e})")
        assert err <= BF16_TOL, err
        if name == "mid":
            dropped = tail(hs1.astype(np.float64)) - v_full_ref
            moved = rel_err(dropped, ref)
            print(f"{name}: the same quantity with R_a dropped moves by {moved:.3e}")
            assert moved >= 10 * BF16_TOL, moved
    finally:
        OD.ATTENTION_THREADS = threads
        if name == "small_short":
            m.close()


@pytest.mark.parametrize("name", ["small", "mid", "large"])
def test_bf16_steps_with_rr_are_deterministic(dev, name):
    """Four denoising steps with Residual Rescaling forced on (the first
    establishes the layer state, the next three inject), run twice from the
    same state: the trajectory and every reported statistic are the same bits
    (the GEMM, attention and reduction kernels sum in fixed orders, with no
    atomics), which the decision-trace protocol relies on."""
    from paper_2609_34608_amd import _lib as L
    spec, W, m = model_for(name, dev)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    skip_g, _ = rr_of(spec, L.WAM_RR_FORCE_SKIP)
    cd = to_dev(make_observations(spec, 0)[0], dev)
    x0 = to_dev(make_initial_noise(spec), dev)
    runs = []
    for _ in range(2):
        m.reset_layer_state()
        x = x0.clone()
        infos = m.continue_(0, 4, x, cd, rr=skip_g)
        runs.append((x.cpu().numpy(), infos))
    np.testing.assert_array_equal(runs[0][0], runs[1][0])
    for a, b in zip(runs[0][1], runs[1][1]):
        assert (a.attempted, a.accepted) == (b.attempted, b.accepted)
        for f in ("alpha", "cos", "fit"):
            np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    assert sum(i.accepted for i in runs[0][1]) == 3
