"""GPU parity of the state-continuity diagnostics (Eq. app-layer-errors):
the per-layer relative hidden-state change Delta_l(i) and the output error
E_out(i) of residual reuse against full computation, along the native
trajectory of the fp32 tiny model with residual-rescaling bounds, computed
through the C ABI by the bench harness and by the float64 oracle.  Both are
ratios of norms of fp32 results: agreement to 1e-4 (Delta) and 1e-3 (E_out,
a difference of two nearly equal outputs) absolute."""
import numpy as np
import pytest

from oracle import dit as OD, method as OM, metrics as X
from synth import make_weights, make_initial_noise, make_observations
from gpu_common import device, to_dev, rr_of, f32_sigmas, model_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return device()


def test_layer_diagnostics_match_oracle(dev):
    import bench
    from paper_2609_34608_amd import _lib as L
    spec, W, m = model_for("tiny_rr", dev, bias_std=0.02, gain_std=0.1)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    rr_g, rr_o = rr_of(spec, L.WAM_RR_FORCE_SKIP)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    delta, e_out = bench.layer_diagnostics(m, spec, to_dev(x0, dev), to_dev(cond, dev), rr_g, spec.K)
    # oracle: the same quantities along its own native trajectory
    st = OM.LayerState()
    x = OD.as64(x0)
    d_ref, e_ref = [], []
    for i in range(spec.K):
        hs = [OD.hidden_after(W, spec, x, cond, sig[i], n) for n in range(spec.L + 1)]
        d_ref.append([X.layer_change(hs[l + 1], hs[l]) for l in range(spec.L)])
        v_full = OD.velocity(W, spec, x, cond, sig[i])
        v_reuse, _ = OM.velocity_rr(W, spec, x, cond, sig[i], rr_o, st)
        e_ref.append(X.output_error(v_reuse, v_full))
        x = OM.euler_update(x, v_full, sig[i], sig[i + 1])
    print("Delta_l mean over steps (GPU):", np.round(np.mean(delta, axis=0), 5))
    print("E_out (GPU):", np.round(e_out, 5), " (oracle):", np.round(e_ref, 5))
    np.testing.assert_allclose(delta, d_ref, atol=1e-4)
    np.testing.assert_allclose(e_out, e_ref, atol=1e-3)
    assert e_out[0] == pytest.approx(0.0, abs=1e-6)  # the first step only establishes the state
    assert all(v > 0 for v in e_out[1:])
