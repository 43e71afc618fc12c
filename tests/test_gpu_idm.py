"""GPU parity of independent execution of the video and action branches
(Sec. 3.3; Fast-WAM-IDM profiles of the appendix): single-branch Residual
Rescaling, models with only video or only action tokens, the action model's
condition, and teacher-forced closed-loop pair replans, through the C ABI
against the float64 oracle (fp32 <= 1e-4; bf16 action chunk <= 2e-2)."""
from collections import deque

import numpy as np
import pytest

from oracle import dit as OD, method as OM
from synth import get_pair, make_weights, make_initial_noise, make_observations, make_remap_noise
from gpu_common import device, to_dev, rel_err, rr_of, f32_sigmas

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
BF16_TOL = 2e-2


@pytest.fixture(scope="module")
def dev():
    return device()


def _model(spec, dev, own_stream=False, **wkw):
    from paper_2609_34608_amd import runtime as R
    W = make_weights(spec, **wkw)
    m = R.WamModel(R.config_of(spec), W, device=dev, own_stream=own_stream)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    return W, m, sig


@pytest.mark.parametrize("mode_name", ["AUTO", "FORCE_SKIP", "FORCE_FULL", "MIXED"])
@pytest.mark.parametrize("devdec", [0, 1])
def test_single_branch_rr_matches_oracle(dev, mode_name, devdec):
    """All rows pooled into one branch: per-step alpha / cos / fit of branch 0,
    NaN for branch 1, and the trajectory, on both decision paths."""
    from paper_2609_34608_amd import _lib as L
    spec = get_pair("tiny_idm")[0].replace(Na=16, A=7, B=2)  # both token kinds, pooled
    W, m, sig = _model(spec, dev, bias_std=0.02, gain_std=0.1)
    m.set_option(L.WAM_OPT_DEVICE_DECISION, devdec)
    modes = {"AUTO": (L.WAM_RR_AUTO, {}), "FORCE_SKIP": (L.WAM_RR_FORCE_SKIP, {}),
             "FORCE_FULL": (L.WAM_RR_FORCE_FULL, {}), "MIXED": (L.WAM_RR_AUTO, {"gamma_cos": 0.0, "gamma_fit": 1.02})}
    mode, kw = modes[mode_name]
    rr_g, rr_o = rr_of(spec, mode, single=True, **kw)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    x = to_dev(x0, dev)
    infos = m.continue_(0, spec.K, x, to_dev(cond, dev), rr=rr_g)
    trace = deque(i.accepted for i in infos if i.attempted)
    ref, _, oinfos = OM.denoise(W, spec, x0, cond, sig, 0, spec.K, rr_o, OM.LayerState(), forced=trace)
    assert rel_err(x.cpu().numpy(), ref) <= FP32_TOL
    attempted = 0
    for gi, oi in zip(infos, oinfos):
        assert (gi.attempted, gi.accepted, gi.layers_evaluated) == (oi.attempted, oi.accepted, oi.layers_evaluated)
        if gi.attempted:
            attempted += 1
            np.testing.assert_allclose(gi.alpha, oi.alpha, atol=1e-4)
            np.testing.assert_allclose(gi.cos, oi.cos, atol=1e-4)
            np.testing.assert_allclose(gi.fit, oi.fit, atol=1e-3)
            assert np.all(np.isnan(gi.cos[:, 1]))
    # FORCE_FULL computes every middle without running the gate
    assert attempted == (0 if mode_name == "FORCE_FULL" else spec.K - 1)
    m.close()


def test_video_only_model_matches_oracle(dev):
    """A model without action tokens (the video model of the pair) under
    single-branch RR: chunk and decisions."""
    from paper_2609_34608_amd import _lib as L
    spec = get_pair("tiny_idm")[0]
    W, m, sig = _model(spec, dev, bias_std=0.02, gain_std=0.1)
    rr_g, rr_o = rr_of(spec, L.WAM_RR_AUTO, single=True, gamma_cos=0.0, gamma_fit=1.02)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    x = to_dev(x0, dev)
    infos = m.continue_(0, spec.K, x, to_dev(cond, dev), rr=rr_g)
    trace = deque(i.accepted for i in infos if i.attempted)
    ref, _, _ = OM.denoise(W, spec, x0, cond, sig, 0, spec.K, rr_o, OM.LayerState(), forced=trace)
    assert x.shape[1] == spec.Nv * spec.Cv
    assert rel_err(x.cpu().numpy(), ref) <= FP32_TOL
    m.close()


def test_pack_condition_exact(dev):
    import torch
    from paper_2609_34608_amd import runtime as R
    sv, sa = get_pair("tiny_idm")
    sa = sa.replace(B=3)
    _, m, _ = _model(sa, dev)
    rng = np.random.default_rng(3)
    obs = rng.standard_normal((3, sv.No, sv.Co)).astype(np.float32)
    traj = rng.standard_normal((3, sv.Nv * sv.Cv + 5)).astype(np.float32)  # ctx rows with a larger stride
    out = torch.full((3, sa.No, sa.Co), 7.0, dtype=torch.float32, device=dev)
    m.pack_condition(to_dev(obs, dev), sv.No, sv.Co, to_dev(traj, dev), sv.Nv, sv.Cv, traj.shape[1], out)
    ctx = traj[:, :sv.Nv * sv.Cv].reshape(3, sv.Nv, sv.Cv)
    np.testing.assert_array_equal(out.cpu().numpy(), OM.pack_condition(obs, ctx, sa.Co).astype(np.float32))
    with pytest.raises(R.WamError):  # token counts must add up to No
        m.pack_condition(to_dev(obs, dev), sv.No, sv.Co, to_dev(traj, dev), sv.Nv - 1, sv.Cv, traj.shape[1], out)
    m.close()


def _ra(spec, or_enabled):
    return dict(b0=spec.tr_b0, r=spec.tr_r, shift_action=spec.shift_action, shift_video=spec.shift_video,
                k1=spec.or_k1, tau=spec.or_tau, kappa_max=spec.or_kappa_max, or_enabled=or_enabled)


@pytest.mark.parametrize("graphs", [False, True])
def test_idm_pair_closed_loop_matches_oracle(dev, graphs):
    """Teacher-forced per replan for each model: the oracle starts from the
    device's retained state and follows its RR trace; the action model's
    oracle replan runs under the condition the device packed from the device's
    video output (which is checked exactly against the oracle's packing)."""
    from paper_2609_34608_amd import runtime as R, _lib as L
    sv, sa = get_pair("tiny_idm")
    Wv, mv, sig = _model(sv, dev, own_stream=graphs, bias_std=0.02, gain_std=0.1)
    Wa, ma, _ = _model(sa, dev, own_stream=graphs, bias_std=0.02, gain_std=0.1)
    for m in (mv, ma):
        m.set_option(L.WAM_OPT_DEVICE_DECISION, int(graphs))
        m.set_option(L.WAM_OPT_GRAPHS, int(graphs))
    pair = R.IdmPair(mv, ma, sv.No, sv.Co)
    rr_gv, rr_ov = rr_of(sv, L.WAM_RR_AUTO, single=True)
    rr_ga, rr_oa = rr_of(sa, L.WAM_RR_AUTO, single=True)
    rav, raa = _ra(sv, True), _ra(sa, False)
    rtv = OM.ReplanRuntime(Wv, sv, sig, rr_ov, OM.RuntimeProfile(**rav))
    rta = OM.ReplanRuntime(Wa, sa, sig, rr_oa, OM.RuntimeProfile(**raa))
    rho = sv.ar_rho
    delta = 1.0 / np.sqrt(1 - rho * rho)
    obs = make_observations(sv, sv.control_steps)
    xv_g, xa_g = mv.new_traj(), ma.new_traj()
    paths = []
    for t in range(sv.control_steps):
        c_real = obs[t]
        c_pred = (rho * obs[t - 1]).astype(np.float32) if t > 0 else obs[t]
        if t > 0:
            for m, rt in ((mv, rtv), (ma, rta)):
                xb, xr, kappa = m.get_replan_state()
                rt.set_state(xb.cpu().numpy(), xr.cpu().numpy(), kappa)
        cr, cp = to_dev(c_real, dev), to_dev(c_pred, dev)
        iv, ia = pair.replan(
            cr, xv_g, xa_g, to_dev(make_remap_noise(sv, t), dev), to_dev(make_remap_noise(sa, t), dev),
            video_kw=dict(cond_pred=cp, u_hat=[cp], u=[cr], delta=[delta], weight=[1.0],
                          noise_first=to_dev(make_initial_noise(sv), dev), rr=rr_gv, **rav),
            action_kw=dict(noise_first=to_dev(make_initial_noise(sa), dev), rr=rr_ga, **raa))
        tv = deque(int(d) for d in iv.decision[:iv.steps] if d >= 0)
        ref_v, rinfo_v = rtv.replan(c_real, c_pred, [c_pred], [c_real], [delta], [1.0],
                                    noise_first=make_initial_noise(sv), noise_remap=make_remap_noise(sv, t),
                                    forced=tv)
        assert iv.path == rinfo_v.path and iv.steps == rinfo_v.steps, t
        assert rel_err(xv_g.cpu().numpy(), ref_v) <= FP32_TOL, t
        cond_a = OM.pack_condition(c_real, OD.split_trajectory(sv, xv_g.cpu().numpy())[0], sa.Co)
        np.testing.assert_array_equal(pair.cond_action.cpu().numpy(), cond_a.astype(np.float32))
        ta = deque(int(d) for d in ia.decision[:ia.steps] if d >= 0)
        ref_a, rinfo_a = rta.replan(cond_a, noise_first=make_initial_noise(sa),
                                    noise_remap=make_remap_noise(sa, t), forced=ta)
        assert ia.path == rinfo_a.path and ia.steps == rinfo_a.steps, t
        assert rel_err(xa_g.cpu().numpy(), ref_a) <= FP32_TOL, t
        paths.append((iv.path, ia.path))
    first = (L.WAM_PATH_FIRST, L.WAM_PATH_FIRST)
    assert paths[0] == first and all(p[1] == L.WAM_PATH_DIRECT for p in paths[1:])
    mv.close()
    ma.close()


def test_small_bf16_pair_first_replan(dev):
    """The small pair (bf16) on a 3-step schedule: video from noise, then the
    action model under the observation and the video latent; action chunk
    within 2e-2 of the float64 oracle run on the same packed condition."""
    from paper_2609_34608_amd import runtime as R, _lib as L
    sv, sa = get_pair("idm")
    sv = sv.replace(K=3, tr_b0=1, tr_r=1, or_k1=1)
    sa = sa.replace(K=3, tr_b0=1, tr_r=1)
    Wv, mv, sig = _model(sv, dev)
    Wa, ma, _ = _model(sa, dev)
    pair = R.IdmPair(mv, ma, sv.No, sv.Co)
    rr_gv, rr_ov = rr_of(sv, L.WAM_RR_FORCE_FULL, single=True)
    rr_ga, rr_oa = rr_of(sa, L.WAM_RR_FORCE_FULL, single=True)
    obs = make_observations(sv, 0)[0]
    xv_g, xa_g = mv.new_traj(), ma.new_traj()
    cr = to_dev(obs, dev)
    pair.replan(cr, xv_g, xa_g, to_dev(make_remap_noise(sv, 0), dev), to_dev(make_remap_noise(sa, 0), dev),
                video_kw=dict(cond_pred=cr, noise_first=to_dev(make_initial_noise(sv), dev), rr=rr_gv,
                              **_ra(sv, True)),
                action_kw=dict(noise_first=to_dev(make_initial_noise(sa), dev), rr=rr_ga, **_ra(sa, False)))
    ref_v, _, _ = OM.denoise(Wv, sv, make_initial_noise(sv), obs, sig, 0, sv.K, rr_ov, OM.LayerState())
    assert rel_err(xv_g.cpu().numpy(), ref_v) <= BF16_TOL
    cond_a = OM.pack_condition(obs, OD.split_trajectory(sv, xv_g.cpu().numpy())[0], sa.Co)
    ref_a, _, _ = OM.denoise(Wa, sa, make_initial_noise(sa), cond_a, sig, 0, sa.K, rr_oa, OM.LayerState())
    assert rel_err(OM.action_chunk(sa, xa_g.cpu().numpy()), OM.action_chunk(sa, ref_a)) <= BF16_TOL
    mv.close()
    ma.close()
