"""GPU parity of the replan paths through the separate adaptation calls.

  * Observation Rebinding composed from the single operations (Sec. 3.2):
    remap, prefix under the predicted condition, score, REBIND, continuation
    under the bound real condition, equals wam_replan's accept path bit for
    bit; calls that would interleave with an open replan are refused.
  * Replans with Trajectory Remapping switched off (fresh noise at sigma_0,
    the "w/o TR" variant of the ablation) against the oracle, teacher-forced.
  * Residual Rescaling's accepted path at the small bf16 model's full shape
    (Sec. 3.3, Eq. residual-injection): the change that injection makes to
    the velocity (reuse minus full computation on the same input) against the
    oracle's under the same forced decision, and alpha per branch.
  * The host-decision, device-decision and graph-replay ways of running a
    replan give the same bits at the small bf16 model's shape.
"""
from collections import deque

import numpy as np
import pytest

from oracle import dit as OD, method as OM
from synth import make_initial_noise, make_observations, make_remap_noise
from gpu_common import device, to_dev, rel_err, rr_of, f32_sigmas, model_for

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
BF16_TOL = 2e-2


@pytest.fixture(scope="module")
def dev():
    return device()


def _tiny_replay(dev):
    spec, W, m = model_for("tiny_replay", dev, bias_std=0.02, gain_std=0.1)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    return spec, W, m, sig


def _first_replan(m, spec, obs, dev, rr):
    x_out = m.new_traj()
    m.reset_all()
    m.replan(to_dev(obs[0], dev), x_out, to_dev(make_remap_noise(spec, 0), dev), cond_pred=to_dev(obs[0], dev),
             u_hat=[to_dev(obs[0], dev)], u=[to_dev(obs[0], dev)], delta=[1.0], weight=[1.0],
             noise_first=to_dev(make_initial_noise(spec), dev), rr=rr, b0=spec.tr_b0, r=spec.tr_r,
             shift_action=spec.shift_action, k1=spec.or_k1, tau=spec.or_tau, kappa_max=spec.or_kappa_max)
    return x_out


def test_rebind_composition_equals_replan_accept_path(dev):
    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd.runtime import WamError
    spec, W, m, sig = _tiny_replay(dev)
    m.set_option(L.WAM_OPT_GRAPHS, 0)
    m.set_option(L.WAM_OPT_DEVICE_DECISION, 0)
    rr_g, _ = rr_of(spec, L.WAM_RR_AUTO, gamma_cos=0.0, gamma_fit=1.5)
    rho = spec.ar_rho
    delta = 1.0 / np.sqrt(1 - rho * rho)
    obs = make_observations(spec, 1)
    cr, cp = to_dev(obs[1], dev), to_dev((rho * obs[0]).astype(np.float32), dev)
    b0, r, k1, K = spec.tr_b0, spec.tr_r, spec.or_k1, spec.K
    # wam_replan, accept path
    x_ref = _first_replan(m, spec, obs, dev, rr_g)
    info = m.replan(cr, x_ref, to_dev(make_remap_noise(spec, 1), dev), cond_pred=cp, u_hat=[cp], u=[cr],
                    delta=[delta], weight=[1.0], rr=rr_g, b0=b0, r=r, shift_action=spec.shift_action, k1=k1,
                    tau=spec.or_tau, kappa_max=spec.or_kappa_max)
    assert info.path == L.WAM_PATH_ACCEPT
    # the same from the single operations
    _first_replan(m, spec, obs, dev, rr_g)
    xb, xr, _ = m.get_replan_state()
    x = m.remap(xb, xr, float(sig[r]), float(sig[b0]), spec.shift_action, 0, to_dev(make_remap_noise(spec, 1), dev))
    m.reset_layer_state()
    cap = m.new_traj()
    m.continue_(b0, b0 + k1, x, cp, rr=rr_g, capture_stage=r, x_capture=cap)
    S = m.consistency_score([cp], [cr], [delta], [1.0])
    assert S == pytest.approx(info.S, rel=1e-12) and S < spec.or_tau
    m.rebind(cr)
    m.continue_(b0 + k1, K, x, None, rr=rr_g)  # None: the bound (real) condition
    np.testing.assert_array_equal(x.cpu().numpy(), x_ref.cpu().numpy())
    # after reset nothing is bound: a null condition is an error again
    m.reset_all()
    with pytest.raises(WamError, match="no bound condition"):
        m.continue_(0, 1, x, None)
    with pytest.raises(WamError, match="null rebind condition"):
        m.rebind(None)


def test_open_replan_refuses_state_calls(dev):
    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd.runtime import WamError
    spec, W, m, sig = _tiny_replay(dev)
    m.set_option(L.WAM_OPT_GRAPHS, 0)
    m.set_option(L.WAM_OPT_DEVICE_DECISION, 1)
    obs = make_observations(spec, 1)
    rr_g, _ = rr_of(spec, L.WAM_RR_AUTO)
    _first_replan(m, spec, obs, dev, rr_g)
    c = to_dev(obs[1], dev)
    x_out = m.new_traj()
    a = m.replan_args(c, x_out, to_dev(make_remap_noise(spec, 1), dev), cond_pred=c, u_hat=[c], u=[c],
                      delta=[1.0], weight=[1.0], rr=rr_g, b0=spec.tr_b0, r=spec.tr_r,
                      shift_action=spec.shift_action, k1=spec.or_k1, tau=spec.or_tau,
                      kappa_max=spec.or_kappa_max)
    m.replan_begin(a)
    x = to_dev(make_initial_noise(spec), dev)
    for call in (lambda: m.velocity(0, x, c), lambda: m.continue_(0, 1, x, c), lambda: m.hidden(0, x, c, 1),
                 lambda: m.get_replan_state(), lambda: m.set_schedule(sig), lambda: m.rebind(c),
                 lambda: m.set_option(L.WAM_OPT_ATTENTION, 0), lambda: m.reset_layer_state()):
        with pytest.raises(WamError, match="replan is open"):
            call()
    info = m.replan_end(a)  # the open replan is intact
    assert info.path == L.WAM_PATH_ACCEPT
    m.set_option(L.WAM_OPT_DEVICE_DECISION, 0)


def test_replans_without_remapping_match_oracle(dev):
    """The w/o TR variant: every later replan starts from fresh noise at
    sigma_0 (K steps, the prefix under the predicted condition first),
    teacher-forced against the oracle per replan."""
    from paper_2609_34608_amd import _lib as L
    spec, W, m, sig = _tiny_replay(dev)
    m.set_option(L.WAM_OPT_GRAPHS, 0)
    m.set_option(L.WAM_OPT_DEVICE_DECISION, 0)
    rr_g, rr_o = rr_of(spec, L.WAM_RR_AUTO)
    ra = dict(b0=spec.tr_b0, r=spec.tr_r, shift_action=spec.shift_action, k1=spec.or_k1, tau=spec.or_tau,
              kappa_max=spec.or_kappa_max)
    rho = spec.ar_rho
    delta = 1.0 / np.sqrt(1 - rho * rho)
    obs = make_observations(spec, 4)
    m.reset_all()
    rt = OM.ReplanRuntime(W, spec, sig, rr_o, OM.RuntimeProfile(tr_enabled=False, **ra))
    x_out = m.new_traj()
    for t in range(5):
        c_real = obs[t]
        c_pred = (rho * obs[t - 1]).astype(np.float32) if t > 0 else obs[t]
        if t > 0:
            xb, xr, kappa = m.get_replan_state()
            rt.set_state(xb.cpu().numpy(), xr.cpu().numpy(), kappa)
        cr, cp = to_dev(c_real, dev), to_dev(c_pred, dev)
        info = m.replan(cr, x_out, to_dev(make_remap_noise(spec, t), dev), cond_pred=cp, u_hat=[cp], u=[cr],
                        delta=[delta], weight=[1.0], noise_first=to_dev(make_initial_noise(spec), dev), rr=rr_g,
                        tr_enabled=False, **ra)
        trace = deque(int(d) for d in info.decision[:info.steps] if d >= 0)
        ref, rinfo = rt.replan(c_real, c_pred, [c_pred], [c_real], [delta], [1.0],
                               noise_first=make_initial_noise(spec), noise_remap=make_remap_noise(spec, t),
                               forced=trace)
        assert (info.path, info.steps, info.kappa) == (rinfo.path, rinfo.steps, rinfo.kappa), t
        if t > 0 and info.path != L.WAM_PATH_FORCED:
            assert info.steps == spec.K  # prefix + continuation from sigma_0
        assert rel_err(x_out.cpu().numpy(), ref) <= FP32_TOL, t


def test_small_bf16_injection_matches_oracle(dev):
    """Residual injection at the small model's full shape (bf16, T = 864,
    boundaries (2, 4, 10)): the layer state is established at step 0 on
    both sides; at step 1 (the device's own latent as input) the velocity
    with reuse forced minus the velocity with the middle computed is compared
    with the oracle's, and alpha per branch likewise.  Dropping the retained
    residual or taking alpha = 1 moves that difference by far more than the
    tolerance (tests/test_oracle_sensitivity.py)."""
    from paper_2609_34608_amd import _lib as L
    spec, W, m = model_for("small", dev)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    skip_g, skip_o = rr_of(spec, L.WAM_RR_FORCE_SKIP)
    full_g, _ = rr_of(spec, L.WAM_RR_FORCE_FULL)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    cd = to_dev(cond, dev)
    m.reset_layer_state()
    x = to_dev(x0, dev)
    m.denoise_step(0, x, cd, rr=skip_g)  # no state yet: full compute, establishes (p_a, R_a)
    x1 = x.cpu().numpy()
    v_skip, info = m.velocity(1, x, cd, rr=skip_g)
    assert info.attempted and info.accepted
    v_full, _ = m.velocity(1, x, cd, rr=full_g)
    state = OM.LayerState()
    OM.velocity_rr(W, spec, x0, cond, sig[0], skip_o, state)
    vs_ref, rinfo = OM.velocity_rr(W, spec, x1, cond, sig[1], skip_o, state)
    vf_ref = OD.velocity(W, spec, x1, cond, sig[1])
    e = rel_err(v_skip.cpu().numpy() - v_full.cpu().numpy(), vs_ref - vf_ref)
    ea = float(np.max(np.abs(info.alpha - rinfo.alpha) / np.abs(rinfo.alpha)))
    print(f"small bf16 injection: velocity change rel err {e:.3e}, alpha rel err {ea:.3e}, "
          f"alpha {info.alpha.ravel()}, cos {info.cos.ravel()}")
    assert e <= BF16_TOL, e
    assert ea <= 1e-2, ea


@pytest.mark.parametrize("name", ["tiny_rr", "small"])
def test_free_running_decision_agreement(dev, name):
    """Decision-trace protocol, part (i): the oracle runs free (its own gate,
    its own trajectory) beside the device over a whole chunk with Residual
    Rescaling on, thresholds placed inside the range of the statistics so
    that both decisions occur.  Reported: the agreement rate of the reuse
    decisions and the margin of every flip (the oracle's distance of cos or
    fit from its threshold); a flip is only allowed at a near-tie (margin
    within 1e-2, the bf16 error of the statistics is about 1e-3)."""
    from paper_2609_34608_amd import _lib as L
    kw = dict(bias_std=0.02, gain_std=0.1) if name == "tiny_rr" else {}
    spec, W, m = model_for(name, dev, **kw)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    # statistics of a pass that refreshes at every step (the gate never
    # passes) set the thresholds: cos at its median, fit never binding
    _, never_o = rr_of(spec, L.WAM_RR_AUTO, gamma_cos=1.5)
    _, _, infos = OM.denoise(W, spec, x0, cond, sig, 0, spec.K, never_o, OM.LayerState())
    cos_all = np.concatenate([i.cos.ravel() for i in infos if i.attempted])
    fit_all = np.concatenate([i.fit.ravel() for i in infos if i.attempted])
    g_cos = float(np.float32(np.median(cos_all)))
    g_fit = float(np.float32(np.max(fit_all) * 1.01))
    rr_g, rr_o = rr_of(spec, L.WAM_RR_AUTO, gamma_cos=g_cos, gamma_fit=g_fit)
    m.reset_layer_state()
    x = to_dev(x0, dev)
    got = m.continue_(0, spec.K, x, to_dev(cond, dev), rr=rr_g)
    _, _, ref = OM.denoise(W, spec, x0, cond, sig, 0, spec.K, rr_o, OM.LayerState())
    n_att, agree, flips = 0, 0, []
    for k, (g, r) in enumerate(zip(got, ref)):
        if not (g.attempted and r.attempted):
            assert g.attempted == r.attempted, k
            continue
        n_att += 1
        if g.accepted == r.accepted:
            agree += 1
        else:
            margin = float(min(np.min(np.abs(r.cos - g_cos)), np.min(np.abs(r.fit - g_fit))))
            flips.append((k, margin))
    rate = agree / max(n_att, 1)
    print(f"{name}: free-running decision agreement {agree}/{n_att} = {rate:.3f}; gamma_cos {g_cos:.4f}; "
          f"flips (step, margin): {flips}; device decisions {[int(g.accepted) for g in got if g.attempted]}, "
          f"oracle {[int(r.accepted) for r in ref if r.attempted]}")
    assert n_att >= 3
    for k, margin in flips:
        assert margin <= 1e-2, (k, margin)


@pytest.mark.parametrize("rr_mode", ["AUTO", "FORCE_SKIP"])
def test_exec_modes_agree_at_small_bf16(dev, rr_mode):
    """The three ways of running a replan at the small bf16 model's shape
    (closed-loop replay: TR + OR + RR, action shift 8) give the same bits:
    host decision (the gate read back per step), device decision (a flag
    kernel predicates the inject or middle / refresh launches) and captured
    step graphs replayed with the device decision.  Five replans cover the
    first, accepted and forced-refresh paths; with reuse forced the predicated
    inject runs, with AUTO (every gate fails on these weights) the middle."""
    from paper_2609_34608_amd import _lib as L
    spec0 = model_for("replay", dev)[0]
    rr_g, _ = rr_of(spec0, getattr(L, f"WAM_RR_{rr_mode}"))
    ra = dict(b0=spec0.tr_b0, r=spec0.tr_r, shift_action=spec0.shift_action, shift_video=spec0.shift_video,
              k1=spec0.or_k1, tau=spec0.or_tau, kappa_max=spec0.or_kappa_max)
    rho = spec0.ar_rho
    delta = 1.0 / np.sqrt(1 - rho * rho)
    n_ctrl = 5
    obs = make_observations(spec0, n_ctrl)

    def run(own_stream, devdec, graphs):
        spec, W, m = model_for("replay", dev, own_stream=own_stream)
        m.set_schedule(f32_sigmas(spec.K))
        m.set_option(L.WAM_OPT_DEVICE_DECISION, devdec)
        m.set_option(L.WAM_OPT_GRAPHS, graphs)
        m.reset_all()
        x_out = m.new_traj()
        outs, paths, decisions = [], [], []
        try:
            for t in range(n_ctrl):
                cr = to_dev(obs[t], dev)
                cp = to_dev((rho * obs[t - 1]).astype(np.float32) if t > 0 else obs[t], dev)
                info = m.replan(cr, x_out, to_dev(make_remap_noise(spec, t), dev), cond_pred=cp, u_hat=[cp],
                                u=[cr], delta=[delta], weight=[1.0],
                                noise_first=to_dev(make_initial_noise(spec), dev), rr=rr_g, **ra)
                outs.append(x_out.cpu().numpy())
                paths.append(info.path)
                decisions.append(list(info.decision[:info.steps]))
        finally:
            m.set_option(L.WAM_OPT_GRAPHS, 0)
            m.set_option(L.WAM_OPT_DEVICE_DECISION, 0)
        return outs, paths, decisions

    host = run(False, 0, 0)
    devd = run(False, 1, 0)
    graph = run(True, 1, 1)
    assert host[1] == [L.WAM_PATH_FIRST, L.WAM_PATH_ACCEPT, L.WAM_PATH_ACCEPT, L.WAM_PATH_ACCEPT,
                       L.WAM_PATH_FORCED]
    if rr_mode == "FORCE_SKIP":
        assert any(d == 1 for ds in host[2] for d in ds)
    for other in (devd, graph):
        assert other[1] == host[1] and other[2] == host[2]
        for a, b in zip(host[0], other[0]):
            np.testing.assert_array_equal(a, b)
