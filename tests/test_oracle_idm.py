"""Pins of the oracle's independent execution of the video and action
branches (Sec. 3.3; the Fast-WAM-IDM profiles of the appendix)."""
from collections import deque

import numpy as np
import pytest

from oracle import dit, method as M
from synth import get_pair, make_weights, make_initial_noise, make_observations, make_remap_noise
from conftest import load_golden


def _rr(spec, **kw):
    q, s, e = spec.rr_bounds
    return M.RRProfile(q, s, e, mode=kw.pop("mode", M.RR_AUTO), **kw)


# ---------------------------------------------------------------- RR branches
@pytest.mark.parametrize("cv,ca", [(1.1, 1.2), (1.05, 0.7), (1.2, -0.5)])
def test_single_branch_stats_closed_form(cv, ca):
    """p_i = cv p_a on the video/observation rows and ca p_a on the action rows:
    joint execution gives each branch its own closed form; a single branch
    pools the sums, alpha = (cv |pV|^2 + ca |pA|^2) / (|pV|^2 + |pA|^2) and
    cos = (cv |pV|^2 + ca |pA|^2) / (sqrt(cv^2 |pV|^2 + ca^2 |pA|^2) sqrt(|pV|^2 + |pA|^2))."""
    spec = get_pair("tiny_idm")[0].replace(Na=16, A=7)  # both branches present
    rng = np.random.default_rng(5)
    p_a = rng.standard_normal((spec.T, spec.D))
    rv, ra = M.branch_rows(spec)
    p_i = p_a.copy()
    p_i[rv] *= cv
    p_i[ra] *= ca
    prof = _rr(spec, alpha_min=-10.0, alpha_max=10.0)  # unclamped, to see the pooled value
    nv, na = np.sum(p_a[rv] ** 2), np.sum(p_a[ra] ** 2)
    # joint: per-branch closed forms
    for r, c in ((rv, cv), (ra, ca)):
        al, co, fi, _ = M.rr_branch_stats(p_i[r], p_a[r], prof)
        assert al == pytest.approx(c, rel=1e-12) and co == pytest.approx(np.sign(c), rel=1e-12)
        assert fi == pytest.approx(0.0, abs=1e-12)
    # single: pooled closed forms over all rows
    (rows,) = M.branch_rows(spec, single=True)
    assert len(rows) == spec.T
    al, co, fi, _ = M.rr_branch_stats(p_i[rows], p_a[rows], prof)
    num = cv * nv + ca * na
    assert al == pytest.approx(num / (nv + na), rel=1e-12)
    assert co == pytest.approx(num / (np.sqrt(cv * cv * nv + ca * ca * na) * np.sqrt(nv + na)), rel=1e-12)
    resid = (cv - al) ** 2 * nv + (ca - al) ** 2 * na
    assert fi == pytest.approx(np.sqrt(resid / (cv * cv * nv + ca * ca * na)), rel=1e-10)


def test_single_branch_decides_on_all_rows():
    """Flip the retained action residual of a joint model: joint execution
    rejects (the action branch has cos = -1), a single branch accepts exactly
    when the pooled cosine (|V|^2 - |A|^2) / (|V|^2 + |A|^2) passes."""
    spec = get_pair("tiny_idm")[0].replace(Na=16, A=7)
    W = make_weights(spec)
    x = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    sig = M.flow_schedule(spec.K)
    rv, ra = M.branch_rows(spec)
    results = {}
    for single in (False, True):
        st = M.LayerState()
        M.velocity_rr(W, spec, x, cond, sig[1], _rr(spec, mode=M.RR_FORCE_FULL, single=single), st)
        st.p_a = st.p_a.copy()
        st.p_a[:, ra] *= -1.0
        _, info = M.velocity_rr(W, spec, x, cond, sig[1], _rr(spec, single=single), st)
        results[single] = info
    # the same x and sigma: p_i equals the unflipped p_a
    assert not results[False].accepted and results[False].cos[0, 1] == pytest.approx(-1.0, abs=1e-12)
    st = M.LayerState()
    M.velocity_rr(W, spec, x, cond, sig[1], _rr(spec, mode=M.RR_FORCE_FULL), st)
    nv, na = np.sum(st.p_a[0, rv] ** 2), np.sum(st.p_a[0, ra] ** 2)
    pooled = (nv - na) / (nv + na)
    assert results[True].cos[0, 0] == pytest.approx(pooled, rel=1e-10)
    assert np.isnan(results[True].cos[0, 1])
    assert results[True].accepted == (pooled >= 0.80 and results[True].fit[0, 0] <= 0.60)


# ---------------------------------------------------------------- pair
def test_pack_condition_brute_force():
    rng = np.random.default_rng(1)
    obs = rng.standard_normal((2, 3, 5))
    ctx = rng.standard_normal((2, 4, 2))
    out = M.pack_condition(obs, ctx, 6)
    for b in range(2):
        for t in range(7):
            for c in range(6):
                if t < 3:
                    want = obs[b, t, c] if c < 5 else 0.0
                else:
                    want = ctx[b, t - 3, c] if c < 2 else 0.0
                assert out[b, t, c] == want


def test_idm_profiles_match_schedule_table():
    """The small pair's profiles are Table app-schedules' Fast-WAM-IDM rows:
    video 10 / 2+4 / 6 (entry stage 4), action 10 / 5 / 5 (entry stage 5)."""
    video, action = get_pair("idm")
    rows = {r[1]: r for r in load_golden("denoising_steps.csv") if r[0] == "fastwam_idm"}
    for spec, traj in ((video, "video"), (action, "action")):
        _, _, first, a, b, refresh, b0 = rows[traj]
        assert spec.K == int(first) and spec.tr_b0 == int(b0)
        assert spec.or_k1 == int(a) and spec.K - spec.tr_b0 - spec.or_k1 == int(b)
        assert spec.K - spec.tr_b0 == int(refresh)
    assert video.tr_r == 5 and video.shift_video == 0  # stage 5 -> stage 4, no temporal shift
    assert action.tr_r == action.tr_b0 == 5 and action.shift_action == 10  # stage 5, ten positions


def _pair_runtime(name, K=None, tau=1e9):
    sv, sa = get_pair(name)
    rts = []
    for spec, or_on in ((sv, True), (sa, False)):
        k = K or spec.K
        prof = M.RuntimeProfile(b0=spec.tr_b0, r=spec.tr_r, k1=spec.or_k1, tau=tau,
                                kappa_max=spec.or_kappa_max, shift_action=spec.shift_action,
                                shift_video=spec.shift_video, or_enabled=or_on)
        rts.append(M.ReplanRuntime(make_weights(spec), spec, M.flow_schedule(k), _rr(spec, single=True), prof))
    return M.IdmPairRuntime(*rts)


def test_idm_pair_step_counts_and_condition():
    """Tiny pair with the small pair's schedules (K = 10): the video model runs
    10, then 2 + 4 on an accepted prefix and 2 + 6 on a rejected one; the action
    model runs 10, then 5 under the real observation; the action model's
    condition is the observation followed by the video model's new latent."""
    pair = _pair_runtime("tiny_idm", K=10)
    sv, sa = pair.video.spec, pair.action.spec
    pair.video.p.b0, pair.video.p.r, pair.video.p.k1 = 4, 5, 2
    pair.action.p.b0, pair.action.p.r = 5, 5
    obs = make_observations(sv, 3)
    nf = (make_initial_noise(sv), make_initial_noise(sa))
    xv, xa, iv, ia = pair.replan(obs[0], noise_first=nf)
    assert iv.steps == 10 and ia.steps == 10
    c = pair.action_condition(obs[0], xv)
    assert np.array_equal(c[:, :sv.No, :sv.Co], obs[0])
    assert np.array_equal(c[:, sv.No:, :sv.Cv], dit.split_trajectory(sv, xv)[0])
    assert not np.any(c[:, sv.No:, sv.Cv:]) and not np.any(c[:, :sv.No, sv.Co:])
    nr = (make_remap_noise(sv, 1), make_remap_noise(sa, 1))
    xv, xa, iv, ia = pair.replan(obs[1], obs[1], [obs[1]], [obs[1]], [1.0], [1.0], noise_remap=nr)
    assert iv.path == M.PATH_ACCEPT and iv.steps == 6
    assert ia.path == M.PATH_DIRECT and ia.steps == 5
    pair.video.p.tau = 0.0
    nr = (make_remap_noise(sv, 2), make_remap_noise(sa, 2))
    _, _, iv, ia = pair.replan(obs[2], obs[2], [obs[2]], [obs[2]], [1.0], [1.0], noise_remap=nr)
    assert iv.path == M.PATH_REJECT and iv.steps == 8 and ia.steps == 5
