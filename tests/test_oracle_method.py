"""Pins of the oracle's solver and adaptation operators.

Each test ties the oracle to something other than itself: numbers the paper
prints (tests/golden, each with its table or section), closed forms of the
equations, invariants, and brute force on tiny inputs.
"""
from collections import deque

import numpy as np
import pytest

from oracle import dit, method as M
from synth import get_workload, make_weights, make_initial_noise, make_observations, make_remap_noise
from conftest import load_golden


# ---------------------------------------------------------------- schedule
def test_schedule_reproduces_printed_noise_levels():
    for name, K, shift, stage, printed, dec in load_golden("noise_levels.csv"):
        sig = M.flow_schedule(int(K), float(shift))
        assert round(sig[int(stage)], int(dec)) == pytest.approx(float(printed), abs=1e-12), name


def test_schedule_endpoints_and_monotone():
    for K in (1, 4, 10, 20):
        for S in (1.0, 3.0, 5.0):
            sig = M.flow_schedule(K, S)
            assert sig[0] == 1.0 and sig[-1] == 0.0
            assert np.all(np.diff(sig) < 0)


def test_step_counts_match_schedule_table():
    """accepted a+b = refresh = K - b0 for every row of Table app-schedules."""
    for model, traj, first, a, b, refresh, b0 in load_golden("denoising_steps.csv"):
        K = int(first)
        assert int(a) + int(b) == int(refresh) == K - int(b0), (model, traj)


def test_runtime_step_counts_follow_schedule_table():
    """The runtime performs k1 + (K-b0-k1) steps on an accepted prefix and
    K-b0 on a refresh, for each printed profile."""
    spec = get_workload("tiny")
    W = make_weights(spec)
    for model, traj, first, a, b, refresh, b0 in load_golden("denoising_steps.csv"):
        K, a, b0 = int(first), int(a), int(b0)
        if a == 0:
            continue  # no anticipatory prefix in this profile
        sig = M.flow_schedule(K)
        prof = M.RuntimeProfile(b0=b0, r=b0, k1=a, tau=1e9, kappa_max=3)
        rt = M.ReplanRuntime(W, spec, sig, None, prof)
        obs = make_observations(spec, 2)
        x0 = make_initial_noise(spec)
        _, i0 = rt.replan(obs[0], noise_first=x0)
        assert i0.steps == K
        _, i1 = rt.replan(obs[1], obs[1], [obs[1]], [obs[1]], [1.0], [1.0],
                          noise_remap=make_remap_noise(spec, 1))
        assert i1.path == M.PATH_ACCEPT and i1.steps == int(refresh)
        prof.tau = 0.0  # S = 0 is not < 0: reject, restart from the remapped init
        _, i2 = rt.replan(obs[2], obs[2], [obs[2]], [obs[2]], [1.0], [1.0],
                          noise_remap=make_remap_noise(spec, 2))
        assert i2.path == M.PATH_REJECT and i2.steps == a + int(refresh)


# ---------------------------------------------------------------- RR
def test_layer_counts_match_layer_table():
    for name, L, q, s, e, evaluated in load_golden("rr_layers.csv"):
        p = M.RRProfile(int(q), int(s), int(e))
        p.validate(int(L))
        assert p.evaluated_after_reuse(int(L)) == int(evaluated), name


def _thr(model):
    for m, gc, gf, amin, amax, eps in load_golden("rr_thresholds.csv"):
        if m == model:
            return float(gc), float(gf), float(amin), float(amax), float(eps)
    raise KeyError(model)


@pytest.mark.parametrize("c,alpha,fit", [(1.1, 1.1, 0.0), (0.9, 1.0, 0.1 / 0.9),
                                         (0.8, 1.0, 0.25), (2.0, 1.25, 0.375), (1.0, 1.0, 0.0)])
def test_rr_closed_form_scaled_probe(c, alpha, fit):
    """p_i = c p_a: alpha = clamp(c), cos = 1, fit = |c - alpha| / |c|."""
    rng = np.random.default_rng(0)
    p_a = rng.standard_normal(500)
    p_i = c * p_a
    gc, gf, amin, amax, eps = _thr("fastwam_idm")
    a = M.rr_alpha(p_i, p_a, eps, amin, amax)
    assert a == pytest.approx(alpha, abs=1e-12)
    assert M.rr_cos(p_i, p_a) == pytest.approx(1.0, abs=1e-12)
    assert M.rr_fit(p_i, p_a, a) == pytest.approx(fit, abs=1e-12)


def test_rr_gate_against_printed_thresholds():
    rng = np.random.default_rng(1)
    p_a = rng.standard_normal(300)
    cases = {  # c -> {model: pass?}
        0.8: {"cosmos_policy": False, "fastwam_idm": True},
        2.0: {"motus": True, "cosmos_policy": False},
        1.1: {"cosmos_policy": True, "fastwam_idm": True, "motus": True},
        -1.0: {"cosmos_policy": False, "fastwam_idm": False, "motus": False},
    }
    for c, exp in cases.items():
        p_i = c * p_a
        for model, want in exp.items():
            gc, gf, amin, amax, eps = _thr(model)
            a = M.rr_alpha(p_i, p_a, eps, amin, amax)
            got = M.rr_gate(M.rr_cos(p_i, p_a), M.rr_fit(p_i, p_a, a), gc, gf)
            assert got == want, (c, model)


def test_rr_orthogonal_and_degenerate():
    p_a = np.array([1.0, 0.0, 0.0, 0.0])
    p_i = np.array([0.0, 2.0, 0.0, 0.0])
    assert M.rr_cos(p_i, p_a) == 0.0
    a = M.rr_alpha(p_i, p_a, 1e-8, 1.0, 1.25)
    assert a == 1.0  # least-squares factor 0 is clamped to alpha_min
    assert not M.rr_gate(M.rr_cos(p_i, p_a), M.rr_fit(p_i, p_a, a), 0.8, 0.6)
    # zero probe residual: rejected (refresh)
    z = np.zeros(4)
    assert not M.rr_gate(M.rr_cos(z, p_a), M.rr_fit(z, p_a, 1.0), -1.0, 1e9)
    # eps floor of the denominator: mean(p_a^2) below eps uses eps
    tiny = np.full(4, 1e-6)
    assert M.rr_alpha(tiny * 1e3, tiny, 1e-8, -1e9, 1e9) == pytest.approx(1e-9 / 1e-8)


def test_rr_alpha_is_least_squares_brute_force():
    """Unclamped alpha minimises ||p_i - a p_a|| (scan over a grid)."""
    rng = np.random.default_rng(2)
    p_a = rng.standard_normal(50)
    p_i = 1.13 * p_a + 0.3 * rng.standard_normal(50)
    a = M.rr_alpha(p_i, p_a, 1e-8, -10, 10)
    grid = np.linspace(0.5, 2.0, 150001)
    err = [np.sum((p_i - g * p_a) ** 2) for g in grid[::100]]
    best = grid[::100][int(np.argmin(err))]
    assert abs(a - best) < 2e-3


@pytest.fixture(scope="module")
def rr_model():
    spec = get_workload("tiny_rr").replace(B=2)
    W = make_weights(spec, bias_std=0.02, weight_std=0.05)
    x = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    return spec, W, x, cond


def _prof(spec, **kw):
    q, s, e = spec.rr_bounds
    return M.RRProfile(q, s, e, **kw)


def test_identity_adaptation(rr_model):
    """The same step twice: cos = 1, alpha = 1, fit = 0, accepted, and the
    injected h_e equals the exactly computed one (output = full compute)."""
    spec, W, x, cond = rr_model
    st = M.LayerState()
    prof = _prof(spec)
    v1, i1 = M.velocity_rr(W, spec, x, cond, 0.7, prof, st)
    assert not i1.attempted and st.valid
    pa, Ra = st.p_a.copy(), st.R_a.copy()
    v2, i2 = M.velocity_rr(W, spec, x, cond, 0.7, prof, st)
    assert i2.attempted and i2.accepted
    np.testing.assert_allclose(i2.cos, 1.0, atol=1e-12)
    np.testing.assert_allclose(i2.alpha, 1.0, atol=1e-12)
    np.testing.assert_allclose(i2.fit, 0.0, atol=1e-7)
    np.testing.assert_array_equal(st.p_a, pa)  # accepted reuse keeps the state
    np.testing.assert_array_equal(st.R_a, Ra)
    v_full = dit.velocity(W, spec, x, cond, 0.7)
    np.testing.assert_allclose(v2, v_full, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(v1, v_full)
    assert i2.layers_evaluated == prof.evaluated_after_reuse(spec.L)


def test_force_full_is_bit_identical_to_native(rr_model):
    spec, W, x, cond = rr_model
    sig = M.flow_schedule(spec.K)
    st = M.LayerState()
    x_rr, _, infos = M.denoise(W, spec, x, cond, sig, 0, spec.K, _prof(spec, mode=M.RR_FORCE_FULL), st)
    x_nat, _, _ = M.denoise(W, spec, x, cond, sig, 0, spec.K, None, M.LayerState())
    np.testing.assert_array_equal(x_rr, x_nat)
    # a gate that can never pass (gamma_cos > 1) is also the native path
    x_g, _, infos = M.denoise(W, spec, x, cond, sig, 0, spec.K, _prof(spec, gamma_cos=1.5), M.LayerState())
    np.testing.assert_array_equal(x_g, x_nat)
    assert sum(i.attempted for i in infos) == spec.K - 1 and not any(i.accepted for i in infos)


def test_injection_formula_by_rows(rr_model):
    """FORCE_SKIP: h_e = h_s + alpha_b R_a per branch rows — checked by
    running the layers by hand."""
    spec, W, x, cond = rr_model
    prof = _prof(spec, mode=M.RR_FORCE_SKIP)
    st = M.LayerState()
    M.velocity_rr(W, spec, x, cond, 0.9, prof, st)
    x2 = x * 0.9 + 0.1
    v, info = M.velocity_rr(W, spec, x2, cond, 0.6, prof, st)
    q, s, e = spec.rr_bounds
    c = dit.cond_vector(W, 0.6)
    h = dit.embed_tokens(W, spec, x2, cond)
    h_q = dit.run_layers(W, spec, h, c, 0, q)
    h_s = dit.run_layers(W, spec, h_q, c, q, s)
    h_e = h_s.copy()
    for b in range(spec.B):
        for t in range(spec.T):
            br = 1 if spec.Nv <= t < spec.Nv + spec.Na else 0
            h_e[b, t] = h_s[b, t] + info.alpha[b, br] * st.R_a[b, t]
    ref = dit.final_layer(W, spec, dit.run_layers(W, spec, h_e, c, e, spec.L), c)
    np.testing.assert_allclose(v, ref, rtol=1e-13, atol=1e-13)
    # per-branch alpha from its own rows only
    p_i = h_s - h_q
    rv, ra = M.branch_rows(spec)
    for b in range(spec.B):
        assert info.alpha[b, 1] == M.rr_alpha(p_i[b, ra], st.p_a[b, ra], prof.eps, prof.alpha_min, prof.alpha_max)


def test_refresh_replaces_state(rr_model):
    spec, W, x, cond = rr_model
    prof = _prof(spec, gamma_cos=1.5)  # always refresh
    st = M.LayerState()
    M.velocity_rr(W, spec, x, cond, 0.9, prof, st)
    x2 = -x
    M.velocity_rr(W, spec, x2, cond, 0.4, prof, st)
    c = dit.cond_vector(W, 0.4)
    q, s, e = spec.rr_bounds
    h_q = dit.run_layers(W, spec, dit.embed_tokens(W, spec, x2, cond), c, 0, q)
    h_s = dit.run_layers(W, spec, h_q, c, q, s)
    h_e = dit.run_layers(W, spec, h_s, c, s, e)
    np.testing.assert_array_equal(st.p_a, h_s - h_q)
    np.testing.assert_array_equal(st.R_a, h_e - h_s)


# ---------------------------------------------------------------- Euler
def test_euler_constant_velocity():
    sig = M.flow_schedule(7, 3.0)
    x0 = np.array([0.3, -1.2, 2.0])
    v = np.array([1.5, 0.25, -3.0])
    x = x0
    for k in range(7):
        x = M.euler_update(x, v, sig[k], sig[k + 1])
    np.testing.assert_allclose(x, x0 - v, atol=1e-14)


def test_euler_linear_velocity_product_form():
    sig = M.flow_schedule(5)
    lam = 0.37
    x = np.array([1.0, -2.0])
    prod = 1.0
    for k in range(5):
        x = M.euler_update(x, lam * x, sig[k], sig[k + 1])
        prod *= 1 + lam * (sig[k + 1] - sig[k])
    np.testing.assert_allclose(x, prod * np.array([1.0, -2.0]), rtol=1e-14)


def test_euler_recovers_data_under_exact_flow_velocity():
    """x_sigma = (1-sigma) x0 + sigma eps has velocity eps - x0: Euler lands on x0."""
    rng = np.random.default_rng(3)
    x0, eps = rng.standard_normal(10), rng.standard_normal(10)
    sig = M.flow_schedule(10, 5.0)
    x = eps.copy()
    for k in range(10):
        x = M.euler_update(x, eps - x0, sig[k], sig[k + 1])
    np.testing.assert_allclose(x, x0, atol=1e-13)


# ---------------------------------------------------------------- TR
@pytest.fixture(scope="module")
def traj_spec():
    return get_workload("tiny").replace(B=2)


def test_direction_unit_rms_and_sigma_independent(traj_spec):
    sp = traj_spec
    rng = np.random.default_rng(4)
    xr, xb = rng.standard_normal((2, sp.B, sp.traj))
    d1 = M.tr_direction(sp, xr, xb, 0.3)
    d2 = M.tr_direction(sp, xr, xb, 7.0)
    np.testing.assert_allclose(d1, d2, rtol=1e-13)
    dv, da = dit.split_trajectory(sp, d1)
    for b in range(sp.B):
        assert np.sqrt(np.mean(dv[b] ** 2)) == pytest.approx(1.0, abs=1e-13)
        assert np.sqrt(np.mean(da[b] ** 2)) == pytest.approx(1.0, abs=1e-13)
    with pytest.raises(ValueError):
        M.tr_direction(sp, xr, xb, 0.0)


def test_remap_round_trip(traj_spec):
    """Shift 0 and sigma_b0 = rms(x^r - x_bar) per branch gives x_init = x^r
    when both branches share that rms."""
    sp = traj_spec.replace(B=1)
    rng = np.random.default_rng(5)
    xb = rng.standard_normal((1, sp.traj))
    dlt = rng.standard_normal((1, sp.traj))
    dv, da = dit.split_trajectory(sp, dlt)
    dv = dv / np.sqrt(np.mean(dv ** 2)) * 0.42
    da = da / np.sqrt(np.mean(da ** 2)) * 0.42
    xr = xb + dit.join_trajectory(sp, dv, da)
    d = M.tr_direction(sp, xr, xb, 0.9)
    x_init = M.tr_remap(sp, xb, d, 0.42, 0, 0, np.zeros_like(xb))
    np.testing.assert_allclose(x_init, xr, atol=1e-13)


def test_remap_shift_index_map_brute_force(traj_spec):
    sp = traj_spec
    rng = np.random.default_rng(6)
    xb, d, eps = rng.standard_normal((3, sp.B, sp.traj))
    sb0 = 0.55
    for shift_a, shift_v in ((0, 0), (3, 0), (5, 2), (sp.Na, 0), (sp.Na + 4, sp.Nv)):
        out = M.tr_remap(sp, xb, d, sb0, shift_a, shift_v, eps)
        nv = sp.Nv * sp.Cv
        for b in range(sp.B):
            for j in range(sp.Na):
                for ch in range(sp.A):
                    idx = nv + j * sp.A + ch
                    if j + shift_a < sp.Na:
                        src = nv + (j + shift_a) * sp.A + ch
                        ref = xb[b, src] + sb0 * d[b, src]
                    else:
                        ref = sb0 * eps[b, idx]
                    assert out[b, idx] == pytest.approx(ref, abs=1e-14)
            for j in range(sp.Nv):
                for ch in range(sp.Cv):
                    idx = j * sp.Cv + ch
                    if j + shift_v < sp.Nv:
                        src = (j + shift_v) * sp.Cv + ch
                        ref = xb[b, src] + sb0 * d[b, src]
                    else:
                        ref = sb0 * eps[b, idx]
                    assert out[b, idx] == pytest.approx(ref, abs=1e-14)


def test_remap_empty_mapping_is_fresh_noise(traj_spec):
    """M = empty and sigma_b0 = sigma_0 = 1 reduces to the native initialisation."""
    sp = traj_spec
    rng = np.random.default_rng(7)
    xb, d, eps = rng.standard_normal((3, sp.B, sp.traj))
    out = M.tr_remap(sp, xb, d, 1.0, sp.Na, sp.Nv, eps)
    np.testing.assert_array_equal(out, eps)


# ---------------------------------------------------------------- OR
def test_or_score_examples():
    assert M.or_score([0.3], [2.0]) == pytest.approx(0.3)
    assert M.or_score([0.1, 0.2], [0.5, 0.5]) == pytest.approx(0.15811388300841897, abs=1e-15)
    assert M.or_score([0.1, 0.2], [1.0, 0.0]) == pytest.approx(0.1)
    u = np.array([1.0, 2.0, 3.0, 4.0])
    uh = u + np.array([0.5, -0.5, 0.5, -0.5])
    assert M.or_component_error(uh, u, 2.0) == pytest.approx(0.25)


def test_or_accept_strict_comparisons():
    assert M.or_accept(0.1, 0.12, 0, 3)
    assert not M.or_accept(0.12, 0.12, 0, 3)
    assert not M.or_accept(0.0, 0.12, 3, 3)
    assert M.or_accept(0.0, 0.12, 2, 3)


def _kappa_sequence(kappa_max, n, S=0.0, tau=1.0):
    seq, kappa = [], 0
    for _ in range(n):
        if kappa < kappa_max:
            if M.or_accept(S, tau, kappa, kappa_max):
                kappa += 1
                seq.append("A")
            else:
                kappa = 0
                seq.append("R")
        else:
            kappa = 0
            seq.append("F")
    return "".join(seq)


def test_kappa_sequence_and_coverage_bound():
    assert _kappa_sequence(3, 8) == "AAAFAAAF"
    assert _kappa_sequence(1, 6) == "AFAFAF"
    for model, rr_acc, rr_skip, or_acc, cov, kmax in load_golden("reuse_statistics.csv"):
        kmax = int(kmax)
        bound = kmax / (kmax + 1)  # every prefix accepted
        assert float(cov) / 100 <= bound
        # coverage = r_OR * N_start / N_noninitial and at least kmax/(kmax+1)
        # of the non-initial replans start a prefix
        assert (float(cov) / float(or_acc)) >= bound - 1e-9


def test_runtime_kappa_pattern(rr_model):
    spec, W, x, cond = rr_model
    spec = spec.replace(B=1)
    W = make_weights(spec)
    sig = M.flow_schedule(spec.K)
    rt = M.ReplanRuntime(W, spec, sig, None, M.RuntimeProfile(b0=2, r=2, k1=1, tau=1.0, kappa_max=2))
    obs = make_observations(spec, 6)
    rt.replan(obs[0], noise_first=make_initial_noise(spec))
    paths = []
    for t in range(1, 7):
        _, info = rt.replan(obs[t], obs[t], [obs[t]], [obs[t]], [1.0], [1.0],
                            noise_remap=make_remap_noise(spec, t))
        paths.append(info.path)
    assert paths == [M.PATH_ACCEPT, M.PATH_ACCEPT, M.PATH_FORCED] * 2
    r, cov = (rt.counters.n_bind / rt.counters.n_start, rt.counters.n_bind / rt.counters.n_noninitial)
    assert r == 1.0 and cov == pytest.approx(4 / 6)


# ---------------------------------------------------------------- runtime
def test_perfect_prediction_accepted_equals_direct_run(rr_model):
    """u_hat = u (S = 0): prefix under c_hat = c plus continuation equals the
    K-b0 steps all under c, exactly."""
    spec, W, x, cond = rr_model
    sig = M.flow_schedule(spec.K)
    obs = make_observations(spec, 1)
    rr = _prof(spec)
    common = dict(b0=1, r=2, shift_action=2, k1=1)
    a = M.ReplanRuntime(W, spec, sig, rr, M.RuntimeProfile(**common, tau=0.5))
    b = M.ReplanRuntime(W, spec, sig, rr, M.RuntimeProfile(**common, or_enabled=False))
    for rt in (a, b):
        rt.replan(obs[0], noise_first=make_initial_noise(spec))
    xa, ia = a.replan(obs[1], obs[1], [obs[1]], [obs[1]], [1.0], [1.0], noise_remap=make_remap_noise(spec, 1))
    xb, ib = b.replan(obs[1], noise_remap=make_remap_noise(spec, 1))
    assert ia.path == M.PATH_ACCEPT and ia.S == 0.0 and ib.path == M.PATH_DIRECT
    np.testing.assert_array_equal(xa, xb)
    np.testing.assert_array_equal(a.x_r, b.x_r)


def test_tr_disabled_with_b0_zero_is_native(rr_model):
    spec, W, x, cond = rr_model
    sig = M.flow_schedule(spec.K)
    obs = make_observations(spec, 1)
    rt = M.ReplanRuntime(W, spec, sig, None, M.RuntimeProfile(b0=0, r=1, tr_enabled=False, or_enabled=False))
    rt.replan(obs[0], noise_first=make_initial_noise(spec))
    noise = make_remap_noise(spec, 1)
    x1, info = rt.replan(obs[1], noise_remap=noise)
    ref, _, _ = M.denoise(W, spec, noise, obs[1], sig, 0, spec.K, None, M.LayerState())
    np.testing.assert_array_equal(x1, ref)
    assert info.steps == spec.K


def test_forced_decision_trace_overrides_gate(rr_model):
    spec, W, x, cond = rr_model
    sig = M.flow_schedule(spec.K)
    st = M.LayerState()
    trace = deque([True, False, True])
    _, _, infos = M.denoise(W, spec, x, cond, sig, 0, spec.K, _prof(spec, gamma_cos=1.5), st, forced=trace)
    assert [i.accepted for i in infos] == [False, True, False, True]
    assert not trace
