"""Oracle of the solver and the three state-adaptation operators (float64).

TEST INFRASTRUCTURE ONLY — never called by the product path.

Follows the paper's method section:
  * Trajectory Remapping, Sec. 3.1: denoising direction Eq.(direction) with the
    unit-RMS normalisation of the trajectory-profile appendix
    Eq.(app-transport-rms), remapped initialisation Eq.(transport);
  * Observation Rebinding, Sec. 3.2: consistency score Eq.(bind-discrepancy),
    acceptance S < tau and kappa < kappa_max, kappa reset on refresh, forced
    refresh at kappa_max;
  * Residual Rescaling, Sec. 3.3: layer partition 0<q<s<e<L, retained residuals
    Eq.(crr-reference), rescaling factor Eq.(crr-alpha), gate Eq.(crr-gate),
    injection Eq.(residual-injection), refresh on failure;
  * joint runtime, Sec. 3.4, with the denoising-step counts of the schedules
    table in the trajectory-profile appendix (accepted a+b = refresh = K-b0).

The flow solver (rectified-flow Euler) and its sigma schedule are readings:
the paper only says "diffusion or flow".  The shifted schedule
sigma = S s / (1 + (S-1) s), s = 1 - k/K reproduces the noise levels the paper
prints for Fast-WAM-IDM (stage 4 -> 0.88235, stage 5 -> 0.83333 at S = 5,
K = 10) and the uniform one the ~0.7 of Motus at stage 3.

Parity status: every function here is pinned in tests/test_oracle_method.py
by printed values, closed forms or brute force (schedule, step and layer
counts, alpha/cos/fit closed forms, remap round trip and index map, the
two-component score example, the kappa sequence, Euler invariants, full
re-denoise == no-reuse path).
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field

import numpy as np

from . import dit

f64 = np.float64

RR_OFF, RR_AUTO, RR_FORCE_SKIP, RR_FORCE_FULL = 0, 1, 2, 3

PATH_FIRST, PATH_ACCEPT, PATH_REJECT, PATH_FORCED, PATH_DIRECT = 0, 1, 2, 3, 4


# --------------------------------------------------------------------------
# schedule and solver
# --------------------------------------------------------------------------
def flow_schedule(K: int, shift: float = 1.0) -> np.ndarray:
    """sigma_k = S s / (1 + (S-1) s) with s = 1 - k/K, k = 0..K (sigma_0=1, sigma_K=0)."""
    s = 1.0 - np.arange(K + 1, dtype=f64) / K
    return shift * s / (1.0 + (shift - 1.0) * s)


def euler_update(x, v, sigma_k, sigma_k1):
    """One Euler step of the flow ODE: x + (sigma_{k+1} - sigma_k) v."""
    return dit.as64(x) + (f64(sigma_k1) - f64(sigma_k)) * dit.as64(v)


# --------------------------------------------------------------------------
# Residual Rescaling (Sec. 3.3)
# --------------------------------------------------------------------------
@dataclass
class RRProfile:
    q: int
    s: int
    e: int
    alpha_min: float = 1.0
    alpha_max: float = 1.25
    eps: float = 1e-8
    gamma_cos: float = 0.80
    gamma_fit: float = 0.60
    mode: int = RR_AUTO
    # False: the two jointly executed branches (video + observation rows,
    # action rows) each get an alpha and must both pass (Sec. 3.3, joint
    # execution).  True: the model's whole token set is one branch, as for each
    # model of an independently executed pair (Sec. 3.3, independent execution).
    single: bool = False

    def validate(self, L: int):
        if self.mode != RR_OFF and not (0 < self.q < self.s < self.e < L):
            raise ValueError(f"need 0<q<s<e<L, got q={self.q} s={self.s} e={self.e} L={L}")

    def evaluated_after_reuse(self, L: int) -> int:
        """Layers evaluated on an accepted step: head + probe + tail = s + (L-e)."""
        return self.s + (L - self.e)


def rr_alpha(p_i, p_a, eps, alpha_min, alpha_max) -> float:
    """Eq.(crr-alpha): clamp(mean(p_i*p_a) / max(mean(p_a*p_a), eps), amin, amax)."""
    p_i, p_a = dit.as64(p_i).ravel(), dit.as64(p_a).ravel()
    if p_i.size == 0:  # an empty branch: nothing to rescale (and its gate fails)
        return float(alpha_min)
    num = np.mean(p_i * p_a)
    den = max(np.mean(p_a * p_a), eps)
    return float(np.clip(num / den, alpha_min, alpha_max))


def rr_cos(p_i, p_a) -> float:
    """cos(p_i, p_a); 0 when either vector is zero (which fails the gate)."""
    p_i, p_a = dit.as64(p_i).ravel(), dit.as64(p_a).ravel()
    ni, na = np.linalg.norm(p_i), np.linalg.norm(p_a)
    if ni == 0.0 or na == 0.0:
        return 0.0
    return float(np.dot(p_i, p_a) / (ni * na))


def rr_fit(p_i, p_a, alpha) -> float:
    """||p_i - alpha p_a||_2 / ||p_i||_2; +inf when p_i is zero."""
    p_i, p_a = dit.as64(p_i).ravel(), dit.as64(p_a).ravel()
    ni = np.linalg.norm(p_i)
    if ni == 0.0:
        return float("inf")
    return float(np.linalg.norm(p_i - alpha * p_a) / ni)


def rr_gate(cos, fit, gamma_cos, gamma_fit, p_a_zero=False) -> bool:
    """Eq.(crr-gate): cos >= gamma_cos and fit <= gamma_fit (a zero residual fails)."""
    if p_a_zero or not np.isfinite(fit):
        return False
    return bool(cos >= gamma_cos and fit <= gamma_fit)


def rr_branch_stats(p_i, p_a, prof: RRProfile):
    """alpha (Eq. crr-alpha), cos and relative fit (Eq. crr-gate) of one
    branch of one sample, and whether it passes the gate."""
    alpha = rr_alpha(p_i, p_a, prof.eps, prof.alpha_min, prof.alpha_max)
    cos = rr_cos(p_i, p_a)
    fit = rr_fit(p_i, p_a, alpha)
    return alpha, cos, fit, rr_gate(cos, fit, prof.gamma_cos, prof.gamma_fit, p_a_zero=not np.any(p_a))


def branch_rows(spec, single: bool = False):
    """Row indices (within one sample) of the branches RR checks: the two
    jointly executed ones, V = video and observation rows and A = action rows,
    or (single) all rows as one branch."""
    if single:
        return (np.arange(spec.T),)
    v = np.r_[0:spec.Nv, spec.Nv + spec.Na:spec.T]
    a = np.arange(spec.Nv, spec.Nv + spec.Na)
    return v, a


@dataclass
class RRStepInfo:
    attempted: bool = False
    accepted: bool = False
    alpha: np.ndarray | None = None  # [B, 2] (branch 0 = V, 1 = A)
    cos: np.ndarray | None = None
    fit: np.ndarray | None = None
    layers_evaluated: int = 0
    layers_skipped: int = 0
    rr_active: bool = False


class LayerState:
    """Retained exact layer state (p_a, R_a), Eq.(crr-reference)."""

    def __init__(self):
        self.p_a = None
        self.R_a = None

    def reset(self):
        self.p_a = None
        self.R_a = None

    @property
    def valid(self) -> bool:
        return self.p_a is not None


def velocity_rr(W, spec, x, cond, sigma, prof: RRProfile | None, state: LayerState,
                forced: deque | None = None):
    """Denoiser prediction with Residual Rescaling inside the forward pass.

    Returns (v, RRStepInfo).  ``forced`` (decision-trace protocol) supplies the
    accept/reject decision of each attempt instead of the gate; the
    statistics are still computed and reported.
    """
    L = spec.L
    c = dit.cond_vector(W, sigma)
    h = dit.embed_tokens(W, spec, x, cond)
    info = RRStepInfo(layers_evaluated=L)
    if prof is None or prof.mode == RR_OFF:
        h = dit.run_layers(W, spec, h, c, 0, L)
        return dit.final_layer(W, spec, h, c), info
    prof.validate(L)
    q, s, e = prof.q, prof.s, prof.e
    info.rr_active = True
    h = dit.run_layers(W, spec, h, c, 0, q)
    h_q = h
    h = dit.run_layers(W, spec, h, c, q, s)
    h_s = h
    p_i = h_s - h_q

    accept = False
    if state.valid and prof.mode in (RR_AUTO, RR_FORCE_SKIP):
        info.attempted = True
        B = spec.B
        rows = branch_rows(spec, prof.single)
        # [B, 2] statistics; with a single branch column 1 stays NaN (no branch)
        alpha = np.full((B, 2), np.nan)
        cosv = np.full((B, 2), np.nan)
        fitv = np.full((B, 2), np.nan)
        ok = True
        for b in range(B):
            for br, r in enumerate(rows):
                alpha[b, br], cosv[b, br], fitv[b, br], passed = rr_branch_stats(
                    p_i[b, r], state.p_a[b, r], prof)
                ok &= passed
        info.alpha, info.cos, info.fit = alpha, cosv, fitv
        if forced is not None:
            accept = bool(forced.popleft())
        elif prof.mode == RR_FORCE_SKIP:
            accept = True
        else:
            accept = ok

    if accept:
        # Eq.(residual-injection): h_e = h_s + alpha R_a, per sample and branch.
        h_e = h_s.copy()
        for b in range(spec.B):
            for br, r in enumerate(branch_rows(spec, prof.single)):
                h_e[b, r] = h_s[b, r] + info.alpha[b, br] * state.R_a[b, r]
        info.accepted = True
        info.layers_skipped = e - s
        info.layers_evaluated = L - (e - s)
    else:
        # full middle from h_s, then refresh (or establish) the layer state
        h_e = dit.run_layers(W, spec, h_s, c, s, e)
        state.p_a = p_i
        state.R_a = h_e - h_s
    h = dit.run_layers(W, spec, h_e, c, e, L)
    return dit.final_layer(W, spec, h, c), info


def denoise(W, spec, x, cond, sigmas, k_from: int, k_to: int, prof: RRProfile | None,
            state: LayerState, capture_stage: int | None = None, forced: deque | None = None):
    """Euler steps k_from..k_to-1; returns (x at stage k_to, captured latent, infos).

    The latent at stage ``capture_stage`` (if visited, k_from <= r <= k_to) is
    returned as the retained intermediate latent x^r.
    """
    x = dit.as64(x).copy()
    captured = None
    infos = []
    for k in range(k_from, k_to):
        if capture_stage == k:
            captured = x.copy()
        v, info = velocity_rr(W, spec, x, cond, sigmas[k], prof, state, forced)
        x = euler_update(x, v, sigmas[k], sigmas[k + 1])
        infos.append(info)
    if capture_stage == k_to:
        captured = x.copy()
    return x, captured, infos


# --------------------------------------------------------------------------
# Trajectory Remapping (Sec. 3.1)
# --------------------------------------------------------------------------
def _branches(spec, x):
    """Per-sample views [video (Nv, Cv), action (Na, A)] of a [B, traj] array."""
    return dit.split_trajectory(spec, x)


def unit_rms(v):
    """N(v) = v / sqrt(mean(v^2)) (Eq. app-transport-rms); 0 if v is zero; an
    empty branch (a model without video or without action tokens) stays empty."""
    v = dit.as64(v)
    if v.size == 0:
        return v.copy()
    r = np.sqrt(np.mean(v * v))
    return v / r if r > 0 else np.zeros_like(v)


def tr_direction(spec, x_r, x_bar, sigma_r):
    """Eq.(direction): d = N((x^r - x_bar) / sigma_r), normalised per sample and
    per branch over the complete trajectory of that branch."""
    if not sigma_r > 0:
        raise ValueError("sigma_r must be > 0")
    diff = (dit.as64(x_r) - dit.as64(x_bar)) / f64(sigma_r)
    dv, da = _branches(spec, diff)
    out_v = np.stack([unit_rms(dv[b]) for b in range(spec.B)])
    out_a = np.stack([unit_rms(da[b]) for b in range(spec.B)])
    return dit.join_trajectory(spec, out_v, out_a)


def shift_slots(a, shift: int):
    """Remapping operator A: target slot j takes source slot j + shift.

    Returns (shifted, mapped) where mapped[j] says whether slot j is in M
    (i.e. j + shift is a valid source slot)."""
    n = a.shape[0]
    out = np.zeros_like(a)
    mapped = np.zeros(n, bool)
    for j in range(n):
        if j + shift < n:
            out[j] = a[j + shift]
            mapped[j] = True
    return out, mapped


def tr_remap(spec, x_bar, d, sigma_b0, shift_action: int, shift_video: int, noise):
    """Eq.(transport): x[j] = A(x_bar)[j] + sigma_b0 A(d)[j] for j in M, else
    fresh noise sigma_b0 * eps[j] (eps ~ N(0,1) supplied by the caller).

    Returns (x_init [B, traj], mapped mask per branch)."""
    if shift_action < 0 or shift_video < 0:
        raise ValueError("shifts must be >= 0")
    xbv, xba = _branches(spec, x_bar)
    dv, da = _branches(spec, d)
    nv, na = _branches(spec, noise)
    outv = np.empty_like(xbv)
    outa = np.empty_like(xba)
    for b in range(spec.B):
        for src_x, src_d, eps, shift, out in ((xbv[b], dv[b], nv[b], shift_video, outv),
                                              (xba[b], da[b], na[b], shift_action, outa)):
            sx, mapped = shift_slots(src_x, shift)
            sd, _ = shift_slots(src_d, shift)
            out[b] = np.where(mapped[:, None], sx + f64(sigma_b0) * sd, f64(sigma_b0) * eps)
    return dit.join_trajectory(spec, outv, outa)


# --------------------------------------------------------------------------
# Observation Rebinding (Sec. 3.2)
# --------------------------------------------------------------------------
def or_component_error(u_hat, u, delta) -> float:
    """e_m = sqrt(mean(((u_hat - u) / delta)^2))."""
    r = (dit.as64(u_hat) - dit.as64(u)) / f64(delta)
    return float(np.sqrt(np.mean(r * r)))


def or_score(errors, weights) -> float:
    """S = sqrt(sum_m w_m e_m^2 / sum_m w_m)."""
    e = dit.as64(errors)
    w = dit.as64(weights)
    return float(np.sqrt(np.sum(w * e * e) / np.sum(w)))


def or_accept(S: float, tau: float, kappa: int, kappa_max: int) -> bool:
    """Rebinding proceeds only when S < tau and kappa < kappa_max."""
    return bool(S < tau and kappa < kappa_max)


# --------------------------------------------------------------------------
# joint runtime (Sec. 3.4)
# --------------------------------------------------------------------------
@dataclass
class RuntimeProfile:
    b0: int
    r: int
    shift_action: int = 0
    shift_video: int = 0
    k1: int = 0
    tau: float = 0.5
    kappa_max: int = 3
    tr_enabled: bool = True
    or_enabled: bool = True
    rr_first: bool = True  # RR allowed during the first replan
    rr_prefix: bool = True  # RR allowed on the anticipatory prefix and its continuation
    rr_refresh: bool = True  # RR allowed on a refresh from the remapped initialisation


@dataclass
class ReplanInfo:
    path: int
    S: float | None
    kappa: int
    steps: int
    rr_infos: list = field(default_factory=list)


@dataclass
class ReuseCounters:
    """Counters of the reuse-statistics appendix, Eq.(app-reuse-rates) and
    Eq.(app-rebinding-rates)."""
    n_attempt: int = 0
    n_reuse: int = 0
    b_skip: int = 0
    b_dense: int = 0
    n_start: int = 0
    n_bind: int = 0
    n_noninitial: int = 0

    def add_steps(self, infos, L):
        for i in infos:
            if i.rr_active:
                self.b_dense += L
                self.b_skip += i.layers_skipped
            self.n_attempt += int(i.attempted)
            self.n_reuse += int(i.accepted)


class ReplanRuntime:
    """Closed-loop replan state machine: TR -> OR prefix -> check -> rebind or
    restart, with RR inside every denoising step."""

    def __init__(self, W, spec, sigmas, rr: RRProfile | None, prof: RuntimeProfile):
        self.W, self.spec, self.sigmas = W, spec, dit.as64(sigmas)
        self.rr, self.p = rr, prof
        self.K = len(sigmas) - 1
        self.x_bar = None
        self.x_r = None
        self.kappa = 0
        self.layer = LayerState()
        self.counters = ReuseCounters()
        if not (0 <= prof.b0 < self.K):
            raise ValueError("b0 out of range")
        if prof.tr_enabled and not (prof.b0 <= prof.r < self.K):
            raise ValueError("need b0 <= r < K so that x^r is retained with sigma_r > 0")
        if prof.or_enabled and not (0 < prof.k1 < self.K - prof.b0):
            raise ValueError("need 0 < k1 < K - b0")

    def _rr(self, allowed: bool):
        return self.rr if (allowed and self.rr is not None) else None

    def set_state(self, x_bar, x_r, kappa):
        """Teacher forcing: adopt an externally supplied replan state."""
        self.x_bar = dit.as64(x_bar).copy()
        self.x_r = dit.as64(x_r).copy()
        self.kappa = int(kappa)

    def replan(self, cond_real, cond_pred=None, u_hat=None, u=None, deltas=None,
               weights=None, noise_first=None, noise_remap=None, forced: deque | None = None):
        sp, p, sig = self.spec, self.p, self.sigmas
        K = self.K
        first = self.x_bar is None
        self.layer.reset()
        if first:
            x, xr, infos = denoise(self.W, sp, noise_first, cond_real, sig, 0, K,
                                   self._rr(p.rr_first), self.layer, p.r, forced)
            self.counters.add_steps(infos, sp.L)
            self.x_bar, self.x_r = x, xr
            return x, ReplanInfo(PATH_FIRST, None, self.kappa, K, infos)

        self.counters.n_noninitial += 1
        if p.tr_enabled:
            d = tr_direction(sp, self.x_r, self.x_bar, sig[p.r])
            x_init = tr_remap(sp, self.x_bar, d, sig[p.b0], p.shift_action, p.shift_video,
                              noise_remap)
            entry = p.b0
        else:
            x_init = dit.as64(noise_remap).copy()  # fresh N(0,1) at sigma_0 = 1
            entry = 0
        S = None
        all_infos = []
        if p.or_enabled and self.kappa < p.kappa_max:
            self.counters.n_start += 1
            x_pre, xr_pre, infos = denoise(self.W, sp, x_init, cond_pred, sig, entry,
                                           entry + p.k1, self._rr(p.rr_prefix), self.layer,
                                           p.r, forced)
            self.counters.add_steps(infos, sp.L)
            all_infos += infos
            errs = [or_component_error(a, b, dl) for a, b, dl in zip(u_hat, u, deltas)]
            S = or_score(errs, weights)
            if or_accept(S, p.tau, self.kappa, p.kappa_max):
                self.kappa += 1
                self.counters.n_bind += 1
                path = PATH_ACCEPT
                x, xr, infos = denoise(self.W, sp, x_pre, cond_real, sig, entry + p.k1, K,
                                       self._rr(p.rr_prefix), self.layer, p.r, forced)
                xr = xr if xr is not None else xr_pre
            else:
                self.kappa = 0
                path = PATH_REJECT
                self.layer.reset()
                x, xr, infos = denoise(self.W, sp, x_init, cond_real, sig, entry, K,
                                       self._rr(p.rr_refresh), self.layer, p.r, forced)
        else:
            path = PATH_FORCED if p.or_enabled else PATH_DIRECT
            if p.or_enabled:
                self.kappa = 0
            x, xr, infos = denoise(self.W, sp, x_init, cond_real, sig, entry, K,
                                   self._rr(p.rr_refresh), self.layer, p.r, forced)
        self.counters.add_steps(infos, sp.L)
        all_infos += infos
        self.x_bar, self.x_r = x, xr
        steps = len(all_infos)
        return x, ReplanInfo(path, S, self.kappa, steps, all_infos)


# --------------------------------------------------------------------------
# independent execution of the video and action branches (Sec. 3.3; the
# Fast-WAM-IDM profiles of the appendix)
# --------------------------------------------------------------------------
def pack_condition(obs, ctx, Co: int):
    """Condition tokens of the action model of an independently executed pair:
    the observation tokens followed by the video model's latent tokens (the
    action model reads the predicted video), each zero-padded to Co channels.
    obs [B, n_obs, c_obs], ctx [B, n_ctx, c_ctx] -> [B, n_obs + n_ctx, Co]."""
    obs, ctx = dit.as64(obs), dit.as64(ctx)
    B, n_obs, c_obs = obs.shape
    _, n_ctx, c_ctx = ctx.shape
    if c_obs > Co or c_ctx > Co:
        raise ValueError("channels exceed Co")
    out = np.zeros((B, n_obs + n_ctx, Co))
    out[:, :n_obs, :c_obs] = obs
    out[:, n_obs:, :c_ctx] = ctx
    return out


class IdmPairRuntime:
    """Video and action executed as two models with their own replan state,
    schedule and RR decision.  Each control step runs the video model's
    replan under the observation, then the action model's under the
    observation plus the video model's new latent."""

    def __init__(self, video: ReplanRuntime, action: ReplanRuntime):
        sv, sa = video.spec, action.spec
        if sv.Na != 0 or sa.Nv != 0:
            raise ValueError("video model has no action tokens, action model no video tokens")
        if sa.No < sv.Nv or sa.Co < max(sv.Co, sv.Cv):
            raise ValueError("action condition must hold the observation and the video tokens")
        if action.p.or_enabled:
            raise ValueError("the action model runs under the real observation only")
        self.video, self.action = video, action

    def action_condition(self, obs, x_video):
        sv = self.video.spec
        ctx = dit.split_trajectory(sv, x_video)[0]
        return pack_condition(obs, ctx, self.action.spec.Co)

    def replan(self, obs_real, obs_pred=None, u_hat=None, u=None, deltas=None, weights=None,
               noise_first=(None, None), noise_remap=(None, None), forced=(None, None)):
        xv, info_v = self.video.replan(obs_real, obs_pred, u_hat, u, deltas, weights,
                                       noise_first[0], noise_remap[0], forced[0])
        cond_a = self.action_condition(obs_real, xv)
        xa, info_a = self.action.replan(cond_a, None, None, None, None, None,
                                        noise_first[1], noise_remap[1], forced[1])
        return xv, xa, info_v, info_a


def action_chunk(spec, x):
    """Action rows of a trajectory, [B, Na, A]."""
    return dit.split_trajectory(spec, x)[1]
