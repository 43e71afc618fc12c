"""Oracle of the paper's timing, reuse and diagnostic statistics (float64).

TEST INFRASTRUCTURE ONLY.

  * mean time per replan and speedup: Eq.(app-mean-speedup), timing appendix;
  * observation-to-action latency: Eq.(app-o2a);
  * RR acceptance / layer-skip fraction: Eq.(app-reuse-rates);
  * OR acceptance / replan coverage: Eq.(app-rebinding-rates);
  * trajectory cosine and relative L2: Eq.(app-trajectory-similarity);
  * action RMSE: Eq.(app-action-rmse) (here over every action dimension);
  * layer change and output error: Eq.(app-layer-errors).

Parity status: mean/speedup pinned by recomputing the speedups the paper
prints in its efficiency and ablation tables (tests/golden); the rest pinned
by closed-form cases.
"""
from __future__ import annotations

import numpy as np

f64 = np.float64


def mean_time_per_replan_ms(fg_s, bg_s, replans):
    """1000 * sum_j (f_j + b_j) / sum_j r_j (durations in seconds)."""
    return 1000.0 * (np.sum(np.asarray(fg_s, f64)) + np.sum(np.asarray(bg_s, f64))) / np.sum(replans)


def mean_o2a_ms(o2a_s, replans):
    return 1000.0 * np.sum(np.asarray(o2a_s, f64)) / np.sum(replans)


def o2a(t_obs, t_ready):
    """Eq.(app-o2a): T = t_ready - t_obs."""
    return f64(t_ready) - f64(t_obs)


def speedup(native_ms, method_ms):
    return f64(native_ms) / f64(method_ms)


def rr_rates(n_reuse, n_attempt, b_skip, b_dense):
    """(r_RR, f_skip) = (N_reuse / N_attempt, B_skip / B_dense)."""
    r = n_reuse / n_attempt if n_attempt else float("nan")
    f = b_skip / b_dense if b_dense else float("nan")
    return r, f


def or_rates(n_bind, n_start, n_noninitial):
    """(r_OR, coverage) = (N_bind / N_start, N_bind / N_noninitial)."""
    r = n_bind / n_start if n_start else float("nan")
    c = n_bind / n_noninitial if n_noninitial else float("nan")
    return r, c


def cosine(a, b):
    a, b = np.asarray(a, f64).ravel(), np.asarray(b, f64).ravel()
    return float(np.dot(a, b) / (np.linalg.norm(a) * np.linalg.norm(b)))


def rel_l2(x, ref):
    """||x - ref|| / ||ref|| (the reference is the denominator)."""
    x, ref = np.asarray(x, f64).ravel(), np.asarray(ref, f64).ravel()
    return float(np.linalg.norm(x - ref) / np.linalg.norm(ref))


def action_rmse(a, a_ref):
    """sqrt(mean over actions and dimensions of (a - a_ref)^2)."""
    d = np.asarray(a, f64) - np.asarray(a_ref, f64)
    return float(np.sqrt(np.mean(d * d)))


def layer_change(h_next, h):
    """Delta_l = ||h_{l+1} - h_l|| / ||h_l||."""
    return rel_l2(h_next, h)


def output_error(y_reuse, y_full):
    """E_out = ||y_reuse - y_full|| / ||y_full||."""
    return rel_l2(y_reuse, y_full)


def max_rel_err(y, y_ref):
    """max_i |y_i - ref_i| / max_i |ref_i| (the parity measure)."""
    y, y_ref = np.asarray(y, f64), np.asarray(y_ref, f64)
    return float(np.max(np.abs(y - y_ref)) / np.max(np.abs(y_ref)))
