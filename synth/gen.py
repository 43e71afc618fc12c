"""Seeded generators for weights, noise and observations.

Random streams (numpy PCG64 through ``default_rng``), one per purpose:

    [seed, 0]      weight matrices and embedding tables, N(0, 0.02^2), drawn
                   tensor by tensor in manifest order, row-major
    [seed, 1]      initial noise of the first replan, N(0, 1)
    [seed, 2]      first observation o_0 ~ N(0, 1/(1-rho^2)) (stationary AR(1))
    [seed, 3, t]   unit-normal noise for the unmapped slots of replan t
    [seed, 4]      AR(1) innovations eta_t ~ N(0, 1)
    [seed, 5]      optional non-zero biases (tests only)
    [seed, 6]      optional non-unit QK-norm gains (tests only)

In bf16 mode every weight value is rounded to the nearest bf16 (ties to even),
so that both the fp64 CPU oracle and the device path see exactly the same
numbers.  All arrays are float32 in host memory.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np

from .workloads import WorkloadSpec

TIME_EMB_DIM = 256  # sinusoidal timestep features fed to the conditioning MLP


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # add half an ulp of bf16 minus one, plus the lsb that is kept (ties to
    # even), then truncate; 32-bit wrap-around only ever reaches bits that
    # the mask drops
    r = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    r &= np.uint32(0xFFFF0000)
    return r.view(np.float32).reshape(a.shape)


def weight_manifest(w: WorkloadSpec) -> list[tuple[str, tuple[int, ...], str]]:
    """(name, shape, kind) for every parameter, in draw order.

    kind is "w" (matrix / table, N(0, 0.02^2)), "b" (bias, 0 by default) or
    "g" (norm gain, 1 by default).  Linear layers compute y = x @ W + b with W
    stored as [in, out].
    """
    D, F, dh = w.D, w.F, w.dh
    m: list[tuple[str, tuple[int, ...], str]] = [
        ("t_w1", (TIME_EMB_DIM, D), "w"), ("t_b1", (D,), "b"),
        ("t_w2", (D, D), "w"), ("t_b2", (D,), "b"),
        ("in_wv", (w.Cv, D), "w"), ("in_bv", (D,), "b"),
        ("in_wa", (w.A, D), "w"), ("in_ba", (D,), "b"),
        ("in_wo", (w.Co, D), "w"), ("in_bo", (D,), "b"),
    ]
    for l in range(w.L):
        p = f"l{l}."
        m += [
            (p + "mod_w", (D, 6 * D), "w"), (p + "mod_b", (6 * D,), "b"),
            (p + "qkv_w", (D, 3 * D), "w"), (p + "qkv_b", (3 * D,), "b"),
            (p + "q_g", (dh,), "g"), (p + "k_g", (dh,), "g"),
            (p + "proj_w", (D, D), "w"), (p + "proj_b", (D,), "b"),
            (p + "fc1_w", (D, F), "w"), (p + "fc1_b", (F,), "b"),
            (p + "fc2_w", (F, D), "w"), (p + "fc2_b", (D,), "b"),
        ]
    m += [
        ("f_mod_w", (D, 2 * D), "w"), ("f_mod_b", (2 * D,), "b"),
        ("out_wv", (D, w.Cv), "w"), ("out_bv", (w.Cv,), "b"),
        ("out_wa", (D, w.A), "w"), ("out_ba", (w.A,), "b"),
    ]
    return m


def make_weights(w: WorkloadSpec, seed: int | None = None, *, bias_std: float = 0.0,
                 gain_std: float = 0.0, weight_std: float = 0.02) -> "OrderedDict[str, np.ndarray]":
    """Draw all parameters of workload ``w``.

    bias_std / gain_std > 0 give non-zero biases and non-unit QK gains; the
    paper-shaped workloads keep the defaults (biases 0, gains 1) and tests use
    the non-default values so that every parameter is exercised.
    """
    seed = w.seed if seed is None else seed
    rw = np.random.default_rng([seed, 0])
    rb = np.random.default_rng([seed, 5])
    rg = np.random.default_rng([seed, 6])
    out: "OrderedDict[str, np.ndarray]" = OrderedDict()
    for name, shape, kind in weight_manifest(w):
        if kind == "w":
            a = rw.standard_normal(shape, dtype=np.float32) * np.float32(weight_std)
        elif kind == "b":
            if bias_std > 0:
                a = rb.standard_normal(shape, dtype=np.float32) * np.float32(bias_std)
            else:
                a = np.zeros(shape, np.float32)
        else:
            if gain_std > 0:
                a = (1.0 + rg.standard_normal(shape, dtype=np.float32) * gain_std).astype(np.float32)
            else:
                a = np.ones(shape, np.float32)
        if w.dtype == "bf16":
            a = bf16_round(a)
        out[name] = np.ascontiguousarray(a, dtype=np.float32)
    return out


def make_initial_noise(w: WorkloadSpec, seed: int | None = None) -> np.ndarray:
    """Unit-normal noise for the first replan, [B, traj] float32."""
    seed = w.seed if seed is None else seed
    r = np.random.default_rng([seed, 1])
    return r.standard_normal((w.B, w.traj), dtype=np.float32)


def make_remap_noise(w: WorkloadSpec, t: int, seed: int | None = None) -> np.ndarray:
    """Unit-normal noise for the unmapped slots of replan t, [B, traj] float32."""
    seed = w.seed if seed is None else seed
    r = np.random.default_rng([seed, 3, t])
    return r.standard_normal((w.B, w.traj), dtype=np.float32)


def make_observations(w: WorkloadSpec, n_steps: int, seed: int | None = None,
                      rho: float | None = None) -> np.ndarray:
    """AR(1) observation tokens o_0..o_{n_steps}, [n_steps+1, B, No, Co] float32.

    o_0 is drawn from the stationary law N(0, 1/(1-rho^2)); afterwards
    o_{t+1} = rho * o_t + eta_t with eta_t ~ N(0, 1).
    """
    seed = w.seed if seed is None else seed
    rho = w.ar_rho if rho is None else rho
    shape = (w.B, w.No, w.Co)
    r0 = np.random.default_rng([seed, 2])
    ri = np.random.default_rng([seed, 4])
    obs = np.empty((n_steps + 1,) + shape, np.float32)
    std0 = 1.0 / np.sqrt(1.0 - rho * rho) if rho < 1 else 1.0
    obs[0] = r0.standard_normal(shape, dtype=np.float32) * np.float32(std0)
    for t in range(n_steps):
        eta = ri.standard_normal(shape, dtype=np.float32)
        obs[t + 1] = np.float32(rho) * obs[t] + eta
    return obs
