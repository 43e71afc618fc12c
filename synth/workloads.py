"""Synthetic workload shapes.

Each workload is a DiT-style joint video-latent + action-token denoiser shaped
like the world action models the paper evaluates (video latent frames split into
patches, action chunks of 7-dim single-arm or 14-dim bimanual actions, and
observation-conditioning tokens).  The paper's own models need trained weights
and simulators, so these seeded random-init models stand in for them.

Profile constants that the paper prints are used where it prints them:
residual-rescaling bounds alpha in [1, 1.25], eps = 1e-8, and the Fast-WAM-IDM
gate thresholds cos >= 0.80, fit <= 0.60 (appendix on residual rescaling,
tables of layer boundaries and thresholds); the rebinding limit kappa_max = 3
(appendix on observation rebinding).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field


@dataclass(frozen=True)
class WorkloadSpec:
    name: str
    # model shape
    B: int
    L: int
    D: int
    H: int
    F: int
    Nv: int  # video-latent tokens
    Cv: int  # channels per video token
    Na: int  # action tokens (chunk length)
    A: int  # action dimension
    No: int  # observation-conditioning tokens
    Co: int  # channels per observation token
    dtype: str  # "fp32" | "bf16"
    K: int  # native denoising steps
    qk_norm: bool = True
    ln_eps: float = 1e-6
    schedule_shift: float = 1.0
    # residual rescaling layer boundaries 0 < q < s < e < L (None = off)
    rr_bounds: tuple | None = None
    rr_alpha_min: float = 1.0
    rr_alpha_max: float = 1.25
    rr_eps: float = 1e-8
    rr_gamma_cos: float = 0.80
    rr_gamma_fit: float = 0.60
    # trajectory remapping: entry stage b0 and retained stage r
    tr_b0: int = 0
    tr_r: int = 0
    shift_action: int = 0
    shift_video: int = 0
    # observation rebinding
    or_k1: int = 0
    or_tau: float = 0.5
    or_kappa_max: int = 3
    ar_rho: float = 0.9
    control_steps: int = 0
    seed: int = 0
    notes: str = ""

    @property
    def T(self) -> int:
        return self.Nv + self.Na + self.No

    @property
    def dh(self) -> int:
        return self.D // self.H

    @property
    def traj(self) -> int:
        """Trajectory elements per sample: [video Nv*Cv | action Na*A]."""
        return self.Nv * self.Cv + self.Na * self.A

    @property
    def M(self) -> int:
        return self.B * self.T

    def replace(self, **kw) -> "WorkloadSpec":
        return dataclasses.replace(self, **kw)

    def flops_per_layer(self) -> float:
        """Algorithmic FLOPs of one DiT layer: four projections + attention."""
        M, D, F, T, B = self.M, self.D, self.F, self.T, self.B
        gemm = 2.0 * M * D * (3 * D) + 2.0 * M * D * D + 2.0 * M * D * F * 2
        attn = 4.0 * B * T * T * D
        return gemm + attn

    def flops_per_step(self, layers: int | None = None) -> float:
        return self.flops_per_layer() * (self.L if layers is None else layers)


WORKLOADS: dict[str, WorkloadSpec] = {}


def _reg(w: WorkloadSpec) -> WorkloadSpec:
    WORKLOADS[w.name] = w
    return w


# Tiny fp32 model: 2 layers, hidden 128, 4 heads, MLP 512; 64 video tokens
# (one 8x8 frame, 16 ch) + 16 action tokens (7-dim) + 8 obs tokens; 4 steps.
# L = 2 admits no 0<q<s<e<L partition, so residual rescaling is off.
TINY = _reg(WorkloadSpec(
    name="tiny", B=1, L=2, D=128, H=4, F=512, Nv=64, Cv=16, Na=16, A=7, No=8,
    Co=16, dtype="fp32", K=4, rr_bounds=None, tr_b0=2, tr_r=2, or_k1=1,
    notes="tiny fp32 DiT, L2 D128 H4 F512, T=88, K=4"))

# Tiny fp32 model with 4 layers so that residual rescaling (1,2,3) applies.
TINY_RR = _reg(TINY.replace(
    name="tiny_rr", L=4, rr_bounds=(1, 2, 3),
    notes="tiny fp32 DiT with 4 layers for residual-rescaling tests"))

# The same with hidden 256 (head size 64): rows of a width that the
# residual-rescaling gate's per-block partial kernels take (multiples of 256).
TINY_RR256 = _reg(TINY_RR.replace(
    name="tiny_rr256", D=256, H=4,
    notes="tiny fp32 DiT, 4 layers, hidden 256, for the partial-sum residual-rescaling gate"))

# Small bf16 model: 12 layers, hidden 768, 12 heads, MLP 3072; 3 frames of
# 16x16 patches = 768 video tokens + 32 action tokens (7-dim) + 64 obs tokens;
# 10 flow steps; reuse continues from step 5.
SMALL = _reg(WorkloadSpec(
    name="small", B=1, L=12, D=768, H=12, F=3072, Nv=768, Cv=16, Na=32, A=7,
    No=64, Co=16, dtype="bf16", K=10, rr_bounds=(2, 4, 10), tr_b0=5, tr_r=5,
    shift_action=8, or_k1=2,
    notes="small bf16 DiT, L12 D768 H12 F3072, T=864, K=10"))

# Mid bf16 model, batch 4: 24 layers, hidden 1024, 16 heads, MLP 4096;
# 5 frames of 20x20 = 2000 video + 50 action (14-dim) + 256 obs; 16 steps.
MID = _reg(WorkloadSpec(
    name="mid", B=4, L=24, D=1024, H=16, F=4096, Nv=2000, Cv=16, Na=50, A=14,
    No=256, Co=16, dtype="bf16", K=16, rr_bounds=(2, 4, 20), tr_b0=8, tr_r=8,
    shift_action=8, or_k1=3,
    notes="mid bf16 DiT, B4 L24 D1024 H16 F4096, T=2306, K=16"))

# Large bf16 model: 28 layers, hidden 1536, 24 heads, MLP 6144; 8 frames of
# 30x40 = 9600 video + 64 action (14-dim) + 512 obs; 20 steps.
LARGE = _reg(WorkloadSpec(
    name="large", B=1, L=28, D=1536, H=24, F=6144, Nv=9600, Cv=16, Na=64, A=14,
    No=512, Co=16, dtype="bf16", K=20, rr_bounds=(2, 4, 24), tr_b0=10, tr_r=10,
    shift_action=8, or_k1=4,
    notes="large bf16 DiT, L28 D1536 H24 F6144, T=10176, K=20"))

# Closed-loop replay on the small model: 100 control steps, action horizon
# shifted by 8 per step, AR(1) observations (rho 0.9, N(0,1) innovations).
REPLAY = _reg(SMALL.replace(
    name="replay", control_steps=100,
    notes="closed-loop replay on the small model, 100 control steps"))

# A tiny closed-loop replay used by CPU tests and the smoke check.
TINY_REPLAY = _reg(TINY_RR.replace(
    name="tiny_replay", control_steps=6, shift_action=4, tr_b0=2, tr_r=2,
    or_k1=1, notes="tiny closed-loop replay for tests"))


# Independent execution of the video and action branches (Sec. 3.3, the
# Fast-WAM-IDM profiles of the appendix): two models of the small model's
# shape.  Video model: 768 latent + 64 observation tokens, TR from stage 5 into
# stage 4 without a shift, anticipatory prefix 2 + 4 steps, refresh 6.  Action
# model: 32 action tokens conditioned on the 64 observation tokens and the
# video model's 768 latent tokens (condition channels 16), TR into stage 5
# shifted by ten positions, 5 steps under the real observation on every later
# replan.
IDM_VIDEO = _reg(SMALL.replace(
    name="idm_video", Na=0, A=1, tr_b0=4, tr_r=5, shift_action=0, or_k1=2, control_steps=100,
    notes="video model of the independent pair (small shape, no action tokens)"))
IDM_ACTION = _reg(SMALL.replace(
    name="idm_action", Nv=0, No=64 + 768, Co=16, tr_b0=5, tr_r=5, shift_action=10, or_k1=0,
    control_steps=100, seed=1,
    notes="action model of the independent pair (conditioned on observation + video latent)"))

# Tiny fp32 pair for parity tests (4 layers so RR applies; K = 4).
TINY_IDM_VIDEO = _reg(TINY_RR.replace(
    name="tiny_idm_video", Na=0, A=1, tr_b0=1, tr_r=2, or_k1=1, control_steps=6,
    notes="tiny video model of the independent pair"))
TINY_IDM_ACTION = _reg(TINY_RR.replace(
    name="tiny_idm_action", Nv=0, No=8 + 64, Co=16, tr_b0=2, tr_r=2, shift_action=4, or_k1=0,
    control_steps=6, seed=1, notes="tiny action model of the independent pair"))

PAIRS = {"idm": ("idm_video", "idm_action"), "tiny_idm": ("tiny_idm_video", "tiny_idm_action")}


def get_pair(name: str) -> tuple:
    """(video spec, action spec) of an independently executed pair."""
    v, a = PAIRS[name]
    return WORKLOADS[v], WORKLOADS[a]


def get_workload(name: str) -> WorkloadSpec:
    try:
        return WORKLOADS[name]
    except KeyError as exc:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}") from exc
