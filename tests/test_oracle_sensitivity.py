"""Sensitivity pins of the bf16 parity quantity (oracle only, CPU).

The bf16 GPU tests compare each DiT layer's update h_{l+1} - h_l with the
oracle's on the same input, at tolerance BF16_UPDATE_TOL.  That check is
only worth something if a broken contraction would fail it.  Here the
oracle itself shows, at the shapes those tests use, that removing a piece of
the layer moves the compared quantity far beyond the tolerance:

  * attention output zeroed (attention-output projection and bias = 0),
  * MLP output zeroed (MLP-down projection and bias = 0),
  * QKV projection zeroed (q = k = v = 0 before QK-norm),
      each by at least 10 x BF16_UPDATE_TOL;
  * uniform attention probabilities (softmax replaced by 1/T): at least
    5 x BF16_UPDATE_TOL.

The measure is the parity measure max |got - ref| / max |ref|.
"""
import contextlib

import numpy as np
import pytest

from oracle import dit as OD, method as OM
from synth import get_workload, make_weights, make_initial_noise, make_observations
from gpu_common import BF16_UPDATE_TOL


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


@contextlib.contextmanager
def _uniform_softmax():
    orig = OD.softmax
    OD.softmax = lambda s, axis=-1: np.full_like(OD.as64(s), 1.0 / s.shape[axis])
    try:
        yield
    finally:
        OD.softmax = orig


def _zeroed(W, l, names):
    W2 = dict(W)
    for n in names:
        W2[f"l{l}.{n}"] = np.zeros_like(W[f"l{l}.{n}"])
    return W2


def _check(spec, W, k, layers):
    sig = OM.flow_schedule(spec.K).astype(np.float32).astype(np.float64)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    c = OD.cond_vector(W, sig[k])
    h = OD.embed_tokens(W, spec, x0, cond)
    for l in range(max(layers) + 1):
        nxt = OD.dit_layer(W, spec, l, h, c)
        if l in layers:
            ref = nxt - h
            for what, names in (("attention", ("proj_w", "proj_b")), ("mlp", ("fc2_w", "fc2_b")),
                                ("qkv", ("qkv_w", "qkv_b"))):
                moved = _rel(OD.dit_layer(_zeroed(W, l, names), spec, l, h, c) - h, ref)
                assert moved >= 10 * BF16_UPDATE_TOL, (l, what, moved)
            with _uniform_softmax():
                moved = _rel(OD.dit_layer(W, spec, l, h, c) - h, ref)
            assert moved >= 5 * BF16_UPDATE_TOL, (l, "uniform softmax", moved)
        h = nxt


def test_small_model_layers():
    """The small model (replay workload shape, T = 864), a first, a middle
    and the last layer at the first step."""
    spec = get_workload("small")
    _check(spec, make_weights(spec), 0, [0, 6, 11])


@pytest.mark.parametrize("lengths", [(24, 8, 8), (41, 16, 8), (288, 32, 13)])
def test_attention_length_shapes(lengths):
    """The short-sequence attention shapes (T = 40, 65, 333; two heads)."""
    Nv, Na, No = lengths
    spec = get_workload("small").replace(L=2, D=128, H=2, F=512, Nv=Nv, Na=Na, No=No, B=2)
    W = make_weights(spec, bias_std=0.02, gain_std=0.1)
    for k in (0, 6):
        _check(spec, W, k, [0, 1])


@pytest.mark.parametrize("D,H", [(192, 3), (1088, 17)])
def test_odd_head_count_shapes(D, H):
    spec = get_workload("small").replace(L=1, D=D, H=H, F=4 * D, Nv=40, Na=16, No=8, B=2)
    W = make_weights(spec, bias_std=0.02, gain_std=0.1)
    _check(spec, W, 0, [0])


def test_threaded_attention_equals_serial():
    """The per-(sample, head) loop of the oracle's attention gives the same
    bits whether its pairs run one after another or on worker threads."""
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((2, 3, 50, 16)) for _ in range(3))
    serial = OD.attention(q, k, v)
    old = OD.ATTENTION_THREADS
    OD.ATTENTION_THREADS = 4
    try:
        threaded = OD.attention(q, k, v)
    finally:
        OD.ATTENTION_THREADS = old
    np.testing.assert_array_equal(serial, threaded)


def test_small_model_injection_quantity():
    """The residual-injection check at the small model's shape compares the
    velocity change that reuse makes (forced reuse minus full computation on
    the same latent) at tolerance 2e-2.  Dropping the retained residual R_a,
    or injecting p_a in its place, moves that change by at least ten times
    the tolerance."""
    spec = get_workload("small")
    W = make_weights(spec)
    sig = OM.flow_schedule(spec.K).astype(np.float32).astype(np.float64)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    prof = OM.RRProfile(*spec.rr_bounds, mode=OM.RR_FORCE_SKIP)
    st = OM.LayerState()
    v0, _ = OM.velocity_rr(W, spec, x0, cond, sig[0], prof, st)
    x1 = OM.euler_update(x0, v0, sig[0], sig[1])
    vf = OD.velocity(W, spec, x1, cond, sig[1])

    def skip_with(R_a):
        s = OM.LayerState()
        s.p_a, s.R_a = st.p_a, R_a
        v, info = OM.velocity_rr(W, spec, x1, cond, sig[1], prof, s)
        assert info.accepted
        return v - vf

    ref = skip_with(st.R_a)
    for what, R_a in (("zero R_a", np.zeros_like(st.R_a)), ("p_a for R_a", st.p_a)):
        moved = _rel(skip_with(R_a), ref)
        assert moved >= 10 * 2e-2, (what, moved)
