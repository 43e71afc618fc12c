"""GPU parity of the bf16 attention kernels through the C ABI.

Four kernels exist in bf16 mode: the online softmax with a running max, and
(with QK-norm, when the gains bound every score) a fixed softmax reference
equal to that bound, in a software-pipelined form, a plain loop (on these
short grids with the keys split over two wave groups, including groups left
without a key tile), and a ping-pong form whose two wave groups alternate
MFMA and exp2 phases.  Each must match the float64
oracle at every sequence length class: one key tile, an exact multiple of
the tile, a one-key tail, and several tiles with a ragged tail.  Tolerance:
2e-2 (bf16 contractions), max |got-ref| / max |ref|.
"""
import numpy as np
import pytest

from oracle import dit as OD
from synth import get_workload, make_weights, make_initial_noise, make_observations
from gpu_common import device, to_dev, rel_err, f32_sigmas, layer_update_errors, BF16_UPDATE_TOL

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


@pytest.fixture(scope="module")
def dev():
    return device()


# (Nv, Na, No) -> T = 40 (one tile), 64 (exact), 65 (one-key tail), 200, 333
_LENGTHS = [(24, 8, 8), (40, 16, 8), (41, 16, 8), (160, 32, 8), (288, 32, 13)]


def _spec(Nv, Na, No, L=2):
    return get_workload("small").replace(L=L, D=128, H=2, F=512, Nv=Nv, Na=Na, No=No, B=2)


_VARIANTS = ["RUNNING_MAX", "BOUNDED", "PINGPONG", "PLAIN"]


@pytest.mark.parametrize("variant", _VARIANTS)
@pytest.mark.parametrize("lengths", _LENGTHS)
def test_bf16_attention_lengths_match_oracle(dev, lengths, variant):
    from paper_2609_34608_amd import runtime as R, _lib as L
    spec = _spec(*lengths)
    W = make_weights(spec, bias_std=0.02, gain_std=0.1)
    m = R.WamModel(R.config_of(spec), W, device=dev)
    m.set_option(L.WAM_OPT_ATTENTION, getattr(L, "WAM_ATTN_" + variant))
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    for k in (0, 6):
        for l, e in layer_update_errors(m, W, spec, k, x0, cond, sig[k], [0, 1], dev):
            print(f"T={spec.T} {variant} step {k} layer {l} update rel err {e:.3e}")
            assert e <= BF16_UPDATE_TOL, (spec.T, k, l, e)
        v, _ = m.velocity(k, to_dev(x0, dev), to_dev(cond, dev))
        ref = OD.velocity(W, spec, x0, cond, sig[k])
        e = rel_err(v.cpu().numpy(), ref)
        print(f"T={spec.T} {variant} step {k} velocity rel err {e:.3e}")
        assert e <= BF16_TOL, (spec.T, k, e)
    m.close()


def test_attention_kernels_agree(dev):
    """The kernels differ only in the bf16 rounding of P (and the bounded
    forms not at all from each other): their layer updates agree far inside
    the bf16 tolerance."""
    from paper_2609_34608_amd import runtime as R, _lib as L
    spec = _spec(288, 32, 13, L=1)
    W = make_weights(spec, bias_std=0.02, gain_std=0.1)
    m = R.WamModel(R.config_of(spec), W, device=dev)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    outs = {}
    for v in _VARIANTS:
        m.set_option(L.WAM_OPT_ATTENTION, getattr(L, "WAM_ATTN_" + v))
        outs[v] = m.hidden(2, to_dev(x0, dev), to_dev(cond, dev), 1).cpu().numpy()
    h0 = m.hidden(2, to_dev(x0, dev), to_dev(cond, dev), 0).cpu().numpy()
    e = rel_err(outs["BOUNDED"] - h0, outs["RUNNING_MAX"] - h0)
    print(f"bounded vs running-max layer update rel diff {e:.3e}")
    assert e <= 5e-3
    # the pipelined and ping-pong kernels sum the same bf16 P in the same
    # MFMA order; the plain form splits the keys of this short grid over two
    # wave groups, whose partial sums differ from the single sum by fp32
    # rounding only
    np.testing.assert_array_equal(outs["BOUNDED"], outs["PINGPONG"])
    e2 = rel_err(outs["PLAIN"] - h0, outs["BOUNDED"] - h0)
    print(f"key-split vs single-group layer update rel diff {e2:.3e}")
    assert e2 <= 1e-3
    m.close()


def test_large_gains_fall_back_to_running_max(dev):
    """Gains large enough that the score bound exceeds the fixed-reference
    limit: the library takes the running-max kernel, even when a bounded
    kernel is asked for, and still matches."""
    from paper_2609_34608_amd import runtime as R, _lib as L
    spec = _spec(160, 32, 8, L=1)
    W = make_weights(spec, bias_std=0.02)
    for l in range(spec.L):
        W[f"l{l}.q_g"][:] = 2.5
        W[f"l{l}.k_g"][:] = 2.2
    m = R.WamModel(R.config_of(spec), W, device=dev)
    m.set_option(L.WAM_OPT_ATTENTION, L.WAM_ATTN_PINGPONG)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    v, _ = m.velocity(3, to_dev(x0, dev), to_dev(cond, dev))
    ref = OD.velocity(W, spec, x0, cond, sig[3])
    e = rel_err(v.cpu().numpy(), ref)
    print(f"gains 2.5 x 2.2 velocity rel err {e:.3e}")
    assert e <= BF16_TOL
    m.close()


@pytest.mark.parametrize("variant", ["RUNNING_MAX", "BOUNDED", "PINGPONG"])
def test_large_forced_forms_sampled_rows(dev, variant):
    """The forms that the automatic choice does not take at the 16-frame
    shape (T = 10176, 24 heads), run there at their own tile shapes: one
    layer's update on sampled rows against the oracle."""
    from paper_2609_34608_amd import _lib as L
    from gpu_common import model_for
    spec, W, m = model_for("large", dev)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    k = 3
    c = OD.cond_vector(W, sig[k])
    rows = np.unique(np.r_[0, spec.M - 1, spec.T - 1, spec.Nv, spec.Nv + spec.Na,
                           np.random.default_rng(7).integers(0, spec.M, 10)])
    m.set_option(L.WAM_OPT_ATTENTION, getattr(L, "WAM_ATTN_" + variant))
    try:
        h_in = m.hidden(k, to_dev(x0, dev), to_dev(cond, dev), 0).cpu().numpy()
        h_out = m.hidden(k, to_dev(x0, dev), to_dev(cond, dev), 1).cpu().numpy().reshape(-1, spec.D)
    finally:
        m.set_option(L.WAM_OPT_ATTENTION, L.WAM_ATTN_AUTO)
    ref = OD.dit_layer_rows(W, spec, 0, h_in, c, rows)
    h0 = h_in.reshape(-1, spec.D)[rows]
    e = rel_err(h_out[rows] - h0, ref - h0)
    print(f"large {variant} layer 0 sampled-row update rel err {e:.3e}")
    assert e <= BF16_TOL, e


@pytest.mark.parametrize("shape", [dict(Nv=0, Na=16, No=8), dict(Nv=40, Na=16, No=0), dict(Nv=24, Na=1, No=3),
                                   dict(Nv=24, Na=8, No=3, B=16), dict(Nv=63, Na=16, No=1)])
def test_bf16_degenerate_shapes_match_oracle(dev, shape):
    """The bf16 path (GEMM planner, attention forms, final heads) on the
    degenerate shapes: no video tokens, no observation tokens, a one-slot
    action chunk, the maximum batch, and a ragged sequence; the velocity of
    two steps within the bf16 tolerance."""
    from paper_2609_34608_amd import runtime as R
    B = shape.pop("B", 2)
    spec = _spec(**shape).replace(B=B)
    W = make_weights(spec, bias_std=0.02, gain_std=0.1)
    m = R.WamModel(R.config_of(spec), W, device=dev)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    for k in (0, 5):
        for l, e in layer_update_errors(m, W, spec, k, x0, cond, sig[k], [0, 1], dev):
            print(f"{shape} B={B} T={spec.T} step {k} layer {l} update rel err {e:.3e}")
            assert e <= BF16_UPDATE_TOL, (k, l, e)
        v, _ = m.velocity(k, to_dev(x0, dev), to_dev(cond, dev))
        ref = OD.velocity(W, spec, x0, cond, sig[k])
        e = rel_err(v.cpu().numpy(), ref)
        print(f"{shape} B={B} T={spec.T} step {k} velocity rel err {e:.3e}")
        assert e <= BF16_TOL, (k, e)
    m.close()


@pytest.mark.parametrize("D,H", [(192, 3), (1088, 17)])
def test_bf16_odd_head_counts_match_oracle(dev, D, H):
    """bf16 mode with an odd number of heads: the QKV output width 192 H is a
    multiple of 64 but not of 128 (its own GEMM tile); D not a multiple of 256
    takes the generic LayerNorm, and D = 1088 the row-wise final layer."""
    from paper_2609_34608_amd import runtime as R
    spec = get_workload("small").replace(L=1, D=D, H=H, F=4 * D, Nv=40, Na=16, No=8, B=2)
    W = make_weights(spec, bias_std=0.02, gain_std=0.1)
    m = R.WamModel(R.config_of(spec), W, device=dev)
    sig = f32_sigmas(spec.K)
    m.set_schedule(sig)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    for k in (0, 5):
        for l, e in layer_update_errors(m, W, spec, k, x0, cond, sig[k], [0], dev):
            print(f"D={D} H={H} step {k} layer {l} update rel err {e:.3e}")
            assert e <= BF16_UPDATE_TOL, (k, l, e)
        v, _ = m.velocity(k, to_dev(x0, dev), to_dev(cond, dev))
        ref = OD.velocity(W, spec, x0, cond, sig[k])
        e = rel_err(v.cpu().numpy(), ref)
        print(f"D={D} H={H} step {k} velocity rel err {e:.3e}")
        assert e <= BF16_TOL, (k, e)
    m.close()
