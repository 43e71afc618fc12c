"""Pins of the oracle DiT pieces against library routines and closed forms.

The paper does not define the denoiser network, so these tests tie each piece
of the oracle's synthetic DiT to an independent implementation: PyTorch CPU
float64 library routines (layer_norm, rms_norm, gelu, scaled_dot_product_attention,
linear, silu), brute-force loops on tiny inputs, and closed-form values.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import dit
from synth import get_workload, make_weights, make_initial_noise, make_observations

@pytest.fixture(scope="module", autouse=True)
def float64_default():
    """float64 torch references in this module only (restored afterwards, so
    that tensors created by later test modules keep torch's float32 default)."""
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(prev)


def t64(a):
    return torch.from_numpy(np.asarray(a, np.float64))


@pytest.fixture(scope="module")
def rng():
    return np.random.default_rng(1234)


def test_layer_norm_matches_torch(rng):
    x = rng.standard_normal((3, 5, 40)) * 3 + 1
    got = dit.layer_norm(x, 1e-6)
    ref = Fn.layer_norm(t64(x), (40,), eps=1e-6).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_rms_norm_matches_torch(rng):
    x = rng.standard_normal((4, 7, 32))
    got = dit.rms_norm(x, 1e-6)
    ref = Fn.rms_norm(t64(x), (32,), eps=1e-6).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_gelu_tanh_matches_torch(rng):
    x = rng.standard_normal(1000) * 4
    got = dit.gelu_tanh(x)
    ref = Fn.gelu(t64(x), approximate="tanh").numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_silu_matches_torch(rng):
    x = rng.standard_normal(100) * 5
    np.testing.assert_allclose(dit.silu(x), Fn.silu(t64(x)).numpy(), rtol=1e-13)


def test_attention_matches_sdpa_and_brute_force(rng):
    B, H, T, dh = 2, 3, 9, 8
    q, k, v = (rng.standard_normal((B, H, T, dh)) for _ in range(3))
    got = dit.attention(q, k, v)
    ref = Fn.scaled_dot_product_attention(t64(q), t64(k), t64(v)).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)
    # brute force: explicit loops over query, key and feature
    bf = np.zeros_like(got)
    for b in range(B):
        for h in range(H):
            for i in range(T):
                s = [sum(q[b, h, i, d] * k[b, h, j, d] for d in range(dh)) / math.sqrt(dh)
                     for j in range(T)]
                m = max(s)
                w = [math.exp(x - m) for x in s]
                z = sum(w)
                for d in range(dh):
                    bf[b, h, i, d] = sum(w[j] * v[b, h, j, d] for j in range(T)) / z
    np.testing.assert_allclose(got, bf, rtol=1e-11, atol=1e-12)


def test_attention_is_bidirectional(rng):
    """No mask: the first query sees the last key."""
    T, dh = 6, 4
    q = np.zeros((1, 1, T, dh))
    k = np.zeros((1, 1, T, dh))
    v = np.zeros((1, 1, T, dh))
    k[0, 0, -1, 0] = 50.0
    q[0, 0, 0, 0] = 1.0
    v[0, 0, -1, 1] = 7.0
    o = dit.attention(q, k, v)
    assert o[0, 0, 0, 1] > 6.9


def test_timestep_features_closed_form():
    e0 = dit.timestep_features(0.0)
    np.testing.assert_array_equal(e0, np.r_[np.ones(128), np.zeros(128)])
    e = dit.timestep_features(0.001)  # t = 1
    for i in (0, 1, 64, 127):
        f = 10000.0 ** (-i / 128)
        assert e[i] == pytest.approx(math.cos(f), abs=1e-15)
        assert e[128 + i] == pytest.approx(math.sin(f), abs=1e-15)


def test_positional_embedding_brute_force():
    T, D = 11, 12
    pe = dit.positional_embedding(T, D)
    for p in range(T):
        for i in range(D):
            if i < D // 2:
                ref = math.sin(p * 10000.0 ** (-i / (D // 2)))
            else:
                ref = math.cos(p * 10000.0 ** (-(i - D // 2) / (D // 2)))
            assert pe[p, i] == pytest.approx(ref, abs=1e-14)
    np.testing.assert_array_equal(pe[0], np.r_[np.zeros(D // 2), np.ones(D // 2)])


def _torch_layer(W, spec, l, h, c):
    """Independent composition of PyTorch library ops for one DiT block."""
    D, H, dh = spec.D, spec.H, spec.dh
    h = t64(h)
    mod = Fn.linear(Fn.silu(t64(c)), t64(W[f"l{l}.mod_w"]).T, t64(W[f"l{l}.mod_b"]))
    sh1, sc1, g1, sh2, sc2, g2 = torch.chunk(mod, 6)
    u = Fn.layer_norm(h, (D,), eps=spec.ln_eps) * (1 + sc1) + sh1
    qkv = Fn.linear(u, t64(W[f"l{l}.qkv_w"]).T, t64(W[f"l{l}.qkv_b"]))
    q, k, v = torch.chunk(qkv, 3, dim=-1)
    B, T = h.shape[:2]
    q = q.reshape(B, T, H, dh).transpose(1, 2)
    k = k.reshape(B, T, H, dh).transpose(1, 2)
    v = v.reshape(B, T, H, dh).transpose(1, 2)
    q = Fn.rms_norm(q, (dh,), weight=t64(W[f"l{l}.q_g"]), eps=spec.ln_eps)
    k = Fn.rms_norm(k, (dh,), weight=t64(W[f"l{l}.k_g"]), eps=spec.ln_eps)
    o = Fn.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B, T, D)
    h = h + g1 * Fn.linear(o, t64(W[f"l{l}.proj_w"]).T, t64(W[f"l{l}.proj_b"]))
    u = Fn.layer_norm(h, (D,), eps=spec.ln_eps) * (1 + sc2) + sh2
    z = Fn.gelu(Fn.linear(u, t64(W[f"l{l}.fc1_w"]).T, t64(W[f"l{l}.fc1_b"])), approximate="tanh")
    return (h + g2 * Fn.linear(z, t64(W[f"l{l}.fc2_w"]).T, t64(W[f"l{l}.fc2_b"]))).numpy()


@pytest.fixture(scope="module")
def tiny():
    spec = get_workload("tiny").replace(B=2)
    W = make_weights(spec, bias_std=0.05, gain_std=0.2, weight_std=0.08)
    return spec, W


def test_dit_layer_matches_torch_composition(tiny, rng):
    spec, W = tiny
    h = rng.standard_normal((spec.B, spec.T, spec.D))
    c = dit.cond_vector(W, 0.37)
    for l in range(spec.L):
        np.testing.assert_allclose(dit.dit_layer(W, spec, l, h, c), _torch_layer(W, spec, l, h, c),
                                   rtol=1e-10, atol=1e-11)


def test_cond_and_embedding_match_torch(tiny):
    spec, W = tiny
    sigma = 0.61
    e = t64(dit.timestep_features(sigma))
    c_ref = Fn.linear(Fn.silu(Fn.linear(e, t64(W["t_w1"]).T, t64(W["t_b1"]))),
                      t64(W["t_w2"]).T, t64(W["t_b2"])).numpy()
    np.testing.assert_allclose(dit.cond_vector(W, sigma), c_ref, rtol=1e-12, atol=1e-13)

    x = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    h0 = dit.embed_tokens(W, spec, x, cond)
    nv = spec.Nv * spec.Cv
    xv = t64(x[:, :nv]).reshape(spec.B, spec.Nv, spec.Cv)
    xa = t64(x[:, nv:]).reshape(spec.B, spec.Na, spec.A)
    ref = torch.cat([Fn.linear(xv, t64(W["in_wv"]).T, t64(W["in_bv"])),
                     Fn.linear(xa, t64(W["in_wa"]).T, t64(W["in_ba"])),
                     Fn.linear(t64(cond), t64(W["in_wo"]).T, t64(W["in_bo"]))], dim=1)
    ref = ref + t64(dit.positional_embedding(spec.T, spec.D))
    np.testing.assert_allclose(h0, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_final_layer_matches_torch_and_ignores_obs_rows(tiny, rng):
    spec, W = tiny
    h = rng.standard_normal((spec.B, spec.T, spec.D))
    c = dit.cond_vector(W, 0.2)
    v = dit.final_layer(W, spec, h, c)
    mod = Fn.linear(Fn.silu(t64(c)), t64(W["f_mod_w"]).T, t64(W["f_mod_b"]))
    sh, sc = torch.chunk(mod, 2)
    u = Fn.layer_norm(t64(h), (spec.D,), eps=spec.ln_eps) * (1 + sc) + sh
    vv = Fn.linear(u[:, :spec.Nv], t64(W["out_wv"]).T, t64(W["out_bv"]))
    va = Fn.linear(u[:, spec.Nv:spec.Nv + spec.Na], t64(W["out_wa"]).T, t64(W["out_ba"]))
    ref = torch.cat([vv.reshape(spec.B, -1), va.reshape(spec.B, -1)], 1).numpy()
    np.testing.assert_allclose(v, ref, rtol=1e-12, atol=1e-13)
    h2 = h.copy()
    h2[:, spec.Nv + spec.Na:] += 5.0
    np.testing.assert_array_equal(dit.final_layer(W, spec, h2, c), v)


def test_zero_gates_make_layer_identity(tiny, rng):
    spec, W = tiny
    W0 = dict(W)
    W0["l0.mod_w"] = np.zeros_like(W["l0.mod_w"])
    W0["l0.mod_b"] = np.zeros_like(W["l0.mod_b"])
    h = rng.standard_normal((spec.B, spec.T, spec.D))
    np.testing.assert_array_equal(dit.dit_layer(W0, spec, 0, h, dit.cond_vector(W, 0.5)), h)


def test_layer_rows_equals_full_layer(tiny, rng):
    spec, W = tiny
    h = rng.standard_normal((spec.B, spec.T, spec.D))
    c = dit.cond_vector(W, 0.8)
    full = dit.dit_layer(W, spec, 1, h, c).reshape(-1, spec.D)
    rows = np.array([0, 5, spec.T - 1, spec.T, spec.T + 17, 2 * spec.T - 1])
    np.testing.assert_allclose(dit.dit_layer_rows(W, spec, 1, h, c, rows), full[rows],
                               rtol=1e-12, atol=1e-12)


def test_token_order_and_position_embedding_enter_velocity(tiny):
    """Swapping two video tokens changes the prediction only through the
    position embedding; without it the head is permutation-equivariant."""
    spec, W = tiny
    x = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    v = dit.velocity(W, spec, x, cond, 0.5)
    assert v.shape == (spec.B, spec.traj)
    xs = x.copy().reshape(spec.B, -1)
    Cv = spec.Cv
    xs[:, 0:Cv], xs[:, Cv:2 * Cv] = x[:, Cv:2 * Cv].copy(), x[:, 0:Cv].copy()
    vs = dit.velocity(W, spec, xs, cond, 0.5)
    assert not np.allclose(vs[:, 0:Cv], v[:, Cv:2 * Cv])
