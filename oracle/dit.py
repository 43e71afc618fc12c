"""Oracle DiT denoiser (float64) — test infrastructure, not the product path.

The paper builds on DiT-style denoisers (related work and method section, the
"DiT forward execution" loop) but does not define the network, so the model
below is the synthetic joint video/action DiT used throughout this
repository.  Every choice it makes where the paper is silent is one of the
readings listed in the design notes (adaLN-style shift/scale/gate modulation,
LayerNorm without affine, QK-RMSNorm, tanh GELU, sinusoidal timestep and
position features, token order [video | action | observation]).

Parity status:
  * layer_norm, rms_norm, gelu_tanh, attention: pinned against PyTorch CPU
    float64 library routines and brute-force loops (tests/test_oracle_dit.py).
  * timestep_features, positional_embedding: pinned by closed-form values.
  * dit_layer: pinned against an independent composition of PyTorch library
    ops, and by the zero-gate identity.
  * the network as a whole: parity unpinned by the paper (no printed
    activations exist); pinned only through its pieces.

Conventions: a Linear computes y = x @ W + b with W stored as [in, out].
The trajectory of one sample is the flat vector
[video (Nv x Cv) | action (Na x A)]; the hidden sequence has T = Nv + Na + No
rows in the order [video | action | observation].
"""
from __future__ import annotations

import numpy as np

f64 = np.float64


def as64(a) -> np.ndarray:
    return np.asarray(a, dtype=f64)


# --------------------------------------------------------------------------
# elementwise pieces
# --------------------------------------------------------------------------
def silu(x):
    x = as64(x)
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    """GELU, tanh approximation: x/2 * (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    x = as64(x)
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * (x * x * x))))


def layer_norm(x, eps):
    """LayerNorm over the last axis, biased variance, no affine parameters."""
    x = as64(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x, eps):
    """x / sqrt(mean(x^2) + eps) over the last axis."""
    x = as64(x)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)


def softmax(s, axis=-1):
    s = as64(s)
    m = s.max(axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)


# --------------------------------------------------------------------------
# conditioning and token embedding
# --------------------------------------------------------------------------
def timestep_features(sigma, dim: int = 256):
    """Sinusoidal features of t = 1000*sigma: [cos(t f_i), sin(t f_i)],
    f_i = 10000^(-i/(dim/2)), i = 0 .. dim/2-1."""
    half = dim // 2
    t = 1000.0 * f64(sigma)
    f = 10000.0 ** (-np.arange(half, dtype=f64) / half)
    return np.concatenate([np.cos(t * f), np.sin(t * f)])


def cond_vector(W, sigma):
    """c = SiLU(e(t) @ W1 + b1) @ W2 + b2, a vector of size D."""
    e = timestep_features(sigma, as64(W["t_w1"]).shape[0])
    a = silu(e @ as64(W["t_w1"]) + as64(W["t_b1"]))
    return a @ as64(W["t_w2"]) + as64(W["t_b2"])


def layer_modulation(W, l: int, c):
    """(shift1, scale1, gate1, shift2, scale2, gate2) of layer l, each [D]."""
    m = silu(c) @ as64(W[f"l{l}.mod_w"]) + as64(W[f"l{l}.mod_b"])
    return np.split(m, 6)


def final_modulation(W, c):
    """(shift, scale) of the final layer, each [D]."""
    m = silu(c) @ as64(W["f_mod_w"]) + as64(W["f_mod_b"])
    return np.split(m, 2)


def positional_embedding(T: int, D: int):
    """PE[p, i] = sin(p w_i) for i < D/2, cos(p w_{i-D/2}) otherwise,
    w_i = 10000^(-i/(D/2)); p is the joint row index."""
    half = D // 2
    p = np.arange(T, dtype=f64)[:, None]
    w = 10000.0 ** (-np.arange(half, dtype=f64) / half)
    return np.concatenate([np.sin(p * w), np.cos(p * w)], axis=1)


def split_trajectory(spec, x):
    """[B, traj] -> video [B, Nv, Cv], action [B, Na, A]."""
    x = as64(x).reshape(spec.B, spec.traj)
    nv = spec.Nv * spec.Cv
    return x[:, :nv].reshape(spec.B, spec.Nv, spec.Cv), x[:, nv:].reshape(spec.B, spec.Na, spec.A)


def join_trajectory(spec, xv, xa):
    return np.concatenate([as64(xv).reshape(spec.B, -1), as64(xa).reshape(spec.B, -1)], axis=1)


def embed_tokens(W, spec, x, cond):
    """h0 = [xv W_v + b_v ; xa W_a + b_a ; co W_o + b_o] + PE, shape [B, T, D]."""
    xv, xa = split_trajectory(spec, x)
    co = as64(cond).reshape(spec.B, spec.No, spec.Co)
    hv = xv @ as64(W["in_wv"]) + as64(W["in_bv"])
    ha = xa @ as64(W["in_wa"]) + as64(W["in_ba"])
    ho = co @ as64(W["in_wo"]) + as64(W["in_bo"])
    h = np.concatenate([hv, ha, ho], axis=1)
    return h + positional_embedding(spec.T, spec.D)[None]


# --------------------------------------------------------------------------
# transformer layer
# --------------------------------------------------------------------------
# Worker threads for the loop over (sample, head) pairs in `attention`.  The
# pairs are independent problems, so the result is the same for any count;
# long oracle runs (the full-size chunk fixtures) raise it to the core count.
ATTENTION_THREADS = 1


def attention(q, k, v):
    """Bidirectional softmax attention over all rows, q/k/v [..., T, dh].

    Each (sample, head) pair is an independent attention problem, so they are
    taken one at a time: the T x T score matrix of a single head is the
    largest array held (about 0.8 GB in float64 at T = 10176), where all heads
    at once would need tens of GB.  The result does not depend on this loop.
    """
    q, k, v = as64(q), as64(k), as64(v)
    out = np.empty(q.shape[:-1] + (v.shape[-1],), f64)
    scale = 1.0 / np.sqrt(q.shape[-1])

    def one(idx):
        s = (q[idx] @ k[idx].T) * scale
        out[idx] = softmax(s, axis=-1) @ v[idx]

    pairs = list(np.ndindex(*q.shape[:-2]))
    if ATTENTION_THREADS > 1 and len(pairs) > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(ATTENTION_THREADS) as ex:
            list(ex.map(one, pairs))
    else:
        for idx in pairs:
            one(idx)
    return out


def qkv_heads(W, spec, l, u):
    """Project u [B, T, D] to per-head q, k, v [B, H, T, dh] (after QK-norm)."""
    B, T, D, H, dh = u.shape[0], u.shape[1], spec.D, spec.H, spec.dh
    qkv = u @ as64(W[f"l{l}.qkv_w"]) + as64(W[f"l{l}.qkv_b"])
    q, k, v = qkv[..., :D], qkv[..., D:2 * D], qkv[..., 2 * D:]

    def heads(a):
        return a.reshape(B, T, H, dh).transpose(0, 2, 1, 3)

    q, k, v = heads(q), heads(k), heads(v)
    if spec.qk_norm:
        q = rms_norm(q, spec.ln_eps) * as64(W[f"l{l}.q_g"])
        k = rms_norm(k, spec.ln_eps) * as64(W[f"l{l}.k_g"])
    return q, k, v


def dit_layer(W, spec, l: int, h, c):
    """One DiT block with adaLN modulation (see module header)."""
    h = as64(h)
    sh1, sc1, g1, sh2, sc2, g2 = layer_modulation(W, l, c)
    u = layer_norm(h, spec.ln_eps) * (1.0 + sc1) + sh1
    q, k, v = qkv_heads(W, spec, l, u)
    o = attention(q, k, v)  # [B, H, T, dh]
    o = o.transpose(0, 2, 1, 3).reshape(h.shape)
    h = h + g1 * (o @ as64(W[f"l{l}.proj_w"]) + as64(W[f"l{l}.proj_b"]))
    u = layer_norm(h, spec.ln_eps) * (1.0 + sc2) + sh2
    z = gelu_tanh(u @ as64(W[f"l{l}.fc1_w"]) + as64(W[f"l{l}.fc1_b"]))
    return h + g2 * (z @ as64(W[f"l{l}.fc2_w"]) + as64(W[f"l{l}.fc2_b"]))


def dit_layer_rows(W, spec, l: int, h, c, rows):
    """dit_layer evaluated only at the given rows (indices into B*T).

    Keys and values still come from every row of the same sample, so the
    result equals dit_layer(...)[rows]; used for full-size spot checks.
    """
    h = as64(h)
    B, T, D = h.shape
    sh1, sc1, g1, sh2, sc2, g2 = layer_modulation(W, l, c)
    u = layer_norm(h, spec.ln_eps) * (1.0 + sc1) + sh1
    rows = np.asarray(rows)
    out = np.empty((len(rows), D), f64)
    for b in np.unique(rows // T):
        sel = np.nonzero(rows // T == b)[0]
        r = rows[sel] % T
        qkv_all = u[b] @ as64(W[f"l{l}.qkv_w"]) + as64(W[f"l{l}.qkv_b"])
        H, dh = spec.H, spec.dh
        q = qkv_all[r, :D].reshape(len(r), H, dh).transpose(1, 0, 2)
        k = qkv_all[:, D:2 * D].reshape(T, H, dh).transpose(1, 0, 2)
        v = qkv_all[:, 2 * D:].reshape(T, H, dh).transpose(1, 0, 2)
        if spec.qk_norm:
            q = rms_norm(q, spec.ln_eps) * as64(W[f"l{l}.q_g"])
            k = rms_norm(k, spec.ln_eps) * as64(W[f"l{l}.k_g"])
        o = attention(q, k, v).transpose(1, 0, 2).reshape(len(r), D)
        hr = h[b, r] + g1 * (o @ as64(W[f"l{l}.proj_w"]) + as64(W[f"l{l}.proj_b"]))
        u2 = layer_norm(hr, spec.ln_eps) * (1.0 + sc2) + sh2
        z = gelu_tanh(u2 @ as64(W[f"l{l}.fc1_w"]) + as64(W[f"l{l}.fc1_b"]))
        out[sel] = hr + g2 * (z @ as64(W[f"l{l}.fc2_w"]) + as64(W[f"l{l}.fc2_b"]))
    return out


def final_layer(W, spec, h, c):
    """Final LN + modulation and per-branch output heads -> velocity [B, traj]."""
    sh, sc = final_modulation(W, c)
    u = layer_norm(as64(h), spec.ln_eps) * (1.0 + sc) + sh
    uv = u[:, :spec.Nv]
    ua = u[:, spec.Nv:spec.Nv + spec.Na]
    vv = uv @ as64(W["out_wv"]) + as64(W["out_bv"])
    va = ua @ as64(W["out_wa"]) + as64(W["out_ba"])
    return join_trajectory(spec, vv, va)


def run_layers(W, spec, h, c, lo: int, hi: int):
    for l in range(lo, hi):
        h = dit_layer(W, spec, l, h, c)
    return h


def velocity(W, spec, x, cond, sigma):
    """Full (no reuse) denoiser prediction v(x, sigma, cond), [B, traj]."""
    c = cond_vector(W, sigma)
    h = embed_tokens(W, spec, x, cond)
    h = run_layers(W, spec, h, c, 0, spec.L)
    return final_layer(W, spec, h, c)


def hidden_after(W, spec, x, cond, sigma, n_layers: int):
    """h_n: hidden state after the first n layers (h_0 = DiT input)."""
    c = cond_vector(W, sigma)
    h = embed_tokens(W, spec, x, cond)
    return run_layers(W, spec, h, c, 0, n_layers)
