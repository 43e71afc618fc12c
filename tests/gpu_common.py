"""Helpers shared by the GPU parity tests (device plumbing only)."""
import numpy as np
import pytest
import torch

from oracle import method as OM
from synth import get_workload, make_weights


# Tolerance of the bf16 single-layer update parity (max |got - ref| / max |ref|
# on h_{l+1} - h_l).  The update passes four bf16 roundings of activations
# (LayerNorm output, q/k/v, the attention probabilities and output, the MLP
# hidden), each a relative 2^-9 on an element; the measured errors are
# 2e-3 to 5e-3.  tests/test_oracle_sensitivity.py pins that removing
# attention, the MLP or the QKV projection moves this quantity by at least
# ten times the tolerance, and a uniform softmax by at least five times.
BF16_UPDATE_TOL = 1e-2


def device():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    return torch.device("cuda:0")


def to_dev(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)


def rel_err(got, ref):
    """max_i |got_i - ref_i| / max_i |ref_i| (the parity measure)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))


def rr_of(spec, mode, single=False, **kw):
    """(GPU profile, oracle profile) pair with the workload's RR constants;
    single = one branch over all rows (independent execution)."""
    from paper_2609_34608_amd import runtime as R, _lib as L
    q, s, e = spec.rr_bounds
    p = dict(alpha_min=spec.rr_alpha_min, alpha_max=spec.rr_alpha_max, eps=spec.rr_eps,
             gamma_cos=spec.rr_gamma_cos, gamma_fit=spec.rr_gamma_fit)
    p.update(kw)
    # the device compares in float32 thresholds; give the oracle the same values
    po = {k: float(np.float32(v)) for k, v in p.items()}
    branches = L.WAM_RR_SINGLE if single else L.WAM_RR_JOINT
    return (R.rr_profile(q, s, e, mode, branches=branches, **p),
            OM.RRProfile(q, s, e, mode=mode, single=single, **po))


def f32_sigmas(K, shift=1.0):
    """Schedule as the device sees it (float32), widened for the oracle."""
    return OM.flow_schedule(K, shift).astype(np.float32).astype(np.float64)


_MODELS = {}


def model_for(name, dev, own_stream=False, **wkw):
    """Cached (spec, weights, WamModel) per workload, weight options and stream."""
    from paper_2609_34608_amd import runtime as R
    key = (name, own_stream, tuple(sorted(wkw.items())))
    if key not in _MODELS:
        spec = get_workload(name)
        if "B" in wkw:
            spec = spec.replace(B=wkw["B"])
        W = make_weights(spec, **{k: v for k, v in wkw.items() if k != "B"})
        m = R.WamModel(R.config_of(spec), W, device=dev, own_stream=own_stream)
        _MODELS[key] = (spec, W, m)
    return _MODELS[key]


def layer_update_errors(m, W, spec, k, x0, cond, sigma, layers, dev):
    """Parity of single DiT layers, teacher-forced: for each layer l, the
    device's update h_{l+1} - h_l against the oracle's dit_layer(h_l) - h_l on
    the device's own h_l, every row and column.  Returns [(l, rel_err)]."""
    from oracle import dit as OD
    c = OD.cond_vector(W, sigma)
    xd, cd = to_dev(x0, dev), to_dev(cond, dev)
    out = []
    h_in = m.hidden(k, xd, cd, min(layers)).cpu().numpy()
    for l in range(min(layers), max(layers) + 1):
        h_out = m.hidden(k, xd, cd, l + 1).cpu().numpy()
        if l in layers:
            ref = OD.dit_layer(W, spec, l, h_in, c)
            out.append((l, rel_err(h_out - h_in, ref - h_in)))
        h_in = h_out
    return out
