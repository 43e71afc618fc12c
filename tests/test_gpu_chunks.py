"""GPU parity of whole native action chunks at the mid (B = 4) and large
(T = 10176) workloads, through the C ABI.

The expected values are the float64 oracle's native replan (Sec. 3.4 with
no retained state: K Euler steps from the seeded noise under the first
observation; K = 16 and 20 as the workloads state), written by
tests/golden/make_chunk_goldens.py, which calls only `oracle/` and `synth/`.
The device runs the same seeded inputs step by step; the action rows after
every step are compared (printed), the final chunk and a spread of final
video tokens are gated at the bf16 tolerance 2e-2 (max |got - ref| /
max |ref|).  These chunks are dominated by the embedding and the output
head; the kernels inside each layer are checked on their own by the
layer-update tests.
"""
import os

import numpy as np
import pytest

from oracle import method as OM
from synth import make_initial_noise, make_observations
from gpu_common import device, to_dev, rel_err, f32_sigmas, model_for

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def dev():
    return device()


@pytest.mark.parametrize("name", ["mid", "large"])
def test_native_chunk_matches_oracle_fixture(dev, name):
    path = os.path.join(GOLDEN, f"native_chunk_{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"fixture {os.path.basename(path)} not written yet (tests/golden/make_chunk_goldens.py)")
    fx = np.load(path)
    spec, W, m = model_for(name, dev)
    sig = f32_sigmas(spec.K)
    np.testing.assert_array_equal(sig, fx["sigmas"])
    assert fx["action_per_step"].shape == (spec.K, spec.B, spec.Na, spec.A)
    m.set_schedule(sig)
    x = to_dev(make_initial_noise(spec), dev)
    cond = to_dev(make_observations(spec, 0)[0], dev)
    errs = []
    for k in range(spec.K):
        m.continue_(k, k + 1, x, cond)
        errs.append(rel_err(OM.action_chunk(spec, x.cpu().numpy()), fx["action_per_step"][k]))
    print(f"{name} action rows rel err per step: " + " ".join(f"{e:.2e}" for e in errs))
    xf = x.cpu().numpy()
    ea = rel_err(OM.action_chunk(spec, xf), fx["action_per_step"][-1])
    xv = xf[:, :spec.Nv * spec.Cv].reshape(spec.B, spec.Nv, spec.Cv)
    ev = rel_err(xv[:, fx["video_index"]], fx["video_rows"])
    print(f"{name} final action chunk rel err {ea:.3e}, video rows {ev:.3e}")
    assert ea <= BF16_TOL
    assert ev <= BF16_TOL
