"""Seeded input generators (CPU): the bf16 rounding that both the oracle and
the device path see, against PyTorch's own float32 -> bfloat16 conversion
(round to nearest, ties to even)."""
import numpy as np
import torch

from synth.gen import bf16_round


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.standard_normal(200_000).astype(np.float32) * 0.02,
        rng.standard_normal(1000).astype(np.float32) * 1e30,
        np.array([0.0, -0.0, 1e-45, -1e-45, 3.0e38, -3.0e38, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8],
                 np.float32),
    ])
    got = bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_bf16_round_ties_to_even():
    # 1 + 2^-8 lies halfway between bf16 neighbours 1 and 1 + 2^-7: the even one (1) wins;
    # 1 + 3 * 2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: 1 + 2^-6 is even
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], np.float32)
    np.testing.assert_array_equal(bf16_round(x), np.array([1.0, 1.0 + 2.0 ** -6], np.float32))
