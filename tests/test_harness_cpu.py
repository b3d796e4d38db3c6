"""CPU checks of the parity harness's own arithmetic (no GPU)."""
import numpy as np
import torch

from tests.harness import bf16_round, error_stats


def test_bf16_round_matches_torch_on_float32_values():
    """For float32-representable inputs, rounding straight from float64 agrees with PyTorch's
    float32 -> bfloat16 round-to-nearest-even conversion."""
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000) * s for s in (1e-3, 1.0, 7.0, 300.0)])
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_round(x.astype(np.float64)), ref)


def test_bf16_round_ties_to_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: even significand (1) wins
    assert bf16_round(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    # 1 + 3 * 2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: the even one is 1 + 2^-6
    assert bf16_round(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    assert bf16_round(np.array([-12.34]))[0] == -12.3125   # ulp 2^-4 in [8, 16)
    assert bf16_round(np.array([0.0]))[0] == 0.0


def test_error_stats():
    ref = np.array([[[1.0, 2.0, 3.0]]])
    got = np.array([[[1.0, 2.0, 3.01]]])
    s = error_stats(got, ref)
    assert abs(s["max_abs"] - 0.01) < 1e-12
    assert s["max_abs_vs_bf16_ref"] == abs(3.01 - 3.0)
    assert s["max_ref"] == 3.0
    assert 0.0 < s["rel_l2_max"] < 0.01 and s["cos_min"] > 0.9999
