"""Pins for the oracle's bfloat16 rounding: hand-picked ties and torch's converter."""
import numpy as np
import pytest

from oracle.bf16 import round_bf16


def test_ties_round_to_even():
    # bf16 keeps 8 significant bits: spacing at 1.0 is 2^-7.
    cases = {
        1.0 + 2.0 ** -8: 1.0,                          # halfway, even neighbour is 1.0
        1.0 + 3 * 2.0 ** -8: 1.0 + 2.0 ** -6,          # halfway, even neighbour is above
        1.0 + 2.0 ** -8 + 2.0 ** -20: 1.0 + 2.0 ** -7,  # just above halfway rounds up
        1.0 + 2.0 ** -8 - 2.0 ** -20: 1.0,             # just below halfway rounds down
        -(1.0 + 3 * 2.0 ** -8): -(1.0 + 2.0 ** -6),
        0.0: 0.0,
        3.0: 3.0,
        2.0 ** -130: 2.0 ** -130,                      # subnormal exactly representable
    }
    for x, want in cases.items():
        assert round_bf16(np.float32(x)) == want, x


def test_specials():
    assert np.isinf(round_bf16(np.float32(np.inf)))
    assert np.isnan(round_bf16(np.float32(np.nan)))
    big = np.float32(3.4e38)  # rounds past the largest bf16 to inf
    assert np.isinf(round_bf16(big))


def test_matches_torch_converter():
    torch = pytest.importorskip("torch")
    x = (np.random.default_rng(0).standard_normal(100_000) *
         10.0 ** np.random.default_rng(1).integers(-30, 30, 100_000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(round_bf16(x), ref)
