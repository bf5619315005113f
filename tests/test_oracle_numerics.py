"""Pins of the oracle's rounding helpers (CPU only)."""
import numpy as np
import pytest
import torch

from oracle.numerics import round_bf16, round_f32, silu, sigmoid


def test_bf16_ties_to_even_hand_values():
    one = 1.0
    ulp = 2.0 ** -7                      # bf16 spacing in [1, 2)
    cases = {
        one + ulp / 2: one,              # halfway, even neighbour is 1.0
        one + 1.5 * ulp: one + 2 * ulp,  # halfway, even neighbour is 1 + 2ulp
        one + 0.49 * ulp: one,
        one + 0.51 * ulp: one + ulp,
        -(one + 1.5 * ulp): -(one + 2 * ulp),
        3.0: 3.0,
        0.0: 0.0,
        2.0 ** -130: 2.0 ** -130,        # bf16 subnormal (spacing 2^-133)
        2.0 ** -134: 0.0,                # half of the smallest subnormal: tie to 0
        3 * 2.0 ** -134: 2.0 ** -132,    # 1.5 subnormal ulps -> even (2 ulps)
    }
    for v, want in cases.items():
        assert round_bf16(np.array([v]))[0] == want, v


def test_bf16_matches_torch_conversion_on_random_floats():
    rng = np.random.default_rng(0)
    a = np.concatenate([
        rng.standard_normal(100000).astype(np.float32),
        (rng.standard_normal(20000) * 1e-38).astype(np.float32),
        (rng.standard_normal(20000) * 1e30).astype(np.float32),
    ])
    # exact ties: low 16 bits = 0x8000
    bits = rng.integers(0, 2**31, size=5000, dtype=np.uint32) & 0xFFFF0000
    ties = (bits | 0x8000).view(np.float32)
    a = np.concatenate([a, ties[np.isfinite(ties)]])
    want = torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy()
    got = round_bf16(a.astype(np.float64))
    np.testing.assert_array_equal(got, want)


def test_bf16_overflow_and_specials():
    big = float(np.ldexp(255.0 / 128.0, 127))
    assert round_bf16(np.array([big]))[0] == big
    assert np.isinf(round_bf16(np.array([np.ldexp(1.0, 128) * 0.999999]))[0])
    out = round_bf16(np.array([np.inf, -np.inf, np.nan]))
    assert out[0] == np.inf and out[1] == -np.inf and np.isnan(out[2])


def test_round_f32_is_ieee():
    v = np.array([1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24, 0.1])
    got = round_f32(v)
    assert got[0] == 1.0 and got[1] == 1.0 + 2.0 ** -22
    assert got[2] == float(np.float32(0.1))


def test_silu_sigmoid_closed_forms():
    assert silu(np.array([0.0]))[0] == 0.0
    a = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(sigmoid(a) + sigmoid(-a), 1.0, rtol=0, atol=1e-15)
    np.testing.assert_allclose(silu(a) - silu(-a), a, rtol=0, atol=1e-12)
    t = torch.tensor(a, dtype=torch.float64)
    np.testing.assert_allclose(silu(a), torch.nn.functional.silu(t).numpy(), rtol=1e-14, atol=1e-300)
