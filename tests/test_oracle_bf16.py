"""The oracle's bf16 rounding (the optional bf16 weight copy of the step) against
PyTorch's float32 -> bfloat16 conversion, a library routine, on every upper half
of the fp32 bit pattern combined with the lower halves that decide rounding
(zero, one, just below, at and above the midpoint, all ones, and random ones):
every exponent, subnormals, ties to even, the carry into the exponent and the
overflow to infinity.  NaN maps to a quiet NaN of the same sign."""
import numpy as np
import torch

import oracle


def _patterns(seed=0):
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    rng = np.random.default_rng(seed)
    lows = np.concatenate([np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32),
                           rng.integers(0, 1 << 16, size=10, dtype=np.uint32)])
    return (hi[:, None] | lows[None, :]).ravel()


def test_round_bf16_matches_torch_on_all_exponents_and_ties():
    u = _patterns()
    x = u.view(np.float32)
    got = oracle.round_bf16(x)
    finite_or_inf = ~np.isnan(x)
    want = torch.from_numpy(x[finite_or_inf]).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(got[finite_or_inf], want.view(np.uint16))


def test_round_bf16_nan_is_quiet_with_sign():
    u = _patterns(1)
    x = u.view(np.float32)
    nan = np.isnan(x)
    got = oracle.round_bf16(x[nan])
    assert np.all((got & 0x7F80) == 0x7F80) and np.all((got & 0x0040) != 0)
    assert np.array_equal(got >> 15, (u[nan] >> 31).astype(np.uint16))


def test_round_bf16_known_values():
    x = np.array([1.0, -2.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 3.4028235e38, np.inf, -0.0,
                  2.0 ** -133], np.float32)
    # 1+2^-8 is a tie and rounds to the even 1.0; 1+3*2^-8 is a tie rounding up to 1+2^-6;
    # the largest float rounds to infinity; 2^-133 is a bf16 subnormal, kept exactly.
    assert oracle.round_bf16(x).tolist() == [0x3F80, 0xC000, 0x3F80, 0x3F82, 0x7F80, 0x7F80,
                                             0x8000, 0x0001]
