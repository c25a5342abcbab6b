"""Pins of the oracle's bf16 rounding (`oracle.to_bf16`).

The layer chain rounds every stage's float64 result to bf16 with it, and the
library's interface fixes that conversion as round to nearest, ties to even
(through float32, as a float32 accumulator is rounded). It is pinned here
against two things it shares no code with:

* an exact reference built from the definition with rational arithmetic: the
  two bf16 neighbours of a float32 value, the nearer one, ties to the one
  with an even last bit, beyond the largest finite value to infinity;
* torch's float64 -> bfloat16 conversion (a library routine, which also goes
  through float32).

The hand-picked cases are chosen so that truncation, round-half-up,
round-half-away-from-zero and a missing carry into the exponent each fail.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle


def _f32_from_bits(u):
    return np.array([u], dtype=np.uint32).view(np.float32)[0]


def _bf16_value(h):
    """Exact value of bf16 bits h (finite) as a Fraction."""
    f = np.array([h << 16], dtype=np.uint32).view(np.float32)[0]
    return Fraction(float(f))


def _rne_reference(f32):
    """Nearest-even bf16 bits of a float32 value, from the definition."""
    f32 = np.float32(f32)
    u = int(np.array([f32], dtype=np.float32).view(np.uint32)[0])
    sign = u & 0x80000000
    mag = u & 0x7FFFFFFF
    if mag >= 0x7F800000:  # inf stays inf (NaN is not in the oracle's data)
        return (sign >> 16) | (mag >> 16)
    lo = mag >> 16          # magnitude truncated toward zero: the lower neighbour
    hi = lo + 1             # the upper neighbour (0x7F80 is +inf)
    x = Fraction(float(np.array([mag], dtype=np.uint32).view(np.float32)[0]))
    vlo = _bf16_value(lo)
    if hi == 0x7F80:
        # past the largest finite bf16, the "upper neighbour" is infinity: the
        # rounding boundary is where the next finite step would have been
        vhi = vlo + (vlo - _bf16_value(lo - 1))
    else:
        vhi = _bf16_value(hi)
    dlo, dhi = x - vlo, vhi - x
    if dlo < dhi:
        r = lo
    elif dhi < dlo:
        r = hi
    else:
        r = lo if lo % 2 == 0 else hi
    return (sign >> 16) | r


# (float32 bits, expected bf16 bits)
CASES = [
    (0x3F808000, 0x3F80),  # 1 + half an ulp: tie, lower neighbour even -> down
    (0x3F818000, 0x3F82),  # tie, lower neighbour odd -> up (round-to-odd-free)
    (0x3F808001, 0x3F81),  # just above the tie -> up (truncation gives 0x3F80)
    (0x3F817FFF, 0x3F81),  # just below the tie -> down
    (0xBF808000, 0xBF80),  # negative tie, even -> toward zero (half-away gives 0xBF81)
    (0xBF818000, 0xBF82),  # negative tie, odd -> away from zero
    (0xBF808001, 0xBF81),  # negative, just past the tie
    (0x3F7FFFFF, 0x3F80),  # carry into the exponent: 0.99999994 -> 1.0
    (0x407F8000, 0x4080),  # tie with odd lower 0x407F -> up, carrying into the exponent
    (0x7F7F7FFF, 0x7F7F),  # just below the tie above the largest finite value
    (0x7F7F8000, 0x7F80),  # tie between the largest finite (odd) and inf -> inf
    (0x7F7FFFFF, 0x7F80),  # float32 max -> inf
    (0xFF7F8000, 0xFF80),  # same, negative -> -inf
    (0x7F800000, 0x7F80),  # +inf
    (0xFF800000, 0xFF80),  # -inf
    (0x00000000, 0x0000),  # +0
    (0x80000000, 0x8000),  # -0 keeps its sign
    (0x00008000, 0x0000),  # subnormal tie, even lower (0) -> 0
    (0x00018000, 0x0002),  # subnormal tie, odd lower -> up
    (0x00008001, 0x0001),  # subnormal just above the tie
    (0x00007FFF, 0x0000),  # below half of the smallest bf16 subnormal -> 0
    (0x80018000, 0x8002),  # negative subnormal tie, odd lower
    (0x007F8000, 0x0080),  # largest subnormal tie (odd 0x007F) -> smallest normal
]


@pytest.mark.parametrize("bits,expected", CASES)
def test_hand_picked_cases(bits, expected):
    f = _f32_from_bits(bits)
    # the case table itself is checked against the rational reference
    assert _rne_reference(f) == expected, hex(_rne_reference(f))
    got = int(oracle.to_bf16(np.array([float(f)]))[0])
    assert got == expected, (hex(bits), hex(got), hex(expected))


def test_random_float32_against_rational_reference():
    rng = np.random.default_rng(5)
    # random bit patterns cover every exponent, subnormals included; ties are
    # forced in a quarter of them
    u = rng.integers(0, 0x7F800000, size=3000, dtype=np.uint64).astype(np.uint32)
    u[::4] = (u[::4] & 0xFFFF0000) | 0x8000
    u[1::8] |= 0x80000000
    f = u.view(np.float32)
    got = oracle.to_bf16(f.astype(np.float64))
    ref = np.array([_rne_reference(v) for v in f], dtype=np.uint16)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(hex(int(u[i])), hex(int(got[i])), hex(int(ref[i]))) for i in bad[:5]]


def test_float64_against_torch():
    rng = np.random.default_rng(6)
    v = np.concatenate([
        rng.standard_normal(20000) * np.exp(rng.uniform(-60, 60, 20000)),
        rng.standard_normal(2000) * 1e-40,     # below the float32 normal range
        np.array([3.3961e38, 3.4e38, -3.39e38, 1e39, -1e39, 0.0, -0.0]),
    ])
    got = oracle.to_bf16(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(v[i], hex(int(got[i])), hex(int(ref[i]))) for i in bad[:5]]


def test_shape_is_kept():
    v = np.arange(24, dtype=np.float64).reshape(2, 3, 4) / 7
    out = oracle.to_bf16(v)
    assert out.shape == (2, 3, 4) and out.dtype == np.uint16
