"""CPU checks of the parity helpers themselves (tests/parity.py)."""
import numpy as np

import oracle as O
from tests.parity import _bf16_ambiguity


def _next_bf16_up(x):
    """The bf16 value after positive bf16 x, from its bit pattern."""
    b = np.asarray(x, np.float32).view(np.uint32) >> 16
    return ((b + 1) << 16).astype(np.uint32).view(np.float32).astype(np.float64)


def test_bf16_ulp_is_the_spacing_of_bf16_values():
    rng = np.random.default_rng(0)
    x = np.exp2(rng.uniform(-20, 20, 2000)) * rng.uniform(1.0, 2.0, 2000)
    r = O.bf16_round(x)
    _, ulp = _bf16_ambiguity(x, np.abs(x))
    lo = np.where(r <= x, r, r - ulp)          # the bf16 neighbours of x
    # spacing measured from the bit patterns, in the binade of x
    gap = _next_bf16_up(lo) - lo
    np.testing.assert_array_equal(ulp, gap)


def test_midpoints_are_ambiguous_and_representable_values_are_not():
    base = np.array([3.03125, 0.0322265625, 1.5, 100.0])    # bf16 values
    _, ulp = _bf16_ambiguity(base, np.abs(base))
    amb_mid, _ = _bf16_ambiguity(base + 0.5 * ulp, np.abs(base) * 1e-3)
    amb_rep, _ = _bf16_ambiguity(base, np.abs(base) * 1e-3)
    assert amb_mid.all() and not amb_rep.any()


def test_fp8_ulp_is_the_spacing_of_e4m3_values():
    from tests.parity import _fp8_ambiguity
    vals = np.array(sorted({abs(float(O.fp8_round(np.float32(v)))) for v in
                            np.linspace(-448, 448, 20001)} | set(O.fp8_round(
                                np.exp2(np.linspace(-9, 8.8, 5000))))))
    vals = vals[vals > 0]
    _, ulp = _fp8_ambiguity(vals[:-1], vals[:-1])
    np.testing.assert_array_equal(ulp, np.diff(vals))
