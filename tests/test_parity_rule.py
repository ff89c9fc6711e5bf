"""CPU checks of the parity helpers themselves (tests/parity.py)."""
import numpy as np
import pytest

import oracle as O
from tests.parity import TIGHT_EMUL, _bf16_ambiguity, check_rows


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

def test_tight_bound_covers_gamma_33():
    u = 2.0 ** -24
    gamma = 33 * u / (1 - 33 * u)
    assert gamma <= TIGHT_EMUL < 1.1 * gamma


def test_float32_sum_of_bf16_products_within_gamma_33():
    """32 exact bf16 x bf16 products and a mean term summed in float32 (any
    order) stay within gamma_33 times the absolute-value sum."""
    rng = np.random.default_rng(0)
    z = O.bf16_round(rng.standard_normal((4000, 32)))
    c = O.bf16_round(rng.standard_normal((4000, 32)) * rng.uniform(0.01, 100, (4000, 1)))
    b = rng.standard_normal(4000) * 10
    exact = np.sum(z * c, axis=1) + b
    prods = (z * c).astype(np.float32)
    assert np.array_equal(prods.astype(np.float64), z * c)  # 16 significant bits: exact
    for order in (np.arange(32), np.arange(32)[::-1], rng.permutation(32)):
        acc = b.astype(np.float32)
        for e in order:
            acc = (acc + prods[:, e]).astype(np.float32)
        bound = TIGHT_EMUL * (np.sum(np.abs(z * c), axis=1) + np.abs(b))
        assert np.all(np.abs(acc - exact) <= bound)


def _row(n=200, k=64, seed=0):
    rng = np.random.default_rng(seed)
    s = rng.standard_normal((1, n))
    order = np.argsort(-s[0], kind="stable")
    return s, order


def test_check_rows_swaps():
    k = 64
    s, order = _row()
    a, b = order[k - 1], order[k]
    gap = s[0, a] - s[0, b]
    lim = np.array([s.shape[1]])
    G = order[:k].copy()
    G[k - 1] = b  # the GPU kept the 65th instead of the 64th
    G = G[np.argsort(-s[0, G], kind="stable")][None, :]
    # exact list: passes; the swapped one on a non-exempt row fails
    assert check_rows(order[None, :k], None, s, np.full_like(s, 1e-12), lim, k) == (1, 0, 0)
    with pytest.raises(AssertionError, match="non-exempt"):
        check_rows(G, None, s, np.full_like(s, 1e-12), lim, k)
    # exempt and within both bounds: one differing row, logged with its gap
    eps = np.full_like(s, gap)
    log = []
    assert check_rows(G, None, s, eps, lim, k, tight=np.full_like(s, 0.6 * gap), log=log) == (1, 1, 1)
    assert len(log) == 1 and log[0][0] == 0 and np.isclose(log[0][1], gap)
    # exempt under eps but beyond the tight bound: rejected
    with pytest.raises(AssertionError, match="unexplainable"):
        check_rows(G, None, s, eps, lim, k, tight=np.full_like(s, 0.4 * gap))
