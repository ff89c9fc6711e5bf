"""CPU checks of the parity rules themselves (tests/parity.py): the swap bound
used for rows whose GPU set differs from the oracle's, and check_rows'
handling of exempt, non-exempt and tightly bounded rows, on planted lists."""
import numpy as np
import pytest

import oracle as O
from tests.parity import TIGHT_EMUL, check_rows


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
