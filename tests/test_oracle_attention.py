"""Pins of the oracle's reading of the index's winners: RoPE, key
reconstruction from codes, and attention over the selected keys."""
import numpy as np
from scipy.special import softmax

import oracle as O
import workloads as W


def test_rope_is_a_position_rotation():
    """Norm-preserving, identity at position 0, additive in the position, and
    scores depend only on the relative position (the RoPE property)."""
    rng = np.random.default_rng(0)
    d = 128
    q, k = rng.standard_normal((2, d))
    for p in (0, 1, 77, 4095, 1 << 20):
        assert abs(np.linalg.norm(O.rope(q, p)) - np.linalg.norm(q)) < 1e-10
    np.testing.assert_array_equal(O.rope(q, 0), q)
    np.testing.assert_allclose(O.rope(O.rope(q, 300), 45), O.rope(q, 345), atol=1e-10)
    for i, j in ((5, 9), (1000, 17), (4095, 4095)):
        np.testing.assert_allclose(O.rope(q, i) @ O.rope(k, j), q @ O.rope(k, j - i), rtol=1e-10)


def test_rope_pairs_and_angles():
    """Dims m and m + d/2 rotate together by pos * theta^(-2m/d): checked with
    unit vectors against the plain 2-D rotation."""
    d, pos = 8, 3
    for m in range(d // 2):
        e = np.zeros(d)
        e[m] = 1.0
        ang = pos * O.ROPE_THETA ** (-2.0 * m / d)
        want = np.zeros(d)
        want[m], want[m + d // 2] = np.cos(ang), np.sin(ang)
        np.testing.assert_allclose(O.rope(e, pos), want, atol=1e-15)


def test_reconstruction_at_full_rank_is_exact():
    """r = d: M_d = I, so mu + B_q c reproduces every key."""
    inp = W.make_layer(W.SPECS["single_head_d128"].with_(N=200))
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 128)
    keys = inp["keys"][0, 0].astype(np.float64)
    khat = O.reconstruct_keys(cal["B_q"], cal["mu"], O.codes(cal["B_k"], cal["mu"], keys))
    np.testing.assert_allclose(khat, keys, atol=1e-9 * np.abs(keys).max())


def test_sparse_attention_special_cases():
    """Selecting every key is dense softmax attention (scipy); the order of the
    selected indices and padding (-1) do not matter; a
    single selected key returns its value."""
    rng = np.random.default_rng(2)
    N, d = 40, 16
    q = rng.standard_normal((3, d))
    keys, values = rng.standard_normal((2, N, d))
    pos = np.array([39, 50, 1000])
    idx = np.tile(np.arange(N), (3, 1))
    got = O.sparse_attention(q, pos, keys, values, idx)
    kr = O.rope(keys, np.arange(N))
    for i in range(3):
        p = softmax(kr @ O.rope(q[i], pos[i]) / np.sqrt(d))
        np.testing.assert_allclose(got[i], p @ values, rtol=1e-12, atol=1e-12)
    perm = np.concatenate([rng.permutation(N), -np.ones(10, int)])
    np.testing.assert_allclose(O.sparse_attention(q, pos, keys, values, np.tile(perm, (3, 1))),
                               got, rtol=1e-12, atol=1e-12)
    one = np.full((3, 5), -1)
    one[:, 2] = 7
    np.testing.assert_allclose(O.sparse_attention(q, pos, keys, values, one),
                               np.tile(values[7], (3, 1)), atol=1e-15)
