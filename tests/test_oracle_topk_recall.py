"""Pins of the oracle's selection, recall and storage rounding."""
import heapq
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_2x2.json")


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["topk_cases"])
def test_topk_hand_cases(case):
    got = O.topk_row(np.array(case["scores"]), case["limit"], case["k"])
    assert got.tolist() == case["idx"]


def _nlargest(s, limit, k):
    """Independent route: heapq over (score, -index) pairs."""
    best = heapq.nlargest(k, ((float(s[j]), -j) for j in range(limit)))
    out = [-j for _, j in best]
    return out + [O.PAD_IDX] * (k - len(out))


def test_topk_matches_heap_selection_random_and_tied():
    rng = np.random.default_rng(0)
    for trial in range(300):
        n = int(rng.integers(1, 300))
        k = int(rng.integers(1, 80))
        if trial % 3 == 0:
            s = rng.integers(0, 5, n).astype(np.float64)  # many exact ties
        else:
            s = rng.standard_normal(n)
        limit = int(rng.integers(1, n + 1))
        assert O.topk_row(s, limit, k).tolist() == _nlargest(s, limit, k)


def test_topk_exhaustive_tiny():
    """Every score pattern over a 3-letter alphabet for n <= 6, every k."""
    for n in range(1, 7):
        for pat in itertools.product([0.0, 1.0, 2.0], repeat=n):
            s = np.array(pat)
            for k in range(1, n + 2):
                got = O.topk_row(s, n, k).tolist()
                want = sorted(range(n), key=lambda j: (-s[j], j))[:k]
                want += [O.PAD_IDX] * (k - len(want))
                assert got == want


def test_candidate_limits_causal_inclusive():
    np.testing.assert_array_equal(O.candidate_limits(3, 10, np.array([0, 4, 20])), [1, 5, 10])
    np.testing.assert_array_equal(O.candidate_limits(2, 7), [7, 7])


def test_recall_hits_against_sorted_intersection():
    rng = np.random.default_rng(1)
    a = np.stack([rng.choice(500, 64, replace=False) for _ in range(50)])
    e = np.stack([rng.choice(500, 64, replace=False) for _ in range(50)])
    e[:10] = a[:10][:, ::-1]  # identical sets in another order
    want = np.array([np.intersect1d(a[i], e[i]).size for i in range(50)])
    np.testing.assert_array_equal(O.recall_hits(a, e), want)
    assert np.all(O.recall_hits(a[:10], e[:10]) == 64)
    padded = np.full((1, 64), O.PAD_IDX)
    padded[0, :3] = [4, 5, 6]
    assert O.recall_hits(padded, padded)[0] == 3


def test_margin_condition_preserves_topk():
    """Proposition 2: if every score moves by at most eps and the top-k margin
    exceeds 2 eps, the top-k set is unchanged; when the margin is below 2 eps a
    perturbation can swap the k-th and (k+1)-th."""
    rng = np.random.default_rng(2)
    k = 64
    for _ in range(200):
        s = rng.standard_normal(1000)
        srt = np.sort(s)[::-1]
        gap = srt[k - 1] - srt[k]
        eps = 0.49 * gap
        s2 = s + rng.uniform(-eps, eps, s.size)
        assert set(O.topk_row(s, 1000, k)) == set(O.topk_row(s2, 1000, k))
    s = rng.standard_normal(1000)
    order = np.argsort(-s)
    gap = s[order[k - 1]] - s[order[k]]
    s2 = s.copy()
    s2[order[k - 1]] -= 0.6 * gap
    s2[order[k]] += 0.6 * gap
    assert set(O.topk_row(s, 1000, k)) != set(O.topk_row(s2, 1000, k))


def test_bf16_round_matches_torch_conversion():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(100000) * 10.0 ** rng.integers(-20, 20, 100000),
                        rng.standard_normal(1000)]).astype(np.float32)
    # exact midpoints between neighbouring bf16 values: ties go to even
    mids = (np.arange(1, 2001, dtype=np.uint32) << 16) + np.uint32(0x3F800000 + 0x8000)
    x = np.concatenate([x, mids.view(np.float32), -mids.view(np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.bf16_round(x), want)


def test_f32_round():
    x = np.array([1.0 + 2.0 ** -30, 1.0 / 3.0, -7.25])
    np.testing.assert_array_equal(O.f32_round(x), x.astype(np.float32).astype(np.float64))


def test_score_scale_covers_float32_rounding():
    """The tolerance scale S_ij: scores computed entirely in float32 from the
    same factors stay within 1e-5 * S_ij of the float64 scores."""
    rng = np.random.default_rng(4)
    d, r = 128, 32
    Bq = rng.standard_normal((d, r))
    Bk = rng.standard_normal((d, r))
    mu = rng.standard_normal(d) * 0.1
    q = rng.standard_normal((64, d)) * 3
    keys = rng.standard_normal((256, d)) * 0.01
    s, *_ = O.index_scores(Bq, Bk, mu, q, keys)
    f = np.float32
    c32 = ((keys.astype(f) - mu.astype(f)) @ Bk.astype(f))
    z32 = q.astype(f) @ Bq.astype(f)
    b32 = q.astype(f) @ mu.astype(f)
    s32 = (z32 @ c32.T + b32[:, None]).astype(np.float64)
    S = O.score_scale(Bq, Bk, mu, q, keys)
    assert np.max(np.abs(s32 - s) / S) < 1e-5


def test_norm_scale_covers_float32_on_the_layer():
    """The parity scale T_ij = ||z|| ||c|| + |b| on SAKI's own factors (LLaMA-
    shaped layer, head 0, 400 causal rows): float32 codes, query sketches and
    scores (factors rounded to float32, as the library stores them) stay
    within 1e-5 T_ij of the float64 scores, and each float32 code and sketch
    element within tests.parity.AMBIG_REL times its absolute-value sum of
    the exact one, the bounds the GPU parity tests rely on.  The magnitude
    scale S_ij of the factored computation is far larger (cancellation in
    B_q^T q and B_k^T (k - mu))."""
    from tests.parity import AMBIG_REL
    spec = W.SPECS["llama31_8b_layer"].with_(H_q=4, H_kv=1)
    inp = W.make_layer(spec)
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 32)
    Bq, Bk, mu = cal["B_q"], cal["B_k"], cal["mu"]
    q = inp["queries"][0, 0][-400:].astype(np.float64)
    keys = inp["keys"][0, 0].astype(np.float64)
    s, z, b, c = O.index_scores(Bq, Bk, mu, q, keys)
    f = np.float32
    c32 = ((keys.astype(f) - mu.astype(f)) @ Bk.astype(f)).astype(np.float64)
    z32 = (q.astype(f) @ Bq.astype(f)).astype(np.float64)
    b32 = (q.astype(f) @ mu.astype(f)).astype(np.float64)
    s32 = z32 @ c32.T + b32[:, None]
    T = O.norm_scale(Bq, Bk, mu, q, keys)
    assert np.max(np.abs(s32 - s) / T) < 1e-5
    assert np.max(np.abs(c32 - c) / (np.abs(keys - mu) @ np.abs(Bk))) < AMBIG_REL
    assert np.max(np.abs(z32 - z) / (np.abs(q) @ np.abs(Bq))) < AMBIG_REL
    assert np.median(O.score_scale(Bq, Bk, mu, q, keys) / T) > 50


def test_fp8_round_matches_torch_e4m3fn():
    """fp8 E4M3 code storage against torch's float8_e4m3fn conversion (round
    to nearest even) inside the format's range, subnormals and exact
    midpoints between neighbouring values included."""
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.standard_normal(50000) * 10.0 ** rng.uniform(-4, 2.5, 50000),
                        rng.uniform(-2.0 ** -6, 2.0 ** -6, 5000)]).astype(np.float32)
    vals = torch.arange(0, 0x7F, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mids = 0.5 * (vals[1:] + vals[:-1])
    x = np.concatenate([x, mids, -mids, vals, -vals]).astype(np.float32)
    x = x[np.abs(x) <= 448.0]
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.fp8_round(x), want)


def test_fp8_format_constants_and_saturation():
    """Largest finite E4M3 value 448, smallest normal 2^-6, smallest
    subnormal 2^-9; magnitudes beyond 448 saturate (reading: no infinities)."""
    x = np.array([448.0, 2.0 ** -6, 2.0 ** -9, 1.0, 1.0625, 1.125, 3.0 * 2 ** -10,
                  5.0 * 2 ** -11, 449.0, 1e6, -1e6, 0.0])
    want = np.array([448.0, 2.0 ** -6, 2.0 ** -9, 1.0, 1.0, 1.125, 2.0 ** -8,
                     2.0 ** -9, 448.0, 448.0, -448.0, 0.0])
    np.testing.assert_array_equal(O.fp8_round(x), want)
