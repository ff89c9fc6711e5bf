"""Parity rules between the GPU path and the oracle (helpers for the tests).

Per-score tolerance.  Every tolerance is relative to the scale
T_ij = ||z_i||_2 ||c_j||_2 + |b_i| of the exact query sketch, code and mean
term (oracle.norm_scale; by Cauchy-Schwarz T_ij bounds |s_hat_ij|).  The GPU
must agree with the oracle within eps_ij = tol * T_ij: tol = 1e-5 for float32
sketches (the float32 forward error of the factored score, measured at under
7e-7 T_ij on the synthetic layers).  bf16 sketches are compared (a) with the
exact oracle at tol = 2e-2 and (b) with the bf16-emulating oracle at
tol = 1e-5, where eps_ij also admits a one-ulp bf16 difference in any code or
query-sketch element whose exact value lies within AMBIG_REL times its
absolute-value sum of a bf16 rounding midpoint (the GPU's float32 value of
such an element may fall on the other side of the midpoint, and then both
roundings are correct).

Top-k sets.  Following Proposition 2, a row is tie-exempt when the oracle's
k-th and (k+1)-th scores are closer than the sum of their tolerances; then
several sets are correct, and every swap between the GPU set G and the oracle
set L must be explainable,
max_{l in L\\G}(s_l - eps_l) <= min_{j in G\\L}(s_j + eps_j).  Rows with a wider
margin must match exactly.
"""
from __future__ import annotations

import numpy as np

import oracle as O

TOL_F32 = 1e-5
TOL_BF16_EXACT = 2e-2
# bf16 codes and z against exact ones: each rounding costs at most 2^-8 of the
# element (half of a 7-bit fraction step), so by Cauchy-Schwarz
# |s_gpu - s_exact| <= (2^-8 + 2^-8 + 2^-16 + fp32 sum) ||z|| ||c|| < 2e-2 T_ij.
# fp8 E4M3 codes against exact codes: rounding a normal code costs at most 2^-4
# of its magnitude (half of a 3-bit fraction step) and a subnormal one (below
# 2^-6) at most 2^-10; with z's bf16 rounding,
# |s_gpu - s_exact| <= (2^-4 + 2^-8 + 2^-12) ||z|| ||c|| + 2^-10 (1 + 2^-8) ||z||_1
# + fp32 sum < 7e-2 T_ij + FP8_SUBNORMAL_ABS * ||z||_1.
TOL_FP8_EXACT = 7e-2
FP8_SUBNORMAL_ABS = 2.0 ** -10 * (1 + 2.0 ** -8)
# Bound on the float32 computation error of one code or query-sketch element,
# relative to its absolute-value sum: the largest error seen in float32
# (2.8e-7 on the LLaMA-shaped layer's codes and sketches) times 3.5; the GPU's
# exported float32 codes are checked against the same bound.
AMBIG_REL = 1e-6
# Rigorous bound on the GPU's float32 evaluation of one score from bf16 (or
# fp8 widened to bf16) codes and query sketches: the r <= 32 products per MFMA
# are exact and are summed with the mean term in float32, so
# |fl(s) - s| <= gamma_33 (sum_e |z_e c_e| + |b|) <= gamma_33 T_ij with
# gamma_33 = 33 u / (1 - 33 u), u = 2^-24 (1.97e-6).  A row whose GPU set
# differs from the oracle's must be a swap within this bound (plus the one-ulp
# allowance of codes and sketch elements near a rounding midpoint), five times
# narrower than the per-score tolerance.
TIGHT_EMUL = 2e-6


def _bf16_ambiguity(exact, abs_sum):
    """Elements whose bf16 rounding may legitimately differ, and the size of
    one bf16 ulp at each element."""
    r = O.bf16_round(exact)
    mag = np.maximum(np.abs(exact), 1e-300)
    ulp = np.exp2(np.floor(np.log2(mag)) - 7.0)  # bf16 spacing in [2^e, 2^(e+1)): 2^(e-7)
    dist_mid = np.abs(0.5 * ulp - np.abs(exact - r))
    amb = dist_mid <= AMBIG_REL * abs_sum + 2.0 ** -24 * mag
    return amb, ulp


def _fp8_ambiguity(exact, abs_sum):
    """As _bf16_ambiguity for fp8 E4M3 codes: the spacing is 2^(e-3) in
    [2^e, 2^(e+1)) for e >= -6 and 2^-9 below 2^-6 (subnormals)."""
    r = O.fp8_round(exact)
    mag = np.maximum(np.abs(exact), 1e-300)
    ulp = np.where(mag < 2.0 ** -6, 2.0 ** -9, np.exp2(np.floor(np.log2(mag)) - 3.0))
    dist_mid = np.abs(0.5 * ulp - np.abs(exact - r))
    amb = (dist_mid <= AMBIG_REL * abs_sum + 2.0 ** -24 * mag) & (mag < O.E4M3_MAX)
    return amb, ulp


def oracle_head(B_q, B_k, mu, q, keys, mode: str, tight: bool = False):
    """Oracle scores and per-score tolerances of one head.

    mode: "f32" (exact codes, tol 1e-5), "bf16_exact" (exact codes, tol 2e-2),
    "bf16_emul" (bf16-rounded codes and z, tol 1e-5 plus ambiguity),
    "fp8_exact" (exact codes, tol 7e-2 plus the subnormal term), "fp8_emul"
    (fp8 codes, bf16 z, tol 1e-5 plus ambiguity).
    Returns (s [Q, N], eps [Q, N]), and with `tight` (emulating modes only)
    also the swap bound TIGHT_EMUL * T plus ambiguity."""
    q = np.asarray(q, np.float64)
    keys = np.asarray(keys, np.float64)
    T = O.norm_scale(B_q, B_k, mu, q, keys)
    if mode in ("f32", "bf16_exact", "fp8_exact"):
        s, z, _, _ = O.index_scores(B_q, B_k, mu, q, keys, "f64")
        tol = {"f32": TOL_F32, "bf16_exact": TOL_BF16_EXACT, "fp8_exact": TOL_FP8_EXACT}[mode]
        eps = tol * T
        if mode == "fp8_exact":
            eps = eps + FP8_SUBNORMAL_ABS * np.abs(z).sum(axis=1)[:, None]
        return s, eps
    assert mode in ("bf16_emul", "fp8_emul")
    s, z, b, c = O.index_scores(B_q, B_k, mu, q, keys, mode[:-5])
    c_ex = O.codes(B_k, mu, keys)
    z_ex, _ = O.query_sketch(B_q, mu, q)
    code_amb = _fp8_ambiguity if mode == "fp8_emul" else _bf16_ambiguity
    amb_c, ulp_c = code_amb(c_ex, np.abs(keys - mu) @ np.abs(B_k))
    amb_z, ulp_z = _bf16_ambiguity(z_ex, np.abs(q) @ np.abs(B_q))
    extra = np.abs(z) @ (amb_c * ulp_c).T + (amb_z * ulp_z) @ np.abs(c).T
    if tight:
        return s, TOL_F32 * T + extra, TIGHT_EMUL * T + extra
    return s, TOL_F32 * T + extra


def check_rows(gpu_idx, gpu_score, s, eps, limits, k, tight=None, log=None):
    """Validate GPU top-k rows against oracle scores.  Raises AssertionError
    with the first offending row; returns (rows, exempt rows, differing rows).
    With `tight` (per-score bounds, e.g. oracle_head's third result) a
    differing row's swap must be explainable within them instead of eps;
    `log` (a list) receives (row, gap, bound) of each differing row, gap being
    the oracle's best dropped score minus its worst kept one."""
    n_exempt = n_diff = 0
    for i in range(s.shape[0]):
        lim = int(limits[i])
        m = min(k, lim)
        gi = np.asarray(gpu_idx[i])
        assert np.all(gi[m:] == -1), f"row {i}: expected {k - m} pads"
        G = gi[:m]
        assert np.all((G >= 0) & (G < lim)), f"row {i}: index out of range {G}"
        assert len(set(G.tolist())) == m, f"row {i}: duplicate indices"
        if gpu_score is not None:
            gs = np.asarray(gpu_score[i], np.float64)
            assert np.all(np.isneginf(gs[m:])), f"row {i}: pad scores"
            err = np.abs(gs[:m] - s[i, G])
            bad = err > eps[i, G]
            assert not bad.any(), (f"row {i}: score error {err[bad][:4]} > eps "
                                   f"{eps[i, G][bad][:4]} at idx {G[bad][:4]}")
            for a in range(m - 1):  # sorted by (score desc, index asc)
                assert gs[a] > gs[a + 1] or (gs[a] == gs[a + 1] and G[a] < G[a + 1]), \
                    f"row {i}: order at {a}"
        full = O.topk_row(s[i], lim, min(k + 1, lim))
        L = full[:m]
        exempt = False
        if lim > k:
            a, b = full[k - 1], full[k]
            exempt = (s[i, a] - s[i, b]) <= eps[i, a] + eps[i, b]
        n_exempt += exempt
        sG, sL = set(G.tolist()), set(L.tolist())
        if sG == sL:
            continue
        n_diff += 1
        assert exempt, f"row {i}: sets differ on a non-exempt row"
        out = np.array(sorted(sL - sG))
        inn = np.array(sorted(sG - sL))
        bnd = eps if tight is None else tight
        lo_out = np.max(s[i, out] - bnd[i, out])
        hi_in = np.min(s[i, inn] + bnd[i, inn])
        assert lo_out <= hi_in, f"row {i}: unexplainable swap {out} <-> {inn}"
        if log is not None:
            a, b = out[np.argmax(s[i, out])], inn[np.argmin(s[i, inn])]
            log.append((i, s[i, a] - s[i, b], bnd[i, a] + bnd[i, b]))
    return s.shape[0], n_exempt, n_diff
